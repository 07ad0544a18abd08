// wise_kernels.hpp — host-side launchers of the libwise kernels.  Shapes are
// validated by the C ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace wise {

// Validated geometry: bh = batch * heads, nb = n / block; gq = heads /
// kv_heads query heads share one key-value head.
struct Dims {
  int bh, n, d, block, nb, heads, gq;
  float scale;
};

constexpr int kMaxSelectBlocks = 1024;  // selection keeps a row's candidates in LDS

hipError_t launch_dense(const Dims& s, const void* q, const void* k, const void* v, void* o,
                        float* lse, float* acc, void* ws, hipStream_t st);
size_t mass_workspace_bytes(const Dims& s);
int dense_query_tile(const Dims& s);   // queries per dense work-group: 64, 128 or 256
hipError_t launch_sparse(const Dims& s, const void* q, const void* k, const void* v,
                         const int32_t* row_ptr, const int32_t* col_idx, const int32_t* order,
                         void* o, float* lse, hipStream_t st);
// Blocks of 64 keys (groups of 4 rows at head_dim 128, else 2) and of 128
// keys at head_dim 128 (groups of 2 rows): work-groups of consecutive rows
// over the union of their supports (sparse_group_rows(s) rows per group; 0:
// not available, and launch_sparse_grouped runs launch_sparse instead).
int sparse_group_rows(const Dims& s);
hipError_t launch_sparse_grouped(const Dims& s, const void* q, const void* k, const void* v,
                                 const int32_t* row_ptr, const int32_t* col_idx, void* o,
                                 float* lse, hipStream_t st);
hipError_t launch_select(const Dims& s, const float* acc, float tau, uint32_t flags,
                         int32_t* row_ptr, int32_t* col_idx, int32_t* row_order, void* ws,
                         hipStream_t st);
size_t select_workspace_bytes(const Dims& s);
hipError_t launch_select_noalloc(const Dims& s, const float* acc, float tau, uint32_t flags,
                                 int32_t* row_ptr, int32_t* col_idx, int32_t* row_order,
                                 hipStream_t st);
int mask_words(const Dims& s);
hipError_t launch_select_step(const Dims& s, const float* r, float tau, uint64_t* mask,
                              hipStream_t st);
hipError_t launch_support_from_masks(const Dims& s, const uint64_t* masks, int n_masks,
                                     uint32_t flags, int32_t* row_ptr, int32_t* col_idx,
                                     int32_t* row_order, void* ws, hipStream_t st);
hipError_t launch_mask_union(const Dims& s, const uint64_t* masks, int n_masks, uint64_t* out,
                             hipStream_t st);
hipError_t launch_mask_overlap(const Dims& s, const uint64_t* a, const uint64_t* b,
                               int64_t* counts, hipStream_t st);
hipError_t launch_support_mass(const Dims& s, const float* r, const int32_t* row_ptr,
                               const int32_t* col_idx, double* row_mass, double* totals,
                               hipStream_t st);

}  // namespace wise
