// wise_kernels.hpp — host-side launchers of the libwise kernels.  Shapes are
// validated by the C ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace wise {

// Validated geometry: bh = batch * heads, nb = n / block.
struct Dims {
  int bh, n, d, block, nb;
  float scale;
};

constexpr int kMaxSelectBlocks = 1024;  // selection keeps a row's candidates in LDS

hipError_t launch_dense(const Dims& s, const void* q, const void* k, const void* v, void* o,
                        float* lse, hipStream_t st);
hipError_t launch_mass(const Dims& s, const void* q, const void* k, const float* lse, float* acc,
                       hipStream_t st);
hipError_t launch_sparse(const Dims& s, const void* q, const void* k, const void* v,
                         const int32_t* row_ptr, const int32_t* col_idx, const int32_t* order,
                         void* o, float* lse, hipStream_t st);
hipError_t launch_select(const Dims& s, const float* acc, float tau, uint32_t flags,
                         int32_t* row_ptr, int32_t* col_idx, int32_t* row_order, void* ws,
                         hipStream_t st);
size_t select_workspace_bytes(const Dims& s);

}  // namespace wise
