// wise_api.hip — the C ABI of libwise (declared in include/wise.h).
//
// Every entry point validates its arguments on the host before touching the
// HIP runtime, so an invalid call returns its status without launching
// anything (and without needing a GPU).  Valid calls only enqueue kernels on
// the caller's stream.
#include <math.h>
#include <stdint.h>

#include "wise.h"
#include "wise_kernels.hpp"

namespace {

constexpr int64_t kI32Max = 2147483647;

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// Geometry checks shared by all calls; fills the validated dims.
wise_status check_shape(const wise_shape* s, wise::Dims* out) {
  if (s == nullptr) return WISE_ERR_NULL;
  if (s->batch <= 0 || s->heads <= 0 || s->seq_len <= 0 || s->head_dim <= 0 || s->block <= 0)
    return WISE_ERR_SHAPE;
  if (s->head_dim != 64 && s->head_dim != 96 && s->head_dim != 128) return WISE_ERR_UNSUPPORTED;
  if (s->block != 16 && s->block != 32 && s->block != 64 && s->block != 128)
    return WISE_ERR_UNSUPPORTED;
  if (s->seq_len % s->block != 0) return WISE_ERR_SHAPE;
  if (s->block < 64 && s->seq_len % 64 != 0) return WISE_ERR_SHAPE;   // 64-key dense tiles
  const int32_t kvh = s->kv_heads == 0 ? s->heads : s->kv_heads;
  if (kvh <= 0 || s->heads % kvh != 0) return WISE_ERR_SHAPE;
  if (isnan(s->scale) || isinf(s->scale)) return WISE_ERR_RANGE;
  const int64_t bh = (int64_t)s->batch * s->heads;
  const int64_t nb = s->seq_len / s->block;
  // CSR offsets are int32: every admissible block pair must be addressable.
  if (bh * nb > kI32Max || bh * nb * (nb + 1) / 2 > kI32Max) return WISE_ERR_SHAPE;
  out->bh = (int)bh;
  out->n = s->seq_len;
  out->d = s->head_dim;
  out->block = s->block;
  out->nb = (int)nb;
  out->heads = s->heads;
  out->gq = s->heads / kvh;
  out->scale = s->scale > 0.f ? s->scale : 1.0f / sqrtf((float)s->head_dim);
  return WISE_OK;
}

wise_status check_qkvo(const void* q, const void* k, const void* v, const void* o) {
  if (!q || !k || !v || !o) return WISE_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16))
    return WISE_ERR_SHAPE;
  return WISE_OK;
}

wise_status from_hip(hipError_t e) { return e == hipSuccess ? WISE_OK : WISE_ERR_HIP; }

}  // namespace

extern "C" {

wise_status wise_dense_attn_accum(const wise_shape* s, const void* q, const void* k,
                                  const void* v, void* o, float* lse, float* acc, void* workspace,
                                  size_t workspace_bytes, void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if ((st = check_qkvo(q, k, v, o)) != WISE_OK) return st;
  if (acc != nullptr && workspace == nullptr) return WISE_ERR_NULL;
  if ((lse && !aligned(lse, 4)) || (acc && !aligned(acc, 4)) ||
      (acc && !aligned(workspace, 256)))
    return WISE_ERR_SHAPE;
  if (acc == nullptr)
    return from_hip(wise::launch_dense(d, q, k, v, o, lse, nullptr, nullptr, (hipStream_t)hip_stream));
  // The workspace is linear in the head count: when it holds fewer than all
  // heads, the heads run in consecutive launches of as many whole key-value
  // groups as fit (the launches share the stream, so they reuse it in
  // turn).  Per head the work and its order are the same either way.
  const size_t full = wise::mass_workspace_bytes(d);
  const size_t group = full / (size_t)d.bh * (size_t)d.gq;
  if (workspace_bytes < group) return WISE_ERR_WORKSPACE;
  const int per = workspace_bytes >= full ? d.bh : (int)(workspace_bytes / group) * d.gq;
  const size_t qkv_head = (size_t)d.n * d.d * 2;   // bytes of one head of q, k, v, o
  for (int h0 = 0; h0 < d.bh; h0 += per) {
    wise::Dims c = d;
    c.bh = per < d.bh - h0 ? per : d.bh - h0;
    const size_t kv0 = (size_t)(h0 / d.gq);
    const hipError_t e = wise::launch_dense(
        c, (const char*)q + h0 * qkv_head, (const char*)k + kv0 * qkv_head,
        (const char*)v + kv0 * qkv_head, (char*)o + h0 * qkv_head,
        lse ? lse + (size_t)h0 * d.n : nullptr, acc + (size_t)h0 * d.nb * d.nb, workspace,
        (hipStream_t)hip_stream);
    if (e != hipSuccess) return WISE_ERR_HIP;
  }
  return WISE_OK;
}

wise_status wise_select_support(const wise_shape* s, const float* acc, float tau, uint32_t flags,
                                int32_t* row_ptr, int32_t* col_idx, int32_t* row_order,
                                void* workspace, size_t workspace_bytes, void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if (!acc || !row_ptr || !col_idx || !workspace) return WISE_ERR_NULL;
  if (d.nb > wise::kMaxSelectBlocks) return WISE_ERR_UNSUPPORTED;
  if (!(tau > 0.f && tau <= 1.f)) return WISE_ERR_RANGE;
  if (flags & ~(uint32_t)(WISE_FORCE_SINK | WISE_FORCE_DIAG)) return WISE_ERR_RANGE;
  if (workspace_bytes < wise::select_workspace_bytes(d)) return WISE_ERR_WORKSPACE;
  if (!aligned(acc, 4) || !aligned(row_ptr, 4) || !aligned(col_idx, 4) ||
      (row_order && !aligned(row_order, 4)) || !aligned(workspace, 256))
    return WISE_ERR_SHAPE;
  return from_hip(wise::launch_select(d, acc, tau, flags, row_ptr, col_idx, row_order, workspace,
                                      (hipStream_t)hip_stream));
}

wise_status wise_select_support_noalloc(const wise_shape* s, const float* acc, float tau,
                                        uint32_t flags, int32_t* row_ptr, int32_t* col_idx,
                                        int32_t* row_order, void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if (!acc || !row_ptr || !col_idx) return WISE_ERR_NULL;
  if (d.nb > wise::kMaxSelectBlocks) return WISE_ERR_UNSUPPORTED;
  if (!(tau > 0.f && tau <= 1.f)) return WISE_ERR_RANGE;
  if (flags & ~(uint32_t)(WISE_FORCE_SINK | WISE_FORCE_DIAG)) return WISE_ERR_RANGE;
  if (wise::select_workspace_bytes(d) > (size_t)WISE_NOALLOC_SCRATCH_BYTES) return WISE_ERR_WORKSPACE;
  if (!aligned(acc, 4) || !aligned(row_ptr, 4) || !aligned(col_idx, 4) ||
      (row_order && !aligned(row_order, 4)))
    return WISE_ERR_SHAPE;
  return from_hip(wise::launch_select_noalloc(d, acc, tau, flags, row_ptr, col_idx, row_order,
                                              (hipStream_t)hip_stream));
}

wise_status wise_sparse_attn(const wise_shape* s, const void* q, const void* k, const void* v,
                             const int32_t* row_ptr, const int32_t* col_idx,
                             const int32_t* row_order, void* o, float* lse, void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if ((st = check_qkvo(q, k, v, o)) != WISE_OK) return st;
  if (!row_ptr || !col_idx) return WISE_ERR_NULL;
  if (!aligned(row_ptr, 4) || !aligned(col_idx, 4) || (row_order && !aligned(row_order, 4)) ||
      (lse && !aligned(lse, 4)))
    return WISE_ERR_SHAPE;
  return from_hip(wise::launch_sparse(d, q, k, v, row_ptr, col_idx, row_order, o, lse,
                                      (hipStream_t)hip_stream));
}

wise_status wise_sparse_attn_grouped(const wise_shape* s, const void* q, const void* k,
                                     const void* v, const int32_t* row_ptr,
                                     const int32_t* col_idx, void* o, float* lse,
                                     void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if ((st = check_qkvo(q, k, v, o)) != WISE_OK) return st;
  if (!row_ptr || !col_idx) return WISE_ERR_NULL;
  if (!aligned(row_ptr, 4) || !aligned(col_idx, 4) || (lse && !aligned(lse, 4)))
    return WISE_ERR_SHAPE;
  return from_hip(wise::launch_sparse_grouped(d, q, k, v, row_ptr, col_idx, o, lse,
                                              (hipStream_t)hip_stream));
}

int32_t wise_sparse_group_rows(const wise_shape* s) {
  wise::Dims d;
  if (check_shape(s, &d) != WISE_OK) return -1;
  return wise::sparse_group_rows(d);
}

wise_status wise_select_step(const wise_shape* s, const float* r, float tau, uint64_t* mask,
                             void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if (!r || !mask) return WISE_ERR_NULL;
  if (d.nb > wise::kMaxSelectBlocks) return WISE_ERR_UNSUPPORTED;
  if (!(tau > 0.f && tau <= 1.f)) return WISE_ERR_RANGE;
  if (!aligned(r, 4) || !aligned(mask, 8)) return WISE_ERR_SHAPE;
  return from_hip(wise::launch_select_step(d, r, tau, mask, (hipStream_t)hip_stream));
}

wise_status wise_support_from_masks(const wise_shape* s, const uint64_t* masks, int32_t n_masks,
                                    uint32_t flags, int32_t* row_ptr, int32_t* col_idx,
                                    int32_t* row_order, void* workspace, size_t workspace_bytes,
                                    void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if (!masks || !row_ptr || !col_idx || !workspace) return WISE_ERR_NULL;
  if (d.nb > wise::kMaxSelectBlocks) return WISE_ERR_UNSUPPORTED;
  if (n_masks < 1) return WISE_ERR_SHAPE;
  if (flags & ~(uint32_t)(WISE_FORCE_SINK | WISE_FORCE_DIAG)) return WISE_ERR_RANGE;
  if (workspace_bytes < wise::select_workspace_bytes(d)) return WISE_ERR_WORKSPACE;
  if (!aligned(masks, 8) || !aligned(row_ptr, 4) || !aligned(col_idx, 4) ||
      (row_order && !aligned(row_order, 4)) || !aligned(workspace, 256))
    return WISE_ERR_SHAPE;
  return from_hip(wise::launch_support_from_masks(d, masks, n_masks, flags, row_ptr, col_idx,
                                                  row_order, workspace,
                                                  (hipStream_t)hip_stream));
}

wise_status wise_mask_union(const wise_shape* s, const uint64_t* masks, int32_t n_masks,
                            uint64_t* out, void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if (!masks || !out) return WISE_ERR_NULL;
  if (n_masks < 1) return WISE_ERR_SHAPE;
  if (!aligned(masks, 8) || !aligned(out, 8)) return WISE_ERR_SHAPE;
  return from_hip(wise::launch_mask_union(d, masks, n_masks, out, (hipStream_t)hip_stream));
}

wise_status wise_mask_overlap(const wise_shape* s, const uint64_t* a, const uint64_t* b,
                              int64_t* counts, void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if (!a || !b || !counts) return WISE_ERR_NULL;
  if (!aligned(a, 8) || !aligned(b, 8) || !aligned(counts, 8)) return WISE_ERR_SHAPE;
  return from_hip(wise::launch_mask_overlap(d, a, b, counts, (hipStream_t)hip_stream));
}

wise_status wise_support_mass(const wise_shape* s, const float* r, const int32_t* row_ptr,
                              const int32_t* col_idx, double* row_mass, double* totals,
                              void* hip_stream) {
  wise::Dims d;
  wise_status st = check_shape(s, &d);
  if (st != WISE_OK) return st;
  if (!r || !row_ptr || !col_idx || !row_mass) return WISE_ERR_NULL;
  if (!aligned(r, 4) || !aligned(row_ptr, 4) || !aligned(col_idx, 4) || !aligned(row_mass, 8) ||
      (totals && !aligned(totals, 8)))
    return WISE_ERR_SHAPE;
  return from_hip(wise::launch_support_mass(d, r, row_ptr, col_idx, row_mass, totals,
                                            (hipStream_t)hip_stream));
}

size_t wise_mass_workspace_min_bytes(const wise_shape* s) {
  wise::Dims d;
  if (check_shape(s, &d) != WISE_OK) return 0;
  return wise::mass_workspace_bytes(d) / (size_t)d.bh * (size_t)d.gq;
}

size_t wise_mass_workspace_bytes(const wise_shape* s) {
  wise::Dims d;
  if (check_shape(s, &d) != WISE_OK) return 0;
  return wise::mass_workspace_bytes(d);
}

int32_t wise_mask_words(const wise_shape* s) {
  wise::Dims d;
  if (check_shape(s, &d) != WISE_OK) return -1;
  return wise::mask_words(d);
}

size_t wise_select_workspace_bytes(const wise_shape* s) {
  wise::Dims d;
  if (check_shape(s, &d) != WISE_OK) return 0;
  return wise::select_workspace_bytes(d);
}

int64_t wise_support_capacity(const wise_shape* s) {
  wise::Dims d;
  if (check_shape(s, &d) != WISE_OK) return -1;
  return (int64_t)d.bh * d.nb * (d.nb + 1) / 2;
}

const char* wise_status_string(wise_status st) {
  switch (st) {
    case WISE_OK: return "WISE_OK: success";
    case WISE_ERR_NULL: return "WISE_ERR_NULL: a required pointer is NULL";
    case WISE_ERR_SHAPE:
      return "WISE_ERR_SHAPE: invalid geometry, seq_len not a multiple of block (of 64 for blocks "
             "16 and 32), heads not a multiple of kv_heads, size beyond int32 CSR indexing, or a "
             "misaligned pointer";
    case WISE_ERR_UNSUPPORTED:
      return "WISE_ERR_UNSUPPORTED: head_dim must be 64/96/128, block 16/32/64/128, "
             "seq_len/block <= 1024 for selection";
    case WISE_ERR_RANGE: return "WISE_ERR_RANGE: tau outside (0, 1], bad scale or unknown flag bits";
    case WISE_ERR_WORKSPACE: return "WISE_ERR_WORKSPACE: workspace smaller than required";
    case WISE_ERR_HIP: return "WISE_ERR_HIP: a kernel launch failed";
  }
  return "unknown wise_status";
}

int32_t wise_abi_version(void) { return WISE_ABI_VERSION; }

}  // extern "C"
