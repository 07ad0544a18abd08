/*
 * wise.h — C ABI of libwise, the gfx950 (MI355X) hot path of WISE
 * (Working-set Inference with Support Exploitation) for recurrent-depth
 * language models.
 *
 * The method (paper, Section 5): during the first t_d recurrent steps run
 * full causal attention and pool its probabilities into per
 * (query-block, key-block) masses (Section 5.1, eq. "block_attention_mass");
 * pick, per query block, the smallest set of key blocks whose pooled mass
 * reaches a threshold (Section 5.1, eq. "block_working_set"); for every later
 * step restrict attention to that fixed block support while Q/K/V are
 * recomputed (Section 5.2, eq. "wise_attention").  The support is kept as a
 * device-resident CSR schedule (Appendix B, "Sparse-kernel implementation").
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every tensor argument is a DEVICE pointer owned by the caller,
 *    contiguous, row-major.  The library allocates nothing: scratch space
 *    comes in as caller-owned workspaces sized by the *_workspace_bytes
 *    queries, except for wise_select_support_noalloc, which uses a fixed
 *    device array of its own (WISE_NOALLOC_SCRATCH_BYTES per GPU).
 *  - bf16 tensors are raw IEEE bfloat16 storage (uint16, round-to-nearest-even
 *    when produced by the library).
 *  - Shapes: q, o are [batch][heads][seq_len][head_dim]; k, v are
 *    [batch][kv_heads][seq_len][head_dim] (kv_heads = heads without
 *    grouped-query attention); lse is [batch][heads][seq_len]; acc is
 *    [batch][heads][nb][nb] with nb = seq_len / block.  CSR row
 *    r = (b * heads + h) * nb + qb: masses, supports and rows stay per query
 *    head, and query head h reads key-value head h / (heads / kv_heads).
 *  - Every call validates its arguments on the host BEFORE touching the
 *    device and returns a status; on any error nothing is launched and no
 *    output is written.  On success the work is only enqueued on
 *    `hip_stream` (a hipStream_t, NULL = default stream) and the call
 *    returns; device-side faults surface at the caller's next
 *    synchronisation.  WISE_ERR_HIP carries a failed launch.
 *  - Calls are stateless and re-entrant; calls on different streams with
 *    disjoint outputs may run concurrently.  No C++ exception crosses the ABI.
 *  - A successful call enqueues kernels only: no allocation, memset, copy or
 *    synchronisation, so calls may be captured in a HIP graph (the graph
 *    then reads whatever the captured buffers hold at replay time).
 *  - Supported: head_dim in {64, 96, 128}; block in {16, 32, 64, 128} (the
 *    block sizes of the paper's block-size sweep, Appendix "Block-Size
 *    Tradeoff"); seq_len % block == 0, and seq_len % 64 == 0 for blocks 16
 *    and 32 (the dense kernel's key tiles); nb <= 1024 for wise_select_support,
 *    wise_select_step and wise_support_from_masks.
 *  - Support bitmasks (the union mode and the diagnostics): uint64
 *    [rows][words], words = wise_mask_words(s) = ceil(nb / 64); bit
 *    (kb & 63) of word kb >> 6 of row r is set iff key block kb belongs to
 *    that row's set.  Several masks "back to back" means mask i starts at
 *    element i * rows * words.
 *  - Alignment: q, k, v, o 16 bytes; workspace 256 bytes; masks, counts
 *    and fp64 arrays 8 bytes; every other pointer 4 bytes.  A misaligned
 *    pointer is WISE_ERR_SHAPE.
 */
#ifndef WISE_H
#define WISE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WISE_ABI_VERSION 6

typedef enum {
  WISE_OK = 0,
  WISE_ERR_NULL = 1,        /* a required pointer is NULL                    */
  WISE_ERR_SHAPE = 2,       /* non-positive dimension, seq_len % block != 0
                               (% 64 for blocks 16, 32), heads % kv_heads != 0,
                               a size that overflows int32 indexing, or a
                               misaligned pointer                            */
  WISE_ERR_UNSUPPORTED = 3, /* head_dim or block outside the supported set   */
  WISE_ERR_RANGE = 4,       /* tau outside (0, 1] / NaN, non-finite scale,
                               or unknown flag bit                           */
  WISE_ERR_WORKSPACE = 5,   /* workspace smaller than the size query returns */
  WISE_ERR_HIP = 6          /* a HIP launch reported an error                */
} wise_status;

/* Problem geometry shared by all calls.  scale <= 0 selects 1/sqrt(head_dim),
 * the softmax temperature of the paper's attention (Section 3, eq.
 * "recurrent_attention").  kv_heads: key-value heads for grouped-query
 * attention (the paper's second backbone shares 8 key-value heads among 32
 * query heads, Appendix B); 0 means kv_heads = heads; heads must be a
 * multiple of it. */
typedef struct {
  int32_t batch;
  int32_t heads;
  int32_t seq_len;
  int32_t head_dim;
  int32_t block;
  float scale;
  int32_t kv_heads;
} wise_shape;

/* Selection flags: blocks forced into every support after the cumulative-mass
 * cut.  The paper's own selection is flags = 0; the default used by this
 * library's callers is WISE_FORCE_SINK | WISE_FORCE_DIAG. */
enum {
  WISE_FORCE_SINK = 1u, /* key block 0 (the attention-sink block)     */
  WISE_FORCE_DIAG = 2u  /* key block qb (the causal diagonal block)   */
};

/*
 * wise_dense_attn_accum — full causal attention of one recurrent step,
 * optionally pooling its probabilities into block masses.
 *
 *   O = softmax(Q K^T * scale + M) V,  M the causal mask (key j <= query i)
 *       (Section 3, eq. "recurrent_attention")
 *   lse_i = log sum_{j<=i} exp(scale * q_i . k_j)      (natural log)
 *   if acc != NULL, for every kb <= qb:
 *     acc[b][h][qb][kb] += (1/block) * sum_{i in I_qb} sum_{j in I_kb, j<=i} A_ij
 *       (Section 5.1, eq. "block_attention_mass"); entries kb > qb untouched.
 *
 *   q       : bf16 [batch][heads][seq_len][head_dim], read-only.
 *   k, v    : bf16 [batch][kv_heads][seq_len][head_dim], read-only.
 *   o       : bf16, same shape as q, written.
 *   lse     : fp32 [batch][heads][seq_len] or NULL.
 *   acc     : fp32 [batch][heads][nb][nb] or NULL (plain dense attention).
 *             Read-modify-written in the same pass as the attention: the
 *             caller zeroes it before the first step it should sum.  Each
 *             acc row is owned by one work-group: no float atomics, bitwise
 *             deterministic.
 *   workspace, workspace_bytes : device scratch, 256-byte aligned, used
 *             only when acc != NULL (then required); contents on entry are
 *             ignored.  wise_mass_workspace_bytes(s) bytes let one launch
 *             cover every head; any smaller size down to
 *             wise_mass_workspace_min_bytes(s) (one key-value group of
 *             heads) runs the heads in consecutive launches of as many
 *             whole groups as fit, with the same results bit for bit.  It holds one fp32 per (query, 64-key span, or
 *             block-sized span for blocks 16 and 32, up to the query's tile)
 *             between the attention and its epilogue.
 * Errors: WISE_ERR_NULL (q, k, v, o NULL, or acc set with workspace NULL),
 *         WISE_ERR_SHAPE, WISE_ERR_UNSUPPORTED, WISE_ERR_WORKSPACE, WISE_ERR_HIP.
 */
wise_status wise_dense_attn_accum(const wise_shape* s, const void* q,
                                  const void* k, const void* v, void* o,
                                  float* lse, float* acc, void* workspace,
                                  size_t workspace_bytes, void* hip_stream);

/*
 * wise_select_support — per query block, the smallest set of key blocks whose
 * accumulated mass reaches tau of the row total (Section 5.1, eq.
 * "block_working_set", the arg-min over admissible blocks), plus the blocks
 * named in `flags`, emitted as CSR.
 *
 * Per row (b, h, qb), with v_kb = acc[b][h][qb][kb] for kb = 0..qb:
 *   1. order the candidates by (v descending, kb ascending);
 *   2. c_k = sum of the first k ordered masses, summed in that order in
 *      fp64 (c_0 = 0), total = c_{qb+1};
 *   3. k* = min{ k >= 0 : c_k >= tau * total }   (fp64);
 *   4. S = first k* ordered blocks  U  {0 if SINK}  U  {qb if DIAG};
 *      S empty (total == 0 and flags == 0) -> S = {qb};
 *   5. col_idx[row_ptr[r] .. row_ptr[r+1]) = S in ascending order.
 *
 *   acc       : fp32 [batch][heads][nb][nb], read-only (entries kb > qb ignored).
 *   tau       : 0 < tau <= 1.
 *   flags     : OR of WISE_FORCE_* bits.
 *   row_ptr   : int32 [rows + 1], rows = batch*heads*nb; row_ptr[0] = 0,
 *               row_ptr[rows] = nnz.
 *   col_idx   : int32 [wise_support_capacity(s)]; the first nnz are written.
 *   row_order : int32 [rows] or NULL: the schedule for wise_sparse_attn
 *               (Appendix B, "execution-metadata preparation"): rows grouped
 *               by (batch, head) in ascending order, and within a head by
 *               support size descending, ties by row id ascending.
 *   workspace : device scratch of at least wise_select_workspace_bytes(s)
 *               bytes; contents on entry are ignored.
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE, WISE_ERR_UNSUPPORTED, WISE_ERR_RANGE,
 *         WISE_ERR_WORKSPACE, WISE_ERR_HIP.
 */
wise_status wise_select_support(const wise_shape* s, const float* acc,
                                float tau, uint32_t flags, int32_t* row_ptr,
                                int32_t* col_idx, int32_t* row_order,
                                void* workspace, size_t workspace_bytes,
                                void* hip_stream);

/* Bytes of the library's own per-device selection scratch (see
 * wise_select_support_noalloc). */
#define WISE_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20)

/*
 * wise_select_support_noalloc — wise_select_support without a caller
 * workspace, for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc).
 *
 * Same selection, CSR, row order, arguments and errors as
 * wise_select_support, minus the workspace.  The per-row counts and
 * bitmasks live instead in a device array of WISE_NOALLOC_SCRATCH_BYTES
 * inside the library: every GPU the library runs on holds its own copy
 * until the process ends, and its address is looked up on the first call on
 * each device (the current device at the call).  The call performs no
 * allocation, free, memset or copy: it only enqueues the selection kernels.
 * Every row's scratch entries are written before they are read, so the
 * array's contents from earlier calls do not matter; but all calls on one
 * GPU share the array, so calls that overlap on one GPU (different streams
 * without ordering, different host threads) race and must not be issued.
 * Limit: wise_select_workspace_bytes(s) <= WISE_NOALLOC_SCRATCH_BYTES
 * (4 MiB: e.g. 28,160 rows of 128 blocks need 0.56 MiB), else
 * WISE_ERR_WORKSPACE and nothing is launched.
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE, WISE_ERR_UNSUPPORTED, WISE_ERR_RANGE,
 *         WISE_ERR_WORKSPACE, WISE_ERR_HIP (also a failed address lookup).
 */
wise_status wise_select_support_noalloc(const wise_shape* s, const float* acc,
                                        float tau, uint32_t flags,
                                        int32_t* row_ptr, int32_t* col_idx,
                                        int32_t* row_order, void* hip_stream);

/*
 * wise_sparse_attn — attention of one late recurrent step restricted to a
 * block support (Section 5.2, eq. "wise_attention"):
 *   O = softmax(Q K^T * scale + M + R) V,  R_ij = 0 if kb(j) in S_{qb(i)},
 *   -inf otherwise.  Q/K/V are this step's; only the support is reused.
 *
 *   q         : bf16 [batch][heads][seq_len][head_dim], read-only.
 *   k, v      : bf16 [batch][kv_heads][seq_len][head_dim], read-only.
 *   row_ptr   : int32 [rows + 1], col_idx : int32 [nnz] — a CSR whose rows
 *               list key-block ids in strictly ascending order with every id
 *               <= qb (as written by wise_select_support).  Ids outside
 *               0..qb are skipped on the device (never read out of bounds);
 *               ordering and uniqueness are trusted, not re-checked.
 *   row_order : int32 [rows], a permutation of 0..rows-1, or NULL for the
 *               identity.  Schedule slot s runs row row_order[s]; slots are
 *               dealt to the 8 XCDs in contiguous ranges (slot s on XCD
 *               s / (rows / 8) when rows % 8 == 0), so rows of one head placed
 *               together share an L2.
 *   o         : bf16, same shape as q, written.  A row with an empty support
 *               writes zeros (and lse = -inf).
 *   lse       : fp32 [batch][heads][seq_len] or NULL.
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE, WISE_ERR_UNSUPPORTED, WISE_ERR_HIP.
 */
wise_status wise_sparse_attn(const wise_shape* s, const void* q, const void* k,
                             const void* v, const int32_t* row_ptr,
                             const int32_t* col_idx, const int32_t* row_order,
                             void* o, float* lse, void* hip_stream);

/*
 * wise_sparse_attn_grouped — the same late step (Section 5.2, eq.
 * "wise_attention"), bit for bit the same outputs as wise_sparse_attn, run
 * by work-groups of wise_sparse_group_rows(s) consecutive query blocks of a
 * head (block 64: 4 at head_dim 128, 2 otherwise; block 128: 2 at head_dim
 * 128) over the union of their supports: each staged key tile serves all of
 * the group's rows that hold it, and every row attends only its own blocks.
 * Faster than wise_sparse_attn when consecutive rows' supports nearly
 * coincide (dense supports: measured 12% at density 0.91 with 4 rows of 64
 * keys, 10% at 0.95 with 2 rows), slower when they differ (27% slower at
 * density 0.43 with 4 rows); the caller picks, e.g. by the support's
 * density against the break-even of the group shape.  Where grouping is unavailable (block 16
 * or 32, block 128 below head_dim 128, more than 1024 key blocks, or
 * seq_len not a multiple of the group's queries: 256 at head_dim 128, else
 * 128; wise_sparse_group_rows(s) == 0) the call runs wise_sparse_attn's
 * kernel.  Arguments as wise_sparse_attn, without
 * row_order (groups are issued heaviest first, per head).
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE, WISE_ERR_UNSUPPORTED, WISE_ERR_HIP.
 */
wise_status wise_sparse_attn_grouped(const wise_shape* s, const void* q,
                                     const void* k, const void* v,
                                     const int32_t* row_ptr,
                                     const int32_t* col_idx, void* o,
                                     float* lse, void* hip_stream);

/* Query blocks per work-group of wise_sparse_attn_grouped: 4 or 2, or 0
 * where it runs wise_sparse_attn's kernel (-1 for an invalid shape). */
int32_t wise_sparse_group_rows(const wise_shape* s);

/*
 * wise_select_step — one discovery step's own support B_q^(t, eta), the set
 * that the paper's temporal union collects (Section 5.1, eq.
 * "block_working_set"), as a bitmask.
 *
 * Per row, steps 1-4 of wise_select_support on that step's masses with no
 * forced blocks (flags = 0): the heaviest k* blocks, k* the first prefix of
 * the (mass desc, block asc) order whose fp64 sum reaches tau of the row
 * total; an empty set (row total 0) becomes {qb}.
 *
 *   r     : fp32 [batch][heads][nb][nb], read-only: ONE step's block masses
 *           (wise_dense_attn_accum pooling into a zeroed buffer gives them).
 *   tau   : 0 < tau <= 1.
 *   mask  : uint64 [rows][words], every word written.
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE, WISE_ERR_UNSUPPORTED, WISE_ERR_RANGE,
 *         WISE_ERR_HIP.
 */
wise_status wise_select_step(const wise_shape* s, const float* r, float tau,
                             uint64_t* mask, void* hip_stream);

/*
 * wise_support_from_masks — the paper's working set of Section 5.1, eq.
 * "block_working_set": per row, the union of n_masks per-step sets (masks
 * back to back, e.g. the window steps t_d-3..t_d from wise_select_step),
 * plus the blocks named in `flags`, emitted as CSR and row order exactly as
 * wise_select_support emits them.  Bits of key blocks past the diagonal are
 * ignored; an empty union with flags = 0 becomes {qb}.
 *
 *   masks     : uint64 [n_masks][rows][words], read-only.  n_masks >= 1.
 *   flags, row_ptr, col_idx, row_order, workspace, workspace_bytes: as for
 *               wise_select_support (same workspace size).
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE (also n_masks < 1),
 *         WISE_ERR_UNSUPPORTED, WISE_ERR_RANGE, WISE_ERR_WORKSPACE, WISE_ERR_HIP.
 */
wise_status wise_support_from_masks(const wise_shape* s, const uint64_t* masks,
                                    int32_t n_masks, uint32_t flags,
                                    int32_t* row_ptr, int32_t* col_idx,
                                    int32_t* row_order, void* workspace,
                                    size_t workspace_bytes, void* hip_stream);

/*
 * wise_mask_union — out = bitwise OR of n_masks masks stored back to back:
 * the rolling working set W_q^(t) of Appendix C ("Stability of the Deployed
 * Working Set") when the masks are the per-step sets of steps
 * max(1, t-3)..t.
 *
 *   masks : uint64 [n_masks][rows][words], read-only.  n_masks >= 1.
 *   out   : uint64 [rows][words], written; it may coincide with one of the
 *           masks (each word is read before it is written), any other
 *           overlap is undefined.
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE (also n_masks < 1), WISE_ERR_HIP.
 */
wise_status wise_mask_union(const wise_shape* s, const uint64_t* masks,
                            int32_t n_masks, uint64_t* out, void* hip_stream);

/*
 * wise_mask_overlap — sizes of the intersection and union of two masks read
 * as sets of (row, key block): counts[0] = |A & B|, counts[1] = |A | B|.
 * Their ratio is the adjacent rolling-set Jaccard J_roll of Appendix C
 * ("Stability of the Deployed Working Set") for A = W^(t-1), B = W^(t).
 *
 *   a, b   : uint64 [rows][words], read-only.
 *   counts : int64 [2], device, written.
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE, WISE_ERR_HIP.
 */
wise_status wise_mask_overlap(const wise_shape* s, const uint64_t* a,
                              const uint64_t* b, int64_t* counts,
                              void* hip_stream);

/*
 * wise_support_mass — attention mass a block support retains from one step
 * of unrestricted attention: the retained future full-attention mass of
 * Section 7.1 and Appendix B (evaluation metrics), computed from that step's
 * block masses r (eq. "block_attention_mass").  Since each query's
 * probabilities sum to 1, sum_rows inside / sum_rows total is the fraction
 * of all causal attention mass that falls inside the support.
 *
 *   r        : fp32 [batch][heads][nb][nb], read-only: one step's masses.
 *   row_ptr, col_idx : a CSR support as for wise_sparse_attn (ids outside
 *              0..qb are skipped).
 *   row_mass : fp64 [rows][2], written: (sum of r[row][kb] over the row's
 *              blocks, sum of r[row][kb] over kb <= qb), each summed in fp64
 *              in a fixed order (bitwise reproducible).
 *   totals   : fp64 [2] or NULL, written: the two columns of row_mass summed
 *              over all rows, in a fixed order.
 * Errors: WISE_ERR_NULL, WISE_ERR_SHAPE, WISE_ERR_HIP.
 */
wise_status wise_support_mass(const wise_shape* s, const float* r,
                              const int32_t* row_ptr, const int32_t* col_idx,
                              double* row_mass, double* totals,
                              void* hip_stream);

/* Bytes of device workspace wise_dense_attn_accum needs when it pools block
 * masses: one fp32 per (query, E-key span up to the end of its tile of T
 * queries), E = block for blocks 16 and 32 and 64 otherwise, T = 256 for head_dim 128
 * when it divides seq_len, else 128 when it divides seq_len, else 64:
 * batch * heads * T * (T / E) * m (m + 1) / 2 * 4 with m = seq_len / T
 * (about half of seq_len^2 / E floats per head; 0 for an invalid shape). */
size_t wise_mass_workspace_bytes(const wise_shape* s);

/* The smallest workspace wise_dense_attn_accum accepts with acc != NULL:
 * wise_mass_workspace_bytes(s) / (batch * heads) * (heads / kv_heads), the
 * share of one key-value group of query heads (0 for an invalid shape). */
size_t wise_mass_workspace_min_bytes(const wise_shape* s);

/* 64-bit words per row of a support bitmask: ceil(nb / 64)
 * (-1 for an invalid shape). */
int32_t wise_mask_words(const wise_shape* s);

/* Bytes of device workspace wise_select_support needs for shape s
 * (0 for an invalid shape). */
size_t wise_select_workspace_bytes(const wise_shape* s);

/* Upper bound on nnz: batch * heads * nb * (nb + 1) / 2, the number of
 * causally admissible block pairs (-1 for an invalid shape). */
int64_t wise_support_capacity(const wise_shape* s);

/* Static, NUL-terminated description of a status code. */
const char* wise_status_string(wise_status st);

/* WISE_ABI_VERSION of the loaded library. */
int32_t wise_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WISE_H */
