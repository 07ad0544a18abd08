// select.hip — support selection and CSR schedule construction on gfx950.
//
// Paper Section 5.1, eq. (block_working_set): per query block, the smallest
// set of admissible key blocks whose mass reaches the threshold, i.e. the
// heaviest k* blocks with k* the first prefix of the descending order that
// reaches tau * total.  The schedule is a device-resident CSR (Appendix B,
// "Sparse-kernel implementation") plus a longest-support-first row order.
//
//   select_rows_kernel   one wave per row: rank every candidate by
//                        (mass desc, block asc), sum the ordered masses
//                        sequentially in fp64 (the same association as a
//                        left-to-right prefix sum), cut, add forced blocks,
//                        emit a bitmask and a count
//   scan_kernel          exclusive scan of counts -> row_ptr
//   scatter_kernel       bitmask -> ascending col_idx
//   order_kernel         per (batch, head): its rows by count descending
//                        (ties by row id), heads in ascending order
//
// The paper's own working set (Section 5.1, eq. block_working_set) is the
// union over the discovery window of per-step sets B_q^(t, eta).  For it the
// per-row kernel runs on one step's masses with no forced blocks and leaves
// the step's bitmask with the caller; union_rows_kernel ORs any number of
// such masks, adds the forced blocks, and feeds the same scan / scatter /
// order kernels.  Two diagnostics close the file: the (intersection, union)
// sizes of two masks (the adjacent rolling-set Jaccard of Appendix C,
// "Stability of the Deployed Working Set") and the attention mass a support
// retains from one step's block masses (Section 7.1 and Appendix B, the
// retained future full-attention mass).
#include <mutex>

#include "wise.h"
#include "wise_device.hpp"
#include "wise_kernels.hpp"

namespace wise {

constexpr int kSelWaves = 4;        // rows per work-group in the per-row kernels
constexpr int kOrderThreads = 256;

// Orderable 32-bit image of a float: unsigned order == float order.
__device__ __forceinline__ uint32_t float_key(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// E = candidates per lane (ceil(nb / 64) rounded up to a power of two).
template <int E>
__global__ void __launch_bounds__(kSelWaves * 64)
select_rows_kernel(const float* __restrict__ acc, int rows, int nb, double tau, uint32_t flags,
                   int32_t* __restrict__ counts, uint64_t* __restrict__ masks, int words) {
  extern __shared__ __attribute__((aligned(16))) uint64_t sel_smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = blockIdx.x * kSelWaves + wave;
  const bool active = row < rows;
  uint64_t* keys = sel_smem + (size_t)wave * 2 * nb;   // [nb] sort keys, later prefixes
  double* sv = (double*)(keys + nb);                    // [nb] masses in sorted order
  const int qb = active ? row % nb : 0;
  const int cnt = active ? qb + 1 : 0;
  const float* v = acc + (size_t)(active ? row : 0) * nb;

  // 1. composite keys: mass descending, then block index ascending
  float x[E];
  uint64_t key[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int b = lane + 64 * e;
    x[e] = 0.f;
    key[e] = 0;
    if (b < cnt) {
      x[e] = v[b];
      key[e] = ((uint64_t)float_key(x[e]) << 32) | (uint32_t)(~(uint32_t)b);
      keys[b] = key[e];
    }
  }
  __syncthreads();
  // 2. rank = number of candidates ordered before this one
  int rank[E];
#pragma unroll
  for (int e = 0; e < E; ++e) rank[e] = 0;
  for (int c = 0; c < cnt; ++c) {
    const uint64_t kc = keys[c];
#pragma unroll
    for (int e = 0; e < E; ++e) rank[e] += (kc > key[e]) ? 1 : 0;
  }
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (lane + 64 * e < cnt) sv[rank[e]] = (double)x[e];
  __syncthreads();
  // 3. sequential fp64 prefix sums in sorted order (identical in every lane)
  double* pre = (double*)keys;
  double run = 0.0;
  for (int r = 0; r < cnt; ++r) {
    run += sv[r];
    if (lane == 0) pre[r] = run;
  }
  __syncthreads();
  // 4. k* = min{k >= 0 : c_k >= tau * total}, c_0 = 0
  const double thr = tau * run;
  int kstar = cnt;
  if (thr <= 0.0) {
    kstar = 0;
  } else {
    for (int r = lane; r < cnt; r += 64)
      if (pre[r] >= thr) { kstar = min(kstar, r + 1); break; }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) kstar = min(kstar, __shfl_xor(kstar, off, 64));
  }
  // 5. selection bitmask, forced blocks, empty -> diagonal
  int total = 0;
  uint64_t mword[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int b = lane + 64 * e;
    bool s = false;
    if (b < cnt)
      s = rank[e] < kstar || (b == 0 && (flags & 1u)) || (b == qb && (flags & 2u));
    mword[e] = __builtin_amdgcn_ballot_w64(s);
    total += __builtin_popcountll(mword[e]);
  }
  if (total == 0) {
    mword[qb >> 6] |= 1ull << (qb & 63);
    total = 1;
  }
  if (active && lane == 0) {
    if (counts != nullptr) counts[row] = total;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (e < words) masks[(size_t)row * words + e] = mword[e];
  }
}

// Inclusive scan of one value per thread over a 1024-thread block.
__device__ __forceinline__ int block_scan_1024(int x, int* wsum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (wave == 0) {
    int w = lane < 16 ? wsum[lane] : 0;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const int y = __shfl_up(w, off, 64);
      if (lane >= off) w += y;
    }
    if (lane < 16) wsum[lane] = w;
  }
  __syncthreads();
  const int add = wave > 0 ? wsum[wave - 1] : 0;
  __syncthreads();
  return x + add;
}

// row_ptr[0] = 0, row_ptr[r+1] = counts[0] + ... + counts[r].
__global__ void __launch_bounds__(1024)
scan_kernel(const int32_t* __restrict__ counts, int rows, int32_t* __restrict__ row_ptr) {
  __shared__ int wsum[16];
  __shared__ int carry;
  if (threadIdx.x == 0) {
    carry = 0;
    row_ptr[0] = 0;
  }
  __syncthreads();
  for (int base = 0; base < rows; base += 1024) {
    const int r = base + threadIdx.x;
    const int x = r < rows ? counts[r] : 0;
    const int inc = block_scan_1024(x, wsum);
    const int c0 = carry;
    if (r < rows) row_ptr[r + 1] = c0 + inc;
    __syncthreads();
    if (threadIdx.x == 1023) carry = c0 + inc;
    __syncthreads();
  }
}

// col_idx[row_ptr[r] ..] = set bits of the row's mask, ascending.
__global__ void __launch_bounds__(kSelWaves * 64)
scatter_kernel(const uint64_t* __restrict__ masks, const int32_t* __restrict__ row_ptr, int rows,
               int words, int32_t* __restrict__ col_idx) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kSelWaves + (threadIdx.x >> 6);
  if (row >= rows) return;
  int pos = row_ptr[row];
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int e = 0; e < words; ++e) {
    const uint64_t m = masks[(size_t)row * words + e];
    if ((m >> lane) & 1ull) col_idx[pos + __builtin_popcountll(m & below)] = 64 * e + lane;
    pos += __builtin_popcountll(m);
  }
}

// Row order: one work-group per (batch, head).  Row r of the head lands at
// rank(r) = #{rows with a larger count} + #{earlier rows with the same count}.
__global__ void __launch_bounds__(kOrderThreads)
order_kernel(const int32_t* __restrict__ counts, int nb, int32_t* __restrict__ order) {
  extern __shared__ int32_t o_smem[];
  const int base = blockIdx.x * nb;
  for (int r = threadIdx.x; r < nb; r += kOrderThreads) o_smem[r] = counts[base + r];
  __syncthreads();
  for (int r = threadIdx.x; r < nb; r += kOrderThreads) {
    const int c = o_smem[r];
    int rank = 0;
    for (int t = 0; t < nb; ++t) {
      const int ct = o_smem[t];
      rank += (ct > c || (ct == c && t < r)) ? 1 : 0;
    }
    order[base + rank] = base + r;
  }
}

// Workspace layout: counts | masks, each 256-B aligned.
struct SelectWs {
  size_t counts, masks, total;
  int words;
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int mask_words(const Dims& s) { return (s.nb + 63) / 64; }

static SelectWs select_ws(const Dims& s) {
  SelectWs w;
  const size_t rows = (size_t)s.bh * s.nb;
  w.words = mask_words(s);
  w.counts = 0;
  w.masks = align256(w.counts + rows * 4);
  w.total = align256(w.masks + rows * w.words * 8);
  return w;
}

size_t select_workspace_bytes(const Dims& s) { return select_ws(s).total; }

// Per-row selection of every row: counts (may be null) and bitmasks.
static void launch_rows(const Dims& s, const float* acc, float tau, uint32_t flags,
                        int32_t* counts, uint64_t* masks, hipStream_t st) {
  const int rows = s.bh * s.nb, words = mask_words(s);
  const int groups = (rows + kSelWaves - 1) / kSelWaves;
  const size_t smem = (size_t)kSelWaves * 2 * s.nb * sizeof(uint64_t);
  const dim3 sg(groups), sb(kSelWaves * 64);
  const double dtau = (double)tau;
  if (s.nb <= 64)
    hipLaunchKernelGGL(select_rows_kernel<1>, sg, sb, smem, st, acc, rows, s.nb, dtau, flags, counts, masks, words);
  else if (s.nb <= 128)
    hipLaunchKernelGGL(select_rows_kernel<2>, sg, sb, smem, st, acc, rows, s.nb, dtau, flags, counts, masks, words);
  else if (s.nb <= 256)
    hipLaunchKernelGGL(select_rows_kernel<4>, sg, sb, smem, st, acc, rows, s.nb, dtau, flags, counts, masks, words);
  else if (s.nb <= 512)
    hipLaunchKernelGGL(select_rows_kernel<8>, sg, sb, smem, st, acc, rows, s.nb, dtau, flags, counts, masks, words);
  else
    hipLaunchKernelGGL(select_rows_kernel<16>, sg, sb, smem, st, acc, rows, s.nb, dtau, flags, counts, masks, words);
}

// counts + masks (in the workspace) -> row_ptr, col_idx, row_order.
static void launch_csr(const Dims& s, const int32_t* counts, const uint64_t* masks,
                       int32_t* row_ptr, int32_t* col_idx, int32_t* row_order, hipStream_t st) {
  const int rows = s.bh * s.nb;
  const int groups = (rows + kSelWaves - 1) / kSelWaves;
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(1024), 0, st, counts, rows, row_ptr);
  hipLaunchKernelGGL(scatter_kernel, dim3(groups), dim3(kSelWaves * 64), 0, st, masks, row_ptr,
                     rows, mask_words(s), col_idx);
  if (row_order != nullptr)
    hipLaunchKernelGGL(order_kernel, dim3(s.bh), dim3(kOrderThreads), (size_t)s.nb * sizeof(int32_t),
                       st, counts, s.nb, row_order);
}

hipError_t launch_select(const Dims& s, const float* acc, float tau, uint32_t flags,
                         int32_t* row_ptr, int32_t* col_idx, int32_t* row_order, void* ws,
                         hipStream_t st) {
  const SelectWs w = select_ws(s);
  char* base = (char*)ws;
  auto* counts = (int32_t*)(base + w.counts);
  auto* masks = (uint64_t*)(base + w.masks);
  launch_rows(s, acc, tau, flags, counts, masks, st);
  launch_csr(s, counts, masks, row_ptr, col_idx, row_order, st);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Selection with no caller workspace (wise_select_support_noalloc): the
// per-row counts and bitmasks live in `scratch`, a file-scope device array of
// WISE_NOALLOC_SCRATCH_BYTES that every GPU the library runs on holds until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory, so kernels only ever receive the address the runtime
// reports for the current device, looked up once per device.  Every row's
// count and mask words are written before they are read, so nothing in the
// array needs clearing; calls that overlap on one device share it and race.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[WISE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex scratch_mutex;
static void* scratch_addr[kMaxDevices];

static hipError_t device_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    scratch_addr[dev] = p;
  }
  *out = scratch_addr[dev];
  return hipSuccess;
}

hipError_t launch_select_noalloc(const Dims& s, const float* acc, float tau, uint32_t flags,
                                 int32_t* row_ptr, int32_t* col_idx, int32_t* row_order,
                                 hipStream_t st) {
  if (select_workspace_bytes(s) > (size_t)WISE_NOALLOC_SCRATCH_BYTES) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = device_scratch(&ws);
  if (e != hipSuccess) return e;
  return launch_select(s, acc, tau, flags, row_ptr, col_idx, row_order, ws, st);
}

// ---------------------------------------------------------------------------
// Temporal union of per-step supports
// ---------------------------------------------------------------------------

hipError_t launch_select_step(const Dims& s, const float* r, float tau, uint64_t* mask,
                              hipStream_t st) {
  launch_rows(s, r, tau, 0u, nullptr, mask, st);
  return hipGetLastError();
}

constexpr int kMaskThreads = 256;

// One thread per row: OR of the row's words over every mask, bits past the
// diagonal dropped, forced blocks added, an empty row given its diagonal.
__global__ void __launch_bounds__(kMaskThreads)
union_rows_kernel(const uint64_t* __restrict__ masks, int n_masks, size_t slab, int rows, int nb,
                  int words, uint32_t flags, int32_t* __restrict__ counts,
                  uint64_t* __restrict__ out) {
  const int row = blockIdx.x * kMaskThreads + threadIdx.x;
  if (row >= rows) return;
  const int qb = row % nb;
  const size_t base = (size_t)row * words;
  int total = 0;
  for (int w = 0; w < words; ++w) {
    uint64_t m = 0;
    for (int i = 0; i < n_masks; ++i) m |= masks[(size_t)i * slab + base + w];
    const int lo = 64 * w;
    const uint64_t keep = qb < lo ? 0ull : (qb - lo >= 63 ? ~0ull : (~0ull >> (63 - (qb - lo))));
    m &= keep;
    if (w == 0 && (flags & 1u)) m |= 1ull;
    if (w == (qb >> 6) && (flags & 2u)) m |= 1ull << (qb & 63);
    out[base + w] = m;
    total += __builtin_popcountll(m);
  }
  if (total == 0) {
    out[base + (qb >> 6)] = 1ull << (qb & 63);
    total = 1;
  }
  counts[row] = total;
}

hipError_t launch_support_from_masks(const Dims& s, const uint64_t* masks, int n_masks,
                                     uint32_t flags, int32_t* row_ptr, int32_t* col_idx,
                                     int32_t* row_order, void* ws, hipStream_t st) {
  const SelectWs w = select_ws(s);
  char* base = (char*)ws;
  auto* counts = (int32_t*)(base + w.counts);
  auto* umask = (uint64_t*)(base + w.masks);
  const int rows = s.bh * s.nb;
  const size_t slab = (size_t)rows * w.words;
  hipLaunchKernelGGL(union_rows_kernel, dim3((rows + kMaskThreads - 1) / kMaskThreads),
                     dim3(kMaskThreads), 0, st, masks, n_masks, slab, rows, s.nb, w.words, flags,
                     counts, umask);
  launch_csr(s, counts, umask, row_ptr, col_idx, row_order, st);
  return hipGetLastError();
}

// out[x] = OR over i of masks[i * slab + x]; out may be one of the masks.
__global__ void __launch_bounds__(kMaskThreads)
mask_union_kernel(const uint64_t* masks, int n_masks, size_t slab, uint64_t* out) {
  for (size_t x = (size_t)blockIdx.x * kMaskThreads + threadIdx.x; x < slab;
       x += (size_t)gridDim.x * kMaskThreads) {
    uint64_t m = 0;
    for (int i = 0; i < n_masks; ++i) m |= masks[(size_t)i * slab + x];
    out[x] = m;
  }
}

hipError_t launch_mask_union(const Dims& s, const uint64_t* masks, int n_masks, uint64_t* out,
                             hipStream_t st) {
  const size_t slab = (size_t)s.bh * s.nb * mask_words(s);
  const size_t blocks = (slab + kMaskThreads - 1) / kMaskThreads;
  hipLaunchKernelGGL(mask_union_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)),
                     dim3(kMaskThreads), 0, st, masks, n_masks, slab, out);
  return hipGetLastError();
}

// Sum over a 1024-thread block; the result is valid in thread 0.
template <typename T>
__device__ __forceinline__ T block_sum_1024(T x, T* wsum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  if (lane == 0) wsum[wave] = x;
  __syncthreads();
  T t = 0;
  if (threadIdx.x == 0)
    for (int i = 0; i < 16; ++i) t += wsum[i];
  return t;
}

// counts[0] = |A & B|, counts[1] = |A | B| (set bits), one work-group.
__global__ void __launch_bounds__(1024)
mask_overlap_kernel(const uint64_t* __restrict__ a, const uint64_t* __restrict__ b, size_t slab,
                    int64_t* __restrict__ counts) {
  __shared__ long long wsum[16];
  long long inter = 0, uni = 0;
  for (size_t x = threadIdx.x; x < slab; x += 1024) {
    const uint64_t p = a[x], q = b[x];
    inter += __builtin_popcountll(p & q);
    uni += __builtin_popcountll(p | q);
  }
  const long long ti = block_sum_1024(inter, wsum);
  __syncthreads();
  const long long tu = block_sum_1024(uni, wsum);
  if (threadIdx.x == 0) {
    counts[0] = ti;
    counts[1] = tu;
  }
}

hipError_t launch_mask_overlap(const Dims& s, const uint64_t* a, const uint64_t* b,
                               int64_t* counts, hipStream_t st) {
  const size_t slab = (size_t)s.bh * s.nb * mask_words(s);
  hipLaunchKernelGGL(mask_overlap_kernel, dim3(1), dim3(1024), 0, st, a, b, slab, counts);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Retained attention mass of a support
// ---------------------------------------------------------------------------

// One wave per row: row_mass[row] = (sum of r over the row's CSR blocks
// kb <= qb, sum of r over kb <= qb), in fp64, lane-strided then a fixed
// butterfly, so the result is bitwise reproducible.
__global__ void __launch_bounds__(kSelWaves * 64)
row_mass_kernel(const float* __restrict__ r, const int32_t* __restrict__ row_ptr,
                const int32_t* __restrict__ col_idx, int rows, int nb,
                double* __restrict__ row_mass) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kSelWaves + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int qb = row % nb;
  const float* v = r + (size_t)row * nb;
  double inside = 0.0, total = 0.0;
  for (int kb = lane; kb <= qb; kb += 64) total += (double)v[kb];
  for (int e = row_ptr[row] + lane; e < row_ptr[row + 1]; e += 64) {
    const int kb = col_idx[e];
    if (kb >= 0 && kb <= qb) inside += (double)v[kb];
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    inside += __shfl_xor(inside, off, 64);
    total += __shfl_xor(total, off, 64);
  }
  if (lane == 0) {
    row_mass[2 * (size_t)row] = inside;
    row_mass[2 * (size_t)row + 1] = total;
  }
}

__global__ void __launch_bounds__(1024)
mass_total_kernel(const double* __restrict__ row_mass, int rows, double* __restrict__ totals) {
  __shared__ double wsum[16];
  double inside = 0.0, total = 0.0;
  for (int x = threadIdx.x; x < rows; x += 1024) {
    inside += row_mass[2 * (size_t)x];
    total += row_mass[2 * (size_t)x + 1];
  }
  const double ti = block_sum_1024(inside, wsum);
  __syncthreads();
  const double tt = block_sum_1024(total, wsum);
  if (threadIdx.x == 0) {
    totals[0] = ti;
    totals[1] = tt;
  }
}

hipError_t launch_support_mass(const Dims& s, const float* r, const int32_t* row_ptr,
                               const int32_t* col_idx, double* row_mass, double* totals,
                               hipStream_t st) {
  const int rows = s.bh * s.nb;
  hipLaunchKernelGGL(row_mass_kernel, dim3((rows + kSelWaves - 1) / kSelWaves),
                     dim3(kSelWaves * 64), 0, st, r, row_ptr, col_idx, rows, s.nb, row_mass);
  if (totals != nullptr)
    hipLaunchKernelGGL(mass_total_kernel, dim3(1), dim3(1024), 0, st, row_mass, rows, totals);
  return hipGetLastError();
}

}  // namespace wise
