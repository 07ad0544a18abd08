// block_mass.hip — block-pooled softmax mass (paper Section 5.1, eq.
// block_attention_mass): acc[qb][kb] += r_qb,kb, the mean over the block's
// queries of the attention probability that falls in key block kb.  The
// kernel recomputes S = Q K^T against the row log-sum-exp the dense kernel
// wrote, so a probability is exp(s * scale - lse) with no second softmax
// pass.
//
// One work-group per (batch, head, query block), NW = block/32 waves, each
// wave 32 queries.  With 32-key blocks a 64-key tile spans two key blocks,
// and the wave pools each half of its scores into its own block.  S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = K from
// LDS, B = Q^T in registers), so every lane holds 32 scores of one query.
// K tiles of 64 keys are staged global -> registers -> LDS, the loads of
// the next tile issued before the current one is computed.  The group owns
// its acc row, so the read-modify-write needs no atomics and the reduction
// order is fixed.
#include "wise_device.hpp"
#include "wise_kernels.hpp"

namespace wise {

namespace {

constexpr int kMassKStride(int d) { return d + 8; }   // LDS K row stride (bf16): 16 B pad

// Global -> register -> LDS staging of one 64-key K tile.
template <int D, int NT>
struct KStage {
  static constexpr int kRowChunks = D / 8;                    // 16-B chunks per key row
  static constexpr int kChunks = kKeyTile * kRowChunks;
  static constexpr int kPer = (kChunks + NT - 1) / NT;
  static constexpr int kStride = kMassKStride(D);

  u32x4_t kr[kPer];

  __device__ __forceinline__ static int chunk(int tid, int i) { return tid + i * NT; }
  __device__ __forceinline__ static bool live(int tid, int i) {
    return kChunks % NT == 0 || chunk(tid, i) < kChunks;
  }

  __device__ __forceinline__ void load(const uint16_t* kt, int tid) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (live(tid, i)) {
        const int ch = chunk(tid, i);
        const uint32_t off = (uint32_t)((ch / kRowChunks) * D + (ch % kRowChunks) * 8);
        kr[i] = *(const u32x4_t*)(kt + off);
      }
    }
  }

  __device__ __forceinline__ void store(uint16_t* ks, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (live(tid, i)) {
        const int ch = chunk(tid, i);
        const int key = ch / kRowChunks, c8 = (ch % kRowChunks) * 8;
        *(u32x4_t*)(ks + key * kStride + c8) = kr[i];
      }
    }
  }
};

// Tile-local key of register r of S^T tile t in a lane of half-wave h (K
// rows stored in natural order: MFMA row m is key m).
__device__ __forceinline__ int mass_key(int t, int r, int h) {
  return 32 * t + 8 * (r >> 2) + 4 * h + (r & 3);
}

}  // namespace

template <int D, int NW>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
block_mass_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                  const float* __restrict__ lse, float* __restrict__ acc, int n, int nb,
                  int heads, int gq, Sched sc, float c) {
  constexpr int kNT = NW * 64, kB = NW * 32;
  constexpr int kStride = kMassKStride(D);
  __shared__ __attribute__((aligned(16))) uint16_t ks[kKeyTile * kStride];
  __shared__ float red[NW];
  int bh, item;
  if (!sched_slot(sc, bh, item)) return;
  const int qb = nb - 1 - item;   // the last (longest) query blocks first
  const size_t hoff = (size_t)bh * n * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q0 = qb * kB + 32 * wave;
  const int qi = q0 + (lane & 31);
  float* arow = acc + ((size_t)bh * nb + qb) * nb;

  // Q^T B-operand fragments, one per 16-dim chunk.
  u32x4_t qf[D / 16];
  {
    const uint16_t* row = Q + hoff + (size_t)qi * D + 8 * (lane >> 5);
#pragma unroll
    for (int k = 0; k < D / 16; ++k) qf[k] = *(const u32x4_t*)(row + 16 * k);
  }
  const float nl = -lse[(size_t)bh * n + qi] * kLog2e;   // -log2 of the row normaliser
  const uint16_t* Kh = K + (size_t)kv_head(bh, heads, gq) * n * D;
  KStage<D, kNT> st;
  st.load(Kh, tid);
  if constexpr (kB == 32) {
    // Tile it holds key blocks 2it (s[0]) and 2it+1 (s[1]); keys past the
    // query are masked, which also drops a block 2it+1 > qb whole.
    const int ntiles = (qb + 2) / 2;
    for (int it = 0; it < ntiles; ++it) {
      st.store(ks, tid);
      __syncthreads();
      if (it + 1 < ntiles) st.load(Kh + (size_t)(it + 1) * kKeyTile * D, tid);
      const int key0 = it * kKeyTile;
      const uint16_t* a0 = ks + (lane & 31) * kStride + 8 * (lane >> 5);
      const uint16_t* a1 = a0 + 32 * kStride;
      f32x16_t s[2] = {f32x16_t{}, f32x16_t{}};
#pragma unroll
      for (int k = 0; k < D / 16; ++k) {
        s[0] = mfma32x32x16(*(const u32x4_t*)(a0 + 16 * k), qf[k], s[0]);
        s[1] = mfma32x32x16(*(const u32x4_t*)(a1 + 16 * k), qf[k], s[1]);
      }
      const bool diag = key0 + kKeyTile - 1 > q0;
      float part[2] = {0.f, 0.f};
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool keep = !diag || key0 + mass_key(t, r, lane >> 5) <= qi;
          part[t] += keep ? fast_exp2(__builtin_fmaf(s[t][r], c, nl)) : 0.f;
        }
      const float b0 = wave_sum(part[0]), b1 = wave_sum(part[1]);
      if (lane == 0) {
        arow[2 * it] += b0 * (1.f / kB);
        if (2 * it + 1 <= qb) arow[2 * it + 1] += b1 * (1.f / kB);
      }
      __syncthreads();
    }
    return;
  }
  constexpr int kTPB = kB / kKeyTile;
  const int ntiles = (qb + 1) * kTPB;
  float blk = 0.f;
  for (int it = 0; it < ntiles; ++it) {
    st.store(ks, tid);
    __syncthreads();
    if (it + 1 < ntiles) st.load(Kh + (size_t)(it + 1) * kKeyTile * D, tid);
    const int key0 = it * kKeyTile;
    float part = 0.f;
    if (key0 <= q0) {
      const uint16_t* a0 = ks + (lane & 31) * kStride + 8 * (lane >> 5);
      const uint16_t* a1 = a0 + 32 * kStride;
      f32x16_t s[2] = {f32x16_t{}, f32x16_t{}};
#pragma unroll
      for (int k = 0; k < D / 16; ++k) {
        s[0] = mfma32x32x16(*(const u32x4_t*)(a0 + 16 * k), qf[k], s[0]);
        s[1] = mfma32x32x16(*(const u32x4_t*)(a1 + 16 * k), qf[k], s[1]);
      }
      const bool diag = it >= qb * kTPB && key0 + kKeyTile - 1 > q0;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool keep = !diag || key0 + mass_key(t, r, lane >> 5) <= qi;
          part += keep ? fast_exp2(__builtin_fmaf(s[t][r], c, nl)) : 0.f;
        }
    }
    blk += wave_sum(part);
    const bool last = (it % kTPB) == kTPB - 1;
    if (last && lane == 0) red[wave] = blk;
    __syncthreads();
    if (last) {
      if (tid == 0) {
        float tot = 0.f;
#pragma unroll
        for (int i = 0; i < NW; ++i) tot += red[i];
        arow[it / kTPB] += tot * (1.f / kB);
      }
      blk = 0.f;
    }
  }
}

template <int D>
static hipError_t launch_mass_d(const Dims& s, const void* q, const void* k, const float* lse,
                                float* acc, hipStream_t st) {
  const float c = s.scale * kLog2e;
  const auto* Q = (const uint16_t*)q;
  const auto* K = (const uint16_t*)k;
  const Sched sc = make_sched(s.bh, s.nb, (size_t)s.n * D * 2 / s.gq);
  const dim3 grid(sched_grid(sc));
  if (s.block == 32)
    hipLaunchKernelGGL((block_mass_kernel<D, 1>), grid, dim3(64), 0, st, Q, K, lse, acc, s.n,
                       s.nb, s.heads, s.gq, sc, c);
  else if (s.block == 64)
    hipLaunchKernelGGL((block_mass_kernel<D, 2>), grid, dim3(128), 0, st, Q, K, lse, acc, s.n,
                       s.nb, s.heads, s.gq, sc, c);
  else
    hipLaunchKernelGGL((block_mass_kernel<D, 4>), grid, dim3(256), 0, st, Q, K, lse, acc, s.n,
                       s.nb, s.heads, s.gq, sc, c);
  return hipGetLastError();
}

hipError_t launch_mass(const Dims& s, const void* q, const void* k, const float* lse, float* acc,
                       hipStream_t st) {
  switch (s.d) {
    case 64: return launch_mass_d<64>(s, q, k, lse, acc, st);
    case 96: return launch_mass_d<96>(s, q, k, lse, acc, st);
    default: return launch_mass_d<128>(s, q, k, lse, acc, st);
  }
}

}  // namespace wise
