// attention.hip — the attention kernels of libwise on gfx950:
//
//   dense_attn_kernel   causal flash attention, O and natural-log LSE
//                       (paper Section 3, eq. recurrent_attention), and
//                       optionally the block-pooled attention mass
//                       (Section 5.1, eq. block_attention_mass)
//   sparse_attn_kernel  attention restricted to a CSR block support
//   sparse_group_kernel (Section 5.2, eq. wise_attention): one work-group
//   sparse_row16_kernel per row; groups of consecutive rows over the union
//                       of their supports (the same outputs, for dense
//                       supports); one wave per row of 16-key blocks
//
// Shared tile engine.  A wave owns 32 consecutive queries.  For each tile of
// 64 keys (32 for 32-key blocks) it computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (A = K from
// LDS, B = Q^T held in registers for the whole row), so every lane ends up
// holding 32 scores of ONE query.  The row max needs one cross-lane step
// (lanes l and l^32 share a query), the row sum none until the end, and the
// probabilities are already in the B-operand layout of O^T = V^T P^T: they are
// packed to bf16 in place and fed straight to the second MFMA chain.  V stays
// row-major in LDS and its A-operand fragments are read transposed with
// ds_read_b64_tr_b16; the 32-byte row pad makes those reads, like the 128-bit
// K reads, free of bank conflicts.  Softmax is
// online in base 2 with the exact running max (so the largest probability of
// a row is exactly 1 in bf16); the O rescale is skipped, wave-uniformly, on
// tiles that raise no row's max.
//
// Work order: see sched_slot (heaviest items of every head first, heads
// grouped per XCD).
#include "wise_device.hpp"
#include "wise_kernels.hpp"

namespace wise {

// ---------------------------------------------------------------------------
// Global -> register -> LDS staging of one tile of KT keys (64, or 32 for
// 32-key blocks; K rows permuted so the S^T accumulator comes out in PV
// operand order; V rows in natural order).  Loads for the next tile are
// issued before the current one is computed, so the memory latency hides
// behind the MFMA work; stores go to an LDS tile no wave still reads: after
// the barrier that retires it, or, in the 8-wave dense group, into its
// second buffer.
// ---------------------------------------------------------------------------
template <int D, int NT, bool kWithV, int KT = kKeyTile>
struct TileStage {
  using G = Geo<D>;
  static_assert(KT == 32 || KT == 64, "key tile");
  static constexpr int kRowChunks = D / 8;                    // 16-B chunks per key row
  static constexpr int kChunks = KT * kRowChunks;             // per tensor
  static constexpr int kPer = (kChunks + NT - 1) / NT;

  u32x4_t kr[kPer];
  u32x4_t vr[kWithV ? kPer : 1];

  // Chunk i of this thread: key row ch / kRowChunks, column (ch % kRowChunks) * 8.
  __device__ __forceinline__ static int chunk(int tid, int i) { return tid + i * NT; }
  __device__ __forceinline__ static bool live(int tid, int i) {
    return kChunks % NT == 0 || chunk(tid, i) < kChunks;
  }

  // rk, rv: the head's K and V; key0: this tile's first key row (uniform,
  // a scalar byte offset), per-lane offsets constant across tiles.
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                       int key0, int tid) {
    const uint32_t soff = (uint32_t)key0 * (D * 2);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (live(tid, i)) {
        const int ch = chunk(tid, i);
        const uint32_t off = (uint32_t)((ch / kRowChunks) * D + (ch % kRowChunks) * 8) * 2;
        kr[i] = buffer_load16(rk, off, soff);
        if constexpr (kWithV) vr[i] = buffer_load16(rv, off, soff);
      }
    }
  }

  __device__ __forceinline__ void store(uint16_t* ks, uint16_t* vs, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (live(tid, i)) {
        const int ch = chunk(tid, i);
        const int key = ch / kRowChunks, c8 = (ch % kRowChunks) * 8;
        *(u32x4_t*)(ks + k_lds_row(key) * G::kKStride + c8) = kr[i];
        if constexpr (kWithV) *(u32x4_t*)(vs + key * G::kVStride + c8) = vr[i];
      }
    }
  }
};

// Tile-local key held by register r of S^T tile t in a lane of half-wave h.
__device__ __forceinline__ int score_key(int t, int r, int h) {
  const int j = r >> 2, i = r & 3;
  return 32 * t + 16 * (j >> 1) + 8 * h + 4 * (j & 1) + i;
}

// ---------------------------------------------------------------------------
// Per-wave state and steps of the tile engine.
// ---------------------------------------------------------------------------
template <int D>
struct WaveRows {
  using G = Geo<D>;
  u32x4_t qf[G::kDChunks];   // Q^T B-operand fragments, one per 16-dim chunk
  f32x16_t o[G::kDTiles];    // O^T accumulator, 32 dims x 32 queries per tile
  float m;                   // running max of scale*log2(e)*s (per query)
  float l;                   // running sum over this lane's half of the keys
  float hs[4];               // last tile's per-part sums (softmax_pv<H, P>, P > 0)

  __device__ __forceinline__ void load_q(const uint16_t* qg, int q0, int lane) {
    const uint16_t* row = qg + (size_t)(q0 + (lane & 31)) * D + 8 * (lane >> 5);
#pragma unroll
    for (int c = 0; c < G::kDChunks; ++c) qf[c] = *(const u32x4_t*)(row + 16 * c);
  }

  __device__ __forceinline__ void reset() {
#pragma unroll
    for (int t = 0; t < G::kDTiles; ++t) o[t] = f32x16_t{};
    m = -INFINITY;
    l = 0.f;
  }

  // S^T of one LDS tile of 32*H keys: s[t] covers LDS rows 32t..32t+31.
  template <int H>
  __device__ __forceinline__ void scores(const uint16_t* ks, int lane, f32x16_t s[H]) const {
    const uint16_t* a0 = ks + (lane & 31) * G::kKStride + 8 * (lane >> 5);
    const uint16_t* a1 = a0 + 32 * G::kKStride;
    f32x16_t s0{}, s1{};
#pragma unroll
    for (int c = 0; c < G::kDChunks; ++c) {
      s0 = mfma32x32x16(*(const u32x4_t*)(a0 + 16 * c), qf[c], s0);
      if constexpr (H == 2) s1 = mfma32x32x16(*(const u32x4_t*)(a1 + 16 * c), qf[c], s1);
    }
    s[0] = s0;
    if constexpr (H == 2) s[1] = s1;
  }

  // Causal mask inside a tile: key0 + local key > query -> -inf.
  template <int H>
  __device__ __forceinline__ static void mask(f32x16_t s[H], int key0, int qi, int lane) {
    const int h = lane >> 5;
#pragma unroll
    for (int t = 0; t < H; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (key0 + score_key(t, r, h) > qi) s[t][r] = -INFINITY;
  }

  // Online softmax of one tile and O^T += V^T P^T.  With kParts = 2 (4) the
  // sums of this lane's probabilities over each 32-key half (16-key quarter)
  // of the tile are kept in hs[] (the row sum then adds the parts).
  template <int H, int kParts = 0>
  __device__ __forceinline__ void softmax_pv(f32x16_t s[H], const uint16_t* vt, int lane, float c) {
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < H; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[t][r]);
    mx = pair_max(mx) * c;
    const bool grow = mx > m;
    if (__builtin_amdgcn_ballot_w64(grow)) {
      const float mn = grow ? mx : m;
      const float alpha = (mn == m) ? 1.f : fast_exp2(m - mn);
      l *= alpha;
      // In-place multiply: keeps O in the same registers on both sides of the
      // branch (a plain `*=` lets the allocator rename O and copy all of it
      // back on the path that skips the rescale).
#pragma unroll
      for (int t = 0; t < G::kDTiles; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) asm volatile("v_mul_f32 %0, %0, %1" : "+v"(o[t][r]) : "v"(alpha));
      m = mn;
    }
    const float mb = (m == -INFINITY) ? 0.f : m;
    u32x4_t pb[2 * H];
    // The tile's probabilities are summed on their own and added to the row
    // sum once per tile: a long row (16K keys per lane at 32K) then carries
    // rounding error ~ tiles * eps instead of ~ keys * eps.
    float ts = 0.f;
#pragma unroll
    for (int t = 0; t < H; ++t) {
      float th = 0.f, tq[2] = {0.f, 0.f};
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(__builtin_fmaf(s[t][r], c, -mb));
        s[t][r] = p;
        if constexpr (kParts == 4) tq[r >> 3] += p;
        else if constexpr (kParts == 2) th += p;
        else ts += p;
      }
      if constexpr (kParts == 4) {
        hs[2 * t] = tq[0];
        hs[2 * t + 1] = tq[1];
        ts += tq[0] + tq[1];
      } else if constexpr (kParts == 2) {
        hs[t] = th;
        ts += th;
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          pb[2 * t + u][e] = pack_bf16x2(s[t][8 * u + 2 * e], s[t][8 * u + 2 * e + 1]);
    }
    // A = V^T fragment: lane L needs V[16ks + 8(L/32) + e][32t + L%32], e = 0..7,
    // fetched as two transpose reads of 4 keys each (see lds_read_tr16).
    l += ts;
    const uint16_t* a = vt + (8 * (lane >> 5) + ((lane >> 2) & 3)) * G::kVStride +
                        16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#pragma unroll
    for (int ks = 0; ks < 2 * H; ++ks)
#pragma unroll
      for (int t = 0; t < G::kDTiles; ++t) {
        const u32x2_t lo = lds_read_tr16(a + (16 * ks) * G::kVStride + 32 * t);
        const u32x2_t hi = lds_read_tr16(a + (16 * ks + 4) * G::kVStride + 32 * t);
        o[t] = mfma32x32x16(u32x4_t{lo[0], lo[1], hi[0], hi[1]}, pb[ks], o[t]);
      }
  }

  // One tile: S^T, the causal mask when the tile reaches past this wave's
  // first query (only ever on diagonal tiles, and only instantiated for
  // them), online softmax and PV.
  template <bool kMask, int H = 2, int kParts = 0>
  __device__ __forceinline__ void attend(const uint16_t* ks, const uint16_t* vt, int lane,
                                         float c, int key0, int q0) {
    f32x16_t s[H];
    scores<H>(ks, lane, s);
    if constexpr (kMask) {
      if (key0 + 32 * H - 1 > q0) mask<H>(s, key0, q0 + (lane & 31), lane);
    }
    softmax_pv<H, kParts>(s, vt, lane, c);
  }

  // log2 of the last tile's probability mass per query, unnormalised (taken
  // against the running max m): entries 0..3 for the four 16-key quarters
  // (E = 16), 0 and 1 for the two 32-key halves (E = 32) or entry 0 for the
  // whole tile (E = 64).  -inf for no mass.
  template <int E>
  __device__ __forceinline__ void tile_log_mass(float out[4]) const {
    if constexpr (E == 16) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float x = pair_sum(hs[t]);
        out[t] = x > 0.f ? m + __builtin_log2f(x) : -INFINITY;
      }
    } else if constexpr (E == 32) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const float x = pair_sum(hs[t]);
        out[t] = x > 0.f ? m + __builtin_log2f(x) : -INFINITY;
      }
    } else {
      const float x = pair_sum(hs[0] + hs[1]);
      out[0] = x > 0.f ? m + __builtin_log2f(x) : -INFINITY;
    }
  }

  // log2 of the row normaliser: lse / ln 2.
  __device__ __forceinline__ float lse2() const { return m + __builtin_log2f(pair_sum(l)); }

  // O = O^T / l written as bf16 rows; lse in natural log.  Only the first
  // nq of the wave's 32 query columns are written.
  __device__ __forceinline__ void finish(uint16_t* og, float* lse, int q0, int lane,
                                         int nq = 32) const {
    const float lt = pair_sum(l);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int q = q0 + (lane & 31), h = lane >> 5;
    if ((lane & 31) >= nq) return;
    uint16_t* row = og + (size_t)q * D + 4 * h;
#pragma unroll
    for (int t = 0; t < G::kDTiles; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u32x2_t w;
        w[0] = pack_bf16x2(o[t][4 * j] * inv, o[t][4 * j + 1] * inv);
        w[1] = pack_bf16x2(o[t][4 * j + 2] * inv, o[t][4 * j + 3] * inv);
        *(u32x2_t*)(row + 32 * t + 8 * j) = w;
      }
    if (lse != nullptr && h == 0) lse[q] = lt > 0.f ? (m + __builtin_log2f(lt)) * kLn2 : -INFINITY;
  }
};

// ---------------------------------------------------------------------------
// Dense causal attention.  A work-group of NW waves owns 32*NW consecutive
// queries of one (batch, head); heavier (later) query tiles are issued first.
//
// With BM > 0 the kernel also pools the attention mass into blocks of BM keys
// and BM queries (Section 5.1, eq. block_attention_mass):
//   acc[qb][kb] += (1/BM) sum_{i in qb} sum_{j in kb, j <= i} A_ij.
// A_ij = 2^(s_ij - lse2_i) needs the row normaliser, known only after the
// row's last tile, so every tile leaves per query the log2 of its
// unnormalised mass (against the running max of that moment) in a workspace
// entry of E = min(BM, 64) keys (only spans up to the query tile's end are
// stored), and the epilogue, once lse2 is known, turns
// each entry into 2^(entry - lse2), sums it over the wave's 32 queries and
// then over the waves and entries of each (query block, key block).  The
// group owns the acc rows of its query blocks: no atomics, and the sums run
// in a fixed order, so the result is bitwise reproducible.
// ---------------------------------------------------------------------------
constexpr int kMassChunk = 256;   // workspace entries reduced per epilogue pass
constexpr int kMassBatch = 16;    // entry loads in flight per half-wave in the epilogue

// Waves per SIMD the register allocator must leave room for.  Two by default
// (the d-128 tiles hold 190-250 VGPRs).  The four-wave dense group at d 96
// and the one-wave 32-key sparse group at d 96 fit in 168 VGPRs (three
// waves), the 32-key sparse group at d 64 in 128 (four): more resident waves
// hide more of each one's staging latency (2-6% on those kernels).
constexpr int dense_waves_per_simd(int d, int nw) { return d == 96 && nw == 4 ? 3 : 2; }
constexpr int sparse_waves_per_simd(int d, int kt) {
  return kt != 32 ? 2 : d == 64 ? 4 : d == 96 ? 3 : 2;
}

template <int D, int NW, int BM>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(dense_waves_per_simd(D, NW))))
dense_attn_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                  const uint16_t* __restrict__ V, uint16_t* __restrict__ O,
                  float* __restrict__ lse, int n, int heads, int gq, Sched sc, float c,
                  float* __restrict__ acc, float* __restrict__ mws) {
  using G = Geo<D>;
  constexpr int kNT = NW * 64, kQT = NW * 32;
  constexpr bool kMass = BM > 0;
  constexpr int kE = BM > 0 && BM < 64 ? BM : 64;   // keys per workspace entry
  constexpr int kEPT = kKeyTile / kE;               // entries per 64-key tile
  constexpr int kParts = kMass ? (kE == 16 ? 4 : 2) : 0;
  // An 8-wave group fills its CU alone (two waves per SIMD), so no other
  // group runs while it waits at a barrier: it keeps two LDS tiles and stages
  // tile it+1 into the other one right after computing tile it, one barrier
  // per tile.  Smaller groups share a CU three or four at a time, which a
  // second buffer would halve; they stage and compute around two barriers.
  constexpr int kBufs = NW == 8 ? 2 : 1;
  __shared__ __attribute__((aligned(16))) uint16_t ks[kBufs * G::kKElems];
  __shared__ __attribute__((aligned(16))) uint16_t vt[kBufs * G::kVElems];
  int bh, item;
  if (!sched_slot(sc, bh, item)) return;
  const int qt = sc.items - 1 - item;
  const size_t hoff = (size_t)bh * n * D;
  const size_t kvoff = (size_t)kv_head(bh, heads, gq) * n * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int qbase = qt * kQT, q0 = qbase + 32 * wave;
  // Workspace: per head, per query tile qt, (qt+1)*kQT/kE entries of kQT
  // queries each (only the spans up to the tile's last query), query-minor.
  const int nq = sc.items;
  const size_t per_tile = (size_t)kQT * (kQT / kE);
  float* ew = kMass ? mws + per_tile * ((size_t)bh * nq * (nq + 1) / 2 + (size_t)qt * (qt + 1) / 2) +
                          32 * wave + (lane & 31)
                    : nullptr;

  WaveRows<D> w;
  w.load_q(Q + hoff, q0, lane);
  w.reset();
  // Per-tile mass entries of this lane's query (lanes 0..31 write them).
  auto put_mass = [&](int it) {
    if constexpr (kMass) {
      float lm[4];
      w.template tile_log_mass<kE>(lm);
      if (lane < 32) {
#pragma unroll
        for (int t = 0; t < kEPT; ++t) ew[(size_t)(it * kEPT + t) * kQT] = lm[t];
      }
    }
  };
  // Tiles 0 .. nfull-1 lie wholly below every query of the group; the last
  // kQT/64 tiles hold the diagonal and are masked per wave.
  const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(K + kvoff), rv = buffer_rsrc(V + kvoff);
  const int ntiles = (qbase + kQT) / kKeyTile;
  const int nfull = qbase / kKeyTile;
  TileStage<D, kNT, true> st;
  st.load(rk, rv, 0, tid);
  if constexpr (kBufs == 2) {
    st.store(ks, vt, tid);
    if (ntiles > 1) st.load(rk, rv, kKeyTile, tid);
    __syncthreads();
    // Buffer (it+1)&1 was last read by tile it-1, which every wave finished
    // before the previous barrier.
    auto stage_next = [&](int it) {
      if (it + 1 < ntiles) {
        const int nx = (it + 1) & 1;
        st.store(ks + nx * G::kKElems, vt + nx * G::kVElems, tid);
        if (it + 2 < ntiles) st.load(rk, rv, (it + 2) * kKeyTile, tid);
      }
      __syncthreads();
    };
    int it = 0;
    for (; it < nfull; ++it) {
      const int cu = it & 1;
      w.template attend<false, 2, kParts>(ks + cu * G::kKElems, vt + cu * G::kVElems, lane, c,
                                         it * kKeyTile, q0);
      put_mass(it);
      stage_next(it);
    }
    for (; it < ntiles; ++it) {
      const int cu = it & 1;
      if (it * kKeyTile <= q0) {
        w.template attend<true, 2, kParts>(ks + cu * G::kKElems, vt + cu * G::kVElems, lane, c,
                                          it * kKeyTile, q0);
        put_mass(it);
      }
      stage_next(it);
    }
  } else {
    for (int it = 0; it < nfull; ++it) {
      st.store(ks, vt, tid);
      __syncthreads();
      st.load(rk, rv, (it + 1) * kKeyTile, tid);
      w.template attend<false, 2, kParts>(ks, vt, lane, c, it * kKeyTile, q0);
      put_mass(it);
      __syncthreads();
    }
    for (int it = nfull; it < ntiles; ++it) {
      st.store(ks, vt, tid);
      __syncthreads();
      if (it + 1 < ntiles) st.load(rk, rv, (it + 1) * kKeyTile, tid);
      if (it * kKeyTile <= q0) {
        w.template attend<true, 2, kParts>(ks, vt, lane, c, it * kKeyTile, q0);
        put_mass(it);
      }
      __syncthreads();
    }
  }
  w.finish(O + hoff, lse ? lse + (size_t)bh * n : nullptr, q0, lane);
  if constexpr (kMass) {
    // Epilogue: entries 0 .. elast of this wave were written above (the
    // tiles it attended); later ones hold no mass for its queries.  A
    // 16-query block is half of a wave's queries: its sums run over 16-lane
    // rows, and each wave feeds two query blocks.
    constexpr int kSub = BM < 32 ? 32 / BM : 1;     // query blocks per wave
    constexpr int kWPB = BM < 32 ? 1 : BM / 32;     // waves (or wave halves) per query block
    constexpr int kQB = kQT / BM;                   // query blocks of the group
    constexpr int kBE = BM / kE;                    // entries per key block
    static_assert(kQB >= 1 && kQT % BM == 0, "mass block larger than the group");
    __shared__ float red[NW * kSub][kMassChunk];
    const float l2 = w.lse2();
    const int elast = (q0 + 31) / kE;
    const int nb = n / BM;
    const int eend = (qbase + kQT - 1) / kE + 1;    // entries any wave of the group wrote
    const int hsel = lane >> 5;                     // each half-wave takes every other entry
    for (int c0 = 0; c0 < eend; c0 += kMassChunk) {
      const int cend = min(c0 + kMassChunk, eend);
      for (int e0 = c0; e0 < cend; e0 += 2 * kMassBatch) {
        float x[kMassBatch];
#pragma unroll
        for (int u = 0; u < kMassBatch; ++u) {      // all loads first, then the sums
          const int e = e0 + 2 * u + hsel;
          x[u] = e < cend && e <= elast ? ew[(size_t)e * kQT] : -INFINITY;
        }
#pragma unroll
        for (int u = 0; u < kMassBatch; ++u) {
          const int e = e0 + 2 * u + hsel;
          if constexpr (kSub == 2) {
            const float y = row16_sum(fast_exp2(x[u] - l2));
            if ((lane & 15) == 0 && e < cend) red[2 * wave + ((lane >> 4) & 1)][e - c0] = y;
          } else {
            const float y = half_wave_sum(fast_exp2(x[u] - l2));
            if ((lane & 31) == 0 && e < cend) red[wave][e - c0] = y;
          }
        }
      }
      __syncthreads();
      const int b0 = c0 / kBE, b1 = (min(c0 + kMassChunk, eend) + kBE - 1) / kBE;
      for (int x = tid; x < kQB * (b1 - b0); x += kNT) {
        const int j = x / (b1 - b0), kb = b0 + x % (b1 - b0);
        const int qb = qbase / BM + j;
        if (kb > qb) continue;
        float sum = 0.f;
#pragma unroll
        for (int wv = 0; wv < kWPB; ++wv)
#pragma unroll
          for (int u = 0; u < kBE; ++u) sum += red[j * kWPB + wv][kb * kBE + u - c0];
        acc[((size_t)bh * nb + qb) * nb + kb] += sum * (1.f / BM);
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// Block-sparse attention over a CSR support.  One work-group per (batch,
// head, query block) row, NW = block/32 waves; key tiles of KT = min(block,
// 64) keys, so a 32-key block is one 32-key tile and a one-wave group.
// Schedule slot s (a logical id, contiguous per XCD) runs row order[s];
// wise_select_support writes the rows of each head together, longest support
// first, so an XCD works through a few heads at a time and their K/V tiles
// stay in its L2.
// ---------------------------------------------------------------------------
template <int D, int NW, int KT>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(sparse_waves_per_simd(D, KT))))
sparse_attn_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                   const uint16_t* __restrict__ V, const int32_t* __restrict__ row_ptr,
                   const int32_t* __restrict__ col_idx, const int32_t* __restrict__ order,
                   uint16_t* __restrict__ O, float* __restrict__ lse, int n, int nb, int rows,
                   int heads, int gq, Sched sc, float c) {
  using G = Geo<D>;
  constexpr int kNT = NW * 64, kB = NW * 32, kTPB = kB / KT, kH = KT / 32;
  static_assert(kTPB >= 1 && kB % KT == 0, "block / key tile");
  __shared__ __attribute__((aligned(16))) uint16_t ks[KT * G::kKStride];
  __shared__ __attribute__((aligned(16))) uint16_t vt[KT * G::kVStride];
  int sh, sit;
  if (!sched_slot(sc, sh, sit)) return;
  const int row = order ? order[sh * nb + sit] : sh * nb + (nb - 1 - sit);
  if ((unsigned)row >= (unsigned)rows) return;
  const int bh = row / nb, qb = row % nb;
  const size_t hoff = (size_t)bh * n * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q0 = qb * kB + 32 * wave;
  const int beg = row_ptr[row];
  int nent = row_ptr[row + 1] - beg;
  // Ids past the diagonal form a suffix of the ascending row: dropping them
  // leaves the diagonal block, when present, as the last entry, the one the
  // masked tail below handles.
  while (nent > 0 && col_idx[beg + nent - 1] > qb) --nent;
  const size_t kvoff = (size_t)kv_head(bh, heads, gq) * n * D;
  const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(K + kvoff), rv = buffer_rsrc(V + kvoff);

  // Tile it of the row: entry it / kTPB, sub-tile it % kTPB.  Ids outside
  // 0..qb are skipped (their tile is never loaded out of bounds nor used).
  auto tile_key = [&](int it, bool& ok) {
    const int kb = col_idx[beg + it / kTPB];
    ok = (unsigned)kb <= (unsigned)qb;
    return ok ? kb * kB + (it % kTPB) * KT : 0;
  };

  WaveRows<D> w;
  w.load_q(Q + hoff, q0, lane);
  w.reset();
  TileStage<D, kNT, true, KT> st;
  const int ntiles = nent * kTPB;
  // Entries are ascending, so only the last one can be the diagonal block:
  // every earlier tile lies wholly below this group's queries.
  const int nfull = (nent - 1) * kTPB;
  bool ok = false;
  int key0 = ntiles > 0 ? tile_key(0, ok) : 0;
  if (ntiles > 0) st.load(rk, rv, key0, tid);
  for (int it = 0; it < nfull; ++it) {
    st.store(ks, vt, tid);
    __syncthreads();
    bool ok_next;
    const int key_next = tile_key(it + 1, ok_next);
    st.load(rk, rv, key_next, tid);
    if (ok && key0 + KT - 1 < qb * kB) w.template attend<false, kH>(ks, vt, lane, c, key0, q0);
    __syncthreads();
    key0 = key_next;
    ok = ok_next;
  }
  for (int it = max(nfull, 0); it < ntiles; ++it) {
    st.store(ks, vt, tid);
    __syncthreads();
    bool ok_next = false;
    const int key_next = (it + 1 < ntiles) ? tile_key(it + 1, ok_next) : 0;
    if (it + 1 < ntiles) st.load(rk, rv, key_next, tid);
    if (ok && key0 <= q0) w.template attend<true, kH>(ks, vt, lane, c, key0, q0);
    __syncthreads();
    key0 = key_next;
    ok = ok_next;
  }
  w.finish(O + hoff, lse ? lse + (size_t)bh * n : nullptr, q0, lane);
}

// ---------------------------------------------------------------------------
// Block-sparse attention over groups of consecutive rows of BR-key blocks:
// the dense kernel's work-group (NW waves, 32 NW queries: 4 rows of 64 or 2
// of 128 keys at head_dim 128, 2 rows of 64 otherwise) walks the ascending
// union of its rows' supports in 64-key tiles, staging each tile once for all
// its waves, and each wave attends only the tiles its own row holds (its
// diagonal block masked, tiles wholly past its queries skipped), so every row
// gets exactly its own attention, in the one-row kernel's tile order.  Where
// consecutive rows' supports nearly coincide (dense supports) the union adds
// few tiles and every staged tile feeds 2-4 times the queries of the one-row
// group; where they differ, the union walk costs more than it saves.  The
// membership of each row and the union are built in LDS as bitmasks (up to
// 1024 key blocks).
// ---------------------------------------------------------------------------
constexpr int kGroupMaskWords = 16;

template <int D, int NW, int BR>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
sparse_group_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                    const uint16_t* __restrict__ V, const int32_t* __restrict__ row_ptr,
                    const int32_t* __restrict__ col_idx, uint16_t* __restrict__ O,
                    float* __restrict__ lse, int n, int nb, int heads, int gq, Sched sc,
                    float c) {
  using G = Geo<D>;
  constexpr int kNT = NW * 64, kQT = NW * 32, kR = kQT / BR;   // rows per group
  constexpr int kTPB = BR / kKeyTile, kWR = BR / 32;           // tiles per block, waves per row
  static_assert(kR >= 2 && kQT % BR == 0 && BR % kKeyTile == 0, "group of rows");
  constexpr int kW = kGroupMaskWords;
  constexpr int kBufs = NW == 8 ? 2 : 1;
  __shared__ __attribute__((aligned(16))) uint16_t ks[kBufs * G::kKElems];
  __shared__ __attribute__((aligned(16))) uint16_t vt[kBufs * G::kVElems];
  __shared__ unsigned long long rmask[kR][kW];   // membership per row of the group
  __shared__ unsigned long long umask[kW];       // their union
  int bh, item;
  if (!sched_slot(sc, bh, item)) return;
  const int qt = sc.items - 1 - item;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int qbase = qt * kQT, q0 = qbase + 32 * wave;
  const int qb0 = qt * kR, mine = wave / kWR;     // the group's first row; this wave's row
  const size_t hoff = (size_t)bh * n * D;
  const size_t kvoff = (size_t)kv_head(bh, heads, gq) * n * D;
  const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(K + kvoff), rv = buffer_rsrc(V + kvoff);
  const int words = (nb + 63) >> 6;

  WaveRows<D> w;
  w.load_q(Q + hoff, q0, lane);
  // The group's first tile is its union's lowest block: block 0 wherever a
  // row holds the sink block, so that tile's loads start before the
  // supports are read (and are reissued for another first block).
  TileStage<D, kNT, true> st;
  st.load(rk, rv, 0, tid);
  w.reset();
  // The group's rows are consecutive CSR rows: their entries form one range,
  // read in one pass.
  const int row0 = bh * nb + qb0;
  int bound[kR + 1];
#pragma unroll
  for (int r = 0; r <= kR; ++r) bound[r] = row_ptr[row0 + r];
  for (int i = tid; i < (kR + 1) * kW; i += kNT) {
    if (i < kR * kW) rmask[i / kW][i % kW] = 0ull;
    else umask[i - kR * kW] = 0ull;
  }
  __syncthreads();
  // Valid ids (0..qb) of every row of the group into the bitmasks.
  for (int e = bound[0] + tid; e < bound[kR]; e += kNT) {
    const int kb = col_idx[e];
    int r = 0;
#pragma unroll
    for (int j = 1; j < kR; ++j) r += e >= bound[j];
    if ((unsigned)kb <= (unsigned)(qb0 + r)) {
      const unsigned long long bit = 1ull << (kb & 63);
      atomicOr(&rmask[r][kb >> 6], bit);
      atomicOr(&umask[kb >> 6], bit);
    }
  }
  __syncthreads();
  // The 64-key tiles of the union's blocks in ascending order (the same
  // sequence in every wave; block cb's tiles are cb * kTPB + 0 .. kTPB - 1),
  // each with this wave's membership.  The walk holds the union's and its
  // row's current 64-block words as wave-uniform values and reads LDS only
  // when it moves on to the next word, so no tile waits on an LDS read for
  // its membership between the barrier and its MFMAs.
  auto uniform64 = [](unsigned long long x) {
    const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)x);
    const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(x >> 32));
    return ((unsigned long long)hi << 32) | lo;
  };
  int wi = 0, cb = 0, sub = kTPB - 1;
  unsigned long long cur = uniform64(umask[0]), mw = uniform64(rmask[mine][0]);
  bool cm = false;                                  // this wave's row holds block cb
  auto next = [&](int& tile, bool& mem) {
    if (sub + 1 < kTPB) {
      tile = cb * kTPB + ++sub;
      mem = cm;
      return true;
    }
    while (cur == 0ull) {
      if (++wi >= words) return false;
      cur = uniform64(umask[wi]);
      mw = uniform64(rmask[mine][wi]);
    }
    const int bit = __builtin_ctzll(cur);
    cb = (wi << 6) + bit;
    cur &= cur - 1ull;
    cm = (mw >> bit) & 1ull;
    sub = 0;
    tile = cb * kTPB;
    mem = cm;
    return true;
  };
  // One instance of the tile step for every tile (it masks only a tile that
  // reaches past the wave's first query): a second, unmasked instance for
  // the tiles below the diagonal costs registers and code for nothing.
  auto attend = [&](const uint16_t* kt, const uint16_t* vv, int tile, bool mem) {
    const int key0 = tile * kKeyTile;
    if (!mem || key0 > q0) return;
    w.template attend<true>(kt, vv, lane, c, key0, q0);
  };

  int kb = 0, kb1 = 0, kb2 = 0;     // tiles: current, next, the one after
  bool m0 = false, m1 = false, m2 = false;
  bool have = next(kb, m0);
  if (have && kb != 0) st.load(rk, rv, kb * kKeyTile, tid);
  if constexpr (kBufs == 2) {
    // Double-buffered as the dense 8-wave group: tile i+1 is stored into the
    // idle buffer right after tile i is computed, one barrier per tile.
    if (have) {
      st.store(ks, vt, tid);
      bool h1 = next(kb1, m1);
      if (h1) st.load(rk, rv, kb1 * kKeyTile, tid);
      __syncthreads();
      for (int it = 0;; ++it) {
        const int cu = it & 1;
        attend(ks + cu * G::kKElems, vt + cu * G::kVElems, kb, m0);
        bool h2 = false;
        if (h1) {
          const int nx = (it + 1) & 1;
          st.store(ks + nx * G::kKElems, vt + nx * G::kVElems, tid);
          h2 = next(kb2, m2);
          if (h2) st.load(rk, rv, kb2 * kKeyTile, tid);
        }
        __syncthreads();
        if (!h1) break;
        kb = kb1;
        m0 = m1;
        kb1 = kb2;
        m1 = m2;
        h1 = h2;
      }
    }
  } else {
    while (have) {
      st.store(ks, vt, tid);
      __syncthreads();
      const bool more = next(kb1, m1);
      if (more) st.load(rk, rv, kb1 * kKeyTile, tid);
      attend(ks, vt, kb, m0);
      __syncthreads();
      kb = kb1;
      m0 = m1;
      have = more;
    }
  }
  w.finish(O + hoff, lse ? lse + (size_t)bh * n : nullptr, q0, lane);
}

// ---------------------------------------------------------------------------
// Block-sparse attention for 16-key blocks.  One one-wave work-group per
// (batch, head, query block) row, as for 32-key blocks; the row's 16 queries
// fill both halves of the wave's 32 MFMA columns (lanes n and n + 16 hold the
// same query, and only the first copy is written).  A 32-key tile is any two
// consecutive blocks of the row's support, staged as LDS rows 0-15 and
// 16-31, so every tile key belongs to the row; a last tile with one block
// stages it twice and masks the copy.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : 2)))
sparse_row16_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                    const uint16_t* __restrict__ V, const int32_t* __restrict__ row_ptr,
                    const int32_t* __restrict__ col_idx, const int32_t* __restrict__ order,
                    uint16_t* __restrict__ O, float* __restrict__ lse, int n, int nb, int rows,
                    int heads, int gq, Sched sc, float c) {
  using G = Geo<D>;
  constexpr int kRowChunks = D / 8;                 // 16-byte chunks per key row
  constexpr int kPer = 32 * kRowChunks / 64;        // chunks per lane and tensor
  __shared__ __attribute__((aligned(16))) uint16_t ks[32 * G::kKStride];
  __shared__ __attribute__((aligned(16))) uint16_t vt[32 * G::kVStride];
  int sh, sit;
  if (!sched_slot(sc, sh, sit)) return;
  const int row = order ? order[sh * nb + sit] : sh * nb + (nb - 1 - sit);
  if ((unsigned)row >= (unsigned)rows) return;
  const int bh = row / nb, qb = row % nb;
  const size_t hoff = (size_t)bh * n * D;
  const int lane = threadIdx.x;
  const int q0 = 16 * qb;
  const size_t kvoff = (size_t)kv_head(bh, heads, gq) * n * D;
  const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(K + kvoff), rv = buffer_rsrc(V + kvoff);

  // The row's valid ids (0..qb) in order; the last can be the diagonal.
  int e = row_ptr[row];
  const int end = row_ptr[row + 1];
  auto next_id = [&]() {
    while (e < end) {
      const int kb = col_idx[e++];
      if ((unsigned)kb <= (unsigned)qb) return kb;
    }
    return -1;
  };
  // Tile: blocks a and b (b < 0: a alone).
  auto next_tile = [&](int& a, int& b) {
    a = next_id();
    b = a < 0 ? -1 : next_id();
    return a >= 0;
  };

  WaveRows<D> w;
  {
    const uint16_t* qr = Q + hoff + (size_t)(q0 + (lane & 15)) * D + 8 * (lane >> 5);
#pragma unroll
    for (int cc = 0; cc < G::kDChunks; ++cc) w.qf[cc] = *(const u32x4_t*)(qr + 16 * cc);
  }
  w.reset();
  // Staging: chunk i of this lane is key row r_i (0..31) of the tile, dims
  // 8 * (ch % kRowChunks); rows 0-15 come from block a, 16-31 from block b
  // (from a again when the tile has one block).
  u32x4_t kr[kPer], vr[kPer];
  auto load = [&](int a, int b) {
    const int bb = b < 0 ? a : b;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int ch = lane + 64 * i, r = ch / kRowChunks;
      const int key = (r < 16 ? 16 * a : 16 * bb - 16) + r;
      const uint32_t off = (uint32_t)(key * D + (ch % kRowChunks) * 8) * 2;
      kr[i] = buffer_load16(rk, off, 0);
      vr[i] = buffer_load16(rv, off, 0);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int ch = lane + 64 * i, r = ch / kRowChunks, c8 = (ch % kRowChunks) * 8;
      *(u32x4_t*)(ks + k_lds_row(r) * G::kKStride + c8) = kr[i];
      *(u32x4_t*)(vt + r * G::kVStride + c8) = vr[i];
    }
  };

  int a = -1, b = -1, an = -1, bn = -1;
  bool have = next_tile(a, b);
  if (have) load(a, b);
  const int qi = q0 + (lane & 15), h = lane >> 5;
  while (have) {
    store();
    __syncthreads();
    const bool more = next_tile(an, bn);
    if (more) load(an, bn);
    f32x16_t sc[1];
    w.template scores<1>(ks, lane, sc);
    if (!more) {
      // the last tile: the diagonal block (if present) and a masked copy
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int blk = r < 8 ? a : b;
        const int key = 16 * blk + 8 * h + (r & 7);
        if (blk < 0 || key > qi) sc[0][r] = -INFINITY;
      }
    }
    w.template softmax_pv<1>(sc, vt, lane, c);
    __syncthreads();
    a = an;
    b = bn;
    have = more;
  }
  w.finish(O + hoff, lse ? lse + (size_t)bh * n : nullptr, q0, lane, 16);
}

// ---------------------------------------------------------------------------
// Launchers (shapes already validated by the C ABI layer).
// ---------------------------------------------------------------------------
template <int D, int NW, int BM>
static void launch_dense_nw(const Dims& s, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            uint16_t* O, float* lse, float* acc, float* ws, hipStream_t st) {
  const Sched sc = make_sched(s.bh, s.n / (NW * 32), (size_t)s.n * D * 4 / s.gq);
  hipLaunchKernelGGL((dense_attn_kernel<D, NW, BM>), dim3(sched_grid(sc)), dim3(NW * 64), 0, st,
                     Q, K, V, O, lse, s.n, s.heads, s.gq, sc, s.scale * kLog2e, acc, ws);
}

template <int D, int NW>
static void launch_dense_bm(const Dims& s, const uint16_t* Q, const uint16_t* K,
                            const uint16_t* V, uint16_t* O, float* lse, float* acc, float* ws,
                            hipStream_t st) {
  if (acc == nullptr) return launch_dense_nw<D, NW, 0>(s, Q, K, V, O, lse, acc, ws, st);
  if (s.block == 16) return launch_dense_nw<D, NW, 16>(s, Q, K, V, O, lse, acc, ws, st);
  if (s.block == 32) return launch_dense_nw<D, NW, 32>(s, Q, K, V, O, lse, acc, ws, st);
  if (s.block == 64) return launch_dense_nw<D, NW, 64>(s, Q, K, V, O, lse, acc, ws, st);
  if constexpr (NW >= 4) launch_dense_nw<D, NW, 128>(s, Q, K, V, O, lse, acc, ws, st);
}

template <int D>
static hipError_t launch_dense_d(const Dims& s, const void* q, const void* k, const void* v,
                                 void* o, float* lse, float* acc, float* ws, hipStream_t st) {
  const auto* Q = (const uint16_t*)q;
  const auto* K = (const uint16_t*)k;
  const auto* V = (const uint16_t*)v;
  // Queries per group (dense_query_tile): 256 for d 128 (each staged K/V tile
  // then feeds twice the MFMA work; 6-8% faster at 4K-32K, slower at d 64
  // and 96), else 128 when they divide n (always so for 128-key blocks).
  const int qt = dense_query_tile(s);
  if constexpr (D == 128) {
    if (qt == 256) {
      launch_dense_bm<D, 8>(s, Q, K, V, (uint16_t*)o, lse, acc, ws, st);
      return hipGetLastError();
    }
  }
  if (qt == 128) launch_dense_bm<D, 4>(s, Q, K, V, (uint16_t*)o, lse, acc, ws, st);
  else launch_dense_bm<D, 2>(s, Q, K, V, (uint16_t*)o, lse, acc, ws, st);
  return hipGetLastError();
}

hipError_t launch_dense(const Dims& s, const void* q, const void* k, const void* v, void* o,
                        float* lse, float* acc, void* ws, hipStream_t st) {
  switch (s.d) {
    case 64: return launch_dense_d<64>(s, q, k, v, o, lse, acc, (float*)ws, st);
    case 96: return launch_dense_d<96>(s, q, k, v, o, lse, acc, (float*)ws, st);
    default: return launch_dense_d<128>(s, q, k, v, o, lse, acc, (float*)ws, st);
  }
}

int dense_query_tile(const Dims& s) {
  if (s.d == 128 && s.n % 256 == 0) return 256;
  return s.n % 128 == 0 ? 128 : 64;
}

size_t mass_workspace_bytes(const Dims& s) {
  // Matches dense_attn_kernel: tiles of T = dense_query_tile queries,
  // entries of E keys, tile qt holding (qt+1)*T/E entries of T queries.
  const size_t e = s.block < 64 ? s.block : 64;
  const size_t qt = (size_t)dense_query_tile(s);
  const size_t nq = s.n / qt;
  return (size_t)s.bh * qt * (qt / e) * (nq * (nq + 1) / 2) * sizeof(float);
}

template <int D>
static hipError_t launch_sparse_d(const Dims& s, const void* q, const void* k, const void* v,
                                  const int32_t* rp, const int32_t* ci, const int32_t* order,
                                  void* o, float* lse, hipStream_t st) {
  const float c = s.scale * kLog2e;
  const auto* Q = (const uint16_t*)q;
  const auto* K = (const uint16_t*)k;
  const auto* V = (const uint16_t*)v;
  const int rows = s.bh * s.nb;
  const Sched sc = make_sched(s.bh, s.nb, (size_t)s.n * D * 4 / s.gq);
  const dim3 grid(sched_grid(sc));
  if (s.block == 16)
    hipLaunchKernelGGL((sparse_row16_kernel<D>), grid, dim3(64), 0, st, Q, K, V, rp, ci, order,
                       (uint16_t*)o, lse, s.n, s.nb, rows, s.heads, s.gq, sc, c);
  else if (s.block == 32)
    hipLaunchKernelGGL((sparse_attn_kernel<D, 1, 32>), grid, dim3(64), 0, st, Q, K, V, rp, ci,
                       order, (uint16_t*)o, lse, s.n, s.nb, rows, s.heads, s.gq, sc, c);
  else if (s.block == 64)
    hipLaunchKernelGGL((sparse_attn_kernel<D, 2, 64>), grid, dim3(128), 0, st, Q, K, V, rp, ci,
                       order, (uint16_t*)o, lse, s.n, s.nb, rows, s.heads, s.gq, sc, c);
  else
    hipLaunchKernelGGL((sparse_attn_kernel<D, 4, 64>), grid, dim3(256), 0, st, Q, K, V, rp, ci,
                       order, (uint16_t*)o, lse, s.n, s.nb, rows, s.heads, s.gq, sc, c);
  return hipGetLastError();
}

template <int D, int NW, int BR = 64>
static void launch_group_nw(const Dims& s, const void* q, const void* k, const void* v,
                            const int32_t* rp, const int32_t* ci, void* o, float* lse,
                            hipStream_t st) {
  const Sched sc = make_sched(s.bh, s.n / (NW * 32), (size_t)s.n * D * 4 / s.gq);
  hipLaunchKernelGGL((sparse_group_kernel<D, NW, BR>), dim3(sched_grid(sc)), dim3(NW * 64), 0, st,
                     (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, rp, ci,
                     (uint16_t*)o, lse, s.n, s.nb, s.heads, s.gq, sc, s.scale * kLog2e);
}

int sparse_group_rows(const Dims& s) {
  if (s.nb > 64 * kGroupMaskWords) return 0;
  const int qt = dense_query_tile(s);
  if (s.block == 64) return qt >= 128 ? qt / 64 : 0;
  if (s.block == 128) return qt == 256 ? 2 : 0;
  return 0;
}

hipError_t launch_sparse_grouped(const Dims& s, const void* q, const void* k, const void* v,
                                 const int32_t* rp, const int32_t* ci, void* o, float* lse,
                                 hipStream_t st) {
  const int rows = sparse_group_rows(s);
  if (s.block == 128) {
    if (rows == 2 && s.d == 128) launch_group_nw<128, 8, 128>(s, q, k, v, rp, ci, o, lse, st);
    else return launch_sparse(s, q, k, v, rp, ci, nullptr, o, lse, st);
  } else if (rows == 4 && s.d == 128) launch_group_nw<128, 8>(s, q, k, v, rp, ci, o, lse, st);
  else if (rows == 2 && s.d == 128) launch_group_nw<128, 4>(s, q, k, v, rp, ci, o, lse, st);
  else if (rows == 2 && s.d == 96) launch_group_nw<96, 4>(s, q, k, v, rp, ci, o, lse, st);
  else if (rows == 2 && s.d == 64) launch_group_nw<64, 4>(s, q, k, v, rp, ci, o, lse, st);
  else return launch_sparse(s, q, k, v, rp, ci, nullptr, o, lse, st);
  return hipGetLastError();
}

hipError_t launch_sparse(const Dims& s, const void* q, const void* k, const void* v,
                         const int32_t* rp, const int32_t* ci, const int32_t* order, void* o,
                         float* lse, hipStream_t st) {
  switch (s.d) {
    case 64: return launch_sparse_d<64>(s, q, k, v, rp, ci, order, o, lse, st);
    case 96: return launch_sparse_d<96>(s, q, k, v, rp, ci, order, o, lse, st);
    default: return launch_sparse_d<128>(s, q, k, v, rp, ci, order, o, lse, st);
  }
}

}  // namespace wise
