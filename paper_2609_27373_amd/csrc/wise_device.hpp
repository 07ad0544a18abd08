// wise_device.hpp — gfx950 device helpers of the libwise attention kernels:
// vector types, the bf16 MFMA wrapper, buffer loads, packing, cross-lane
// helpers, the tile geometry and the work order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wise {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));

constexpr int kKeyTile = 64;    // keys per LDS tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// D (32 x 32, fp32) += A (32 x 16, bf16) * B (16 x 32, bf16).
// Lane l holds A[l % 32][8*(l/32) .. +7], B[8*(l/32) .. +7][l % 32];
// C element (m, n) sits in lane n + 32*((m/4) % 2), register 4*(m/8) + m%4.
__device__ __forceinline__ f32x16_t mfma32x32x16(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// LDS transpose read (ds_read_b64_tr_b16).  Within each 16-lane group g,
// output lane 16g + i, element j is the 16-bit word at
// (address supplied by lane 16g + 4j + i/4) + (i % 4).
__device__ __forceinline__ u32x2_t lds_read_tr16(const uint16_t* p) {
  auto r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4_t*)(const_cast<uint16_t*>(p)));
  return __builtin_bit_cast(u32x2_t, r);
}

// Buffer resource over `base` for raw 16-byte loads (32-bit byte offsets:
// the head's base stays in scalar registers and a tile needs no 64-bit
// address arithmetic per lane).  Offsets past num_records read as zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ u32x4_t buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                 uint32_t soff) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Two fp32 -> packed bf16x2 (round to nearest even), lo in bits 0..15.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Combine x with the value held by lane l ^ 32 (the other half of the wave
// holding the same query column).  permlane32_swap leaves one register with
// the low half-wave replicated and the other with the high half replicated,
// so max / sum of the two is the pair result in every lane, computed in the
// same order in both lanes.
__device__ __forceinline__ float pair_max(float x) {
  uint32_t u = __builtin_bit_cast(uint32_t, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  uint32_t u = __builtin_bit_cast(uint32_t, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Cross-lane sums on the VALU, in a fixed order (bitwise reproducible).
template <int kCtrl>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), kCtrl, 0xF, 0xF, true));
}

// Sum of x over this lane's 16-lane row, in every lane of the row: quad
// butterflies, then the half-row and row mirrors (DPP).
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_mov<0xB1>(x);    // quad_perm [1,0,3,2]
  x += dpp_mov<0x4E>(x);    // quad_perm [2,3,0,1]
  x += dpp_mov<0x141>(x);   // row_half_mirror
  x += dpp_mov<0x140>(x);   // row_mirror
  return x;
}

// Sum of x over the 32 lanes of this lane's half-wave, in every lane: the
// two 16-lane row sums added through permlane16_swap.
__device__ __forceinline__ float half_wave_sum(float x) {
  x = row16_sum(x);
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

// Tile geometry of the attention kernels for head dimension D.
template <int D>
struct Geo {
  static_assert(D == 64 || D == 96 || D == 128, "head_dim");
  static constexpr int kKStride = D + 8;          // LDS K row stride (bf16): 16 B pad
  static constexpr int kVStride = D + 16;         // LDS V row stride (bf16): 32 B pad
  static constexpr int kDChunks = D / 16;         // MFMA k-steps of S^T = K Q^T
  static constexpr int kDTiles = D / 32;          // MFMA m-tiles of O^T = V^T P^T
  static constexpr int kKElems = kKeyTile * kKStride;
  static constexpr int kVElems = kKeyTile * kVStride;
};

// Row of the LDS K tile that holds tile-local key `key`.  S^T = K Q^T puts
// tile row m at accumulator position (m/8, (m/4)%2, m%4); swapping bits 2 and
// 3 of the key makes each lane's 8 consecutive accumulator entries hold 8
// consecutive keys, which is exactly the B-operand layout of O^T = V^T P^T.
__device__ __forceinline__ int k_lds_row(int key) {
  return (key & ~12) | ((key & 4) << 1) | ((key & 8) >> 1);
}

// Key-value head of flattened query head bh = b * heads + h when gq query
// heads share one key-value head: b * (heads / gq) + h / gq.
__device__ __forceinline__ int kv_head(int bh, int heads, int gq) {
  return gq == 1 ? bh : (bh / heads) * (heads / gq) + (bh % heads) / gq;
}

// Work order of the attention and block-mass grids.  A grid covers
// heads * items pieces of work, `item` counting from the heaviest piece of a
// head (0) to the lightest.  The hardware deals work-groups round-robin over
// the 8 XCDs in id order, so an XCD receives every 8th id.  When the heads
// split evenly enough over 8 XCDs (at least 8 heads, the busiest XCD within
// 10% of an even share), each XCD owns a contiguous range of heads, so a
// head's K/V stays in one L2; an XCD with one head fewer than per_xcd, and a
// short last group, leave empty slots that return at once.  An XCD walks its
// heads in groups of `group` heads, item-major inside a group: the heaviest
// items of the group's heads start together, so no long item is left for the
// tail (head-major order would leave them there), while only `group` heads
// compete for the L2 at a time.  Otherwise the whole grid is item-major.
struct Sched {
  int heads, items, group, per_xcd;   // per_xcd == 0: whole grid item-major
};

// Host: the schedule for `heads` x `items` pieces whose heads each stream
// kv_bytes of K/V.  Group size:
//  - a head of 4 MiB of K/V or more (16K and 32K tokens at d 128): as many
//    heads as fit 16 MiB, so the rows in flight on an XCD walk the same few
//    heads' keys in ascending order together and hit each other's tiles in
//    L2 (measured: 32K / 32 heads, one head at a time, 8% faster sparse and
//    4% faster dense than four interleaved heads, which fetched 16 times the
//    algorithmic bytes; 16K, two at a time, 9% and 6%);
//  - otherwise every head of the XCD when 8 divides the head count
//    (measured at 4K / 32 heads / block 64: interleaving 2 heads at a time
//    keeps more K/V in L2, 112 instead of 154 MiB fetched per sparse launch,
//    but balances worse and runs 5% slower; that grid runs in about two
//    rounds of resident work-groups per XCD);
//  - otherwise as many heads as fit about 3 MiB of the 4 MiB L2 (many heads
//    per XCD, many rounds of work).
inline Sched make_sched(int heads, int items, size_t kv_bytes) {
  Sched s{heads, items, 1, 0};
  const int per = (heads + 7) / 8;
  // The busiest XCD holds `per` heads against an even share of heads / 8:
  // partition only while that costs at most 10%.
  if (heads >= 8 && 80 * per <= 11 * heads) {
    s.per_xcd = per;
    if (kv_bytes >= (size_t)(4u << 20)) {
      const size_t fit = (size_t)(16u << 20) / kv_bytes;
      s.group = (int)(fit > (size_t)s.per_xcd ? (size_t)s.per_xcd : fit);
    } else if (heads % 8 == 0) {
      s.group = s.per_xcd;
    } else {
      const size_t fit = kv_bytes > 0 ? (size_t)(3u << 20) / kv_bytes : 1;
      s.group = (int)(fit < 1 ? 1 : (fit > (size_t)s.per_xcd ? (size_t)s.per_xcd : fit));
    }
  }
  return s;
}

inline unsigned sched_grid(const Sched& s) {
  return (unsigned)(s.per_xcd ? 8 * s.per_xcd * s.items : s.heads * s.items);
}

// Device: (head, item) of this work-group; false for an empty slot.
__device__ __forceinline__ bool sched_slot(const Sched& s, int& head, int& item) {
  const int b = blockIdx.x;
  if (s.per_xcd == 0) {
    head = b % s.heads;
    item = b / s.heads;
    return true;
  }
  const int x = b & 7, j = b >> 3;
  const int lo = (x * s.heads) >> 3, cnt = (((x + 1) * s.heads) >> 3) - lo;
  const int g = j / (s.group * s.items);
  if (g * s.group >= cnt) return false;
  const int gh = min(s.group, cnt - g * s.group);
  const int r = j - g * s.group * s.items;
  head = lo + g * s.group + r % gh;
  item = r / gh;
  return item < s.items;   // a short last group leaves empty slots
}

}  // namespace wise
