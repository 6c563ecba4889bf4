// Device helpers shared by the gfx950 kernels: vector types, MFMA wrapper, loads, wave reductions
// and the XCD-aware tile mapping.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cosa_internal.h"

namespace cosa {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// D = A * B + C for A 32x16, B 16x32 (bf16), C/D 32x32 (fp32). Operand layout (wave64):
// lane l supplies A row (l % 32) / B column (l % 32) and eight consecutive k of the 16, the lane
// half (l / 32) selecting which eight. D element (row, col) sits in lane col + 32 * ((row / 4) % 2),
// register 4 * (row / 8) + row % 4.
__device__ __forceinline__ f32x16_t mfma32x32x16(const bf16x8_t& a, const bf16x8_t& b,
                                                 const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ u32x4_t ldg16(const void* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(const u32x4_t& v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

// Cross-lane reductions without the LDS crossbar (ds_bpermute costs an LDS round trip per step):
// v_permlane32_swap exchanges the two 32-lane halves, DPP moves data within rows of 16 lanes, and
// v_readlane takes the last step into a scalar.

// Both halves' values of each lane pair (l, l ^ 32): lo gets lane l % 32, hi lane l % 32 + 32.
__device__ __forceinline__ void half_pair(float v, float& lo, float& hi) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned a = r[0], b = r[1];
  lo = __builtin_bit_cast(float, a);
  hi = __builtin_bit_cast(float, b);
}

// max / sum of v over the lane pair (l, l ^ 32), the same in both lanes.
__device__ __forceinline__ float half_max(float v) {
  float lo, hi;
  half_pair(v, lo, hi);
  return fmaxf(lo, hi);
}
__device__ __forceinline__ float half_sum(float v) {
  float lo, hi;
  half_pair(v, lo, hi);
  return lo + hi;
}

// Lane permutation within rows of 16 (every lane's source lane exists for the patterns used here,
// so the bound-control zero fill never applies; with it the compiler can fold the move into the
// arithmetic instruction that consumes it).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  const int u = __builtin_bit_cast(int, v);
  const int r = __builtin_amdgcn_mov_dpp(u, CTRL, 0xF, 0xF, true);
  return __builtin_bit_cast(float, r);
}

// max of v over each row of 16 lanes, in every lane of the row.
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_mov<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_mov<0x141>(v));  // row_half_mirror: lane i <- 7 - i within 8
  v = fmaxf(v, dpp_mov<0x140>(v));  // row_mirror: lane i <- 15 - i within 16
  return v;
}

// max of v over the wave, as a wave-uniform value.
__device__ __forceinline__ float wave_max(float v) {
  v = row16_max(half_max(v));  // rows 0 and 1 now cover lanes {0-15, 32-47} and {16-31, 48-63}
  const int a = __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0);
  const int b = __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16);
  return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}

// First block of the packed sequence that holds block i (0 without packing), and that sequence's
// index: a binary search over the block offsets in the kernel arguments (uniform, scalar loads).
__device__ __forceinline__ int pack_first(const SeqPack& sp, int i, int& seq) {
  int lo = 0, hi = sp.n - 1;
  if (hi < 0) {
    seq = 0;
    return 0;
  }
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (sp.cu[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  seq = lo;
  return sp.cu[lo];
}

// XCD-aware tile mapping. Workgroup ids are dealt round-robin to the 8 XCDs, so workgroup p runs on
// XCD p % 8. Tiles are grouped in units of G (the query heads that share one KV head and one list):
// unit u goes to XCD u % 8 and its G heads get consecutive dispatch slots there, so the G
// workgroups reading the same K/V pages share that XCD's L2. Returns false for padding slots.
__device__ __forceinline__ bool map_tile(int p, int G, int n_units, int& unit, int& hh) {
  const int xcd = p & 7;
  const int local = p >> 3;
  hh = local % G;
  unit = (local / G) * 8 + xcd;
  return unit < n_units;
}

}  // namespace cosa
