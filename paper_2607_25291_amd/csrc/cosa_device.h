// Device helpers shared by the gfx950 kernels: vector types, MFMA wrapper, loads, wave reductions
// and the XCD-aware tile mapping.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// Exchange with the lane 32 apart (the other half of the wave).
__device__ __forceinline__ float swap_halves(float v) { return __shfl_xor(v, 32); }

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
