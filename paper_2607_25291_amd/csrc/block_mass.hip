// Exact attention block mass per KV group for gfx950: the ground truth of the proxy-fidelity
// comparison (Sec. 3.2, Property 1: full attention's block mass defines the oracle mask).
//
// One workgroup (b/32 waves) per (batch n, KV head g, query block i); wave w owns 32 query rows.
// For each query head h of the group in turn, pass 1 walks the key blocks j = 0..i and keeps the
// online row max and row sum of exp (fp32, on the transposed MFMA tiles of the attention kernel,
// S^T = K Q^T, one query row per lane); pass 2 walks them again and adds each block's probability
// sum, exp(s - m) / l over the wave's rows and the block's causal keys, to the wave's LDS slot of j.
// The waves' slots are summed in a fixed order at the end, so the result is deterministic. Keys
// are read straight from global memory: this is an analysis kernel, not part of the prefill path.
#include <mutex>

#include "cosa_device.h"
#include "cosa_internal.h"

namespace cosa {
namespace {

struct MassParams {
  const uint16_t* q;
  const uint16_t* k;
  float* mass;
  int Hq, Hkv, L, nb, G;
  float scale_log2;
};

// Sum of v over the wave as a wave-uniform value, in a fixed order (DPP within rows of 16 lanes,
// then the four row sums).
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_mov<0x141>(v);  // row_half_mirror
  v += dpp_mov<0x140>(v);  // row_mirror
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (r0 + r1) + (r2 + r3);
}

template <int BLOCK>
__global__ __attribute__((amdgpu_flat_work_group_size(BLOCK * 2, BLOCK * 2)))
void block_mass_kernel(const MassParams P) {
  constexpr int NW = BLOCK / 32;
  constexpr int KT = BLOCK / 32;
  extern __shared__ float slots[];  // [NW][nb]

  const int unit = blockIdx.x;
  const int i = P.nb - 1 - (unit % P.nb);  // heaviest query blocks first
  const int ng = unit / P.nb;
  const int g = ng % P.Hkv, n = ng / P.Hkv;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  float* slot = slots + w * P.nb;
  for (int j = lane; j <= i; j += 64) slot[j] = 0.f;

  const uint16_t* kbase = P.k + (size_t)ng * P.L * kHeadDim + 8 * half;
  const int qrow = i * BLOCK + w * 32 + l32;
  const int qh = w * 32 + l32 - 4 * half;  // query row within the block, lane-half offset removed

  // S^T tiles of key block j: tile t holds keys 32 t + 8 (r / 4) + 4 half + r % 4 (register r) of
  // query row qrow; -inf above the diagonal of block i.
  auto tiles = [&](int j, const bf16x8_t (&qf)[8], f32x16_t (&s)[KT]) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      const uint16_t* kp = kbase + (size_t)(j * BLOCK + 32 * t + l32) * kHeadDim;
      bf16x8_t kf[8];
#pragma unroll
      for (int c = 0; c < 8; ++c) kf[c] = as_bf16x8(ldg16(kp + 16 * c));
#pragma unroll
      for (int r = 0; r < 16; ++r) s[t][r] = 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) s[t] = mfma32x32x16(kf[c], qf[c], s[t]);
    }
    if (j == i) {  // the sign of (query - key) selects -inf, keeping compare masks out of SGPRs
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int dq = qh - (32 * t + 8 * (r >> 2) + (r & 3));
          asm volatile("" : "+v"(dq));
          const uint32_t masked = (uint32_t)(dq >> 31);
          const float sv = s[t][r];
          const uint32_t bits = __builtin_bit_cast(uint32_t, sv);
          s[t][r] = __builtin_bit_cast(float, (bits & ~masked) | (0xFF800000u & masked));
        }
    }
  };

  for (int hh = 0; hh < P.G; ++hh) {
    const int h = g * P.G + hh;
    bf16x8_t qf[8];
    const uint16_t* qp = P.q + ((size_t)(n * P.Hq + h) * P.L + qrow) * kHeadDim + 8 * half;
#pragma unroll
    for (int c = 0; c < 8; ++c) qf[c] = as_bf16x8(ldg16(qp + 16 * c));

    // Pass 1: row max m (raw logits, equal in both lane halves) and this half's sum of exp.
    float m = -INFINITY, l = 0.f;
    for (int j = 0; j <= i; ++j) {
      f32x16_t s[KT];
      tiles(j, qf, s);
      float mloc = -INFINITY;
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, s[t][r]);
      const float mnew = fmaxf(m, half_max(mloc));
      const float mb = mnew * P.scale_log2;
      float rs = 0.f;
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) rs += __builtin_amdgcn_exp2f(fmaf(s[t][r], P.scale_log2, -mb));
      l = fmaf(l, __builtin_amdgcn_exp2f((m - mnew) * P.scale_log2), rs);
      m = mnew;
    }
    const float inv = 1.f / half_sum(l);
    const float mb = m * P.scale_log2;

    // Pass 2: probability mass of every key block over the wave's rows.
    for (int j = 0; j <= i; ++j) {
      f32x16_t s[KT];
      tiles(j, qf, s);
      float ps = 0.f;
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) ps += __builtin_amdgcn_exp2f(fmaf(s[t][r], P.scale_log2, -mb));
      const float wsum = wave_sum(ps * inv);
      if (lane == 0) slot[j] += wsum;
    }
  }
  __syncthreads();
  float* out = P.mass + ((size_t)ng * P.nb + i) * P.nb;
  for (int j = threadIdx.x; j <= i; j += NW * 64) {
    float a = 0.f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) a += slots[ww * P.nb + j];
    out[j] = a;
  }
}

template <int BLOCK>
hipError_t launch_t(const MassParams& P, int n_units, size_t lds, hipStream_t stream) {
  static std::mutex mu;
  static size_t granted = 0;
  if (lds > 48 * 1024) {
    std::lock_guard<std::mutex> lock(mu);
    if (lds > granted) {
      const hipError_t e =
          hipFuncSetAttribute(reinterpret_cast<const void*>(&block_mass_kernel<BLOCK>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
      granted = lds;
    }
  }
  hipLaunchKernelGGL((block_mass_kernel<BLOCK>), dim3(n_units), dim3(BLOCK * 2), lds, stream, P);
  return hipGetLastError();
}

}  // namespace

size_t block_mass_lds_bytes(const Shape& sh) { return (size_t)(sh.b / 32) * sh.nb * sizeof(float); }

hipError_t launch_block_mass(const Shape& sh, const uint16_t* q, const uint16_t* k, float* mass,
                             hipStream_t stream) {
  MassParams P{q, k, mass, sh.Hq, sh.Hkv, sh.L, sh.nb, sh.G, sh.scale * 1.4426950408889634f};
  const int n_units = sh.B * sh.Hkv * sh.nb;
  const size_t lds = block_mass_lds_bytes(sh);
  return sh.b == 128 ? launch_t<128>(P, n_units, lds, stream) : launch_t<64>(P, n_units, lds, stream);
}

}  // namespace cosa
