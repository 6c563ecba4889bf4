// Ordered-skipping attention (OSK) and the dense causal flash baseline for gfx950.
//
// One workgroup computes one (query head, query block) tile of b rows: b/32 wavefronts, 32 query
// rows each. Per visited key block j the K and V pages are staged through LDS, the logits are formed
// transposed, S^T = K Q^T, with bf16 MFMA 32x32x16 so that every lane owns one query row, and the
// online softmax runs in fp32 (Sec. 3.1). OSK walks the KAP list (Algorithm A, attention loop) and
// after Q K^T decides, for the whole b-row tile at once, whether the value side can be skipped
// (Eq. (skip)); the dense kernel visits j = 0..i in order and never skips.
//
// LDS layouts (b = 128 shown; bank model 64 x 4 B):
//   Ks[key][d]   row-major, the 16-byte chunk c of row `key` stored at chunk c ^ (key % 16):
//                conflict-free both for the coalesced row writes and for the MFMA A-operand reads
//                (lane = key, 16 bytes of d).
//   Vt[d][key']  V transposed, so that the P V MFMA reads eight keys of one d as 16 bytes. Keys are
//                permuted inside every 16 (swap of offset bits 2 and 3) so that those eight keys are
//                exactly the eight the lane holds in P^T (see the S^T register layout), and 8-byte
//                units are XOR-swizzled with 2 * ((d % 16) ^ (d / 16 % 8)) so that both the
//                transposing 8-byte writes and the 16-byte reads are conflict-free.
#include "cosa_device.h"
#include "cosa_internal.h"

namespace cosa {
namespace {

struct AttnParams {
  AttnArgs a;
  int Hq, Hkv, L, nb, G, n_units;
  float scale, scale_log2;
};

template <int BLOCK>
struct TileCfg {
  static constexpr int kWaves = BLOCK / 32;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kKeyTiles = BLOCK / 32;
};

template <int BLOCK>
__device__ __forceinline__ int vt_swizzle(int d) {
  return ((d & 15) ^ ((d >> 4) & 7)) & (BLOCK / 8 - 1);
}

// Stored key-group (4 keys) kq holds the actual key group with bits 0 and 1 of its index swapped.
__device__ __forceinline__ int actual_keygroup(int kq) {
  return (kq & ~3) | ((kq & 1) << 1) | ((kq >> 1) & 1);
}

// Global -> registers for one K/V page. K: 16-byte chunks, 16 consecutive threads per 256-byte row.
// V: every thread takes four consecutive keys (one key group) at one 8-wide d slice, so that it can
// write them transposed; 16 consecutive threads still read whole rows.
template <int BLOCK>
__device__ __forceinline__ void load_page(const uint16_t* __restrict__ kp,
                                          const uint16_t* __restrict__ vp, int tid, u32x4_t (&kr)[8],
                                          u32x4_t (&vr)[8]) {
  constexpr int NT = TileCfg<BLOCK>::kThreads;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int id = u * NT + tid;
    kr[u] = ldg16(kp + (id >> 4) * kHeadDim + (id & 15) * 8);
  }
  const int dg = tid & 15;
#pragma unroll
  for (int u2 = 0; u2 < 2; ++u2) {
    const int kgi = actual_keygroup((tid >> 4) + u2 * (NT / 16));
#pragma unroll
    for (int mm = 0; mm < 4; ++mm) vr[u2 * 4 + mm] = ldg16(vp + (4 * kgi + mm) * kHeadDim + dg * 8);
  }
}

template <int BLOCK>
__device__ __forceinline__ void store_k(uint16_t* Ks, const u32x4_t (&kr)[8], int tid) {
  constexpr int NT = TileCfg<BLOCK>::kThreads;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int id = u * NT + tid;
    const int row = id >> 4, col = id & 15;
    *reinterpret_cast<u32x4_t*>(Ks + row * kHeadDim + ((col ^ (row & 15)) << 3)) = kr[u];
  }
}

template <int BLOCK>
__device__ __forceinline__ void store_vt(uint16_t* Vt, const u32x4_t (&vr)[8], int tid) {
  constexpr int NT = TileCfg<BLOCK>::kThreads;
  const int dg = tid & 15;
#pragma unroll
  for (int u2 = 0; u2 < 2; ++u2) {
    const int kq = (tid >> 4) + u2 * (NT / 16);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = 8 * dg + e;
      const int wd = e >> 1;
      const uint32_t k0 = vr[u2 * 4 + 0][wd], k1 = vr[u2 * 4 + 1][wd];
      const uint32_t k2 = vr[u2 * 4 + 2][wd], k3 = vr[u2 * 4 + 3][wd];
      uint32_t lo, hi;
      if (e & 1) {
        lo = (k0 >> 16) | (k1 & 0xffff0000u);
        hi = (k2 >> 16) | (k3 & 0xffff0000u);
      } else {
        lo = (k0 & 0xffffu) | (k1 << 16);
        hi = (k2 & 0xffffu) | (k3 << 16);
      }
      const int unit = kq ^ (2 * vt_swizzle<BLOCK>(d));
      *reinterpret_cast<u32x2_t*>(Vt + d * BLOCK + unit * 4) = u32x2_t{lo, hi};
    }
  }
}

template <int BLOCK, bool OSK>
__global__ __launch_bounds__(BLOCK * 2) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attention_kernel(const AttnParams P) {
  using Cfg = TileCfg<BLOCK>;
  constexpr int KT = Cfg::kKeyTiles;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BLOCK * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kHeadDim * BLOCK];
  __shared__ float vote[Cfg::kWaves];

  int unit, hh;
  if (!map_tile(blockIdx.x, P.G, P.n_units, unit, hh)) return;
  const int i = P.nb - 1 - (unit % P.nb);  // heaviest query blocks first
  const int ng = unit / P.nb;              // n * Hkv + g
  const int g = ng % P.Hkv, n = ng / P.Hkv;
  const int h = g * P.G + hh;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;

  const size_t kv_off = (size_t)ng * P.L * kHeadDim;
  const size_t qo_off = (size_t)(n * P.Hq + h) * P.L * kHeadDim;
  const int qrow = i * BLOCK + w * 32 + l32;

  // Q^T as the MFMA B operand: lane owns query row qrow, 8 chunks of 16 d (8 per lane half).
  bf16x8_t qf[8];
  {
    const uint16_t* qp = P.a.q + qo_off + (size_t)qrow * kHeadDim + 8 * half;
#pragma unroll
    for (int c = 0; c < 8; ++c) qf[c] = as_bf16x8(ldg16(qp + 16 * c));
  }
  // O^T accumulators: tile dt holds d = 32 dt + 8 (r / 4) + 4 half + r % 4 of row qrow.
  f32x16_t o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;
  float m = -INFINITY;  // running row max (raw logits), identical in both lane halves
  float lsum = 0.f;     // this lane half's partial row sum

  int cnt;
  const int32_t* lst = nullptr;
  if constexpr (OSK) {
    cnt = P.a.count[(size_t)ng * P.nb + i];
    cnt = cnt < P.nb ? cnt : P.nb;
    lst = P.a.order + ((size_t)ng * P.nb + i) * P.nb;
  } else {
    cnt = i + 1;
  }
  const size_t log_off = ((size_t)(n * P.Hq + h) * P.nb + i) * P.nb;
  int ncomp = 0;

  for (int kk = 0; kk < cnt; ++kk) {
    const int j = OSK ? lst[kk] : kk;
    if (OSK && (unsigned)j > (unsigned)i) continue;  // malformed entry: never read out of bounds
    u32x4_t kr[8], vr[8];
    load_page<BLOCK>(P.a.k + kv_off + (size_t)j * BLOCK * kHeadDim,
                     P.a.v + kv_off + (size_t)j * BLOCK * kHeadDim, tid, kr, vr);
    __syncthreads();  // every wave is done with the previous page
    store_k<BLOCK>(Ks, kr, tid);
    store_vt<BLOCK>(Vt, vr, tid);
    __syncthreads();

    // S^T tile t: keys 32 t + 8 (r / 4) + 4 half + r % 4 (register r) of query row qrow.
    f32x16_t s[KT];
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      const int key = 32 * t + l32;
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const bf16x8_t kf = as_bf16x8(*reinterpret_cast<const u32x4_t*>(
            Ks + key * kHeadDim + (((2 * c + half) ^ (key & 15)) << 3)));
        acc = mfma32x32x16(kf, qf[c], acc);
      }
      s[t] = acc;
    }
    if (j == i) {  // diagonal block: causal mask inside the tile
      const int qi = w * 32 + l32;
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
          if (key > qi) s[t][r] = -INFINITY;
        }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, s[t][r]);
    mloc = fmaxf(mloc, swap_halves(mloc));
    const float mnew = fmaxf(m, mloc);

    bool skip = false;
    if constexpr (OSK) {
      // Eq. (skip): the tile votes with the largest (m_loc - m) over its b rows, in nats.
      const float marg = wave_max((mloc - mnew) * P.scale);
      if (lane == 0) vote[w] = marg;
      __syncthreads();
      float dk = vote[0];
#pragma unroll
      for (int ww = 1; ww < Cfg::kWaves; ++ww) dk = fmaxf(dk, vote[ww]);
      skip = P.a.skip_on && (dk < P.a.tau);
      if (tid == 0) {
        if (P.a.visit_log) P.a.visit_log[log_off + kk] = skip ? 2 : 1;
        if (P.a.margin_log) P.a.margin_log[log_off + kk] = dk;
      }
    }
    // A skip implies m_loc < m in every row, so the running max is unchanged either way.
    if (!skip) {
      const float alpha = __builtin_amdgcn_exp2f((m - mnew) * P.scale_log2);
      m = mnew;
      const float mb = mnew * P.scale_log2;
      float rs = 0.f;
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = __builtin_amdgcn_exp2f(fmaf(s[t][r], P.scale_log2, -mb));
          s[t][r] = pv;
          rs += pv;
        }
      lsum = fmaf(lsum, alpha, rs);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
      // O^T += V^T P^T over 16-key chunks kc; P^T chunk kc = registers 8 (kc % 2) .. +7 of tile kc / 2.
#pragma unroll
      for (int kc = 0; kc < BLOCK / 16; ++kc) {
        bf16x8_t pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (__bf16)s[kc >> 1][8 * (kc & 1) + e];
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const int d = 32 * dt + l32;
          const int u = (4 * kc + 2 * half) ^ (2 * vt_swizzle<BLOCK>(d));
          const bf16x8_t vf =
              as_bf16x8(*reinterpret_cast<const u32x4_t*>(Vt + d * BLOCK + u * 4));
          o[dt] = mfma32x32x16(vf, pf, o[dt]);
        }
      }
      ++ncomp;
    }
  }

  lsum += swap_halves(lsum);
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  uint16_t* op = P.a.o + qo_off + (size_t)qrow * kHeadDim;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d0 = 32 * dt + 8 * rg + 4 * half;
      uint32_t wv[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const __bf16 lo = (__bf16)(o[dt][4 * rg + 2 * e] * inv);
        const __bf16 hi = (__bf16)(o[dt][4 * rg + 2 * e + 1] * inv);
        wv[e] = (uint32_t)__builtin_bit_cast(uint16_t, lo) |
                ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
      }
      *reinterpret_cast<u32x2_t*>(op + d0) = u32x2_t{wv[0], wv[1]};
    }
  if constexpr (OSK) {
    if (tid == 0 && P.a.n_computed) P.a.n_computed[(size_t)(n * P.Hq + h) * P.nb + i] = ncomp;
  }
}

template <bool OSK>
hipError_t launch(const Shape& sh, const AttnArgs& a, hipStream_t stream) {
  AttnParams P;
  P.a = a;
  P.Hq = sh.Hq;
  P.Hkv = sh.Hkv;
  P.L = sh.L;
  P.nb = sh.nb;
  P.G = sh.G;
  P.n_units = sh.B * sh.Hkv * sh.nb;
  P.scale = sh.scale;
  P.scale_log2 = sh.scale * 1.4426950408889634f;
  const int slots = (P.n_units + kNumXcd - 1) / kNumXcd * kNumXcd * sh.G;
  if (sh.b == 128) {
    hipLaunchKernelGGL((attention_kernel<128, OSK>), dim3(slots), dim3(256), 0, stream, P);
  } else {
    hipLaunchKernelGGL((attention_kernel<64, OSK>), dim3(slots), dim3(128), 0, stream, P);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_osk_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream) {
  return launch<true>(sh, a, stream);
}

hipError_t launch_dense_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream) {
  return launch<false>(sh, a, stream);
}

}  // namespace cosa
