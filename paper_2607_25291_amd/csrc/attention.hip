// Ordered-skipping attention (OSK) and the dense causal flash baseline for gfx950.
//
// A workgroup computes HPW query heads of one KV group for one query block of b rows: b/32
// wavefronts per head, 32 query rows per wavefront. The K and V pages of each visited key block are
// staged through LDS once and serve every head of the workgroup. Logits are formed transposed,
// S^T = K Q^T, with bf16 MFMA 32x32x16 so that every lane owns one query row; the online softmax
// runs in fp32 (Sec. 3.1). OSK walks the KAP list (Algorithm A, attention loop) and after Q K^T
// decides, for each head's whole b-row tile at once, whether the value side can be skipped
// (Eq. (skip)); the dense kernel visits j = 0..i in order and never skips.
//
// Pipeline (double-buffered LDS, one barrier per page): the next page's global loads are issued
// into registers, Q K^T of the current page runs (and each wave posts its skip-vote value), the
// next K page goes to LDS, barrier, the tile decides, softmax and P V run, the next V page goes to
// LDS. K buffer (k+1)%2 was last read by Q K^T of page k-1 and V buffer (k+1)%2 by P V of page k-1,
// both finished by every wave before the barrier of page k.
//
// LDS layouts (64 banks x 4 bytes; rows padded by 16 bytes so that 16 consecutive rows start in 16
// different 4-bank groups):
//   K  [key][d]  row-major, 272-byte rows. MFMA A-operand reads (lane = key, 16 bytes of d) and the
//                coalesced row writes are conflict-free; read addresses are one base register plus
//                immediates.
//   Vt [d][key'] V transposed, so that the P V MFMA reads eight keys of one d as 16 bytes. Keys are
//                permuted inside every 16 (offset bits 2 and 3 swapped) so that those eight keys are
//                the eight the lane holds in P^T. Row d is stored at row slot d ^ ((d / 16) % 8), which
//                keeps both the 16-byte reads (16 consecutive d) and the transposing 8-byte writes
//                (d = 8 g + e for 16 values of g) conflict-free.
#include "cosa_device.h"
#include "cosa_internal.h"

namespace cosa {
namespace {

struct AttnParams {
  AttnArgs a;
  int Hq, Hkv, L, nb, G, n_units;
  float scale, scale_log2;
};

template <int BLOCK, int HPW>
struct TileCfg {
  static constexpr int kWavesPerHead = BLOCK / 32;
  static constexpr int kWaves = HPW * kWavesPerHead;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kKeyTiles = BLOCK / 32;
  static constexpr int kKChunks = BLOCK * 16 / kThreads;  // 16-byte K chunks per thread
  static constexpr int kVGroups = BLOCK * 4 / kThreads;   // (4-key group, 8-wide d slice) per thread
  static constexpr int kKRow = (kHeadDim + 8) * 2;        // bytes per K row in LDS
  static constexpr int kVRow = (BLOCK + 8) * 2;           // bytes per V^T row in LDS
  static constexpr int kKBytes = BLOCK * kKRow;
  static constexpr int kVBytes = kHeadDim * kVRow;
  static constexpr int kLdsBytes = 2 * (kKBytes + kVBytes);
  static constexpr int kWgPerCu = (160 * 1024) / (kLdsBytes + 256);
  static constexpr int kWavesPerEu = (kWgPerCu * kWaves) / 4 > 1 ? (kWgPerCu * kWaves) / 4 : 1;
};

__device__ __forceinline__ int vt_slot(int d) { return d ^ ((d >> 4) & 7); }

// Stored key-group (4 keys) kq holds the actual key group with bits 0 and 1 of its index swapped.
__device__ __forceinline__ int actual_keygroup(int kq) {
  return (kq & ~3) | ((kq & 1) << 1) | ((kq >> 1) & 1);
}

template <int BLOCK, int HPW>
struct Stage {
  u32x4_t k[TileCfg<BLOCK, HPW>::kKChunks];
  u32x4_t v[TileCfg<BLOCK, HPW>::kVGroups][4];
};

// Per-thread byte offsets of the page copy (fixed for the whole kernel).
template <int BLOCK, int HPW>
struct CopyOffsets {
  int k_glb, k_lds;              // K: chunk u adds u * (threads/16) rows
  int v_glb[TileCfg<BLOCK, HPW>::kVGroups];
  int v_lds[TileCfg<BLOCK, HPW>::kVGroups];
  int v_xor;                     // row-slot XOR of this thread's 8 V^T rows
};

template <int BLOCK, int HPW>
__device__ __forceinline__ CopyOffsets<BLOCK, HPW> copy_offsets(int tid) {
  using Cfg = TileCfg<BLOCK, HPW>;
  CopyOffsets<BLOCK, HPW> c;
  c.k_glb = (tid >> 4) * (kHeadDim * 2) + (tid & 15) * 16;
  c.k_lds = (tid >> 4) * Cfg::kKRow + (tid & 15) * 16;
  const int dg = tid & 15;
#pragma unroll
  for (int u = 0; u < Cfg::kVGroups; ++u) {
    const int kq = (u * Cfg::kThreads + tid) >> 4;
    c.v_glb[u] = 4 * actual_keygroup(kq) * (kHeadDim * 2) + dg * 16;
    c.v_lds[u] = 8 * dg * Cfg::kVRow + kq * 8;
  }
  c.v_xor = dg >> 1;
  return c;
}

// Global -> registers for the page at byte offset `page` of this KV head (buffer loads: the page
// offset is a scalar, per-thread offsets and chunk strides are fixed).
template <int BLOCK, int HPW>
__device__ __forceinline__ void load_page(__amdgpu_buffer_rsrc_t kr, __amdgpu_buffer_rsrc_t vr,
                                          int page, const CopyOffsets<BLOCK, HPW>& c,
                                          Stage<BLOCK, HPW>& st) {
  using Cfg = TileCfg<BLOCK, HPW>;
#pragma unroll
  for (int u = 0; u < Cfg::kKChunks; ++u)
    st.k[u] = __builtin_amdgcn_raw_buffer_load_b128(
        kr, c.k_glb, page + u * (Cfg::kThreads / 16) * kHeadDim * 2, 0);
#pragma unroll
  for (int u = 0; u < Cfg::kVGroups; ++u)
#pragma unroll
    for (int mm = 0; mm < 4; ++mm)
      st.v[u][mm] = __builtin_amdgcn_raw_buffer_load_b128(vr, c.v_glb[u] + mm * kHeadDim * 2,
                                                          page, 0);
}

template <int BLOCK, int HPW>
__device__ __forceinline__ void store_k(char* Kb, const Stage<BLOCK, HPW>& st,
                                        const CopyOffsets<BLOCK, HPW>& c) {
  using Cfg = TileCfg<BLOCK, HPW>;
#pragma unroll
  for (int u = 0; u < Cfg::kKChunks; ++u)
    *reinterpret_cast<u32x4_t*>(Kb + c.k_lds + u * (Cfg::kThreads / 16) * Cfg::kKRow) = st.k[u];
}

template <int BLOCK, int HPW>
__device__ __forceinline__ void store_vt(char* Vb, const Stage<BLOCK, HPW>& st,
                                         const CopyOffsets<BLOCK, HPW>& c) {
  using Cfg = TileCfg<BLOCK, HPW>;
#pragma unroll
  for (int u = 0; u < Cfg::kVGroups; ++u) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int wd = e >> 1;
      const uint32_t k0 = st.v[u][0][wd], k1 = st.v[u][1][wd];
      const uint32_t k2 = st.v[u][2][wd], k3 = st.v[u][3][wd];
      uint32_t lo, hi;
      if (e & 1) {
        lo = (k0 >> 16) | (k1 & 0xffff0000u);
        hi = (k2 >> 16) | (k3 & 0xffff0000u);
      } else {
        lo = (k0 & 0xffffu) | (k1 << 16);
        hi = (k2 & 0xffffu) | (k3 << 16);
      }
      // row d = 8 dg + e lives at slot 8 dg + (e ^ (dg >> 1))
      *reinterpret_cast<u32x2_t*>(Vb + c.v_lds[u] + (e ^ c.v_xor) * Cfg::kVRow) =
          u32x2_t{lo, hi};
    }
  }
}

template <int BLOCK, int HPW, bool OSK>
__global__ __attribute__((amdgpu_flat_work_group_size(TileCfg<BLOCK, HPW>::kThreads,
                                                      TileCfg<BLOCK, HPW>::kThreads)))
__attribute__((amdgpu_waves_per_eu(TileCfg<BLOCK, HPW>::kWavesPerEu,
                                   TileCfg<BLOCK, HPW>::kWavesPerEu)))
void attention_kernel(const AttnParams P) {
  using Cfg = TileCfg<BLOCK, HPW>;
  constexpr int KT = Cfg::kKeyTiles;
  constexpr int WPH = Cfg::kWavesPerHead;
  constexpr int PAGE = BLOCK * kHeadDim * 2;  // bytes of one K or V page in global memory
  __shared__ __attribute__((aligned(16))) char lds[Cfg::kLdsBytes];
  __shared__ float vote[2][Cfg::kWaves];
  auto Kbuf = [&](int b) { return lds + b * Cfg::kKBytes; };
  auto Vbuf = [&](int b) { return lds + 2 * Cfg::kKBytes + b * Cfg::kVBytes; };

  int unit, pair;
  if (!map_tile(blockIdx.x, P.G / HPW, P.n_units, unit, pair)) return;
  const int i = P.nb - 1 - (unit % P.nb);  // heaviest query blocks first
  const int ng = unit / P.nb;              // n * Hkv + g
  const int g = ng % P.Hkv, n = ng / P.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int hw = w / WPH, wl = w % WPH;  // head slot in the workgroup, wave within the head
  const int h = g * P.G + pair * HPW + hw;

  const size_t kv_off = (size_t)ng * P.L * kHeadDim;
  const size_t qo_off = (size_t)(n * P.Hq + h) * P.L * kHeadDim;
  const int qrow = i * BLOCK + wl * 32 + l32;
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(P.a.k + kv_off), (short)0, P.L * kHeadDim * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(P.a.v + kv_off), (short)0, P.L * kHeadDim * 2, 0x00020000);
  const CopyOffsets<BLOCK, HPW> co = copy_offsets<BLOCK, HPW>(tid);

  // Q^T as the MFMA B operand: lane owns query row qrow, 8 chunks of 16 d (8 per lane half).
  bf16x8_t qf[8];
  {
    const uint16_t* qp = P.a.q + qo_off + (size_t)qrow * kHeadDim + 8 * half;
#pragma unroll
    for (int c = 0; c < 8; ++c) qf[c] = as_bf16x8(ldg16(qp + 16 * c));
  }
  // LDS read bases: K rows key = 32 t + l32 (t and the d chunk are immediates); V^T rows
  // d = 32 dt + l32 through the row-slot swizzle (one base per dt, the key chunk is an immediate).
  const int k_rd = l32 * Cfg::kKRow + half * 16;
  int v_rd[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) v_rd[dt] = vt_slot(32 * dt + l32) * Cfg::kVRow + half * 16;

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

  // A malformed list entry (outside [0, i]) is visited as block i but contributes nothing.
  auto entry = [&](int kk, bool& valid) -> int {
    if constexpr (OSK) {
      const int j = lst[kk];
      valid = (unsigned)j <= (unsigned)i;
      return valid ? j : i;
    } else {
      valid = true;
      return kk;
    }
  };

  Stage<BLOCK, HPW> st;
  bool v_cur = false;
  int j_cur = 0;
  if (cnt > 0) {
    j_cur = entry(0, v_cur);
    load_page<BLOCK, HPW>(krs, vrs, j_cur * PAGE, co, st);
    store_k<BLOCK, HPW>(Kbuf(0), st, co);
    store_vt<BLOCK, HPW>(Vbuf(0), st, co);
  }
  __syncthreads();

  for (int kk = 0; kk < cnt; ++kk) {
    const int buf = kk & 1;
    const bool has_next = kk + 1 < cnt;
    bool v_next = false;
    int j_next = 0;
    if (has_next) {
      j_next = entry(kk + 1, v_next);
      load_page<BLOCK, HPW>(krs, vrs, j_next * PAGE, co, st);
    }

    // S^T tile t: keys 32 t + 8 (r / 4) + 4 half + r % 4 (register r) of query row qrow.
    f32x16_t s[KT];
    const char* Kb = Kbuf(buf) + k_rd;
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const bf16x8_t kf = as_bf16x8(
            *reinterpret_cast<const u32x4_t*>(Kb + t * 32 * Cfg::kKRow + c * 32));
        acc = mfma32x32x16(kf, qf[c], acc);
      }
      s[t] = acc;
    }
    if (j_cur == i) {  // diagonal block: causal mask inside the tile
      const int qi = wl * 32 + l32;
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
    const float mnew = v_cur ? fmaxf(m, mloc) : m;
    if constexpr (OSK) {
      // Eq. (skip): each head's b-row tile votes with its largest (m_loc - m), in nats.
      const float marg = wave_max((mloc - mnew) * P.scale);
      if (lane == 0) vote[buf][w] = marg;
    }
    if (has_next) store_k<BLOCK, HPW>(Kbuf(buf ^ 1), st, co);
    __syncthreads();

    bool skip = !v_cur;
    if constexpr (OSK) {
      if (v_cur) {
        float dk = vote[buf][hw * WPH];
#pragma unroll
        for (int ww = 1; ww < WPH; ++ww) dk = fmaxf(dk, vote[buf][hw * WPH + ww]);
        skip = P.a.skip_on && (dk < P.a.tau);
        if (wl == 0 && lane == 0) {
          if (P.a.visit_log) P.a.visit_log[log_off + kk] = skip ? 2 : 1;
          if (P.a.margin_log) P.a.margin_log[log_off + kk] = dk;
        }
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
      if (__any(alpha != 1.f)) {  // the running max moved in some row of this wave
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
      }
      // O^T += V^T P^T over 16-key chunks kc; P^T chunk kc = registers 8 (kc % 2) .. +7 of tile kc / 2.
      const char* Vb = Vbuf(buf);
#pragma unroll
      for (int kc = 0; kc < BLOCK / 16; ++kc) {
        bf16x8_t pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (__bf16)s[kc >> 1][8 * (kc & 1) + e];
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const bf16x8_t vf =
              as_bf16x8(*reinterpret_cast<const u32x4_t*>(Vb + v_rd[dt] + kc * 32));
          o[dt] = mfma32x32x16(vf, pf, o[dt]);
        }
      }
      ++ncomp;
    }
    if (has_next) store_vt<BLOCK, HPW>(Vbuf(buf ^ 1), st, co);
    j_cur = j_next;
    v_cur = v_next;
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
    if (wl == 0 && lane == 0 && P.a.n_computed)
      P.a.n_computed[(size_t)(n * P.Hq + h) * P.nb + i] = ncomp;
  }
}

template <int BLOCK, int HPW, bool OSK>
void launch_t(const AttnParams& P, int G, hipStream_t stream) {
  using Cfg = TileCfg<BLOCK, HPW>;
  const int slots = (P.n_units + kNumXcd - 1) / kNumXcd * kNumXcd * (G / HPW);
  hipLaunchKernelGGL((attention_kernel<BLOCK, HPW, OSK>), dim3(slots), dim3(Cfg::kThreads), 0,
                     stream, P);
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
  const bool pair = (sh.G % 2) == 0;
  if (sh.b == 128) {
    if (pair) launch_t<128, 2, OSK>(P, sh.G, stream);
    else launch_t<128, 1, OSK>(P, sh.G, stream);
  } else {
    if (pair) launch_t<64, 2, OSK>(P, sh.G, stream);
    else launch_t<64, 1, OSK>(P, sh.G, stream);
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
