// KAP block scoring for gfx950 (Sec. 4.2 "Block ranking", Eq. (score); Algorithm A, proxy stage).
//
// One workgroup (8 wavefronts) per (batch n, KV head g, query block i), placed so that each XCD
// serves as few KV heads as possible (their sampled keys then stay in that XCD's L2). Its
// R = G * spb sampled query rows (tokens (i*spb + t) * s of the G heads of group g) stay in
// registers as the MFMA B operand.
// The waves stride over chunks of 32 sampled keys c < (i+1)*spb (tokens c * s), computing the
// transposed logits K~ Q~^T with bf16 MFMA 32x32x16, applying the causal mask over sampled
// positions (c <= r) and sm_scale, and reducing them straight into per-block maxima beta[row][j] held
// in LDS. The softmax -> MaxPool -> MaxNorm chain collapses to Pbar = exp(beta - mu) with mu the row
// maximum (the softmax normaliser cancels in the MaxNorm ratio, exp is monotone), so the score matrix
// is never materialised. A second phase takes mu per row and, per key block j, sums
// exp(beta - mu) over the rows in a fixed order (deterministic) and raises the HRM flag when some
// row attains its maximum there (beta == mu, exact).
#include <mutex>

#include "cosa_device.h"
#include "cosa_internal.h"

namespace cosa {
namespace {

constexpr int kScoreThreads = 512;
constexpr int kScoreWaves = kScoreThreads / 64;

struct KapParams {
  KapScoreArgs a;
  int Hq, Hkv, L, nb, G, s, R, nbp, n_units;
  int nch_all;  // 32-key chunks of all L / s sampled keys of a head (staged layout)
  float scale;
};

// Elements of one staged 32-key chunk: 8 d chunks of 64 lanes x 8 values, in MFMA operand order.
constexpr int kStageChunk = 8 * 64 * 8;

// Row of sampled key c (token c * s) of KV head g, batch n: contiguous K [B, Hkv, L, d], or its
// physical page in a paged cache [n_pages, Hkv, page, d] through the page table (entries outside
// [0, n_pages) read page 0).
template <bool PAGED>
__device__ __forceinline__ const uint16_t* sampled_key_row(const KapParams& P, int n, int g, int c) {
  if constexpr (PAGED) {
    const int t = c * P.s;
    const int log2p = P.a.pg.log2_page;
    int e = P.a.pg.table[(size_t)n * P.a.pg.pages_per_seq + (t >> log2p)];
    e = (e >= 0 && (long long)e < P.a.pg.n_pages) ? e : 0;
    const long long row = (((long long)e * P.Hkv + g) << log2p) + (t & ((1 << log2p) - 1));
    return P.a.k + row * kHeadDim;
  } else {
    return P.a.k + ((size_t)(n * P.Hkv + g) * P.L + (size_t)c * P.s) * kHeadDim;
  }
}

// Staging of the sampled keys in MFMA operand order: wavefront w takes 32-key chunk w of all heads
// (head-major) and writes, for d chunk cc, lane (half, l32) the 8 values d = 16 cc + 8 half .. + 7
// of key 32 * chunk + l32 (zeros past the last sampled key), so that the scoring kernel reads each
// chunk as 8 fully contiguous 1 KiB loads instead of 32 scattered rows per load.
template <bool PAGED>
__global__ __launch_bounds__(256) void stage_keys_kernel(const KapParams P) {
  const int wv = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int NG = P.n_units / P.nb;
  if (wv >= NG * P.nch_all) return;
  const int ng = wv / P.nch_all, chunk = wv % P.nch_all;
  const int c = chunk * 32 + l32;
  u32x4_t v[8];
  if (c < P.L / P.s) {
    const uint16_t* kp = sampled_key_row<PAGED>(P, ng / P.Hkv, ng % P.Hkv, c) + 8 * half;
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) v[cc] = ldg16(kp + 16 * cc);
  } else {
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) v[cc] = u32x4_t{0u, 0u, 0u, 0u};
  }
  uint16_t* op = P.a.kstage + (size_t)wv * kStageChunk + lane * 8;
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) *reinterpret_cast<u32x4_t*>(op + cc * 512) = v[cc];
}

// Unit (ng = n * Hkv + g, query block i) of dispatch slot p. Slot p runs on XCD p % 8, and an
// XCD's L2 holds the sampled keys of the heads it serves: when the NG = B * Hkv heads split evenly
// over the 8 XCDs, XCD x takes heads ng = x (mod 8); when NG divides 8, the 8 / NG XCDs that share a
// head split its query blocks. Either way an XCD streams the keys of as few heads as possible, and
// the heaviest query blocks go first. Other NG keep the plain order. False for padding slots.
__device__ __forceinline__ bool proxy_unit(int p, int NG, int nb, int& ng, int& i) {
  const int x = p & 7, local = p >> 3;
  int rank;  // position in the heaviest-first order of the head's query blocks
  if (NG % 8 == 0) {
    const int per = NG >> 3;
    ng = (local % per) * 8 + x;
    rank = local / per;
  } else if (8 % NG == 0) {
    const int k = 8 / NG;
    ng = x % NG;
    rank = local * k + x / NG;
  } else {
    ng = p / nb;
    rank = p % nb;
    if (ng >= NG) return false;
  }
  i = nb - 1 - rank;
  return rank < nb;
}

// Dispatch slots for NG heads of nb query blocks (see proxy_unit).
int proxy_slots(int NG, int nb) {
  if (NG % 8 != 0 && 8 % NG == 0) return 8 * ((nb + 8 / NG - 1) / (8 / NG));
  return NG * nb;
}

// STAGED: the sampled keys come from the staged copy (P.a.kstage) instead of K itself.
template <int SPB, int RT, bool PAGED, bool STAGED>
__global__ __launch_bounds__(kScoreThreads) void kap_score_kernel(const KapParams P) {
  extern __shared__ float beta[];  // [R][nbp]
  __shared__ float mu[RT * 32];

  int ng, i;
  if (!proxy_unit(blockIdx.x, P.n_units / P.nb, P.nb, ng, i)) return;
  const int g = ng % P.Hkv, n = ng / P.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int nkeys = (i + 1) * SPB;
  const int nchunks = (nkeys + 31) >> 5;
  // Packed sequences: the candidates are the blocks F .. i of block i's own sequence.
  int seq;
  const int F = pack_first(P.a.pack, i, seq);
  const int chunk0 = (F * SPB) >> 5;
  auto cand = [&](int j) { return (unsigned)(j - F) <= (unsigned)(i - F); };

  // Q~^T fragments: row rt*32 + l32 = (head offset hh, sample t) -> token (i*SPB + t) * s.
  bf16x8_t qf[RT][8];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int row = rt * 32 + l32;
    if (row < P.R) {
      const int hh = row / SPB, t = row % SPB;
      const size_t tok = (size_t)(i * SPB + t) * P.s;
      const uint16_t* qp =
          P.a.q + ((size_t)(n * P.Hq + g * P.G + hh) * P.L + tok) * kHeadDim + 8 * half;
#pragma unroll
      for (int c = 0; c < 8; ++c) qf[rt][c] = as_bf16x8(ldg16(qp + 16 * c));
    } else {
#pragma unroll
      for (int c = 0; c < 8; ++c) qf[rt][c] = as_bf16x8(u32x4_t{0u, 0u, 0u, 0u});
    }
  }

  const uint16_t* sbase =
      STAGED ? P.a.kstage + (size_t)ng * P.nch_all * kStageChunk + lane * 8 : nullptr;
  auto load_keys = [&](int chunk, bf16x8_t (&kf)[8]) __attribute__((always_inline)) {
    const int c = chunk * 32 + l32;
    if constexpr (STAGED) {
      if (chunk < nchunks) {
        const uint16_t* sp = sbase + (size_t)chunk * kStageChunk;
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) kf[cc] = as_bf16x8(ldg16(sp + cc * 512));
        return;
      }
    } else if (chunk < nchunks && c < nkeys) {
      const uint16_t* kp = sampled_key_row<PAGED>(P, n, g, c) + 8 * half;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) kf[cc] = as_bf16x8(ldg16(kp + 16 * cc));
      return;
    }
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) kf[cc] = as_bf16x8(u32x4_t{0u, 0u, 0u, 0u});
  };

  auto process = [&](int chunk, const bf16x8_t (&kf)[8]) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) acc = mfma32x32x16(kf[cc], qf[rt][cc], acc);
      // acc[r]: sampled key chunk*32 + 8 (r/4) + 4 half + r%4, row rt*32 + l32. Only a chunk that
      // reaches block i (or the zero-filled keys past the last sample) needs the causal mask; the
      // branch is uniform over the wave.
      const int row = rt * 32 + l32;
      if (chunk * 32 + 31 > i * SPB) {
        const int rs = i * SPB + (row % SPB);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = chunk * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          acc[r] = key > rs ? -INFINITY : acc[r];
        }
      }
      // Block maxima are taken on the raw logits and scaled once: x -> sm_scale * x is monotone
      // under rounding, so the scaled maximum equals the maximum of the scaled logits exactly.
      const bool row_ok = row < P.R;
      float* brow = beta + row * P.nbp;
      if constexpr (SPB == 4) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float bm = fmaxf(fmaxf(acc[4 * q4], acc[4 * q4 + 1]),
                                 fmaxf(acc[4 * q4 + 2], acc[4 * q4 + 3]));
          const int j = chunk * 8 + 2 * q4 + half;
          if (row_ok && cand(j)) brow[j] = bm * P.scale;
        }
      } else if constexpr (SPB == 8) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float bm = fmaxf(fmaxf(acc[4 * q4], acc[4 * q4 + 1]),
                           fmaxf(acc[4 * q4 + 2], acc[4 * q4 + 3]));
          bm = half_max(bm);
          const int j = chunk * 4 + q4;
          if (row_ok && cand(j) && (q4 >> 1) == half) brow[j] = bm * P.scale;
        }
      } else if constexpr (SPB == 16) {
#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2) {
          float bm = acc[8 * b2];
#pragma unroll
          for (int r = 1; r < 8; ++r) bm = fmaxf(bm, acc[8 * b2 + r]);
          bm = half_max(bm);
          const int j = chunk * 2 + b2;
          if (row_ok && cand(j) && b2 == half) brow[j] = bm * P.scale;
        }
      } else {
        float bm = acc[0];
#pragma unroll
        for (int r = 1; r < 16; ++r) bm = fmaxf(bm, acc[r]);
        bm = half_max(bm);
        const int j = chunk;
        if (row_ok && cand(j) && half == 0) brow[j] = bm * P.scale;
      }
    }
  };
  // The next chunk of this wave is loaded while the current one is processed.
  bf16x8_t kcur[8], knext[8];
  load_keys(chunk0 + w, kcur);
  for (int chunk = chunk0 + w; chunk < nchunks; chunk += kScoreWaves) {
    load_keys(chunk + kScoreWaves, knext);
    process(chunk, kcur);
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) kcur[cc] = knext[cc];
  }
  __syncthreads();

  // Row maxima mu (MaxNorm denominator, in the log domain).
  for (int row = w; row < P.R; row += kScoreWaves) {
    float v = -INFINITY;
    for (int j = F + lane; j <= i; j += 64) v = fmaxf(v, beta[row * P.nbp + j]);
    v = wave_max(v);
    if (lane == 0) mu[row] = v;
  }
  __syncthreads();

  float* srow = P.a.score + ((size_t)ng * P.nb + i) * P.nb;
  uint8_t* hrow = P.a.hrm + ((size_t)ng * P.nb + i) * P.nb;
  for (int j = F + tid; j <= i; j += kScoreThreads) {
    float acc = 0.f;
    int flag = 0;
    for (int row = 0; row < P.R; ++row) {
      const float b = beta[row * P.nbp + j];
      const float mr = mu[row];
      acc += __expf(b - mr);  // hardware exp2 of the scaled argument (relative error ~1e-7)
      flag |= (b == mr);
    }
    srow[j] = acc;
    hrow[j] = (uint8_t)flag;
  }
}

template <int SPB, int RT, bool PAGED, bool STAGED>
hipError_t launch_t(const KapParams& P, size_t lds, hipStream_t stream) {
  // Dynamic LDS above the default limit has to be allowed per kernel; remember the largest size
  // granted so far for this instantiation.
  static std::mutex mu;
  static size_t granted = 0;
  if (lds > 48 * 1024) {
    std::lock_guard<std::mutex> lock(mu);
    if (lds > granted) {
      const hipError_t e = hipFuncSetAttribute(
          reinterpret_cast<const void*>(&kap_score_kernel<SPB, RT, PAGED, STAGED>),
          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
      granted = lds;
    }
  }
  hipLaunchKernelGGL((kap_score_kernel<SPB, RT, PAGED, STAGED>),
                     dim3(proxy_slots(P.n_units / P.nb, P.nb)), dim3(kScoreThreads), lds, stream, P);
  return hipGetLastError();
}

template <int SPB, bool PAGED, bool STAGED>
hipError_t launch_rt(const KapParams& P, size_t lds, hipStream_t stream) {
  const int rt = (P.R + 31) / 32;
  if (rt <= 1) return launch_t<SPB, 1, PAGED, STAGED>(P, lds, stream);
  if (rt <= 2) return launch_t<SPB, 2, PAGED, STAGED>(P, lds, stream);
  return launch_t<SPB, 4, PAGED, STAGED>(P, lds, stream);
}

template <int SPB>
hipError_t launch_spb(const KapParams& P, size_t lds, hipStream_t stream) {
  if (P.a.kstage != nullptr) {
    const int waves = (P.n_units / P.nb) * P.nch_all;
    if (P.a.pg.table != nullptr)
      hipLaunchKernelGGL(stage_keys_kernel<true>, dim3((waves + 3) / 4), dim3(256), 0, stream, P);
    else
      hipLaunchKernelGGL(stage_keys_kernel<false>, dim3((waves + 3) / 4), dim3(256), 0, stream, P);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_rt<SPB, false, true>(P, lds, stream);
  }
  if (P.a.pg.table != nullptr) return launch_rt<SPB, true, false>(P, lds, stream);
  return launch_rt<SPB, false, false>(P, lds, stream);
}

}  // namespace

size_t kap_stage_bytes(const Shape& sh) {
  const size_t nch_all = ((size_t)sh.L / sh.s + 31) / 32;
  return (size_t)sh.B * sh.Hkv * nch_all * kStageChunk * sizeof(uint16_t);
}

size_t kap_score_lds_bytes(const Shape& sh) {
  const int R = sh.G * sh.spb;
  if (R > 128) return 0;
  if (sh.spb != 4 && sh.spb != 8 && sh.spb != 16 && sh.spb != 32) return 0;
  const size_t bytes = (size_t)R * (sh.nb + 1) * sizeof(float);
  // LDS per workgroup on gfx950 is 160 KiB; the static part (mu) needs 512 bytes.
  if (bytes + 512 > 160 * 1024) return 0;
  return bytes;
}

hipError_t launch_kap_score(const Shape& sh, const KapScoreArgs& a, hipStream_t stream) {
  KapParams P;
  P.a = a;
  P.Hq = sh.Hq;
  P.Hkv = sh.Hkv;
  P.L = sh.L;
  P.nb = sh.nb;
  P.G = sh.G;
  P.s = sh.s;
  P.R = sh.G * sh.spb;
  P.nbp = sh.nb + 1;
  P.nch_all = (sh.L / sh.s + 31) / 32;
  P.n_units = sh.B * sh.Hkv * sh.nb;
  P.scale = sh.scale;
  const size_t lds = kap_score_lds_bytes(sh);
  switch (sh.spb) {
    case 4: return launch_spb<4>(P, lds, stream);
    case 8: return launch_spb<8>(P, lds, stream);
    case 16: return launch_spb<16>(P, lds, stream);
    default: return launch_spb<32>(P, lds, stream);
  }
}

}  // namespace cosa
