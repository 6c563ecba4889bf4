// KAP block scoring for gfx950 (Sec. 4.2 "Block ranking", Eq. (score); Algorithm A, proxy stage).
//
// A unit is (batch n, KV head g, query block i): its R = G * spb sampled query rows (tokens
// (i*spb + t) * s of the G heads of group g) stay in registers as the MFMA B operand, and the
// waves of a workgroup stride over chunks of 32 sampled keys c < (i+1)*spb (tokens c * s),
// computing the transposed logits K~ Q~^T with bf16 MFMA 32x32x16, applying the causal mask over
// sampled positions (c <= r) and sm_scale, and reducing them straight into per-block maxima
// beta[row][j]. The softmax -> MaxPool -> MaxNorm chain collapses to Pbar = exp(beta - mu) with mu
// the row maximum (the softmax normaliser cancels in the MaxNorm ratio, exp is monotone), so the
// score matrix is never materialised. mu is kept on the fly; a second phase sums exp(beta - mu)
// over the rows of each key block j in a fixed order (deterministic) and raises the HRM flag when
// some row attains its maximum there (beta == mu, exact).
//
// Two kernels share this arithmetic and give bit-identical results:
//   - kap_pair_kernel (staged keys, R <= 32): a persistent workgroup per CU takes two adjacent
//     query blocks of one KV head at a time, so that every key fragment loaded into registers
//     feeds two MFMA tiles (64 rows). The first unit's block maxima live in LDS, the second's in a
//     per-workgroup scratch in global memory (written and read once per item).
//   - kap_score_kernel (every other case): one workgroup per unit, block maxima in LDS.
// Both place work so that each XCD serves as few KV heads as possible (their sampled keys then stay
// in that XCD's L2), heaviest query blocks first.
#include <mutex>

#include "cosa_device.h"
#include "cosa_internal.h"

namespace cosa {
namespace {

#define COSA_LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int kScoreThreads = 512;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kPairMaxWorkgroups = 256;  // persistent grid of kap_pair_kernel (one per CU)
constexpr int kBDepth = 4;  // kap_pair_kernel: passes of unit B's read-back in flight

struct KapParams {
  KapScoreArgs a;
  float* bscr;  // kap_pair_kernel: per-workgroup block maxima of the second unit, [nb][32]
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

// IEEE maximum: no quieting of its inputs (fmaxf would first take each MFMA result's maximum with
// itself); the two differ only on NaN inputs and on the sign of a zero result.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Sampled-key fragments of one 32-key chunk (MFMA A operand) for lane (half, l32): from the staged
// copy through a buffer resource over the head's chunks (the chunk offset a scalar, the lane
// offsets loop-invariant, so no address register is rewritten while loads into the fragment
// registers are in flight), or straight from K (zeros past the last sampled key). A chunk index
// past the last one loads the last chunk again: callers never read it, and every load stays
// unconditional.
template <bool PAGED, bool STAGED>
struct KeyLoader {
  const KapParams& P;
  __amdgpu_buffer_rsrc_t srs;
  int voff0, voff1, n, g, l32, half, nkeys, nchunks;

  __device__ __forceinline__ KeyLoader(const KapParams& P_, int ng, int lane, int nkeys_)
      : P(P_),
        srs(__builtin_amdgcn_make_buffer_rsrc(
            STAGED ? (void*)(P_.a.kstage + (size_t)ng * P_.nch_all * kStageChunk) : nullptr,
            (short)0, STAGED ? P_.nch_all * kStageChunk * 2 : 0, 0x00020000)),
        voff0(lane * 16), voff1(lane * 16 + 4096), n(ng / P_.Hkv), g(ng % P_.Hkv), l32(lane & 31),
        half(lane >> 5), nkeys(nkeys_), nchunks((nkeys_ + 31) >> 5) {}

  __device__ __forceinline__ void operator()(int chunk, bf16x8_t (&kf)[8]) const {
    chunk = min(chunk, nchunks - 1);
    if constexpr (STAGED) {
      const int so = chunk * (kStageChunk * 2);
#pragma unroll
      for (int cc = 0; cc < 8; ++cc)
        kf[cc] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(
            srs, cc < 4 ? voff0 : voff1, so + (cc & 3) * 1024, 0));
    } else {
      const int c = chunk * 32 + l32;
      if (c < nkeys) {
        const uint16_t* kp = sampled_key_row<PAGED>(P, n, g, c) + 8 * half;
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) kf[cc] = as_bf16x8(ldg16(kp + 16 * cc));
      } else {
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) kf[cc] = as_bf16x8(u32x4_t{0u, 0u, 0u, 0u});
      }
    }
  }
};

// A wave's chunks first + 8 k, k < nm, through `process`: chunk k + 1 is loaded while chunk k is
// computed, into two register sets that trade roles from chunk to chunk (a register copy would
// wait for the loads in flight). Every load in the main loop is unconditional, and the last chunks
// run in straight-line code for each possible count, so the wait before a chunk's MFMAs counts
// exactly the younger loads instead of assuming some were skipped. `flush` issues the global
// stores a processed chunk left pending; it runs after the next chunk's loads are issued, so that
// the waits for those loads do not wait for the stores as well.
template <class Load, class Process, class Flush>
__device__ __forceinline__ void wave_chunks(int first, int nchunks, const Load& load,
                                            Process&& process, Flush&& flush) {
  const int nm = first < nchunks ? (nchunks - first + kScoreWaves - 1) / kScoreWaves : 0;
  bf16x8_t kb[2][8];
  // The scheduler barrier keeps a chunk's loads ahead of the previous chunk's MFMAs: left alone,
  // the compiler sinks each load behind the last use of the register it reuses, and the loads
  // then land just before they are needed.
  auto fetch = [&](int chunk, bf16x8_t (&kf)[8]) __attribute__((always_inline)) {
    load(chunk, kf);
    __builtin_amdgcn_sched_barrier(0);
  };
  fetch(first, kb[0]);
  int k = 0;
  for (; k + 2 < nm; k += 2) {
    fetch(first + (k + 1) * kScoreWaves, kb[1]);
    flush();
    process(first + k * kScoreWaves, kb[0]);
    fetch(first + (k + 2) * kScoreWaves, kb[0]);
    flush();
    process(first + (k + 1) * kScoreWaves, kb[1]);
  }
  // nm - k chunks remain (at most 2), the first of them already loaded.
  if (nm - k == 2) {
    fetch(first + (k + 1) * kScoreWaves, kb[1]);
    flush();
    process(first + k * kScoreWaves, kb[0]);
    flush();
    process(first + (k + 1) * kScoreWaves, kb[1]);
  } else if (nm - k == 1) {
    flush();
    process(first + k * kScoreWaves, kb[0]);
  }
  flush();
}

// Logits of one 32-key chunk for one 32-row tile: acc[r] holds sampled key
// chunk*32 + 8 (r/4) + 4 half + r%4 of row l32.
__device__ __forceinline__ f32x16_t chunk_logits(const bf16x8_t (&kf)[8], const bf16x8_t (&qf)[8]) {
  f32x16_t acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) acc = mfma32x32x16(kf[cc], qf[cc], acc);
  return acc;
}

// Causal mask over sampled positions for the rows of query block i (sample ts = row % SPB):
// key > i*SPB + ts is masked. Only a chunk that reaches block i needs it; the branch is uniform
// over the wave.
template <int SPB>
__device__ __forceinline__ void causal_mask(f32x16_t& acc, int chunk, int i, int ts, int half) {
  if (chunk * 32 + 31 > i * SPB) {
    const int rs = i * SPB + ts;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = chunk * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
      acc[r] = key > rs ? -INFINITY : acc[r];
    }
  }
}

// Block maxima of a chunk's logits in the lanes that hold them: keep(slot, j, bm, owner) for each
// block j of the chunk whose maximum this lane holds (slot numbers the calls, 0 .. 3); `owner`
// marks the one lane per (row, block) that stores it. Maxima are taken on the raw logits and scaled once by the caller: x -> sm_scale * x is
// monotone under rounding, so the scaled maximum equals the maximum of the scaled logits exactly.
template <int SPB, class Keep>
__device__ __forceinline__ void block_maxima(const f32x16_t& acc, int chunk, int half, Keep&& keep) {
  if constexpr (SPB == 4) {
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const float bm = vmax(vmax(acc[4 * q4], acc[4 * q4 + 1]), vmax(acc[4 * q4 + 2], acc[4 * q4 + 3]));
      keep(q4, chunk * 8 + 2 * q4 + half, bm, true);
    }
  } else if constexpr (SPB == 8) {
    // Block chunk * 4 + q4 holds keys 8 q4 + 4 half .. + 3 of this lane. Per pair of blocks
    // (2 pr, 2 pr + 1) one swap of lane halves leaves the first block's maximum in lanes 0-31 and
    // the second's in lanes 32-63.
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      const float m0 = vmax(vmax(acc[8 * pr], acc[8 * pr + 1]), vmax(acc[8 * pr + 2], acc[8 * pr + 3]));
      const float m1 =
          vmax(vmax(acc[8 * pr + 4], acc[8 * pr + 5]), vmax(acc[8 * pr + 6], acc[8 * pr + 7]));
      const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, m0),
                                                      __builtin_bit_cast(unsigned, m1), false, false);
      const unsigned r0 = r[0], r1 = r[1];
      keep(pr, chunk * 4 + 2 * pr + half,
           vmax(__builtin_bit_cast(float, r0), __builtin_bit_cast(float, r1)), true);
    }
  } else if constexpr (SPB == 16) {
#pragma unroll
    for (int b2 = 0; b2 < 2; ++b2) {
      float bm = acc[8 * b2];
#pragma unroll
      for (int r = 1; r < 8; ++r) bm = vmax(bm, acc[8 * b2 + r]);
      keep(b2, chunk * 2 + b2, half_max(bm), b2 == half);
    }
  } else {
    float bm = acc[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) bm = vmax(bm, acc[r]);
    keep(0, chunk, half_max(bm), half == 0);
  }
}

// Q~^T fragments of one 32-row tile of unit (ng, i): row l32 = (head offset hh, sample t) -> token
// (i*SPB + t) * s; rows >= R (or an absent unit) are zero.
template <int SPB>
__device__ __forceinline__ void load_query_tile(const KapParams& P, int ng, int i, int row, int half,
                                                bool valid, bf16x8_t (&qf)[8]) {
  if (valid && row < P.R) {
    const int n = ng / P.Hkv, g = ng % P.Hkv;
    const int hh = row / SPB, t = row % SPB;
    const size_t tok = (size_t)(i * SPB + t) * P.s;
    const uint16_t* qp = P.a.q + ((size_t)(n * P.Hq + g * P.G + hh) * P.L + tok) * kHeadDim + 8 * half;
#pragma unroll
    for (int c = 0; c < 8; ++c) qf[c] = as_bf16x8(ldg16(qp + 16 * c));
  } else {
#pragma unroll
    for (int c = 0; c < 8; ++c) qf[c] = as_bf16x8(u32x4_t{0u, 0u, 0u, 0u});
  }
}

// Summation order of a key block's score over its rows (fixed, so that every kernel gives the
// same bits): rows in groups of 4 summed in order, (((e0 + e1) + e2) + e3); the 8 groups of each
// 32 rows as the tree ((g0 + g1) + (g2 + g3)) + ((g4 + g5) + (g6 + g7)), absent groups 0; the
// 32-row blocks in order. e = exp(beta - mu) is the hardware exp2 of beta * log2(e) - mu2, one
// fused multiply-add, with mu2 = mu * log2(e) formed once per row: the argument's rounding error
// is relative to |beta| (about 1e-7 of it, a relative error of e below 1e-5 at the logit ranges
// of attention), and a row's maximum gives e = 1 to within that error. The HRM flag compares beta
// with mu itself, exactly.
constexpr float kLog2e = 1.44269504088896341f;
__device__ __forceinline__ float exp_arg(float b, float m2) { return fmaf(b, kLog2e, -m2); }
__device__ __forceinline__ float group4(const float (&b)[4], const float (&mr)[4],
                                        const float (&mr2)[4], int& fl) {
  float s = __builtin_amdgcn_exp2f(exp_arg(b[0], mr2[0]));
#pragma unroll
  for (int r = 1; r < 4; ++r) s += __builtin_amdgcn_exp2f(exp_arg(b[r], mr2[r]));
#pragma unroll
  for (int r = 0; r < 4; ++r) fl |= (b[r] == mr[r]);
  return s;
}

// Score and HRM flag of key block j from its R block maxima (`beta(row, b)` fills rows row ..
// row + 3), the row maxima mu and mu2 = mu * log2(e).
template <class Beta>
__device__ __forceinline__ void score_column(int R, const float* mu, const float* mu2,
                                             Beta&& beta, float& score, uint8_t& flag) {
  float acc = 0.f;
  int fl = 0;
  for (int rb = 0; rb < R; rb += 32) {  // R = G * spb is a multiple of 4
    float g[8];
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const int row = rb + 4 * p;
      g[p] = 0.f;
      if (row < R) {
        float b[4], mr[4], mr2[4];
        beta(row, b);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          mr[r] = mu[row + r];
          mr2[r] = mu2[row + r];
        }
        g[p] = group4(b, mr, mr2, fl);
      }
    }
    acc += ((g[0] + g[1]) + (g[2] + g[3])) + ((g[4] + g[5]) + (g[6] + g[7]));
  }
  score = acc;
  flag = (uint8_t)fl;
}

// One unit per workgroup. STAGED: the sampled keys come from the staged copy (P.a.kstage).
template <int SPB, int RT, bool PAGED, bool STAGED>
__global__ __launch_bounds__(kScoreThreads) void kap_score_kernel(const KapParams P) {
  extern __shared__ float beta[];  // [R][nbp]
  __shared__ float mu[RT * 32], mu2[RT * 32];
  __shared__ float wmax[kScoreWaves][RT * 32];  // each wave's row maxima

  int ng, i;
  if (!proxy_unit(blockIdx.x, P.n_units / P.nb, P.nb, ng, i)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  // Packed sequences: the candidates are the blocks F .. i of block i's own sequence.
  int seq;
  const int F = pack_first(P.a.pack, i, seq);
  auto cand = [&](int j) { return (unsigned)(j - F) <= (unsigned)(i - F); };

  bf16x8_t qf[RT][8];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) load_query_tile<SPB>(P, ng, i, rt * 32 + l32, half, true, qf[rt]);

  // rmax[rt]: maximum of the scaled block maxima this lane produced for row rt * 32 + l32.
  float rmax[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) rmax[rt] = -INFINITY;
  const KeyLoader<PAGED, STAGED> load(P, ng, lane, (i + 1) * SPB);
  wave_chunks((F * SPB >> 5) + w, load.nchunks, load, [&](int chunk, const bf16x8_t (&kf)[8]) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      f32x16_t acc = chunk_logits(kf, qf[rt]);
      const int row = rt * 32 + l32;
      causal_mask<SPB>(acc, chunk, i, row % SPB, half);
      float* brow = beta + row * P.nbp;
      const bool row_ok = row < P.R;
      block_maxima<SPB>(acc, chunk, half, [&](int, int j, float bm, bool owner) {
        const float bs = bm * P.scale;
        const bool c = cand(j);
        if (row_ok && owner && c) brow[j] = bs;
        rmax[rt] = c ? vmax(rmax[rt], bs) : rmax[rt];
      });
    }
  }, [] {});

  // The two lanes of a row took different blocks; then the waves' maxima meet in LDS.
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const float v = half_max(rmax[rt]);
    if (half == 0) wmax[w][rt * 32 + l32] = v;
  }
  __syncthreads();
  if (tid < P.R) {
    float v = wmax[0][tid];
#pragma unroll
    for (int x = 1; x < kScoreWaves; ++x) v = fmaxf(v, wmax[x][tid]);
    mu[tid] = v;
    mu2[tid] = v * kLog2e;
  }
  __syncthreads();

  float* srow = P.a.score + ((size_t)ng * P.nb + i) * P.nb;
  uint8_t* hrow = P.a.hrm + ((size_t)ng * P.nb + i) * P.nb;
  for (int j = F + tid; j <= i; j += kScoreThreads)
    score_column(P.R, mu, mu2, [&](int row, float (&b)[4]) {
#pragma unroll
      for (int r = 0; r < 4; ++r) b[r] = beta[(row + r) * P.nbp + j];
    }, srow[j], hrow[j]);
}

// Work items of kap_pair_kernel: item q is KV head ng, pair k (units nb-1-2k and nb-2-2k). When the
// NG heads split evenly over the 8 XCDs, q % 8 is the XCD and XCD x takes heads ng = x (mod 8);
// pairs go heaviest first.
__device__ __forceinline__ void pair_item(int q, int NG, int& ng, int& k) {
  if (NG % 8 == 0) {
    const int x = q & 7, local = q >> 3, nh = NG >> 3;
    ng = x + 8 * (local % nh);
    k = local / nh;
  } else {
    ng = q % NG;
    k = q / NG;
  }
}

// One item of kap_pair_kernel and this wave's share of its key chunks (all wave-uniform).
// The chunks [c0, nch) of the key range split three ways:
//   - [c0, cF): chunks holding blocks before unit A's sequence (packed sequences only);
//   - [cF, cM): chunks below every row's diagonal whose blocks are all candidates of both units,
//     dealt round-robin from wave 0 (the fast path);
//   - [cM, nch): chunks reaching a diagonal, dealt from wave 7 down, so that they land on the
//     waves with fewer fast chunks.
// A wave's k-th chunk is seq(k): its prefix chunks, then its fast ones, then its tail ones.
struct PairItem {
  int ng, iA, iB, FA, FB, nch, c0, cF, cM, npre, nfast, ntail;
  bool hasB;
  __amdgpu_buffer_rsrc_t keys;  // the head's staged sampled keys

  __device__ __forceinline__ int seq(int k, int w) const {
    if (k < npre) return c0 + w + kScoreWaves * k;
    k -= npre;
    if (k < nfast) return cF + w + kScoreWaves * k;
    return cM + (kScoreWaves - 1 - w) + kScoreWaves * (k - nfast);
  }
};

template <int SPB>
__device__ __forceinline__ PairItem pair_plan(const KapParams& P, int q, int w) {
  PairItem it;
  int pk;
  pair_item(q, P.n_units / P.nb, it.ng, pk);
  it.iA = P.nb - 1 - 2 * pk;
  it.iB = it.iA - 1;
  it.hasB = it.iB >= 0;
  int seq;
  it.FA = pack_first(P.a.pack, it.iA, seq);
  it.FB = it.hasB ? pack_first(P.a.pack, it.iB, seq) : it.FA;  // FB <= FA
  it.nch = ((it.iA + 1) * SPB + 31) >> 5;
  it.c0 = (it.FB * SPB) >> 5;
  it.cF = max(it.c0, (it.FA * SPB + 31) >> 5);
  it.cM = max(it.cF, it.hasB && it.iB * SPB >= 31 ? (it.iB * SPB - 31) / 32 + 1 : 0);
  it.cM = min(it.cM, it.nch);
  it.cF = min(it.cF, it.cM);
  auto count = [](int from, int to) { return from < to ? (to - from + kScoreWaves - 1) / kScoreWaves : 0; };
  it.npre = count(it.c0 + w, it.cF);
  it.nfast = count(it.cF + w, it.cM);
  it.ntail = count(it.cM + (kScoreWaves - 1 - w), it.nch);
  it.keys = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(P.a.kstage + (size_t)it.ng * P.nch_all * kStageChunk), (short)0,
      P.nch_all * kStageChunk * 2, 0x00020000);
  return it;
}

// Workgroup barrier for LDS data only: __syncthreads() would also wait for every global load in
// flight, the next item's prefetch included.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Two adjacent query blocks iA = nb-1-2k and iB = iA-1 of one KV head per item, R <= 32 rows each:
// tile 0 holds unit A's rows, tile 1 unit B's, and both multiply every key fragment (staged keys).
// A persistent grid of G workgroups (a multiple of 8) walks the items: in round r workgroup
// b = 8c + x takes item q = r*G + 8c' + x with c' = c in even rounds and G/8 - 1 - c in odd ones
// (snake order, so that heavy and light items even out), on the XCD x the item's head maps to.
// While unit A's scores are formed, the next item's query tiles and first two key chunks load.
template <int SPB>
__global__ __launch_bounds__(kScoreThreads) void kap_pair_kernel(const KapParams P) {
  extern __shared__ float beta[];  // unit A: [32][nbp] (rows >= R unused)
  __shared__ float muA[32], muB[32], muA2[32], muB2[32];
  __shared__ float wmax[kScoreWaves][2][32];
  // The item's query rows, [64][256 B] (tile t, row l at 32 t + l), 16-byte slot s of row rho
  // stored at slot s ^ (rho % 16) so that the operand reads hit 16 different slots. Loaded once per
  // workgroup by direct global -> LDS loads, then read by every wave.
  __shared__ __attribute__((aligned(16))) uint16_t qst[64 * kHeadDim];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  const int NG = P.n_units / P.nb, Q = NG * ((P.nb + 1) >> 1);
  const int G = gridDim.x, c8 = blockIdx.x >> 3, x8 = blockIdx.x & 7;
  auto item_q = [&](int r) { return r * G + 8 * ((r & 1) ? (G >> 3) - 1 - c8 : c8) + x8; };
  // Unit B's block maxima, [nb][32] per workgroup.
  float* const bB = P.bscr + (size_t)blockIdx.x * P.nb * 32;
  const bool row_ok = l32 < P.R;
  const int voff0 = lane * 16, voff1 = lane * 16 + 4096;

  // Staged keys of chunk `chunk` (clamped to the item's last one: such a chunk is never read,
  // and every load stays unconditional).
  auto load = [&](const PairItem& it, int chunk, bf16x8_t (&kf)[8]) __attribute__((always_inline)) {
    const int so = min(chunk, it.nch - 1) * (kStageChunk * 2);
#pragma unroll
    for (int cc = 0; cc < 8; ++cc)
      kf[cc] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(it.keys, cc < 4 ? voff0 : voff1,
                                                               so + (cc & 3) * 1024, 0));
  };
  auto fetch = [&](const PairItem& it, int chunk, bf16x8_t (&kf)[8]) __attribute__((always_inline)) {
    load(it, chunk, kf);
    __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the MFMAs that follow
  };

  bf16x8_t qf[2][8], kb0[8], kb1[8];
  // Query rows and first key chunk of item q (the plan is recomputed where it is used, which costs
  // a few scalar instructions and keeps one plan live at a time). Wave w moves query rows
  // 8w .. 8w + 7 (two 1 KiB loads of four rows); a row outside the item (>= R, or unit B absent)
  // loads row 0 of the head group, whose products are never read. The key fetches are
  // unconditional (a chunk the wave does not have loads a clamped one that is never read), so they
  // load straight into the registers the item's loop reads, with no copy.
  auto prefetch = [&](int q) __attribute__((always_inline)) {
    const PairItem nx = pair_plan<SPB>(P, q, w);
    const int n = nx.ng / P.Hkv, g = nx.ng % P.Hkv;
    const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(P.a.q + (size_t)(n * P.Hq + g * P.G) * P.L * kHeadDim), (short)0,
        P.G * P.L * kHeadDim * 2, 0x00020000);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      // Rows rho = r0 + lane / 16 of tile t = r0 / 32: row l = lb + lane / 16 of the tile, with lb
      // a multiple of 4 and so is SPB; hence l / SPB = lb / SPB, l % SPB = lb % SPB + lane / 16,
      // and l < R exactly when lb < R (R a multiple of 4). All but the lane term are wave-uniform
      // (formed in scalar registers, nothing held in vector registers across the item).
      const int r0 = 8 * w + 4 * u;  // first of the four rows
      const int t = r0 >> 5, lb = r0 & 31, lr = lane >> 4;
      const int iu = t ? nx.iB : nx.iA;
      const bool real = lb < P.R && (t == 0 || nx.hasB);
      const int sbase =
          real ? ((lb / SPB) * P.L + (iu * SPB + lb % SPB) * P.s) * (kHeadDim * 2) : 0;
      const int voff = sbase + (real ? lr * P.s * (kHeadDim * 2) : 0) +
                       16 * ((lane & 15) ^ ((lb + lr) & 15));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(qrs, COSA_LDS_PTR(qst + r0 * kHeadDim), 16, voff, 0,
                                               0, 0);
    }
    fetch(nx, nx.seq(nx.npre, w), kb0);
  };
  // The item's second key chunk.
  auto prefetch_k1 = [&](int q) __attribute__((always_inline)) {
    const PairItem nx = pair_plan<SPB>(P, q, w);
    fetch(nx, nx.seq(nx.npre + 1, w), kb1);
  };
  if (item_q(0) >= Q) return;
  prefetch(item_q(0));
  prefetch_k1(item_q(0));

  for (int r = 0;; ++r) {
    const PairItem it = pair_plan<SPB>(P, item_q(r), w);
    // This item's query rows, and the prefetched key chunks (issued during the previous item's
    // scores, so long since landed). A wait the compiler sees: the main loop's waits then start
    // from nothing in flight.
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    lds_barrier();
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int rho = 32 * t + l32;
#pragma unroll
      for (int c = 0; c < 8; ++c)
        qf[t][c] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(
            qst + rho * kHeadDim + 8 * ((2 * c + half) ^ (rho & 15))));
    }
    const int iA = it.iA, iB = it.iB, FA = it.FA, FB = it.FB;
    const bool hasB = it.hasB;
    auto candA = [&](int j) { return (unsigned)(j - FA) <= (unsigned)(iA - FA); };
    auto candB = [&](int j) { return (unsigned)(j - FB) <= (unsigned)(iB - FB); };
    float rmaxA = -INFINITY, rmaxB = -INFINITY;
    float* const browA = beta + l32 * P.nbp;

    auto mma = [&](const bf16x8_t (&kf)[8], f32x16_t& x0, f32x16_t& x1) __attribute__((always_inline)) {
#pragma unroll
      for (int r2 = 0; r2 < 16; ++r2) x0[r2] = x1[r2] = 0.f;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {  // the two tiles' chains interleaved
        x0 = mfma32x32x16(kf[cc], qf[0][cc], x0);
        x1 = mfma32x32x16(kf[cc], qf[1][cc], x1);
      }
    };
    // A fast chunk: no mask, no test, every store unconditional (rows >= R of beta are never
    // read; for SPB >= 16 both lanes of a block store the same value).
    auto epi_fast = [&](int chunk, const f32x16_t& x0, const f32x16_t& x1) __attribute__((always_inline)) {
      block_maxima<SPB>(x0, chunk, half, [&](int, int j, float bm, bool) {
        const float bs = bm * P.scale;
        browA[j] = bs;
        rmaxA = vmax(rmaxA, bs);
      });
      block_maxima<SPB>(x1, chunk, half, [&](int, int j, float bm, bool) {
        const float bs = bm * P.scale;
        bB[j * 32 + l32] = bs;
        rmaxB = vmax(rmaxB, bs);
      });
    };
    // Any other chunk: masks and candidate tests.
    auto process_slow = [&](int chunk, const bf16x8_t (&kf)[8]) __attribute__((always_inline)) {
      f32x16_t a0, a1;
      mma(kf, a0, a1);
      causal_mask<SPB>(a0, chunk, iA, l32 % SPB, half);
      block_maxima<SPB>(a0, chunk, half, [&](int, int j, float bm, bool owner) {
        const float bs = bm * P.scale;
        const bool c = candA(j);
        if (row_ok && owner && c) browA[j] = bs;
        rmaxA = c ? vmax(rmaxA, bs) : rmaxA;
      });
      if (hasB) {
        causal_mask<SPB>(a1, chunk, iB, l32 % SPB, half);
        block_maxima<SPB>(a1, chunk, half, [&](int, int j, float bm, bool) {
          const float bs = bm * P.scale;
          const bool c = candB(j);
          if (c) bB[j * 32 + l32] = bs;
          rmaxB = c ? vmax(rmaxB, bs) : rmaxB;
        });
      }
    };
    // The interleave of one chunk's 16 MFMAs with the previous chunk's epilogue: the epilogue's
    // vector instructions issue in the shadow of the MFMAs instead of after them.
    auto interleave = [] __attribute__((always_inline)) {
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // two VALU
      }
    };
    auto sq = [&](int k) { return it.seq(k, w); };

    // Prefix chunks (packed sequences only), one at a time.
    for (int k = 0; k < it.npre; ++k) {
      bf16x8_t t[8];
      load(it, sq(k), t);
      process_slow(sq(k), t);
    }
    // Fast chunks in pairs, software-pipelined: the MFMAs of one chunk beside the epilogue of the
    // previous one, the keys two chunks ahead loading meanwhile. kb0 and kb1 hold chunks npre and
    // npre + 1 on entry.
    int k = it.npre;
    const int kend = it.npre + it.nfast + it.ntail;
    const int nfp = it.nfast & ~1;
    if (nfp > 0) {
      f32x16_t xa0, xa1, xb0, xb1;
      mma(kb0, xa0, xa1);
      for (int t = 0; t + 2 < nfp; t += 2) {
        fetch(it, sq(k + t + 2), kb0);
        mma(kb1, xb0, xb1);
        epi_fast(sq(k + t), xa0, xa1);
        interleave();
        fetch(it, sq(k + t + 3), kb1);
        mma(kb0, xa0, xa1);
        epi_fast(sq(k + t + 1), xb0, xb1);
        interleave();
      }
      // Past the hot loop a fetch runs only for a chunk the wave has (outside the loop a
      // conditional load costs nothing).
      if (k + nfp < kend) fetch(it, sq(k + nfp), kb0);
      mma(kb1, xb0, xb1);
      epi_fast(sq(k + nfp - 2), xa0, xa1);
      interleave();
      epi_fast(sq(k + nfp - 1), xb0, xb1);
      k += nfp;
      if (k + 1 < kend) fetch(it, sq(k + 1), kb1);
    }
    // The rest (an odd fast chunk and the tail, a few per wave): kb0 and kb1 hold chunks k, k + 1.
    for (; k < kend; ++k) {
      if (k < it.npre + it.nfast) {
        f32x16_t x0, x1;
        mma(kb0, x0, x1);
        epi_fast(sq(k), x0, x1);
      } else {
        process_slow(sq(k), kb0);
      }
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) kb0[cc] = kb1[cc];
      if (k + 2 < kend) fetch(it, sq(k + 2), kb1);
    }

    {
      const float va = half_max(rmaxA), vb = half_max(rmaxB);
      if (half == 0) {
        wmax[w][0][l32] = va;
        wmax[w][1][l32] = vb;
      }
    }
    __syncthreads();  // also orders the scratch stores of every wave before the reads below

    // Unit B's block maxima, read back in passes of 128 key blocks: lane group tid / 4 takes block
    // FB + tid / 4 + 128 m in pass m, lane q = tid % 4 its rows 8q .. 8q + 7 (two 16-byte loads;
    // 4 lanes read one block's 128 bytes). A lane forms the first level of the fixed tree over its
    // two 4-row groups itself, and the other two levels come from two DPP adds. The first kBDepth
    // passes load here, each later one after the pass kBDepth before it is formed, into the
    // registers that pass has just read (no register copy, which would wait for the load). Every
    // load and store is unconditional, in whole rounds, so that the compiler's waits count exactly:
    // a pass past the last repeats its loads, and a store that must not happen (a lane other than
    // q = 0, a block past iB, a padding pass) gets an offset past the end of its row's buffer
    // resource, which drops it. Blocks past nb - 1 read 0 (range check). Unit B's scores come
    // before the next item's prefetch and unit A's scores, so that no load but these is in flight
    // while they form.
    const int q4 = tid & 3, jb0 = FB + (tid >> 2);
    // Without unit B (the last item of an odd nb) one pass runs with every store dropped.
    const int npass = hasB ? (iB - FB + 128) >> 7 : 1;
    const __amdgpu_buffer_rsrc_t brs =
        __builtin_amdgcn_make_buffer_rsrc((void*)bB, (short)0, P.nb * 32 * 4, 0x00020000);
    const int bvoff = jb0 * 128 + 32 * q4;
    auto bload = [&](int m, u32x4_t (&v)[2]) __attribute__((always_inline)) {
      const int o = bvoff + 16384 * min(m, npass - 1);
      v[0] = __builtin_amdgcn_raw_buffer_load_b128(brs, o, 0, 0);
      v[1] = __builtin_amdgcn_raw_buffer_load_b128(brs, o + 16, 0, 0);
    };
    u32x4_t bv[kBDepth][2];
#pragma unroll
    for (int m = 0; m < kBDepth; ++m) bload(m, bv[m]);
    if (tid < 64 && (tid & 31) < P.R) {
      const int t = tid >> 5, row = tid & 31;
      float v = wmax[0][t][row];
#pragma unroll
      for (int x = 1; x < kScoreWaves; ++x) v = fmaxf(v, wmax[x][t][row]);
      (t ? muB : muA)[row] = v;
      (t ? muB2 : muA2)[row] = v * kLog2e;
    }
    lds_barrier();

    float* const srow = P.a.score + ((size_t)it.ng * P.nb + iA) * P.nb;
    uint8_t* const hrow = P.a.hrm + ((size_t)it.ng * P.nb + iA) * P.nb;
    {
      // The lane's rows are formed afresh here (an opaque copy of the lane index): a value kept from
      // the item's start would be spilled, and its reload would wait for every load in flight.
      int q4o = tid & 3;
      asm volatile("" : "+v"(q4o));
      float mb[2][4], mb2[2][4];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) {
          mb[h][r2] = muB[8 * q4o + 4 * h + r2];
          mb2[h][r2] = muB2[8 * q4o + 4 * h + r2];
        }
      // Unit B's output row (query block iB, the row before unit A's): its blocks 0 .. iB.
      const int nB = hasB ? iB + 1 : 0;
      const __amdgpu_buffer_rsrc_t sB = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(hasB ? srow - P.nb : srow), (short)0, nB * 4, 0x00020000);
      const __amdgpu_buffer_rsrc_t hB = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(hasB ? hrow - P.nb : hrow), (short)0, nB, 0x00020000);
      auto pass = [&](int m, const u32x4_t (&v)[2]) __attribute__((always_inline)) {
        // Groups 2q and 2q + 1 (rows 8q .. 8q + 3, 8q + 4 .. 8q + 7), formed on every lane and
        // selected (rows past R hold stale values, absent groups count 0): no branch.
        float g[2];
        int fl = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          float b[4];
#pragma unroll
          for (int r2 = 0; r2 < 4; ++r2) b[r2] = __builtin_bit_cast(float, (uint32_t)v[h][r2]);
          int f = 0;
          g[h] = group4(b, mb[h], mb2[h], f);
          const bool ok = 8 * q4 + 4 * h < P.R;
          g[h] = ok ? g[h] : 0.f;
          fl |= ok ? f : 0;
        }
        float t = g[0] + g[1];                   // (g_2q + g_2q+1)
        t += dpp_mov<0xB1>(t);                   // quad_perm [1,0,3,2]: ((g0 + g1) + (g2 + g3)), ...
        t += dpp_mov<0x4E>(t);                   // quad_perm [2,3,0,1]: the two halves
        fl |= __builtin_amdgcn_mov_dpp(fl, 0xB1, 0xF, 0xF, true);
        fl |= __builtin_amdgcn_mov_dpp(fl, 0x4E, 0xF, 0xF, true);
        const int jo = (q4 == 0 && m < npass) ? jb0 + 128 * m : (1 << 28);  // else dropped
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, t), sB, jo * 4, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b8((uint8_t)fl, hB, jo, 0, 0);
      };
      const int m_last = (npass - 1) / kBDepth * kBDepth;  // first pass of the last round
      for (int m0 = 0; m0 < m_last; m0 += kBDepth) {
#pragma unroll
        for (int mm = 0; mm < kBDepth; ++mm) {
          pass(m0 + mm, bv[mm]);
          __builtin_amdgcn_sched_barrier(0);
          bload(m0 + mm + kBDepth, bv[mm]);
        }
      }
#pragma unroll
      for (int mm = 0; mm < kBDepth; ++mm) pass(m_last + mm, bv[mm]);
    }

    // The next item: its query tiles and first two key chunks load while unit A's scores form.
    // After the last item the current one is fetched again (nothing reads it): an unconditional
    // prefetch loads straight into the registers the next item's loop reads, with no copy.
    // The second key chunk's loads go out after this wave's first column of unit A's scores, so
    // that their issue overlaps that column's arithmetic instead of stalling in one burst.
    const bool more = item_q(r + 1) < Q;
    const int qn = item_q(more ? r + 1 : r);
    prefetch(qn);
    auto column_a = [&](int j) __attribute__((always_inline)) {
      score_column(P.R, muA, muA2, [&](int row, float (&b)[4]) {
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) b[r2] = beta[(row + r2) * P.nbp + j];
      }, srow[j], hrow[j]);
    };
    if (FA + tid <= iA) column_a(FA + tid);
    prefetch_k1(qn);
    for (int j = FA + tid + kScoreThreads; j <= iA; j += kScoreThreads) column_a(j);
    lds_barrier();  // beta and the row maxima are reused by the next item
    if (!more) break;
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // the last (unused) prefetch has landed
}

// Dynamic LDS above the default limit has to be allowed per kernel; remember the largest size
// granted so far for each kernel.
hipError_t allow_lds(const void* fn, size_t lds, std::mutex& mu, size_t& granted) {
  if (lds <= 48 * 1024) return hipSuccess;
  std::lock_guard<std::mutex> lock(mu);
  if (lds > granted) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    granted = lds;
  }
  return hipSuccess;
}

template <int SPB, int RT, bool PAGED, bool STAGED>
hipError_t launch_t(const KapParams& P, size_t lds, hipStream_t stream) {
  static std::mutex mu;
  static size_t granted = 0;
  const hipError_t e = allow_lds(
      reinterpret_cast<const void*>(&kap_score_kernel<SPB, RT, PAGED, STAGED>), lds, mu, granted);
  if (e != hipSuccess) return e;
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

// Persistent grid of kap_pair_kernel: a multiple of 8 workgroups, at most one per CU.
int pair_grid(const Shape& sh) {
  const long long items = (long long)sh.B * sh.Hkv * ((sh.nb + 1) / 2);
  const long long g = (items + 7) / 8 * 8;
  return (int)(g < kPairMaxWorkgroups ? g : kPairMaxWorkgroups);
}

template <int SPB>
hipError_t launch_pair(const KapParams& P, int grid, size_t lds, hipStream_t stream) {
  static std::mutex mu;
  static size_t granted = 0;
  const hipError_t e =
      allow_lds(reinterpret_cast<const void*>(&kap_pair_kernel<SPB>), lds, mu, granted);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((kap_pair_kernel<SPB>), dim3(grid), dim3(kScoreThreads), lds, stream, P);
  return hipGetLastError();
}

size_t stage_keys_bytes(const Shape& sh) {
  const size_t nch_all = ((size_t)sh.L / sh.s + 31) / 32;
  return (size_t)sh.B * sh.Hkv * nch_all * kStageChunk * sizeof(uint16_t);
}

// Dynamic LDS of kap_pair_kernel: unit A's block maxima with 32 rows whatever R (its unconditional
// stores reach them).
size_t pair_lds_bytes(const Shape& sh) { return (size_t)32 * (sh.nb + 1) * sizeof(float); }

bool pair_applies(const Shape& sh) {
  // Static LDS: 2.5 KiB of row maxima (per wave, per row and scaled) and 16 KiB of query rows.
  // The query rows of one head group are addressed by 32-bit offsets.
  return sh.G * sh.spb <= 32 && pair_lds_bytes(sh) + 18944 <= 160 * 1024 &&
         (size_t)sh.G * sh.L * kHeadDim * 2 < ((size_t)1 << 31);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

template <int SPB>
hipError_t launch_spb(const Shape& sh, KapParams& P, size_t lds, hipStream_t stream) {
  if (P.a.kstage != nullptr) {
    const int waves = (P.n_units / P.nb) * P.nch_all;
    if (P.a.pg.table != nullptr)
      hipLaunchKernelGGL(stage_keys_kernel<true>, dim3((waves + 3) / 4), dim3(256), 0, stream, P);
    else
      hipLaunchKernelGGL(stage_keys_kernel<false>, dim3((waves + 3) / 4), dim3(256), 0, stream, P);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (pair_applies(sh)) {
      P.bscr = reinterpret_cast<float*>(reinterpret_cast<char*>(P.a.kstage) +
                                        align256(stage_keys_bytes(sh)));
      return launch_pair<SPB>(P, pair_grid(sh), pair_lds_bytes(sh), stream);
    }
    return launch_rt<SPB, false, true>(P, lds, stream);
  }
  if (P.a.pg.table != nullptr) return launch_rt<SPB, true, false>(P, lds, stream);
  return launch_rt<SPB, false, false>(P, lds, stream);
}

}  // namespace

size_t kap_stage_bytes(const Shape& sh) {
  // Staged sampled keys, then (when the paired kernel runs) its per-workgroup block maxima.
  const size_t keys = stage_keys_bytes(sh);
  if (!pair_applies(sh)) return keys;
  return align256(keys) + (size_t)pair_grid(sh) * sh.nb * 32 * sizeof(float);
}

size_t kap_score_lds_bytes(const Shape& sh) {
  const int R = sh.G * sh.spb;
  if (R > 128) return 0;
  if (sh.spb != 4 && sh.spb != 8 && sh.spb != 16 && sh.spb != 32) return 0;
  const size_t bytes = (size_t)R * (sh.nb + 1) * sizeof(float);
  // LDS per workgroup on gfx950 is 160 KiB; the static part (row maxima, per wave and per row,
  // and scaled) needs at most 5 KiB.
  if (bytes + 5120 > 160 * 1024) return 0;
  return bytes;
}

hipError_t launch_kap_score(const Shape& sh, const KapScoreArgs& a, hipStream_t stream) {
  KapParams P;
  P.a = a;
  P.bscr = nullptr;
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
    case 4: return launch_spb<4>(sh, P, lds, stream);
    case 8: return launch_spb<8>(sh, P, lds, stream);
    case 16: return launch_spb<16>(sh, P, lds, stream);
    default: return launch_spb<32>(sh, P, lds, stream);
  }
}

}  // namespace cosa
