// Flag-grouped sort and stage-1 cut for gfx950 (Sec. 4.2 "Flag-grouped sorting", Eq. (mkap);
// Algorithm A, proxy stage).
//
// One row per (batch n, KV head g, query block i). The causal candidates (j <= i, from the first
// block of the packed sequence when several sequences share the token axis) become 64-bit keys
// (hrm << 63) | (float bits of score << 32) | (0xffffffff - j): scores are non-negative, so their
// bit patterns order like the values, and comparing keys orders by HRM flag, then score, then
// ascending block index. The kept set is the K_i largest keys, in descending key order (the HRM
// group first, each group by descending score). By fraction, K_i follows from the row length
// (integer arithmetic on the budget in millionths): a radix selection over 8-bit digits finds the
// K_i-th largest key, and only the keys at or above it are sorted. Rows of up to 2048 candidates
// take that cut on one wavefront each (keys in registers, no workgroup barrier); longer rows, or
// kept sets over 1024, on a workgroup per row. By top-p the cut depends on the sorted scores, so
// the whole row is sorted by a workgroup, as it is when every candidate is kept. The top-p sums run in fp64 in one fixed order, on
// one lane: the row total over ascending block index, then the running mass down the sorted order
// until it reaches p of the total (each score widens exactly, so the cut depends on nothing but
// that order). Ascending visit order re-sorts the kept set by block index. Keys are distinct, so
// every path yields the one ordering. The row of `order` is written in full: K_i block ids
// followed by -1. Scores are expected to be finite and non-negative (the proxy's are).
#include <mutex>

#include "cosa_device.h"
#include "cosa_internal.h"

namespace cosa {
namespace {

constexpr int kSelThreads = 256;

struct SelParams {
  KapSelectArgs a;
  int nb, n_units;
};

__device__ __forceinline__ uint64_t make_key(uint8_t h, float s, int j) {
  const uint32_t sb = __float_as_uint(s) & 0x7fffffffu;
  return ((uint64_t)(h != 0) << 63) | ((uint64_t)sb << 32) | (uint64_t)(0xffffffffu - (uint32_t)j);
}
__device__ __forceinline__ int key_index(uint64_t key) {
  return (int)(0xffffffffu - (uint32_t)(key & 0xffffffffu));
}
__device__ __forceinline__ float key_score(uint64_t key) {
  return __uint_as_float((uint32_t)(key >> 32) & 0x7fffffffu);
}

// Sort keys[0..n2) in descending order (n2 a power of two).
__device__ void bitonic_desc(uint64_t* keys, int n2, int tid) {
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = tid; t < (n2 >> 1); t += kSelThreads) {
        const int lo = 2 * t - (t & (stride - 1));  // pair t of the stage (stride a power of two)
        const int hi = lo + stride;
        const uint64_t x = keys[lo], y = keys[hi];
        const bool first_half_desc = (lo & size) == 0;
        if (first_half_desc ? (x < y) : (x > y)) {
          keys[lo] = y;
          keys[hi] = x;
        }
      }
      __syncthreads();
    }
  }
}

// Sort keys[0..n2) in descending order within one wavefront (n2 a power of two): lane l takes the
// compare-exchanges l, l + 64, ... of each stage; LDS operations of one wave complete in issue
// order, so the stages need no workgroup barrier.
__device__ void bitonic_desc_wave(uint64_t* keys, int n2, int lane) {
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = lane; t < (n2 >> 1); t += 64) {
        const int lo = 2 * t - (t & (stride - 1));
        const int hi = lo + stride;
        const uint64_t x = keys[lo], y = keys[hi];
        const bool first_half_desc = (lo & size) == 0;
        if (first_half_desc ? (x < y) : (x > y)) {
          keys[lo] = y;
          keys[hi] = x;
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
  }
}

// The keys among keys[0..n) that are the K largest (1 <= K <= n, keys distinct): a most
// significant digit first radix selection over 8-bit digits finds the top bits shared with the
// K-th largest key; on return every key with (key & *mask) >= *prefix is selected, and exactly K
// keys are.
__device__ void select_top(const uint64_t* keys, int n, int K, int tid, uint32_t* hist,
                           uint64_t* sh_prefix, int* sh_rem, int* sh_done, uint64_t* mask_out,
                           uint64_t* prefix_out) {
  if (tid == 0) {
    *sh_prefix = 0ull;
    *sh_rem = K;
    *sh_done = 0;
  }
  uint64_t mask = 0ull;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += kSelThreads) hist[b] = 0u;
    __syncthreads();
    const uint64_t prefix = *sh_prefix;
    if (*sh_done) break;
    for (int t = tid; t < n; t += kSelThreads) {
      const uint64_t key = keys[t];
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane l holds bins 255 - 4 l .. 252 - 4 l: counts in descending digit order
      uint32_t c[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = hist[255 - 4 * tid - q];
      const uint32_t own = c[0] + c[1] + c[2] + c[3];
      uint32_t incl = own;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t up = __shfl_up(incl, d);
        if (tid >= d) incl += up;
      }
      const uint32_t excl = incl - own;
      const uint32_t rem = (uint32_t)*sh_rem;
      if (excl < rem && rem <= incl) {
        uint32_t acc = excl;
        int q = 0;
        while (acc + c[q] < rem) acc += c[q++];
        *sh_prefix = prefix | ((uint64_t)(255 - 4 * tid - q) << shift);
        *sh_rem = (int)(rem - acc);
        if (c[q] == rem - acc) *sh_done = 1;  // every key with this digit is selected
      }
    }
    mask |= 0xFFull << shift;
    __syncthreads();
  }
  *mask_out = mask;
  *prefix_out = *sh_prefix;
}

__global__ __launch_bounds__(kSelThreads) void kap_select_kernel(const SelParams P) {
  extern __shared__ uint64_t keys[];
  __shared__ int kcut;
  __shared__ uint32_t hist[256];
  __shared__ uint64_t sel_prefix;
  __shared__ int sel_rem, sel_done, sel_n;

  const int unit = blockIdx.x;
  const int i = unit % P.nb;
  const int ng = unit / P.nb;
  const int tid = threadIdx.x;
  // Candidates: blocks F .. i (F = 0, or the first block of block i's packed sequence).
  int seq;
  const int F = pack_first(P.a.pack, i, seq);
  const int n = i - F + 1;
  int n2 = 2;
  while (n2 < n) n2 <<= 1;

  const size_t row_off = ((size_t)ng * P.nb + i) * P.nb;
  const float* srow = P.a.score + row_off;
  const uint8_t* hrow = P.a.hrm + row_off;
  for (int t = tid; t < n2; t += kSelThreads)
    keys[t] = t < n ? make_key(hrow[F + t], srow[F + t], F + t) : 0ull;
  __syncthreads();

  int K;
  uint64_t* out = keys;  // the kept keys in descending order, first K entries
  if (P.a.mode == 0) {  // COSA_SELECT_FRACTION: the K largest keys, then only those sorted
    const int64_t k = (P.a.value_micro * (int64_t)n + 999999) / 1000000;
    K = (int)(k < 1 ? 1 : (k > n ? n : k));
    uint64_t mask, prefix;
    select_top(keys, n, K, tid, hist, &sel_prefix, &sel_rem, &sel_done, &mask, &prefix);
    uint64_t* small = keys + n2;
    int k2 = 2;
    while (k2 < K) k2 <<= 1;
    if (tid == 0) sel_n = 0;
    __syncthreads();
    for (int t = tid; t < n; t += kSelThreads) {
      const uint64_t key = keys[t];
      if ((key & mask) >= prefix) small[atomicAdd(&sel_n, 1)] = key;
    }
    for (int t = K + tid; t < k2; t += kSelThreads) small[t] = 0ull;
    __syncthreads();
    if (k2 <= 128) {
      if (tid < 64) bitonic_desc_wave(small, k2, tid);
      __syncthreads();
    } else {
      bitonic_desc(small, k2, tid);
    }
    out = small;
    n2 = k2;
  } else if (P.a.mode == 2) {  // COSA_SELECT_ALL
    bitonic_desc(keys, n2, tid);
    K = n;
  } else {  // COSA_SELECT_TOP_P: shortest prefix reaching p of the row mass
    // The row total in ascending block index, read before the sort permutes the keys; the kept
    // count from the running mass in sorted order. Both are sequential fp64 sums on one lane, so
    // the cut is the same for any launch shape.
    double total = 0.0;
    if (tid == 0)
      for (int t = 0; t < n; ++t) total += (double)key_score(keys[t]);
    __syncthreads();
    bitonic_desc(keys, n2, tid);
    if (tid == 0) {
      const double target = ((double)P.a.value_micro / 1e6) * total;
      double cum = 0.0;
      int k = 0;
      while (k < n) {
        cum += (double)key_score(keys[k]);
        ++k;
        if (cum >= target) break;
      }
      kcut = k;
    }
    __syncthreads();
    K = kcut;
  }

  if (P.a.order_mode == 1) {  // COSA_ORDER_ASCENDING: same kept set by ascending block index
    for (int k = tid; k < n2; k += kSelThreads) {
      const uint64_t key = out[k];
      out[k] = k < K ? (uint64_t)(0xffffffffu - (uint32_t)key_index(key)) : 0ull;
    }
    __syncthreads();
    if (n2 <= 128) {
      if (tid < 64) bitonic_desc_wave(out, n2, tid);
      __syncthreads();
    } else {
      bitonic_desc(out, n2, tid);
    }
  }

  int32_t* orow = P.a.order + row_off;
  for (int k = tid; k < P.nb; k += kSelThreads) orow[k] = k < K ? key_index(out[k]) : -1;
  if (tid == 0) P.a.count[(size_t)ng * P.nb + i] = K;
}

// The fraction cut on one wavefront per row, four rows per workgroup, for rows of at most 64*T
// candidates. Lane l holds candidates l, l + 64, ... of its row as keys in registers. The radix
// selection counts into a 256-bin histogram of the wave's own in LDS; a scan of the counts across
// the lanes and a ballot find the digit. The kept keys are packed by a ballot prefix into the
// wave's LDS and sorted there (by rank when at most 128). No step waits at a workgroup barrier:
// LDS operations of one wave complete in issue order. The digit rule is select_top's, so the kept
// set and the written row are the same. Rows go heaviest first (the last query blocks of every KV
// head lead), and eight waves per SIMD keep the 128K problem's 8192 rows resident at once.
constexpr int kWaveRows = 4;         // rows, one per wavefront, per workgroup
constexpr int kWaveMaxKept = 1024;   // largest kept set the wave path sorts

__device__ __forceinline__ void lds_fence() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Inclusive prefix sum over the 64 lanes: DPP right shifts by 1, 2, 4 and 8 lanes within each row
// of 16 (lanes with no source lane in the row add 0), then the totals of the rows below.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x, int lane) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  const uint32_t r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31);
  const uint32_t r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = lane >> 4;
  return x + (row > 0 ? r0 : 0u) + (row > 1 ? r1 : 0u) + (row > 2 ? r2 : 0u);
}

// Sort n <= 128 distinct keys src[0..n) in descending order into dst[0..n): lane l ranks keys l and
// l + 64 against every key (reads of one address by all lanes are broadcasts) and stores each at
// its rank, the number of larger keys.
__device__ void rank_sort_desc_wave(const uint64_t* src, uint64_t* dst, int n, int lane) {
  const uint64_t a = lane < n ? src[lane] : 0ull;
  const uint64_t b = lane + 64 < n ? src[lane + 64] : 0ull;
  int ra = 0, rb = 0;
#pragma unroll 4
  for (int j = 0; j < n; ++j) {
    const uint64_t x = src[j];
    ra += x > a;
    rb += x > b;
  }
  if (lane < n) dst[ra] = a;
  if (lane + 64 < n) dst[rb] = b;
  lds_fence();
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t b) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
}

template <int T>
__global__ __launch_bounds__(kWaveRows * 64) __attribute__((amdgpu_waves_per_eu(T <= 16 ? 8 : 4)))
void kap_select_wave_kernel(const SelParams P, const int k2max) {
  extern __shared__ uint64_t wave_lds[];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int u = blockIdx.x * kWaveRows + w;
  if (u >= P.n_units) return;
  const int rows_per_block = P.n_units / P.nb;  // batch x KV heads
  const int i = P.nb - 1 - u / rows_per_block;
  const int ng = u % rows_per_block;
  uint64_t* region = wave_lds + (size_t)w * (k2max + 128);
  uint32_t* hist = reinterpret_cast<uint32_t*>(region);  // 256 counts
  uint64_t* kept = region + 128;                          // k2max keys

  int seq;
  const int F = pack_first(P.a.pack, i, seq);
  const int n = i - F + 1;
  const int trow = (n + 63) >> 6;
  const size_t row_off = ((size_t)ng * P.nb + i) * P.nb;
  const float* srow = P.a.score + row_off + F;
  const uint8_t* hrow = P.a.hrm + row_off + F;
  // Key of candidate c (block F + c): high word (hrm << 31) | score bits, low word ~(F + c), never
  // 0. Slots past the row hold key 0, below every candidate: with K <= n they change neither the
  // K-th largest key nor, since the cut keeps exactly the K largest, the kept set, so the counts
  // and the packing need no bounds test. The row is read through buffer resources of n entries,
  // whose reads past the end return 0.
  const __amdgpu_buffer_rsrc_t srs =
      __builtin_amdgcn_make_buffer_rsrc((void*)srow, (short)0, n * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t hrs =
      __builtin_amdgcn_make_buffer_rsrc((void*)hrow, (short)0, n, 0x00020000);
  uint32_t khi[T], klo[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    khi[t] = 0u;
    klo[t] = 0u;
  }
  // The slot loops leave at the row's last slot (a uniform exit: no lane mask per slot).
#pragma unroll
  for (int t = 0; t < T; ++t) {
    if (t >= trow) break;
    const int c = lane + 64 * t;
    const uint32_t sv = __builtin_amdgcn_raw_buffer_load_b32(srs, 4 * c, 0, 0);
    const uint8_t hv = __builtin_amdgcn_raw_buffer_load_b8(hrs, c, 0, 0);
    khi[t] = ((uint32_t)(hv != 0) << 31) | (sv & 0x7fffffffu);
    klo[t] = c < n ? 0xffffffffu - (uint32_t)(F + c) : 0u;
  }
  const int64_t kk = (P.a.value_micro * (int64_t)n + 999999) / 1000000;
  const int K = (int)(kk < 1 ? 1 : (kk > n ? n : kk));

  // Radix selection, most significant 8-bit digit first: (mask, prefix) grow by one digit per pass
  // until the digit's bin holds exactly the keys still wanted.
  uint32_t mhi = 0u, mlo = 0u, phi = 0u, plo = 0u;
  uint32_t rem = (uint32_t)K;
  bool done = false;
  for (int pass = 0; pass < 8 && !done; ++pass) {
    reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0u, 0u, 0u, 0u);
    lds_fence();
    const bool hi_digit = pass < 4;
    const int sh = 24 - 8 * (pass & 3);
    if (hi_digit) {
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if (t >= trow) break;
        if ((khi[t] & mhi) == phi) atomicAdd(&hist[(khi[t] >> sh) & 255u], 1u);
      }
    } else {  // the high word is decided: mhi is all ones
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if (t >= trow) break;
        if (khi[t] == phi && (klo[t] & mlo) == plo) atomicAdd(&hist[(klo[t] >> sh) & 255u], 1u);
      }
    }
    lds_fence();
    // lane l holds bins 255 - 4l .. 252 - 4l, in descending digit order
    const uint4 h4 = reinterpret_cast<const uint4*>(hist)[63 - lane];
    const uint32_t own = h4.x + h4.y + h4.z + h4.w;
    const uint32_t incl = wave_incl_scan(own, lane);
    const uint32_t excl = incl - own;
    const uint64_t hit = __ballot(excl < rem && rem <= incl);  // one lane: counts only grow
    const int L = hit ? __builtin_ctzll(hit) : 0;
    const uint32_t e = __builtin_amdgcn_readlane(excl, L);
    const uint32_t c0 = __builtin_amdgcn_readlane(h4.w, L), c1 = __builtin_amdgcn_readlane(h4.z, L);
    const uint32_t c2 = __builtin_amdgcn_readlane(h4.y, L), c3 = __builtin_amdgcn_readlane(h4.x, L);
    uint32_t acc = e, cnt = c0;
    int q = 0;
    if (acc + c0 < rem) {
      acc += c0, q = 1, cnt = c1;
      if (acc + c1 < rem) {
        acc += c1, q = 2, cnt = c2;
        if (acc + c2 < rem) acc += c2, q = 3, cnt = c3;
      }
    }
    const uint32_t digit = 255u - 4u * (uint32_t)L - (uint32_t)q;
    if (hi_digit) {
      phi |= digit << sh;
      mhi |= 0xFFu << sh;
    } else {
      plo |= digit << sh;
      mlo |= 0xFFu << sh;
    }
    rem -= acc;
    done = cnt == rem;  // every key with this digit is kept
  }

  // Pack the kept keys (exactly K) in candidate order, then sort them.
  const uint64_t mask = ((uint64_t)mhi << 32) | mlo, prefix = ((uint64_t)phi << 32) | plo;
  int base = 0;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    if (t >= trow) break;
    const uint64_t key = ((uint64_t)khi[t] << 32) | klo[t];
    const bool sel = (key & mask) >= prefix;
    const uint64_t b = __ballot(sel);
    const int pos = base + (int)lanes_below(b);
    if (sel && pos < k2max) kept[pos] = key;
    base += __popcll(b);
  }
  lds_fence();
  const uint64_t* out = kept;
  if (K <= 128) {  // rank sort into the histogram's space, which is free now
    if (P.a.order_mode == 1) {  // COSA_ORDER_ASCENDING: same kept set by ascending block index
      for (int k = lane; k < K; k += 64)
        kept[k] = (uint64_t)(0xffffffffu - (uint32_t)key_index(kept[k]));
      lds_fence();
    }
    uint64_t* sorted = reinterpret_cast<uint64_t*>(hist);
    rank_sort_desc_wave(kept, sorted, K, lane);
    out = sorted;
  } else {
    int k2 = 2;
    while (k2 < K) k2 <<= 1;
    for (int k = K + lane; k < k2; k += 64) kept[k] = 0ull;
    lds_fence();
    bitonic_desc_wave(kept, k2, lane);
    if (P.a.order_mode == 1) {
      for (int k = lane; k < k2; k += 64)
        kept[k] = k < K ? (uint64_t)(0xffffffffu - (uint32_t)key_index(kept[k])) : 0ull;
      lds_fence();
      bitonic_desc_wave(kept, k2, lane);
    }
  }
  int32_t* orow = P.a.order + row_off;
  for (int k = lane; k < P.nb; k += 64) orow[k] = k < K ? key_index(out[k]) : -1;
  if (lane == 0) P.a.count[(size_t)ng * P.nb + i] = K;
}

}  // namespace

size_t kap_select_lds_bytes(const Shape& sh) {
  int n2 = 2;
  while (n2 < sh.nb) n2 <<= 1;
  return 2 * (size_t)n2 * sizeof(uint64_t);  // all candidates, then the kept ones
}

hipError_t launch_kap_select(const Shape& sh, const KapSelectArgs& a, hipStream_t stream) {
  SelParams P;
  P.a = a;
  P.nb = sh.nb;
  P.n_units = sh.B * sh.Hkv * sh.nb;
  if (a.mode == 0 && sh.nb <= 64 * 32) {  // COSA_SELECT_FRACTION on rows that fit one wavefront
    const int64_t kmax = (a.value_micro * (int64_t)sh.nb + 999999) / 1000000;
    int k2max = 2;
    while (k2max < kmax) k2max <<= 1;
    if (k2max <= kWaveMaxKept) {
      const dim3 grid((P.n_units + kWaveRows - 1) / kWaveRows), block(kWaveRows * 64);
      const size_t lds = (size_t)kWaveRows * (k2max + 128) * sizeof(uint64_t);
      const int per_lane = (sh.nb + 63) / 64;
      if (per_lane <= 1) hipLaunchKernelGGL(kap_select_wave_kernel<1>, grid, block, lds, stream, P, k2max);
      else if (per_lane <= 2) hipLaunchKernelGGL(kap_select_wave_kernel<2>, grid, block, lds, stream, P, k2max);
      else if (per_lane <= 4) hipLaunchKernelGGL(kap_select_wave_kernel<4>, grid, block, lds, stream, P, k2max);
      else if (per_lane <= 8) hipLaunchKernelGGL(kap_select_wave_kernel<8>, grid, block, lds, stream, P, k2max);
      else if (per_lane <= 16) hipLaunchKernelGGL(kap_select_wave_kernel<16>, grid, block, lds, stream, P, k2max);
      else hipLaunchKernelGGL(kap_select_wave_kernel<32>, grid, block, lds, stream, P, k2max);
      return hipGetLastError();
    }
  }
  // Dynamic LDS above the default limit (long sequences) has to be allowed for the kernel; remember
  // the largest size granted so far.
  const size_t lds = kap_select_lds_bytes(sh);
  static std::mutex mu;
  static size_t granted = 0;
  if (lds > 48 * 1024) {
    std::lock_guard<std::mutex> lock(mu);
    if (lds > granted) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&kap_select_kernel),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)lds);
      if (e != hipSuccess) return e;
      granted = lds;
    }
  }
  hipLaunchKernelGGL(kap_select_kernel, dim3(P.n_units), dim3(kSelThreads), lds, stream, P);
  return hipGetLastError();
}

}  // namespace cosa
