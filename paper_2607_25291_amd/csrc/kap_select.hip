// Flag-grouped sort and stage-1 cut for gfx950 (Sec. 4.2 "Flag-grouped sorting", Eq. (mkap);
// Algorithm A, proxy stage).
//
// One workgroup per (batch n, KV head g, query block i). The causal candidates (j <= i, from the
// first block of the packed sequence when several sequences share the token axis) become 64-bit
// keys  (hrm << 63) | (float bits of score << 32) | (0xffffffff - j): scores are non-negative, so
// their bit patterns order like the values, and comparing keys orders by HRM flag, then score, then
// ascending block index. The kept set is the K_i largest keys, in descending key order (the HRM
// group first, each group by descending score). By fraction, K_i follows from the row length
// (integer arithmetic on the budget in millionths): a radix selection over 8-bit digits finds the
// K_i-th largest key, and only the keys at or above it are sorted (bitonic, in LDS; within one
// wavefront when at most 128). By top-p the cut depends on the sorted scores, so the whole row is
// sorted, as it is when every candidate is kept. The top-p sums run in fp64 in one fixed order, on
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
        const int lo = (t / stride) * 2 * stride + (t % stride);
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

// Sort keys[0..n2) in descending order within one wavefront (n2 a power of two, at most 128): the
// wave's lanes each take one compare-exchange per stage; LDS operations of one wave complete in
// issue order, so the stages need no workgroup barrier.
__device__ void bitonic_desc_wave(uint64_t* keys, int n2, int lane) {
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (lane < (n2 >> 1)) {
        const int lo = (lane / stride) * 2 * stride + (lane % stride);
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
