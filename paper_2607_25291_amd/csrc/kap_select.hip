// Flag-grouped sort and stage-1 cut for gfx950 (Sec. 4.2 "Flag-grouped sorting", Eq. (mkap);
// Algorithm A, proxy stage).
//
// One workgroup per (batch n, KV head g, query block i). The causal candidates (j <= i, from the
// first block of the packed sequence when several sequences share the token axis) become 64-bit
// keys  (hrm << 63) | (float bits of score << 32) | (0xffffffff - j): scores are non-negative, so
// their bit patterns order like the values, and comparing keys orders by HRM flag, then score, then
// ascending block index. A bitonic sort in LDS puts them in descending key order (the HRM group
// first, each group by descending score). The cut K_i is then taken by fraction (integer
// arithmetic on the budget in millionths), by top-p (fp64 prefix sums of the sorted scores), or is
// the whole row; ascending visit order re-sorts the kept set by block index. The row of `order` is
// written in full: K_i block ids followed by -1.
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

__global__ __launch_bounds__(kSelThreads) void kap_select_kernel(const SelParams P) {
  extern __shared__ uint64_t keys[];
  __shared__ double part[kSelThreads];
  __shared__ double total_s;
  __shared__ int kcut;

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
  bitonic_desc(keys, n2, tid);

  int K;
  if (P.a.mode == 2) {  // COSA_SELECT_ALL
    K = n;
  } else if (P.a.mode == 0) {  // COSA_SELECT_FRACTION
    const int64_t k = (P.a.value_micro * (int64_t)n + 999999) / 1000000;
    K = (int)(k < 1 ? 1 : (k > n ? n : k));
  } else {  // COSA_SELECT_TOP_P: shortest prefix reaching p of the row mass
    const int seg = (n + kSelThreads - 1) / kSelThreads;
    const int lo = tid * seg, hi = min(n, lo + seg);
    double ps = 0.0;
    for (int k = lo; k < hi; ++k) ps += (double)key_score(keys[k]);
    part[tid] = ps;
    __syncthreads();
    if (tid == 0) {
      double run = 0.0;
      for (int t = 0; t < kSelThreads; ++t) {
        const double v = part[t];
        part[t] = run;
        run += v;
      }
      total_s = run;
      kcut = n;
    }
    __syncthreads();
    const double target = ((double)P.a.value_micro / 1e6) * total_s;
    double cum = part[tid];
    for (int k = lo; k < hi; ++k) {
      cum += (double)key_score(keys[k]);
      if (cum >= target) {
        atomicMin(&kcut, k + 1);
        break;
      }
    }
    __syncthreads();
    K = kcut;
  }

  if (P.a.order_mode == 1) {  // COSA_ORDER_ASCENDING: same kept set by ascending block index
    for (int k = tid; k < n2; k += kSelThreads) {
      const uint64_t key = keys[k];
      keys[k] = k < K ? (uint64_t)(0xffffffffu - (uint32_t)key_index(key)) : 0ull;
    }
    __syncthreads();
    bitonic_desc(keys, n2, tid);
  }

  int32_t* orow = P.a.order + row_off;
  for (int k = tid; k < P.nb; k += kSelThreads) orow[k] = k < K ? key_index(keys[k]) : -1;
  if (tid == 0) P.a.count[(size_t)ng * P.nb + i] = K;
}

}  // namespace

size_t kap_select_lds_bytes(const Shape& sh) {
  int n2 = 2;
  while (n2 < sh.nb) n2 <<= 1;
  return (size_t)n2 * sizeof(uint64_t);
}

hipError_t launch_kap_select(const Shape& sh, const KapSelectArgs& a, hipStream_t stream) {
  SelParams P;
  P.a = a;
  P.nb = sh.nb;
  P.n_units = sh.B * sh.Hkv * sh.nb;
  hipLaunchKernelGGL(kap_select_kernel, dim3(P.n_units), dim3(kSelThreads),
                     kap_select_lds_bytes(sh), stream, P);
  return hipGetLastError();
}

}  // namespace cosa
