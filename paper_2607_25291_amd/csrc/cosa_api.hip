// C ABI of the CoSA prefill-attention library: host-side validation, workspace layout and launches.
// Every entry point validates all arguments before enqueuing anything (see include/cosa.h).
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "cosa.h"
#include "cosa_internal.h"

static_assert(COSA_MAX_PACKED_SEQS == cosa::kMaxPackedSeqs, "packing limit of the ABI and kernels");

// Workspace of cosa_prefill_noalloc: one copy per GPU, held until the process ends. In host code
// this name is only a handle for hipGetSymbolAddress; the device address of each GPU's copy is
// looked up once per device (scratch_of_device) and used everywhere the host needs the array.
static __device__ __align__(256) unsigned char scratch[COSA_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;

cosa_status fail(cosa_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = std::string(cosa_status_string(st)) + ": " + buf;
  return st;
}

cosa_status ok() {
  g_last_error.clear();
  return COSA_OK;
}

cosa_status hip_fail(hipError_t e, const char* what) {
  return fail(COSA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Validates the problem and fills the internal shape. `empty` is set for B == 0 or L == 0.
cosa_status make_shape(const cosa_problem* p, cosa::Shape& sh, bool& empty) {
  if (!p) return fail(COSA_ERR_INVALID_ARG, "problem is NULL");
  if (p->batch < 0 || p->seq_len < 0)
    return fail(COSA_ERR_INVALID_ARG, "batch (%d) and seq_len (%d) must be >= 0", p->batch,
                p->seq_len);
  if (p->n_q_heads < 1 || p->n_kv_heads < 1 || p->n_q_heads % p->n_kv_heads != 0)
    return fail(COSA_ERR_INVALID_ARG, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)",
                p->n_q_heads, p->n_kv_heads);
  if (p->head_dim < 1 || p->block < 1 || p->stride < 1)
    return fail(COSA_ERR_INVALID_ARG, "head_dim, block and stride must be >= 1");
  if (p->block % p->stride != 0)
    return fail(COSA_ERR_INVALID_ARG, "stride (%d) must divide block (%d)", p->stride, p->block);
  if (!(p->sm_scale >= 0.f) || !isfinite(p->sm_scale))
    return fail(COSA_ERR_INVALID_ARG, "sm_scale must be finite and >= 0 (0 = 1/sqrt(d))");
  if (p->causal != 0 && p->causal != 1)
    return fail(COSA_ERR_INVALID_ARG, "causal must be 0 or 1");
  if (p->causal != 1) return fail(COSA_ERR_UNSUPPORTED, "only causal prefill is supported");
  if (p->head_dim != cosa::kHeadDim)
    return fail(COSA_ERR_UNSUPPORTED, "head_dim %d (supported: 128)", p->head_dim);
  if (p->block != 64 && p->block != 128)
    return fail(COSA_ERR_UNSUPPORTED, "block %d (supported: 64, 128)", p->block);
  if (p->seq_len % p->block != 0)
    return fail(COSA_ERR_UNSUPPORTED, "seq_len %d is not a multiple of block %d", p->seq_len,
                p->block);
  sh.B = p->batch;
  sh.Hq = p->n_q_heads;
  sh.Hkv = p->n_kv_heads;
  sh.L = p->seq_len;
  sh.d = p->head_dim;
  sh.b = p->block;
  sh.s = p->stride;
  sh.nb = p->seq_len / p->block;
  sh.G = p->n_q_heads / p->n_kv_heads;
  sh.spb = p->block / p->stride;
  sh.scale = p->sm_scale > 0.f ? p->sm_scale : (float)(1.0 / sqrt((double)p->head_dim));
  if (sh.nb > 8192) return fail(COSA_ERR_UNSUPPORTED, "%d blocks (supported: <= 8192)", sh.nb);
  // grid sizes and 32-bit index arithmetic inside the kernels
  const long long units = (long long)sh.B * sh.Hkv * sh.nb;
  if (units * sh.G + 8LL * sh.G > (1LL << 30) || (long long)sh.L * cosa::kHeadDim >= (1LL << 31))
    return fail(COSA_ERR_UNSUPPORTED, "problem too large for one launch");
  empty = sh.B == 0 || sh.L == 0;
  return ok();
}

cosa_status check_proxy_limits(const cosa::Shape& sh) {
  if (sh.spb != 4 && sh.spb != 8 && sh.spb != 16 && sh.spb != 32)
    return fail(COSA_ERR_UNSUPPORTED, "block / stride = %d samples per block (supported: 4, 8, 16, 32)",
                sh.spb);
  if (sh.G * sh.spb > 128)
    return fail(COSA_ERR_UNSUPPORTED, "G * samples per block = %d proxy rows (supported: <= 128)",
                sh.G * sh.spb);
  if (cosa::kap_score_lds_bytes(sh) == 0)
    return fail(COSA_ERR_UNSUPPORTED, "proxy block maxima (%d rows x %d blocks) exceed LDS",
                sh.G * sh.spb, sh.nb);
  return ok();
}

cosa_status check_select(const cosa_select* sel, int64_t& micro) {
  if (!sel) return fail(COSA_ERR_INVALID_ARG, "select is NULL");
  if (sel->mode != COSA_SELECT_FRACTION && sel->mode != COSA_SELECT_TOP_P &&
      sel->mode != COSA_SELECT_ALL)
    return fail(COSA_ERR_INVALID_ARG, "unknown select mode %d", (int)sel->mode);
  if (sel->order != COSA_ORDER_KAP && sel->order != COSA_ORDER_ASCENDING)
    return fail(COSA_ERR_INVALID_ARG, "unknown order mode %d", (int)sel->order);
  micro = 1000000;
  if (sel->mode != COSA_SELECT_ALL) {
    if (!(sel->value > 0.f && sel->value <= 1.f))
      return fail(COSA_ERR_INVALID_ARG, "select value %g outside (0, 1]", (double)sel->value);
    micro = (int64_t)floor((double)sel->value * 1e6 + 0.5);
  }
  return ok();
}

cosa_status check_skip(const cosa_skip* sk, const cosa::Shape& sh, int& on, float& tau) {
  on = 0;
  tau = 0.f;
  if (!sk || sk->mode == COSA_SKIP_NONE) return ok();
  if (sk->mode != COSA_SKIP_ROWMAX) return fail(COSA_ERR_INVALID_ARG, "unknown skip mode %d",
                                                (int)sk->mode);
  if (!(sk->delta > 0.f) || !isfinite(sk->delta) || (double)sk->delta > (double)sh.L)
    return fail(COSA_ERR_INVALID_ARG, "skip delta %g outside (0, seq_len = %d]", (double)sk->delta,
                sh.L);
  on = 1;
  tau = (float)log((double)sk->delta / (double)sh.L);  // Eq. (skip): ln(Delta / N)
  return ok();
}

// Validates a paged KV cache description against the problem and fills the internal form.
cosa_status check_paged(const cosa_paged_kv* kv, const cosa::Shape& sh, bool need_v,
                        cosa::KvPages& pg) {
  if (!kv) return fail(COSA_ERR_INVALID_ARG, "paged kv is NULL");
  const int ps = kv->page_size;
  if (ps < 16 || ps > (1 << 20) || (ps & (ps - 1)) != 0)
    return fail(COSA_ERR_INVALID_ARG, "page_size %d is not a power of two in [16, 2^20]", ps);
  if (sh.L % ps != 0)
    return fail(COSA_ERR_INVALID_ARG, "page_size %d does not divide seq_len %d", ps, sh.L);
  if (kv->n_pages < 1) return fail(COSA_ERR_INVALID_ARG, "n_pages (%lld) must be >= 1",
                                   (long long)kv->n_pages);
  if (kv->n_pages > (1LL << 31))
    return fail(COSA_ERR_INVALID_ARG, "n_pages (%lld) exceeds the int32 page numbers of the table",
                (long long)kv->n_pages);
  if (!kv->k_cache || !kv->page_table || (need_v && !kv->v_cache))
    return fail(COSA_ERR_INVALID_ARG, "k_cache%s and page_table must be non-NULL",
                need_v ? ", v_cache" : "");
  pg.table = kv->page_table;
  pg.log2_page = 0;
  while ((1 << pg.log2_page) < ps) ++pg.log2_page;
  pg.pages_per_seq = sh.L / ps;
  pg.n_pages = kv->n_pages;
  return ok();
}

// Validates a packing of several sequences along the token axis and fills the kernel-argument form:
// block offsets and, with skipping on, each sequence's threshold ln(Delta / L_q) (Eq. (skip) with N
// the sequence's own length), computed in double and rounded once to float.
cosa_status check_varlen(const cosa_varlen* vl, const cosa::Shape& sh, const cosa_skip* sk,
                         cosa::SeqPack& sp) {
  if (!vl) return fail(COSA_ERR_INVALID_ARG, "varlen is NULL");
  if (vl->n_seqs < 1 || vl->n_seqs > COSA_MAX_PACKED_SEQS)
    return fail(COSA_ERR_INVALID_ARG, "n_seqs %d outside [1, %d]", vl->n_seqs,
                COSA_MAX_PACKED_SEQS);
  if (!vl->cu_blocks) return fail(COSA_ERR_INVALID_ARG, "cu_blocks is NULL");
  if (vl->cu_blocks[0] != 0)
    return fail(COSA_ERR_INVALID_ARG, "cu_blocks[0] = %d, must be 0", vl->cu_blocks[0]);
  for (int q = 0; q < vl->n_seqs; ++q)
    if (vl->cu_blocks[q + 1] <= vl->cu_blocks[q])
      return fail(COSA_ERR_INVALID_ARG, "cu_blocks must increase strictly (entries %d and %d)", q,
                  q + 1);
  if (vl->cu_blocks[vl->n_seqs] != sh.nb)
    return fail(COSA_ERR_INVALID_ARG, "cu_blocks[n_seqs] = %d, must equal seq_len / block = %d",
                vl->cu_blocks[vl->n_seqs], sh.nb);
  sp = cosa::SeqPack{};
  sp.n = vl->n_seqs;
  for (int q = 0; q <= vl->n_seqs; ++q) sp.cu[q] = vl->cu_blocks[q];
  if (sk && sk->mode == COSA_SKIP_ROWMAX) {
    for (int q = 0; q < vl->n_seqs; ++q) {
      const long long len = (long long)(sp.cu[q + 1] - sp.cu[q]) * sh.b;
      if ((double)sk->delta > (double)len)
        return fail(COSA_ERR_INVALID_ARG, "skip delta %g exceeds the length %lld of sequence %d",
                    (double)sk->delta, len, q);
      sp.tau[q] = (float)log((double)sk->delta / (double)len);
    }
  }
  return ok();
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

cosa_workspace_layout layout_of(const cosa::Shape& sh) {
  const size_t rows = (size_t)sh.B * sh.Hkv * sh.nb;
  const size_t cells = rows * sh.nb;
  cosa_workspace_layout l;
  l.score = 0;
  l.hrm = align256(l.score + cells * sizeof(float));
  l.order = align256(l.hrm + cells * sizeof(uint8_t));
  l.count = align256(l.order + cells * sizeof(int32_t));
  l.keys = align256(l.count + rows * sizeof(int32_t));
  l.queue = align256(l.keys + cosa::kap_stage_bytes(sh));
  l.total = align256(l.queue + cosa::kOskQueueBytes);
  return l;
}

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Device address of `scratch` on the GPU that runs `stream` (the current device for the null
// stream), taken once per device with that device current and kept for later calls.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

cosa_status scratch_of_device(hipStream_t stream, void** addr) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int dev = cur;
  if (stream != nullptr) {
    hipDevice_t sd;
    if ((e = hipStreamGetDevice(stream, &sd)) != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
    dev = (int)sd;
  }
  if (dev < 0 || dev >= kMaxDevices)
    return fail(COSA_ERR_UNSUPPORTED, "device %d (supported: 0 .. %d)", dev, kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return hip_fail(e, "hipSetDevice");
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess && e2 != hipSuccess) e = e2;
    }
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (p == nullptr || reinterpret_cast<uintptr_t>(p) % 256 != 0)
      return fail(COSA_ERR_HIP, "scratch of device %d at %p is not 256-byte aligned", dev, p);
    g_scratch_addr[dev] = p;
  }
  *addr = g_scratch_addr[dev];
  return ok();
}

// Algorithm A end to end; kv == nullptr: contiguous K and V at k, v; vl == nullptr: no packing.
cosa_status prefill(const cosa_problem* problem, const void* q, const void* k, const void* v,
                    const cosa_paged_kv* kv, const cosa_varlen* vl, const cosa_select* select,
                    const cosa_skip* skip, void* workspace, size_t workspace_bytes, void* o,
                    void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int64_t micro = 0;
  if ((st = check_select(select, micro)) != COSA_OK) return st;
  int on = 0;
  float tau = 0.f;
  if ((st = check_skip(skip, sh, on, tau)) != COSA_OK) return st;
  cosa::KvPages pg{};
  if (kv && (st = check_paged(kv, sh, true, pg)) != COSA_OK) return st;
  if (empty) return ok();
  cosa::SeqPack sp{};
  if (vl && (st = check_varlen(vl, sh, skip, sp)) != COSA_OK) return st;
  if ((st = check_proxy_limits(sh)) != COSA_OK) return st;
  if (!q || !k || !v || !o) return fail(COSA_ERR_INVALID_ARG, "q, k, v and o must be non-NULL");
  const cosa_workspace_layout l = layout_of(sh);
  if (!workspace || workspace_bytes < l.total)
    return fail(COSA_ERR_WORKSPACE, "workspace of %zu bytes at %p, need %zu", workspace_bytes,
                workspace, l.total);
  if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0)
    return fail(COSA_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  char* ws = static_cast<char*>(workspace);
  float* score = reinterpret_cast<float*>(ws + l.score);
  uint8_t* hrm = reinterpret_cast<uint8_t*>(ws + l.hrm);
  int32_t* order = reinterpret_cast<int32_t*>(ws + l.order);
  int32_t* count = reinterpret_cast<int32_t*>(ws + l.count);
  uint16_t* keys = reinterpret_cast<uint16_t*>(ws + l.keys);
  uint32_t* queue = reinterpret_cast<uint32_t*>(ws + l.queue);
  const hipStream_t s = as_stream(stream);
  hipError_t e = cosa::launch_kap_score(
      sh, cosa::KapScoreArgs{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), score,
                             hrm, pg, sp, keys},
      s);
  if (e != hipSuccess) return hip_fail(e, "kap_score launch");
  e = cosa::launch_kap_select(
      sh,
      cosa::KapSelectArgs{score, hrm, order, count, (int)select->mode, (int)select->order, micro, sp},
      s);
  if (e != hipSuccess) return hip_fail(e, "kap_select launch");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), order, count,
                   nullptr, nullptr, nullptr, on, tau, pg, nullptr, sp, queue};
  e = cosa::launch_osk_attention(sh, a, s);
  return e == hipSuccess ? ok() : hip_fail(e, "osk_attention launch");
}

}  // namespace

extern "C" {

const char* cosa_status_string(cosa_status status) {
  switch (status) {
    case COSA_OK: return "COSA_OK";
    case COSA_ERR_INVALID_ARG: return "COSA_ERR_INVALID_ARG";
    case COSA_ERR_UNSUPPORTED: return "COSA_ERR_UNSUPPORTED";
    case COSA_ERR_WORKSPACE: return "COSA_ERR_WORKSPACE";
    case COSA_ERR_HIP: return "COSA_ERR_HIP";
  }
  return "COSA_ERR_UNKNOWN";
}

const char* cosa_last_error(void) { return g_last_error.c_str(); }

cosa_status cosa_kap_score(const cosa_problem* problem, const void* q, const void* k, float* score,
                           uint8_t* hrm, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (empty) return ok();
  if ((st = check_proxy_limits(sh)) != COSA_OK) return st;
  if (!q || !k || !score || !hrm)
    return fail(COSA_ERR_INVALID_ARG, "q, k, score and hrm must be non-NULL");
  cosa::KapScoreArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), score, hrm,
                       cosa::KvPages{}};
  const hipError_t e = cosa::launch_kap_score(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "kap_score launch");
}

size_t cosa_kap_score_workspace_bytes(const cosa_problem* problem) {
  cosa::Shape sh;
  bool empty = false;
  if (make_shape(problem, sh, empty) != COSA_OK) return 0;
  return cosa::kap_stage_bytes(sh);
}

cosa_status cosa_kap_score_staged(const cosa_problem* problem, const void* q, const void* k,
                                  void* workspace, size_t workspace_bytes, float* score,
                                  uint8_t* hrm, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (empty) return ok();
  if ((st = check_proxy_limits(sh)) != COSA_OK) return st;
  if (!q || !k || !score || !hrm)
    return fail(COSA_ERR_INVALID_ARG, "q, k, score and hrm must be non-NULL");
  const size_t need = cosa::kap_stage_bytes(sh);
  if (!workspace || workspace_bytes < need)
    return fail(COSA_ERR_WORKSPACE, "workspace of %zu bytes at %p, need %zu", workspace_bytes,
                workspace, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0)
    return fail(COSA_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  cosa::KapScoreArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), score, hrm,
                       cosa::KvPages{}, cosa::SeqPack{}, static_cast<uint16_t*>(workspace)};
  const hipError_t e = cosa::launch_kap_score(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "kap_score launch");
}

cosa_status cosa_kap_score_paged(const cosa_problem* problem, const void* q,
                                 const cosa_paged_kv* kv, float* score, uint8_t* hrm,
                                 void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  cosa::KvPages pg{};
  if ((st = check_paged(kv, sh, false, pg)) != COSA_OK) return st;
  if (empty) return ok();
  if ((st = check_proxy_limits(sh)) != COSA_OK) return st;
  if (!q || !score || !hrm) return fail(COSA_ERR_INVALID_ARG, "q, score and hrm must be non-NULL");
  cosa::KapScoreArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kv->k_cache),
                       score, hrm, pg};
  const hipError_t e = cosa::launch_kap_score(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "kap_score launch");
}

cosa_status cosa_kap_select_ordered(const cosa_problem* problem, const float* score,
                                    const uint8_t* hrm, const cosa_select* select, int32_t* order,
                                    int32_t* count, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int64_t micro = 0;
  if ((st = check_select(select, micro)) != COSA_OK) return st;
  if (empty) return ok();
  if (!score || !hrm || !order || !count)
    return fail(COSA_ERR_INVALID_ARG, "score, hrm, order and count must be non-NULL");
  cosa::KapSelectArgs a{score, hrm, order, count, (int)select->mode, (int)select->order, micro};
  const hipError_t e = cosa::launch_kap_select(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "kap_select launch");
}

cosa_status cosa_osk_attention(const cosa_problem* problem, const void* q, const void* k,
                               const void* v, const int32_t* order, const int32_t* count,
                               const cosa_skip* skip, void* o, uint8_t* visit_log,
                               float* margin_log, int32_t* n_computed, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int on = 0;
  float tau = 0.f;
  if ((st = check_skip(skip, sh, on, tau)) != COSA_OK) return st;
  if (empty) return ok();
  if (!q || !k || !v || !order || !count || !o)
    return fail(COSA_ERR_INVALID_ARG, "q, k, v, order, count and o must be non-NULL");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), order, count,
                   visit_log, margin_log, n_computed, on, tau, cosa::KvPages{}};
  const hipError_t e = cosa::launch_osk_attention(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "osk_attention launch");
}

size_t cosa_osk_attention_queue_bytes(void) { return cosa::kOskQueueBytes; }

cosa_status cosa_osk_attention_queued(const cosa_problem* problem, const void* q, const void* k,
                                      const void* v, const int32_t* order, const int32_t* count,
                                      const cosa_skip* skip, void* o, uint8_t* visit_log,
                                      float* margin_log, int32_t* n_computed, void* queue,
                                      size_t queue_bytes, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int on = 0;
  float tau = 0.f;
  if ((st = check_skip(skip, sh, on, tau)) != COSA_OK) return st;
  if (empty) return ok();
  if (!q || !k || !v || !order || !count || !o)
    return fail(COSA_ERR_INVALID_ARG, "q, k, v, order, count and o must be non-NULL");
  if (!queue || queue_bytes < cosa::kOskQueueBytes)
    return fail(COSA_ERR_WORKSPACE, "queue of %zu bytes at %p, need %zu", queue_bytes, queue,
                cosa::kOskQueueBytes);
  if (reinterpret_cast<uintptr_t>(queue) % 4 != 0)
    return fail(COSA_ERR_INVALID_ARG, "queue must be 4-byte aligned");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), order, count,
                   visit_log, margin_log, n_computed, on, tau, cosa::KvPages{}, nullptr,
                   cosa::SeqPack{}, static_cast<uint32_t*>(queue)};
  const hipError_t e = cosa::launch_osk_attention(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "osk_attention launch");
}

cosa_status cosa_osk_attention_paged(const cosa_problem* problem, const void* q,
                                     const cosa_paged_kv* kv, const int32_t* order,
                                     const int32_t* count, const cosa_skip* skip, void* o,
                                     uint8_t* visit_log, float* margin_log, int32_t* n_computed,
                                     void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int on = 0;
  float tau = 0.f;
  if ((st = check_skip(skip, sh, on, tau)) != COSA_OK) return st;
  cosa::KvPages pg{};
  if ((st = check_paged(kv, sh, true, pg)) != COSA_OK) return st;
  if (empty) return ok();
  if (!q || !order || !count || !o)
    return fail(COSA_ERR_INVALID_ARG, "q, order, count and o must be non-NULL");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kv->k_cache),
                   static_cast<const uint16_t*>(kv->v_cache), static_cast<uint16_t*>(o), order,
                   count, visit_log, margin_log, n_computed, on, tau, pg};
  const hipError_t e = cosa::launch_osk_attention(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "osk_attention launch");
}

cosa_status cosa_dense_attention(const cosa_problem* problem, const void* q, const void* k,
                                 const void* v, void* o, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (empty) return ok();
  if (!q || !k || !v || !o) return fail(COSA_ERR_INVALID_ARG, "q, k, v and o must be non-NULL");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), nullptr, nullptr,
                   nullptr, nullptr, nullptr, 0, 0.f, cosa::KvPages{}};
  const hipError_t e = cosa::launch_dense_attention(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "dense_attention launch");
}

cosa_status cosa_masked_attention(const cosa_problem* problem, const void* q, const void* k,
                                  const void* v, const uint8_t* mask, void* o, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (empty) return ok();
  if (!q || !k || !v || !mask || !o)
    return fail(COSA_ERR_INVALID_ARG, "q, k, v, mask and o must be non-NULL");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), nullptr, nullptr,
                   nullptr, nullptr, nullptr, 0, 0.f, cosa::KvPages{}, mask};
  const hipError_t e = cosa::launch_masked_attention(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "masked_attention launch");
}

cosa_status cosa_block_mass(const cosa_problem* problem, const void* q, const void* k, float* mass,
                            void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (empty) return ok();
  if (!q || !k || !mass) return fail(COSA_ERR_INVALID_ARG, "q, k and mass must be non-NULL");
  if (cosa::block_mass_lds_bytes(sh) > 160 * 1024)
    return fail(COSA_ERR_UNSUPPORTED, "%d blocks exceed the block-mass kernel's LDS", sh.nb);
  const hipError_t e = cosa::launch_block_mass(sh, static_cast<const uint16_t*>(q),
                                               static_cast<const uint16_t*>(k), mass,
                                               as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "block_mass launch");
}

cosa_status cosa_prefill_workspace_layout(const cosa_problem* problem,
                                          cosa_workspace_layout* layout) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (!layout) return fail(COSA_ERR_INVALID_ARG, "layout is NULL");
  *layout = layout_of(sh);
  return ok();
}

size_t cosa_prefill_workspace_bytes(const cosa_problem* problem) {
  cosa_workspace_layout l;
  if (cosa_prefill_workspace_layout(problem, &l) != COSA_OK) return 0;
  return l.total;
}

cosa_status cosa_prefill(const cosa_problem* problem, const void* q, const void* k, const void* v,
                         const cosa_select* select, const cosa_skip* skip, void* workspace,
                         size_t workspace_bytes, void* o, void* stream) {
  return prefill(problem, q, k, v, nullptr, nullptr, select, skip, workspace, workspace_bytes, o,
                 stream);
}

cosa_status cosa_prefill_noalloc(const cosa_problem* problem, const void* q, const void* k,
                                 const void* v, const cosa_select* select, const cosa_skip* skip,
                                 void* o, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int64_t micro = 0;
  if ((st = check_select(select, micro)) != COSA_OK) return st;
  int on = 0;
  float tau = 0.f;
  if ((st = check_skip(skip, sh, on, tau)) != COSA_OK) return st;
  if (empty) return ok();
  const size_t need = layout_of(sh).total;
  if (need > (size_t)COSA_NOALLOC_SCRATCH_BYTES)
    return fail(COSA_ERR_WORKSPACE,
                "the problem needs %zu bytes of workspace; the static scratch holds %zu "
                "(use cosa_prefill with a caller workspace)",
                need, (size_t)COSA_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = scratch_of_device(as_stream(stream), &ws)) != COSA_OK) return st;
  return prefill(problem, q, k, v, nullptr, nullptr, select, skip, ws,
                 (size_t)COSA_NOALLOC_SCRATCH_BYTES, o, stream);
}

cosa_status cosa_prefill_paged(const cosa_problem* problem, const void* q, const cosa_paged_kv* kv,
                               const cosa_select* select, const cosa_skip* skip, void* workspace,
                               size_t workspace_bytes, void* o, void* stream) {
  if (!kv) return fail(COSA_ERR_INVALID_ARG, "paged kv is NULL");
  return prefill(problem, q, kv->k_cache, kv->v_cache, kv, nullptr, select, skip, workspace,
                 workspace_bytes, o, stream);
}

cosa_status cosa_kap_score_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                  const void* q, const void* k, float* score, uint8_t* hrm,
                                  void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (empty) return ok();
  cosa::SeqPack sp{};
  if ((st = check_varlen(varlen, sh, nullptr, sp)) != COSA_OK) return st;
  if ((st = check_proxy_limits(sh)) != COSA_OK) return st;
  if (!q || !k || !score || !hrm)
    return fail(COSA_ERR_INVALID_ARG, "q, k, score and hrm must be non-NULL");
  cosa::KapScoreArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), score, hrm,
                       cosa::KvPages{}, sp};
  const hipError_t e = cosa::launch_kap_score(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "kap_score launch");
}

cosa_status cosa_kap_select_ordered_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                           const float* score, const uint8_t* hrm,
                                           const cosa_select* select, int32_t* order,
                                           int32_t* count, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int64_t micro = 0;
  if ((st = check_select(select, micro)) != COSA_OK) return st;
  if (empty) return ok();
  cosa::SeqPack sp{};
  if ((st = check_varlen(varlen, sh, nullptr, sp)) != COSA_OK) return st;
  if (!score || !hrm || !order || !count)
    return fail(COSA_ERR_INVALID_ARG, "score, hrm, order and count must be non-NULL");
  cosa::KapSelectArgs a{score, hrm, order, count, (int)select->mode, (int)select->order, micro, sp};
  const hipError_t e = cosa::launch_kap_select(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "kap_select launch");
}

cosa_status cosa_osk_attention_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                      const void* q, const void* k, const void* v,
                                      const int32_t* order, const int32_t* count,
                                      const cosa_skip* skip, void* o, uint8_t* visit_log,
                                      float* margin_log, int32_t* n_computed, void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  int on = 0;
  float tau = 0.f;
  if ((st = check_skip(skip, sh, on, tau)) != COSA_OK) return st;
  if (empty) return ok();
  cosa::SeqPack sp{};
  if ((st = check_varlen(varlen, sh, skip, sp)) != COSA_OK) return st;
  if (!q || !k || !v || !order || !count || !o)
    return fail(COSA_ERR_INVALID_ARG, "q, k, v, order, count and o must be non-NULL");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), order, count,
                   visit_log, margin_log, n_computed, on, tau, cosa::KvPages{}, nullptr, sp};
  const hipError_t e = cosa::launch_osk_attention(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "osk_attention launch");
}

cosa_status cosa_dense_attention_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                        const void* q, const void* k, const void* v, void* o,
                                        void* stream) {
  cosa::Shape sh;
  bool empty = false;
  cosa_status st = make_shape(problem, sh, empty);
  if (st != COSA_OK) return st;
  if (empty) return ok();
  cosa::SeqPack sp{};
  if ((st = check_varlen(varlen, sh, nullptr, sp)) != COSA_OK) return st;
  if (!q || !k || !v || !o) return fail(COSA_ERR_INVALID_ARG, "q, k, v and o must be non-NULL");
  cosa::AttnArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), nullptr, nullptr,
                   nullptr, nullptr, nullptr, 0, 0.f, cosa::KvPages{}, nullptr, sp};
  const hipError_t e = cosa::launch_dense_attention(sh, a, as_stream(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "dense_attention launch");
}

cosa_status cosa_prefill_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                const void* q, const void* k, const void* v,
                                const cosa_select* select, const cosa_skip* skip, void* workspace,
                                size_t workspace_bytes, void* o, void* stream) {
  if (!varlen) return fail(COSA_ERR_INVALID_ARG, "varlen is NULL");
  return prefill(problem, q, k, v, nullptr, varlen, select, skip, workspace, workspace_bytes, o,
                 stream);
}

cosa_status cosa_prefill_paged_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                      const void* q, const cosa_paged_kv* kv,
                                      const cosa_select* select, const cosa_skip* skip,
                                      void* workspace, size_t workspace_bytes, void* o,
                                      void* stream) {
  if (!kv) return fail(COSA_ERR_INVALID_ARG, "paged kv is NULL");
  if (!varlen) return fail(COSA_ERR_INVALID_ARG, "varlen is NULL");
  return prefill(problem, q, kv->k_cache, kv->v_cache, kv, varlen, select, skip, workspace,
                 workspace_bytes, o, stream);
}

}  // extern "C"
