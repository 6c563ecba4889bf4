/*
 * cosa.h — C ABI of the CoSA prefill-attention library for AMD Instinct MI355X (gfx950).
 *
 * CoSA ("Accelerating Long-Context Inference via Proxy-Kernel Co-Designed Sparse Attention",
 * arXiv 2607.25291) computes causal prefill attention in two stages:
 *   1. the Kernel-Aware Proxy (KAP, Sec. 4.2) scores query-block x key-block importance from
 *      stride-downsampled Q/K, keeps blocks under a moderate budget and emits, per query block, an
 *      ordered list of key blocks with the "have rowmax" (HRM) blocks first;
 *   2. the Ordered-Skipping Kernel (OSK, Sec. 4.3) is a flash-style attention that visits only the
 *      listed KV pages, in list order, and skips the value side of a block when every row's local
 *      maximum lies below its running maximum by more than ln(Delta/N) (Eq. (skip)).
 * Algorithm A (appendix) gives the complete workflow; cosa_prefill runs it end to end.
 *
 * Conventions for every entry point
 *   - Tensors are device pointers (hipMalloc'd or equivalent) owned by the caller; bf16 tensors are
 *     passed as raw 16-bit storage. Every tensor is dense and contiguous in the layout given.
 *   - Shapes: Q and O [B, Hq, L, d]; K and V [B, Hkv, L, d]; nb = ceil(L / b).
 *     Proxy tensors are per KV head: score, hrm, order [B, Hkv, nb, nb]; count [B, Hkv, nb].
 *     Per-query-head logs: visit_log, margin_log [B, Hq, nb, nb]; n_computed [B, Hq, nb].
 *   - stream is a hipStream_t (NULL: the legacy default stream). All work is enqueued
 *     asynchronously on it; nothing is synchronised and nothing is allocated or freed.
 *   - Arguments are validated on the host before anything is enqueued. On any non-OK status nothing
 *     has been launched and no output has been written; cosa_last_error() then describes the cause.
 *     Faults inside kernels surface at the caller's next synchronisation of the stream.
 *   - Calls on different streams are independent and may run concurrently; the library keeps no
 *     state between calls apart from the loaded kernels.
 *   - batch == 0 or seq_len == 0 is an empty problem: the call validates and returns COSA_OK
 *     without launching anything.
 *
 * Supported problem space (COSA_ERR_UNSUPPORTED otherwise): head_dim == 128, block in {64, 128},
 * causal == 1, seq_len a multiple of block, samples per block (block / stride) in {4, 8, 16, 32},
 * G * (block / stride) <= 128 rows per proxy unit, and nb <= 8192.
 *
 * The *_paged entry points take K and V from a paged KV cache (cosa_paged_kv) instead of the
 * contiguous [B, Hkv, L, d] tensors; everything else is unchanged, and on the same data their
 * results are bit-identical to the contiguous calls.
 */
#ifndef COSA_H_
#define COSA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COSA_OK = 0,
  COSA_ERR_INVALID_ARG = 1, /* NULL required pointer, inconsistent shape, value out of range      */
  COSA_ERR_UNSUPPORTED = 2, /* valid problem outside the supported space listed above             */
  COSA_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than cosa_prefill_workspace_bytes()       */
  COSA_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed                         */
} cosa_status;

/* One attention layer's prefill problem (Algorithm A inputs and parameters). */
typedef struct {
  int32_t batch;      /* B >= 0                                                                   */
  int32_t n_q_heads;  /* Hq >= 1, a multiple of n_kv_heads (grouped-query attention)              */
  int32_t n_kv_heads; /* Hkv >= 1; query head h reads KV head h / (Hq / Hkv)                       */
  int32_t seq_len;    /* L = N of the paper >= 0                                                  */
  int32_t head_dim;   /* d                                                                        */
  int32_t block;      /* b: query block = key block = KV page, in tokens (appendix: b = 128)      */
  int32_t stride;     /* s: proxy downsampling stride (Sec. 4.2), divides b; token r*s is sampled  */
  float sm_scale;     /* logit scale; 0 selects 1/sqrt(head_dim) (Algorithm A)                     */
  int32_t causal;     /* must be 1 (causal prefill)                                               */
} cosa_problem;

/* Stage-1 selection (Sec. 4.2 "Flag-grouped sorting", Eq. (mkap)). */
typedef enum {
  COSA_SELECT_FRACTION = 0, /* K_i = ceil(value * (i + 1)) of the i + 1 causal candidates,        */
                            /* clamped to [1, i + 1]; value is taken at 1e-6 resolution            */
  COSA_SELECT_TOP_P = 1,    /* shortest prefix of the order whose score mass >= value * row total  */
  COSA_SELECT_ALL = 2       /* every causal candidate (value ignored)                              */
} cosa_select_mode;

typedef enum {
  COSA_ORDER_KAP = 0,       /* HRM blocks first, then by descending score; ties by ascending index */
  COSA_ORDER_ASCENDING = 1  /* the same kept set, listed by ascending block index                  */
} cosa_order_mode;

typedef struct {
  cosa_select_mode mode;
  float value;              /* budget B1 or top-p mass p, in (0, 1] (ignored for ALL)             */
  cosa_order_mode order;
} cosa_select;

/* Stage-2 in-kernel skip (Eq. (skip)). */
typedef enum {
  COSA_SKIP_NONE = 0,
  COSA_SKIP_ROWMAX = 1      /* skip a listed block when max_r (m_loc[r] - m[r]) < ln(delta / L)    */
} cosa_skip_mode;

typedef struct {
  cosa_skip_mode mode;
  float delta;              /* skip scale Delta, 0 < delta <= seq_len when mode == ROWMAX          */
} cosa_skip;

/* Visit codes written to visit_log. */
#define COSA_VISIT_COMPUTED 1
#define COSA_VISIT_SKIPPED 2

/* Byte offsets of the proxy tensors inside a cosa_prefill workspace (each 256-byte aligned). */
typedef struct {
  size_t score; /* float   [B, Hkv, nb, nb]                                         */
  size_t hrm;   /* uint8_t [B, Hkv, nb, nb]                                         */
  size_t order; /* int32_t [B, Hkv, nb, nb]                                         */
  size_t count; /* int32_t [B, Hkv, nb]                                             */
  size_t keys;  /* staged sampled keys, cosa_kap_score_workspace_bytes() (scratch)  */
  size_t queue; /* OSK work-queue counters, cosa_osk_attention_queue_bytes() (scratch) */
  size_t total; /* bytes required                                                   */
} cosa_workspace_layout;

/*
 * Paged KV cache (Sec. 4.3 "Physical jumping over pages"; Algorithm A takes paged K and V; appendix
 * D.1: a logical block of b tokens resolves through one or more physical pages when the page size
 * b_p differs from b). The order invariance of Sec. 3.2 is what lets the walk visit pages in any
 * order through such a table.
 *   k_cache, v_cache: bf16 [n_pages, n_kv_heads, page_size, head_dim]; page p of KV head g holds
 *                     page_size consecutive tokens, each a contiguous row of head_dim values.
 *   page_table:       int32 [batch, seq_len / page_size]; entry [n, t / page_size] is the physical
 *                     page holding token t of sequence n (for every KV head).
 *   page_size:        tokens per page, a power of two in [16, 2^20] that divides seq_len.
 *   n_pages:          physical pages in each cache (>= 1).
 * Pointers are device pointers owned by the caller. Table entries are device data and are not
 * checked before launch: an entry outside [0, n_pages) is read as page 0 (the kernels never read
 * outside the caches; the affected outputs are then meaningless).
 */
typedef struct {
  const void* k_cache;
  const void* v_cache;
  const int32_t* page_table;
  int32_t page_size;
  int64_t n_pages;
} cosa_paged_kv;

/*
 * Variable-length packing. Several sequences of different lengths share one call by being
 * concatenated along the token axis of the [B, H, L, d] tensors, each starting on a block boundary
 * and spanning whole blocks: sequence q owns blocks [cu_blocks[q], cu_blocks[q + 1]) (tokens
 * cu_blocks[q] * b .. cu_blocks[q + 1] * b - 1) of every batch entry. Each sequence is an
 * independent causal problem: query block i of sequence q only sees key blocks from cu_blocks[q]
 * up to i (proxy candidates, the stage-1 cut K_i over those i - cu_blocks[q] + 1 candidates, list
 * entries, dense walk), and its skip threshold is ln(delta / L_q) with L_q its own length in tokens
 * (Eq. (skip), N the context length of the sequence). The results for a sequence equal those of a
 * separate call on that sequence alone, with block indices offset by cu_blocks[q].
 *   n_seqs:    1 <= n_seqs <= COSA_MAX_PACKED_SEQS.
 *   cu_blocks: HOST int32 [n_seqs + 1], cu_blocks[0] = 0, strictly increasing,
 *              cu_blocks[n_seqs] = seq_len / block. Read during the call only.
 * With skipping on, delta must not exceed the shortest sequence's length.
 */
#define COSA_MAX_PACKED_SEQS 128
typedef struct {
  int32_t n_seqs;
  const int32_t* cu_blocks;
} cosa_varlen;

/* Human-readable name of a status code (static storage). */
const char* cosa_status_string(cosa_status status);

/* Detail of the most recent failure in the calling thread ("" if none). Valid until the next
 * call into the library from the same thread. */
const char* cosa_last_error(void);

/*
 * KAP block scoring (Sec. 4.2 "Block ranking", Eq. (score); Algorithm A, proxy stage).
 * For every batch n, KV head g and query block i, with the sampled rows r = i*spb .. i*spb+spb-1
 * (spb = b/s, token r*s) of every query head of group g and the sampled keys c <= r (token c*s):
 *   beta[r, j] = max over the sampled keys c of block j of sm_scale * <Q[r*s], K[c*s]>,
 *   Pbar[r, j] = exp(beta[r, j] - max_j' beta[r, j'])      (softmax -> MaxPool -> MaxNorm),
 *   score[n, g, i, j] = sum over the G*spb rows of Pbar[r, j],
 *   hrm[n, g, i, j]   = 1 if some row attains its maximum in block j, else 0,
 * for j <= i; entries j > i are not written. fp32 arithmetic on bf16 inputs; the row sum runs in a
 * fixed order, so results are deterministic.
 */
cosa_status cosa_kap_score(const cosa_problem* problem, const void* q, const void* k,
                           float* score, uint8_t* hrm, void* stream);

/*
 * cosa_kap_score with the sampled keys staged first: a copy of the L / s sampled keys of every KV
 * head is written to the caller's workspace in the order the matrix cores consume them (32-key
 * chunks of 8 KiB), so that the scoring kernel reads 1 KiB contiguous per load instead of 32 rows
 * per load. Results are bit-identical to cosa_kap_score. workspace: device memory of at least
 * cosa_kap_score_workspace_bytes() bytes, 16-byte aligned; its contents are scratch (overwritten,
 * meaningless on return). cosa_prefill and its variants stage the keys inside their own workspace.
 */
size_t cosa_kap_score_workspace_bytes(const cosa_problem* problem);
cosa_status cosa_kap_score_staged(const cosa_problem* problem, const void* q, const void* k,
                                  void* workspace, size_t workspace_bytes, float* score,
                                  uint8_t* hrm, void* stream);

/*
 * Flag-grouped sort and stage-1 cut (Sec. 4.2, Eq. (mkap); Algorithm A, proxy stage).
 * For every (n, g, i): the candidates j <= i are ordered by (hrm desc, score desc, j asc), the
 * leading K_i are kept (per select->mode), and order[n, g, i, :] receives them (or the same set by
 * ascending j for COSA_ORDER_ASCENDING) followed by -1 up to nb; count[n, g, i] = K_i.
 * Reads score/hrm entries j <= i only.
 */
cosa_status cosa_kap_select_ordered(const cosa_problem* problem, const float* score,
                                    const uint8_t* hrm, const cosa_select* select, int32_t* order,
                                    int32_t* count, void* stream);

/*
 * Ordered-skipping attention (Sec. 4.3; Algorithm A, attention loop; Eq. (skip)).
 * Query head h of batch n and query block i walks order[n, g(h), i, 0 .. count-1] in list order:
 * S = sm_scale * Q_i K_j^T (causal mask on the diagonal block), m_loc = rowmax(S), running max
 * m <- max(m, m_loc), margin d = max over the b rows of (m_loc - m) in nats; with
 * skip->mode == ROWMAX the block's value side is skipped when d < tau, tau = ln(delta / L)
 * computed in double and rounded once to float. Otherwise the online-softmax state is updated
 * (P = exp(S - m) rounded to bf16 for the P V product, fp32 accumulation). O = O / l in bf16.
 * order entries must lie in [0, i] and be distinct; count in [1, nb] (not checked on the device).
 * skip may be NULL (no skipping). Optional logs (NULL to omit), indexed by list position k:
 * visit_log (COSA_VISIT_*), margin_log (d in nats), n_computed (computed blocks per tile).
 */
cosa_status cosa_osk_attention(const cosa_problem* problem, const void* q, const void* k,
                               const void* v, const int32_t* order, const int32_t* count,
                               const cosa_skip* skip, void* o, uint8_t* visit_log,
                               float* margin_log, int32_t* n_computed, void* stream);

/*
 * cosa_osk_attention as cosa_prefill runs it: a persistent grid of one workgroup per compute unit
 * that takes (query block, head pair) tiles from eight work queues, one per XCD, heaviest query
 * blocks first; a workgroup drains its own XCD's queue, then the others. Same arguments, results
 * and logs as cosa_osk_attention, bit for bit. queue: device memory of at least
 * cosa_osk_attention_queue_bytes() bytes, 4-byte aligned, owned by the caller; its contents are
 * scratch (reset by the call on the stream, meaningless on return), so calls that may run at the
 * same time need distinct queue buffers. Returns COSA_ERR_WORKSPACE if queue is NULL or too small.
 */
size_t cosa_osk_attention_queue_bytes(void);
cosa_status cosa_osk_attention_queued(const cosa_problem* problem, const void* q, const void* k,
                                      const void* v, const int32_t* order, const int32_t* count,
                                      const cosa_skip* skip, void* o, uint8_t* visit_log,
                                      float* margin_log, int32_t* n_computed, void* queue,
                                      size_t queue_bytes, void* stream);

/*
 * Dense causal flash attention (Sec. 3.1): every key block j <= i in ascending order, same tile
 * code and numerics as cosa_osk_attention without list and skip. The in-house baseline.
 */
cosa_status cosa_dense_attention(const cosa_problem* problem, const void* q, const void* k,
                                 const void* v, void* o, void* stream);

/*
 * Block-sparse attention under a binary block mask with logical skipping (Sec. 3.2, Eq.
 * (proxy-mask); the mask-driven scheme the OSK is compared with in appendix D "Kernel
 * microbenchmark"). Query head h of batch n and query block i visits j = 0 .. i in ascending order
 * and computes block j exactly when mask[n, g(h), i, j] != 0 (u8 [B, Hkv, nb, nb]; entries j > i
 * are not read). A masked block costs a step of the walk but no loads and no arithmetic. Same tile
 * code and numerics as cosa_osk_attention; on the same block set the output equals
 * cosa_osk_attention over the ascending list without skipping, bit for bit. A row with no block
 * selected yields O = 0.
 */
cosa_status cosa_masked_attention(const cosa_problem* problem, const void* q, const void* k,
                                  const void* v, const uint8_t* mask, void* o, void* stream);

/*
 * Exact attention block mass per KV group (analysis; Sec. 3.2, Property 1: the mass that full
 * attention puts on each key block defines the oracle mask a proxy is measured against).
 *   mass[n, g, i, j] = sum over the query heads h of group g and the rows r of query block i of
 *                      sum over the keys c of block j with c <= r of softmax_c(sm_scale Q_h[r].K_g[c])
 * for j <= i (fp32 [B, Hkv, nb, nb]; entries j > i are not written). Each row's probabilities sum
 * to one, so row block i's masses sum to G * b. Two passes over the keys per head (row statistics,
 * then block sums); the summation order is fixed, so results are deterministic. Not on the
 * prefill path: it costs about as much as dense attention.
 */
cosa_status cosa_block_mass(const cosa_problem* problem, const void* q, const void* k, float* mass,
                            void* stream);

/* Workspace size of cosa_prefill (0 if the problem is invalid; see cosa_last_error()). */
size_t cosa_prefill_workspace_bytes(const cosa_problem* problem);

/* Offsets of score/hrm/order/count inside the cosa_prefill workspace. */
cosa_status cosa_prefill_workspace_layout(const cosa_problem* problem,
                                          cosa_workspace_layout* layout);

/*
 * Complete proxy-kernel workflow (Algorithm A): cosa_kap_score_staged, cosa_kap_select_ordered
 * and cosa_osk_attention enqueued back to back on one stream, with the proxy tensors and the staged
 * keys in the caller-provided workspace (at least cosa_prefill_workspace_bytes(), 16-byte
 * aligned; contents on return are the proxy tensors at cosa_prefill_workspace_layout() offsets).
 * skip may be NULL.
 */
cosa_status cosa_prefill(const cosa_problem* problem, const void* q, const void* k, const void* v,
                         const cosa_select* select, const cosa_skip* skip, void* workspace,
                         size_t workspace_bytes, void* o, void* stream);

/* Largest workspace cosa_prefill_noalloc can use: 128 MiB, which holds the workspace of one
 * 128K-token layer with 8 KV heads (120 MiB). */
#define COSA_NOALLOC_SCRATCH_BYTES (128u * 1024u * 1024u)

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): cosa_prefill with its workspace in a static scratch
 * array of the library instead of a caller buffer. Same arguments, results and errors as
 * cosa_prefill otherwise; the caller still owns q, k, v and o.
 *   - Returns COSA_ERR_WORKSPACE and enqueues nothing when cosa_prefill_workspace_bytes(problem)
 *     exceeds COSA_NOALLOC_SCRATCH_BYTES.
 *   - Allocates nothing: no hipMalloc, hipFree or allocating library routine. The scratch array
 *     exists once per GPU the library runs on and is held until the process ends; its device
 *     address is looked up on the first call on each GPU (the GPU of `stream`, the current device
 *     for the null stream).
 *   - Every call on one GPU uses that GPU's single array, which keeps the last call's contents
 *     (they are not exposed). Calls that overlap on one GPU (several streams, or several host
 *     threads) race on it: the caller must serialise them. Whatever must start at zero is cleared
 *     by a kernel on `stream` (no memset node).
 */
cosa_status cosa_prefill_noalloc(const cosa_problem* problem, const void* q, const void* k,
                                 const void* v, const cosa_select* select, const cosa_skip* skip,
                                 void* o, void* stream);

/*
 * cosa_kap_score with K read from a paged cache (kv->v_cache is not used and may be NULL):
 * sampled key c (token c * stride) of KV head g is row (token % page_size) of physical page
 * page_table[n, token / page_size].
 */
cosa_status cosa_kap_score_paged(const cosa_problem* problem, const void* q,
                                 const cosa_paged_kv* kv, float* score, uint8_t* hrm, void* stream);

/*
 * cosa_osk_attention with K and V read from a paged cache: the K and V pages of a listed block j
 * are gathered through page_table (b / page_size physical pages per block when page_size < b, a
 * part of one page otherwise), in list order.
 */
cosa_status cosa_osk_attention_paged(const cosa_problem* problem, const void* q,
                                     const cosa_paged_kv* kv, const int32_t* order,
                                     const int32_t* count, const cosa_skip* skip, void* o,
                                     uint8_t* visit_log, float* margin_log, int32_t* n_computed,
                                     void* stream);

/* cosa_prefill (Algorithm A end to end) on a paged KV cache; same workspace as cosa_prefill. */
cosa_status cosa_prefill_paged(const cosa_problem* problem, const void* q, const cosa_paged_kv* kv,
                               const cosa_select* select, const cosa_skip* skip, void* workspace,
                               size_t workspace_bytes, void* o, void* stream);

/*
 * Packed variable-length forms (cosa_varlen). Each behaves as the call without the suffix applied
 * to every packed sequence separately; proxy entries (score, hrm, order rows) outside a block's own
 * sequence are not read and, for score and hrm, not written.
 */
cosa_status cosa_kap_score_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                  const void* q, const void* k, float* score, uint8_t* hrm,
                                  void* stream);
cosa_status cosa_kap_select_ordered_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                           const float* score, const uint8_t* hrm,
                                           const cosa_select* select, int32_t* order,
                                           int32_t* count, void* stream);
cosa_status cosa_osk_attention_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                      const void* q, const void* k, const void* v,
                                      const int32_t* order, const int32_t* count,
                                      const cosa_skip* skip, void* o, uint8_t* visit_log,
                                      float* margin_log, int32_t* n_computed, void* stream);
cosa_status cosa_dense_attention_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                        const void* q, const void* k, const void* v, void* o,
                                        void* stream);
cosa_status cosa_prefill_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                const void* q, const void* k, const void* v,
                                const cosa_select* select, const cosa_skip* skip, void* workspace,
                                size_t workspace_bytes, void* o, void* stream);
cosa_status cosa_prefill_paged_varlen(const cosa_problem* problem, const cosa_varlen* varlen,
                                      const void* q, const cosa_paged_kv* kv,
                                      const cosa_select* select, const cosa_skip* skip,
                                      void* workspace, size_t workspace_bytes, void* o,
                                      void* stream);

#ifdef __cplusplus
}
#endif

#endif /* COSA_H_ */
