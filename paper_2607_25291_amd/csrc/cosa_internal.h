// Internal interface between the C ABI layer (cosa_api.hip) and the kernel translation units.
// Every launcher enqueues on `stream` and returns the hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace cosa {

constexpr int kHeadDim = 128;
constexpr int kNumXcd = 8;  // MI355X: 8 accelerator complex dies, workgroups dispatched round-robin

// Shape of one validated problem (all sizes in elements).
struct Shape {
  int B, Hq, Hkv, L, d, b, s, nb, G, spb;
  float scale;  // resolved sm_scale
};

// Where a KV head's keys and values live. table == nullptr: contiguous [B, Hkv, L, d] at the K/V
// pointers of the call. Otherwise a paged cache [n_pages, Hkv, page, d] per tensor and a page table
// [B, L / page] of physical page numbers (entries are clamped into [0, n_pages) on the device).
struct KvPages {
  const int32_t* table;
  int log2_page;       // page = 1 << log2_page tokens
  int pages_per_seq;   // L / page
  long long n_pages;
};

// Variable-length packing: n sequences concatenated along the token axis, sequence q owning blocks
// [cu[q], cu[q + 1]) with cu[0] = 0 and cu[n] = nb. Query block i then only sees key blocks from its
// own sequence's first block up to i, and the skip threshold of its sequence, tau[q] = ln(delta /
// L_q) rounded once to float. n == 0: one unpacked sequence per batch entry. Passed by value in the
// kernel arguments (no device memory).
constexpr int kMaxPackedSeqs = 128;
struct SeqPack {
  int n;
  int cu[kMaxPackedSeqs + 1];
  float tau[kMaxPackedSeqs];
};

struct KapScoreArgs {
  const uint16_t* q;
  const uint16_t* k;   // contiguous K, or the paged K cache
  float* score;
  uint8_t* hrm;
  KvPages pg;
  SeqPack pack;
  uint16_t* kstage;    // kap_stage_bytes() of scratch for the staged sampled keys, or nullptr
};

struct KapSelectArgs {
  const float* score;
  const uint8_t* hrm;
  int32_t* order;
  int32_t* count;
  int mode;         // cosa_select_mode
  int order_mode;   // cosa_order_mode
  int64_t value_micro;  // budget or p in millionths
  SeqPack pack;
};

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  const int32_t* order;   // OSK only
  const int32_t* count;   // OSK only
  uint8_t* visit_log;     // optional
  float* margin_log;      // optional
  int32_t* n_computed;    // optional
  int skip_on;
  float tau;              // skip threshold in nats (float32)
  KvPages pg;             // k and v are the paged caches when pg.table != nullptr (OSK only)
  const uint8_t* mask;    // block mask [B, Hkv, nb, nb] (masked walk only)
  SeqPack pack;           // packed sequences (OSK and dense walks); tau per sequence
  uint32_t* queue;        // OSK: kOskQueueBytes of work-queue counters (persistent grid), or nullptr
};

// Work-queue counters of the persistent OSK grid: one 32-bit counter per XCD, 128 bytes apart.
constexpr size_t kOskQueueBytes = kNumXcd * 128;

// LDS bytes the proxy-scoring kernel needs for a shape (0 if the shape is outside its limits).
size_t kap_score_lds_bytes(const Shape& sh);
// Scratch bytes of the staged sampled keys (all L / s of every head, in MFMA operand order).
size_t kap_stage_bytes(const Shape& sh);
size_t kap_select_lds_bytes(const Shape& sh);

hipError_t launch_kap_score(const Shape& sh, const KapScoreArgs& a, hipStream_t stream);
hipError_t launch_kap_select(const Shape& sh, const KapSelectArgs& a, hipStream_t stream);
hipError_t launch_osk_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream);
hipError_t launch_dense_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream);
hipError_t launch_masked_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream);
size_t block_mass_lds_bytes(const Shape& sh);
hipError_t launch_block_mass(const Shape& sh, const uint16_t* q, const uint16_t* k, float* mass,
                             hipStream_t stream);

}  // namespace cosa
