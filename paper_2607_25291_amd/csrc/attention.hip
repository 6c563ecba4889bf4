// Ordered-skipping attention (OSK) and the dense causal flash baseline for gfx950.
//
// A workgroup computes HPW query heads of one KV group for one query block of b rows: b/32
// wavefronts per head, 32 query rows per wavefront. The K and V pages of each visited key block are
// fetched once into LDS and serve every head of the workgroup. Logits are formed transposed,
// S^T = K Q^T, with bf16 MFMA 32x32x16 so that every lane owns one query row; the online softmax
// runs in fp32 (Sec. 3.1). OSK walks the KAP list (Algorithm A, attention loop) and after Q K^T
// decides, for each head's whole b-row tile at once, whether the value side can be skipped
// (Eq. (skip)); the dense kernel visits j = 0..i in order and never skips.
//
// Pages move from HBM straight into LDS (buffer loads with an LDS destination: no registers are
// spent on staging), double-buffered. Each wave works through its pages in two halves,
//   QK(m): Q K^T of page m, the diagonal mask, the new running max and the wave's skip vote;
//   PV(m): the skip decision from the votes, softmax, P V of page m;
// with a workgroup barrier after each half. With two heads in a workgroup the waves of the second
// head start one barrier later, so phase 2m runs QK(m) of head 0 beside PV(m-1) of head 1 and phase
// 2m+1 runs PV(m) of head 0 beside QK(m) of head 1. Waves w and w + 4 share a SIMD: while one
// issues the Q K^T MFMAs the other runs its softmax VALU work and P V MFMAs. The waves of head 0
// fetch K pages (page m+1 at the end of QK(m), after its vote), those of head 1 V pages (page m+1
// at the end of their QK(m)); a single head fetches both. Issuing a page copy stalls the issuing
// wave for about as long as the load path takes to accept it, so it comes after the Q K^T MFMAs:
// in a phase whose P V half computes, the copy then overlaps the partner wave's P V work instead
// of delaying the Q K^T chain. A wave waits for its own copies at the end of its PV half, so every
// copy has the rest of its phase and the next one to land before the barrier that publishes it.
//
// The grid is either one workgroup per tile (query block, head pair) or, when the caller supplies
// work-queue counters, persistent: one workgroup per CU takes tiles from per-XCD queues in the
// order the hardware would run them (see the tile loop below).
// With a paged KV cache (Sec. 4.3 "Physical jumping over pages"; appendix D.1) the copies gather a
// block's rows through the page table; everything from the LDS layouts on is shared.
//
// LDS layouts (one 16-byte slot of 8 values at a time; a direct load writes 64 consecutive slots,
// each lane picks the global slot that belongs there):
//   K [key][d]  256-byte rows, slot s of row r stored at slot s ^ (r % 16). The MFMA A-operand reads
//               (lane = key, 16 bytes of d) of 16 consecutive keys hit 16 different slots.
//   V [key][d]  256-byte rows, slot s of row r stored at slot s ^ 4 (r % 4). P V takes V through
//               transposing LDS reads (ds_read_b64_tr_b16): in each 16-lane group the lane i receives,
//               for k = 0..3, element i % 4 of the 8 bytes addressed by lane 4k + i / 4. Lane i
//               addressing V[key0 + i/4][d0 + 4 (i%4)] therefore receives keys key0..key0+3 of
//               column d0 + i, which is the P^T key set that lane holds from the S^T accumulators.
#include <type_traits>

#include "cosa_device.h"
#include "cosa_internal.h"

namespace cosa {
namespace {

typedef short s16x4_t __attribute__((ext_vector_type(4)));

// A wave-uniform read of data this kernel never writes (the count and first list entries in a
// tile's prologue), through the constant address space: a scalar load, counted apart from the
// vector memory operations (the Q fragments) already in flight. Inside the page loop the list is
// read with vector loads instead: an outstanding scalar load would make every LDS wait a full one.
__device__ __forceinline__ int32_t ld_uniform(const int32_t* p) {
  return *(const __attribute__((address_space(4))) int32_t*)(size_t)p;
}
#define COSA_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// s_waitcnt immediates (vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8): wait for vector
// memory and LDS operations, or for LDS operations only.
constexpr int kVmcntLgkm0 = 0x0070;
constexpr int kLgkm0 = 0xC07F;

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
  static constexpr int kPage = BLOCK * kHeadDim * 2;         // bytes of one K or V page
  static constexpr int kLdsBytes = 4 * kPage;
  static constexpr int kWgPerCu = (160 * 1024) / (kLdsBytes + 256);
  static constexpr int kWavesPerEu = (kWgPerCu * kWaves) / 4 > 1 ? (kWgPerCu * kWaves) / 4 : 1;
};

// Direct global -> LDS copy of one page by NW waves: wave w moves chunks c = u * NW + w (rows
// 4c .. 4c+3). Lane l fills LDS slot l of the chunk (row 4c + l/16, stored slot l%16) with the
// global slot that the layout puts there. The page offset and the chunk offset are scalars.
template <int BLOCK, int NW, bool IS_K>
__device__ __forceinline__ void copy_page(__amdgpu_buffer_rsrc_t rs, char* dst, int page_off,
                                          int w, int lane) {
  constexpr int kChunks = BLOCK * kHeadDim * 2 / 1024;
  static_assert(kChunks % NW == 0, "page chunks must split evenly over the waves");
  // The wave's first chunk in LDS and in the page. Kept opaque so that the per-chunk addresses are
  // formed here (one scalar add each) instead of being held in registers across the page loop.
  int lds0 = (int)(size_t)COSA_LDS(dst) + w * 1024;
  int src0 = page_off + w * 1024;
  asm volatile("" : "+s"(lds0), "+s"(src0));
#pragma unroll
  for (int u = 0; u < kChunks / NW; ++u) {
    const int c = u * NW + w;
    const int row = 4 * c + (lane >> 4);
    const int stored = lane & 15;
    const int slot = IS_K ? (stored ^ (row & 15)) : (stored ^ ((row & 3) << 2));
    const int voff = (lane >> 4) * (kHeadDim * 2) + slot * 16;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rs, (__attribute__((address_space(3))) void*)(size_t)(lds0 + u * NW * 1024), 16, voff,
        src0 + u * NW * 1024, 0, 0);
  }
}

// Paged variant (Sec. 4.3 "Physical jumping over pages"): the block's rows live in physical pages of
// 2^log2p >= 16 tokens of a [n_pages, Hkv, page, d] cache. Wave w moves the consecutive chunks
// w * CPW .. w * CPW + CPW - 1 in runs of four (16 rows): a run starts 16-aligned, so it lies inside
// one physical page whatever the page size, and each run takes one buffer resource, its chunks
// immediate offsets from it (no per-chunk test for a page boundary). Lane k of `tbl` holds the raw
// table entry of the block's k-th page-sized segment (segment 0 when a page holds the block). A run
// reads its entry into a scalar register and forms the page address there (the range clamp, a
// 64-bit multiply by the page stride `pstride` and the add to the head's cache base `cache`), so
// that the copy adds no vector instructions to the wave that issues it; entries outside
// [0, n_pages) read page 0.
template <int BLOCK, int NW, bool IS_K, bool WHOLE>
__device__ __forceinline__ void copy_page_paged(int tbl, uint64_t cache, uint64_t pstride,
                                                unsigned n_pages, int first_row, int log2p,
                                                char* dst, int w, int lane) {
  constexpr int kChunks = BLOCK * kHeadDim * 2 / 1024;
  constexpr int CPW = kChunks / NW;
  static_assert(kChunks % NW == 0 && CPW % 4 == 0, "each wave moves a multiple of 16 rows");
  const int page_mask = (1 << log2p) - 1;
  // Opaque wave index: the per-chunk offsets are formed here instead of being hoisted out of the
  // page loop into scalar registers.
  asm volatile("" : "+s"(w));
  if constexpr (WHOLE) {
    // The block lies inside one physical page (page size >= block): one resource for the wave's
    // chunks, as for a contiguous cache.
    const uint32_t e = (uint32_t)__builtin_amdgcn_readfirstlane(tbl);
    const uint64_t base = cache + (uint64_t)(e < n_pages ? e : 0u) * pstride;
    const int in_page = first_row & page_mask;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(base + (uint64_t)in_page * (kHeadDim * 2)), (short)0, BLOCK * kHeadDim * 2,
        0x00020000);
    int lds0 = (int)(size_t)COSA_LDS(dst) + w * CPW * 1024;
    int src0 = w * CPW * 1024;
    asm volatile("" : "+s"(lds0), "+s"(src0));
#pragma unroll
    for (int u = 0; u < CPW; ++u) {
      // Row 4 (w CPW + u) + lane / 16 of the block; only its residue mod 16 enters the swizzle,
      // and w CPW is a multiple of 4.
      const int row = 4 * (u & 3) + (lane >> 4);
      const int stored = lane & 15;
      const int slot = IS_K ? (stored ^ (row & 15)) : (stored ^ ((row & 3) << 2));
      const int voff = (lane >> 4) * (kHeadDim * 2) + slot * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void*)(size_t)(lds0 + u * 1024), 16, voff,
          src0 + u * 1024, 0, 0);
    }
    return;
  }
#pragma unroll
  for (int run = 0; run < CPW / 4; ++run) {
    const int row0 = (w * CPW + 4 * run) * 4;  // first row of the run within the block
    const int in_page = (first_row + row0) & page_mask;
    const int seg = row0 >> log2p;
    const uint32_t e = (uint32_t)__builtin_amdgcn_readlane(tbl, seg);
    const uint64_t base = cache + (uint64_t)(e < n_pages ? e : 0u) * pstride;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(base + (uint64_t)in_page * (kHeadDim * 2)), (short)0, 16 * kHeadDim * 2,
        0x00020000);
#pragma unroll
    for (int u4 = 0; u4 < 4; ++u4) {
      const int u = 4 * run + u4;
      // Row 4 (w CPW + u) + lane / 16 of the block; only its residue mod 16 enters the swizzle,
      // and w CPW is a multiple of 4.
      const int row = 4 * (u & 3) + (lane >> 4);
      const int stored = lane & 15;
      const int slot = IS_K ? (stored ^ (row & 15)) : (stored ^ ((row & 3) << 2));
      const int voff = (lane >> 4) * (kHeadDim * 2) + slot * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, COSA_LDS(dst + (w * CPW + u) * 1024), 16, voff,
                                               u4 * 1024, 0, 0);
    }
  }
}

// Where the keys and values live: contiguous [B, Hkv, L, d], or a paged cache whose pages are
// smaller than a block (a block spans several pages) or at least a block (one page holds it).
constexpr int kPgNone = 0;
constexpr int kPgSplit = 1;
constexpr int kPgWhole = 2;

// How the key blocks of a query block are walked.
constexpr int kWalkDense = 0;  // j = 0 .. i ascending, every block computed
constexpr int kWalkList = 1;   // OSK: the KAP list in list order, rowmax skip vote
constexpr int kWalkMask = 2;   // j = 0 .. i ascending, blocks whose mask byte is 0 skipped in-loop

// Zeroes the work-queue counters of a persistent OSK launch (one per XCD, 128 bytes apart).
__global__ void queue_reset(uint32_t* queue) {
  if (threadIdx.x < kNumXcd) queue[threadIdx.x * 32] = 0u;
}

template <int BLOCK, int HPW, int WALK, int PG, bool PERSIST>
__global__ __attribute__((amdgpu_flat_work_group_size(TileCfg<BLOCK, HPW>::kThreads,
                                                      TileCfg<BLOCK, HPW>::kThreads)))
__attribute__((amdgpu_waves_per_eu(TileCfg<BLOCK, HPW>::kWavesPerEu,
                                   TileCfg<BLOCK, HPW>::kWavesPerEu)))
void attention_kernel(const AttnParams P) {
  using Cfg = TileCfg<BLOCK, HPW>;
  constexpr bool PAGED = PG != kPgNone;
  constexpr bool OSK = WALK == kWalkList;
  constexpr bool MASKED = WALK == kWalkMask;
  constexpr int KT = Cfg::kKeyTiles;
  constexpr int WPH = Cfg::kWavesPerHead;
  constexpr int PAGE = Cfg::kPage;
  // V buffers first: they get the low 64 KiB, where every transposing read's buffer and key offsets
  // fit the instruction's immediate (the K reads add their buffer base once per d chunk).
  __shared__ __attribute__((aligned(1024))) char v_lds0[PAGE];
  __shared__ __attribute__((aligned(1024))) char v_lds1[PAGE];
  __shared__ __attribute__((aligned(1024))) char k_lds0[PAGE];
  __shared__ __attribute__((aligned(1024))) char k_lds1[PAGE];
  __shared__ float vote[2][Cfg::kWaves];
  __shared__ int tile_slot;

  // Persistent grid (OSK with a work queue): one workgroup per CU takes tiles until none are left.
  // Slot p is the tile the hardware would run as workgroup p; queue x hands out the slots
  // p = x + 8 k, which the hardware would deal to XCD x, heaviest first. A workgroup starts on its
  // own XCD's queue and moves on to the next one when that is empty, so every tile is taken exactly
  // once and every workgroup leaves once all eight queues are empty. Thread 0 claims the next slot
  // during the last page of the current tile, which hides the atomic's latency without holding a
  // slot for long, and broadcasts it through LDS.
  const int n_slots = (P.n_units + kNumXcd - 1) / kNumXcd * kNumXcd * (P.G / HPW);
  int qx = PERSIST ? (int)(__builtin_amdgcn_s_getreg(0xF814) & (kNumXcd - 1)) : 0;  // XCC_ID
  int qtried = 0;
  unsigned k_next = 0u;
  bool have_next = false;
  auto claim = [&]() -> int {
    while (qtried < kNumXcd) {
      const int p = qx + kNumXcd * (int)atomicAdd(&P.a.queue[qx * 32], 1u);
      if (p < n_slots) return p;
      qx = (qx + 1) & (kNumXcd - 1);
      ++qtried;
    }
    return -1;
  };
  for (;;) {
  int unit, pair;
  if constexpr (PERSIST) {
    if (threadIdx.x == 0) {
      int p = -1;
      if (have_next) {
        p = qx + kNumXcd * (int)k_next;
        if (p >= n_slots) {
          qx = (qx + 1) & (kNumXcd - 1);
          ++qtried;
          p = claim();
        }
      } else {
        p = claim();
      }
      have_next = false;
      tile_slot = p;
    }
    __syncthreads();
    const int ps = __builtin_amdgcn_readfirstlane(tile_slot);
    __syncthreads();
    if (ps < 0) return;
    if (!map_tile(ps, P.G / HPW, P.n_units, unit, pair)) continue;
  } else {
    if (!map_tile(blockIdx.x, P.G / HPW, P.n_units, unit, pair)) return;
  }
  const int i = P.nb - 1 - (unit % P.nb);  // heaviest query blocks first
  const int ng = unit / P.nb;              // n * Hkv + g
  const int g = ng % P.Hkv, n = ng / P.Hkv;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, scalar
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

  // Q^T as the MFMA B operand: lane owns query row qrow, 8 chunks of 16 d (8 per lane half). Loaded
  // first: it does not depend on the list, so its latency overlaps the list reads below.
  bf16x8_t qf[8];
  {
    const uint16_t* qp = P.a.q + qo_off + (size_t)qrow * kHeadDim + 8 * half;
#pragma unroll
    for (int c = 0; c < 8; ++c) qf[c] = as_bf16x8(ldg16(qp + 16 * c));
  }

  // Packed sequences: block i only sees the blocks F .. i of its own sequence, whose skip
  // threshold is its own (F = 0 and the call's threshold without packing; the masked walk is
  // never packed).
  int seq;
  const int F = pack_first(P.a.pack, i, seq);
  const float tau = P.a.pack.n > 0 ? P.a.pack.tau[seq] : P.a.tau;
  int cnt;
  const int32_t* lst = nullptr;
  const uint8_t* mrow = nullptr;
  if constexpr (OSK) {
    cnt = ld_uniform(P.a.count + (size_t)ng * P.nb + i);
    cnt = cnt < P.nb ? cnt : P.nb;
    lst = P.a.order + ((size_t)ng * P.nb + i) * P.nb;
  } else {
    cnt = i - F + 1;
    if constexpr (MASKED) mrow = P.a.mask + ((size_t)ng * P.nb + i) * P.nb;
  }
  // List entries, read ahead of their use. A malformed entry (outside [F, i]) is fetched as block
  // i but contributes nothing. With a block mask, a masked block's entry is -1: nothing is fetched
  // or computed for it, but the walk still steps through it (logical skipping).
  auto raw_entry = [&](int kk) -> int {
    if constexpr (OSK) return kk < cnt ? lst[kk] : 0;
    else if constexpr (MASKED) return (kk < cnt && mrow[kk] != 0) ? kk : -1;
    else return F + kk;
  };
  auto listed = [&](int raw) -> bool { return (unsigned)(raw - F) <= (unsigned)(i - F); };
  auto page_of = [&](int raw) -> int { return listed(raw) ? raw : i; };

  // Physical pages of a listed block (paged caches): lane k loads the table entry of the block's k-th
  // page-sized segment (the lanes past the block's segments load entries they do not use, those past
  // the sequence's row read 0), through a buffer resource over the row of sequence n. The entry is
  // checked only where it is used, a page later: a check right after the load would wait for it.
  const int log2p = PAGED ? P.a.pg.log2_page : 0;
  const unsigned n_pages = PAGED ? (unsigned)min(P.a.pg.n_pages, 1LL << 31) : 0u;
  const __amdgpu_buffer_rsrc_t trs = __builtin_amdgcn_make_buffer_rsrc(
      PAGED ? (void*)(P.a.pg.table + (size_t)n * P.a.pg.pages_per_seq) : nullptr, (short)0,
      PAGED ? P.a.pg.pages_per_seq * 4 : 0, 0x00020000);
  auto table_of = [&](int raw) -> int {
    if constexpr (PAGED) {
      const int lp = ((page_of(raw) * BLOCK) >> log2p) + lane;
      return __builtin_amdgcn_raw_buffer_load_b32(trs, lp * 4, 0, 0);
    }
    return 0;
  };
  auto copy_block = [&](auto is_k, auto nwc, int raw, int tbl, char* dst, int wv)
      __attribute__((always_inline)) {
    constexpr bool IS_K = decltype(is_k)::value;
    constexpr int NW = decltype(nwc)::value;
    if constexpr (PAGED) {
      // K or V cache of KV head g; one physical page of one head is page * d elements, pages of
      // consecutive page numbers are Hkv of those apart.
      const uint64_t head_page_bytes = (uint64_t)kHeadDim * 2 << log2p;
      const uint64_t cache = (uint64_t)(IS_K ? P.a.k : P.a.v) + (uint64_t)g * head_page_bytes;
      copy_page_paged<BLOCK, NW, IS_K, PG == kPgWhole>(
          tbl, cache, head_page_bytes * (uint64_t)P.Hkv, n_pages, page_of(raw) * BLOCK, log2p, dst,
          wv, lane);
    } else {
      copy_page<BLOCK, NW, IS_K>(IS_K ? krs : vrs, dst, page_of(raw) * PAGE, wv, lane);
    }
  };

  // Prologue: K and V of page 0.
  auto first_entry = [&](int kk) -> int {
    if constexpr (OSK) return kk < cnt ? ld_uniform(lst + kk) : 0;
    else return raw_entry(kk);
  };
  const int raw0 = __builtin_amdgcn_readfirstlane(first_entry(0));
  const int raw1 = __builtin_amdgcn_readfirstlane(first_entry(1));
  const int raw2 = __builtin_amdgcn_readfirstlane(first_entry(2));
  int tbl_nxt = 0;
  if constexpr (PAGED) {
    // The first block's table entries come through scalar loads (lane k of tbl0 gets entry k), so
    // that its copies start without waiting for the Q fragments' vector loads issued above; the
    // next block's entries load as in the page loop.
    const int nseg = max(BLOCK >> log2p, 1);
    const int32_t* trow = P.a.pg.table + (size_t)n * P.a.pg.pages_per_seq +
                          ((page_of(raw0) * BLOCK) >> log2p);
    int tbl0 = 0;
#pragma unroll
    for (int kseg = 0; kseg < BLOCK / 16; ++kseg) {  // unconditional loads (clamped), issued together
      const int e = ld_uniform(trow + min(kseg, nseg - 1));
      tbl0 = lane == kseg ? e : tbl0;
    }
    tbl_nxt = table_of(raw1);
    if (cnt > 0) {
      copy_block(std::true_type{}, std::integral_constant<int, Cfg::kWaves>{}, raw0, tbl0, k_lds0, w);
      copy_block(std::false_type{}, std::integral_constant<int, Cfg::kWaves>{}, raw0, tbl0, v_lds0,
                 w);
    }
  } else {
    if (cnt > 0 && (!MASKED || listed(raw0))) {
      copy_block(std::true_type{}, std::integral_constant<int, Cfg::kWaves>{}, raw0, 0, k_lds0, w);
      copy_block(std::false_type{}, std::integral_constant<int, Cfg::kWaves>{}, raw0, 0, v_lds0, w);
    }
  }

  // O^T accumulators: tile dt holds d = 32 dt + 8 (r / 4) + 4 half + r % 4 of row qrow.
  f32x16_t o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;
  float m = -INFINITY;  // running row max (raw logits), identical in both lane halves
  float lsum = 0.f;     // this lane half's partial row sum

  // LDS read offsets. K: key 32 t + l32, d slot 2 c + half (t is an immediate). V: transposing
  // reads of rows 32 t + 16 c2 + 8 a + 4 half + (i / 4) and d = 32 dt + 16 g16 + 4 (i % 4), with
  // i = lane % 16 and g16 = (lane / 16) % 2 (t, c2, a are immediates; one offset per dt).
  int k_rd[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) k_rd[c] = l32 * 256 + (((2 * c + half) ^ (l32 & 15)) << 4);
  int v_rd[4];
  {
    const int li = lane & 15, g16 = (lane >> 4) & 1;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int slot = 4 * dt + 2 * g16 + ((li & 3) >> 1);
      v_rd[dt] = (4 * half + (li >> 2)) * 256 + ((slot ^ ((li >> 2) << 2)) << 4) + 8 * (li & 1);
    }
  }
  const size_t log_off = ((size_t)(n * P.Hq + h) * P.nb + i) * P.nb;
  int ncomp = 0;
  // List entries of pages m (cur), m+1 (nxt) and m+2 (nxt2), scalar; pre holds entry m+3 in flight
  // and, for paged caches, tbl_nxt2 the physical pages of entry m+2.
  int cur = raw0, nxt = raw1, nxt2 = raw2;
  int pre = 0, tbl_nxt2 = 0;

  __builtin_amdgcn_s_waitcnt(0);  // prologue pages, list entries and Q fragments
  __syncthreads();

  // State handed from QK(m) to PV(m) of the same wave.
  f32x16_t s[KT];
  float mnew = -INFINITY;
  bool v_pend = false;  // page m is a valid entry

  // QK(m) on K buffer BUF.
  auto qk_half = [&](auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    const char* Kb = BUF ? k_lds1 : k_lds0;
    const int j = page_of(cur);
    v_pend = (OSK || MASKED) ? listed(cur) : true;
    if (MASKED && !v_pend) return;  // a masked block: no Q K^T either
    // S^T tile t: keys 32 t + 8 (r / 4) + 4 half + r % 4 (register r) of query row qrow. The d chunk
    // is the outer loop: the KT tiles are independent accumulation chains. The KT fragments of
    // chunk c + 1 are read from LDS right after the first MFMA of chunk c, so their latency hides
    // behind that chunk's MFMAs (it is exposed when the partner wave has no P V work to fill in).
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[t][r] = 0.f;
    bf16x8_t kf[2][KT];
#pragma unroll
    for (int t = 0; t < KT; ++t)
      kf[0][t] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(Kb + k_rd[0] + t * 32 * 256));
    __builtin_amdgcn_sched_group_barrier(0x100, KT, 0);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      if (c + 1 < 8) {
#pragma unroll
        for (int t = 0; t < KT; ++t)
          kf[(c + 1) & 1][t] =
              as_bf16x8(*reinterpret_cast<const u32x4_t*>(Kb + k_rd[c + 1] + t * 32 * 256));
      }
#pragma unroll
      for (int t = 0; t < KT; ++t) s[t] = mfma32x32x16(kf[c & 1][t], qf[c], s[t]);
      if (c + 1 < 8) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);       // first MFMA of chunk c,
        __builtin_amdgcn_sched_group_barrier(0x100, KT, 0);      // the reads of chunk c + 1,
        __builtin_amdgcn_sched_group_barrier(0x008, KT - 1, 0);  // the rest of chunk c
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, KT, 0);
      }
    }
    if (j == i) {  // diagonal block: causal mask inside the tile
      // key 32 t + 8 (r / 4) + 4 half + r % 4 > query wl*32 + l32, with the lane part moved to the
      // right-hand side so that every compare is against an immediate
      // (the sign of qh - key selects -inf bit by bit, so no compare masks are kept in registers)
      int qh = wl * 32 + l32 - 4 * half;
      asm volatile("" : "+v"(qh));
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int d = qh - (32 * t + 8 * (r >> 2) + (r & 3));
          asm volatile("" : "+v"(d));
          const uint32_t masked = (uint32_t)(d >> 31);  // all ones where key > query
          const float sv = s[t][r];  // bit_cast of a vector element itself reads element 0
          const uint32_t bits = __builtin_bit_cast(uint32_t, sv);
          s[t][r] = __builtin_bit_cast(float, (bits & ~masked) | (0xFF800000u & masked));
        }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, s[t][r]);
    mloc = half_max(mloc);
    mnew = v_pend ? fmaxf(m, mloc) : m;
    if constexpr (OSK) {
      // Eq. (skip): each head's b-row tile votes with its largest (m_loc - m), in nats. Unless
      // that margin is logged, only its comparison with tau matters: the tile is skipped exactly
      // when every row's margin is below tau, so a ballot replaces the cross-lane maximum and the
      // wave votes 0 (some row reaches tau; tau <= 0) or -inf (none does).
      const float d = (mloc - mnew) * P.scale;
      float marg;
      if (P.a.margin_log)
        marg = wave_max(d);
      else
        marg = __ballot(d >= tau) ? 0.f : -INFINITY;
      if (lane == 0) vote[BUF][w] = marg;
    }
  };

  // PV(kk) on V buffer BUF: the votes of this head's waves were posted in the previous phase.
  auto pv_half = [&](int kk, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    const char* Vb = BUF ? v_lds1 : v_lds0;
    bool skip = !v_pend;
    if constexpr (OSK) {
      if (v_pend) {
        float dk = vote[BUF][hw * WPH];
#pragma unroll
        for (int ww = 1; ww < WPH; ++ww) dk = fmaxf(dk, vote[BUF][hw * WPH + ww]);
        skip = P.a.skip_on && (dk < tau);
        if (wl == 0 && lane == 0) {
          if (P.a.visit_log) P.a.visit_log[log_off + kk] = skip ? 2 : 1;
          if (P.a.margin_log) P.a.margin_log[log_off + kk] = dk;
        }
      }
    }
    // A skip implies m_loc < m in every row, so the running max is unchanged either way.
    if (!skip) {
      // A computing P V half is the critical path of its phase (softmax VALU, then its MFMAs,
      // beside the partner's Q K^T): its wave issues first, the partner fills the gaps.
      __builtin_amdgcn_s_setprio(1);
      const float alpha = __builtin_amdgcn_exp2f((m - mnew) * P.scale_log2);
      m = mnew;
      const float mb = mnew * P.scale_log2;
      if (__any(alpha != 1.f)) {  // the running max moved in some row of this wave
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
      }
      // O^T += V^T P^T over 16-key chunks kc = 2 t + c2: P^T element e of the chunk is register
      // 8 c2 + e of tile t (key 32 t + 16 c2 + 8 (e / 4) + 4 half + e % 4); the V^T operand is the
      // matching pair of transposing reads (e / 4 = a). The transposing reads are issued directly
      // so that the chunk and half-row offsets go into the instruction's offset field (the
      // compiler adds them to the address in a VALU op per read otherwise); the explicit wait
      // names the fragments, which hands them to the MFMAs and keeps their registers reserved
      // until the data has landed (the compiler does not see the reads as loads).
      // List and mask walks are software-pipelined: the V^T reads of chunk kc + 1 and the softmax
      // of chunk kc + 2 are issued behind the MFMAs of chunk kc (OSK 2.5 % faster). The dense
      // walk takes the softmax of the whole tile first, which measured 0.6 % faster there. Either
      // way the row sum takes the chunks, and their elements, in order.
      constexpr int KC = BLOCK / 16;
      constexpr bool kPipe = WALK != kWalkDense;
      float rs = 0.f;
      auto softmax_chunk = [&](int kc, bf16x8_t& pf) __attribute__((always_inline)) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = __builtin_amdgcn_exp2f(
              fmaf(s[kc >> 1][8 * (kc & 1) + e], P.scale_log2, -mb));
          rs += pv;
          pf[e] = (__bf16)pv;
        }
      };
      int va[4];
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) va[dt] = (int)(size_t)COSA_LDS(Vb) + v_rd[dt];
      s16x4_t lo[2][4], hi[2][4];
      bf16x8_t pf[KC];
      if constexpr (kPipe) {
        softmax_chunk(0, pf[0]);
        softmax_chunk(1, pf[1]);
      } else {
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) softmax_chunk(kc, pf[kc]);
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(lo[0][dt]) : "v"(va[dt]), "i"(0));
        asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                     : "=v"(hi[0][dt]) : "v"(va[dt]), "i"(8 * 256));
      }
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        const int cb = kc & 1, nx = cb ^ 1;
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(lo[cb][0]), "+v"(lo[cb][1]), "+v"(lo[cb][2]), "+v"(lo[cb][3]),
                       "+v"(hi[cb][0]), "+v"(hi[cb][1]), "+v"(hi[cb][2]), "+v"(hi[cb][3]));
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const bf16x8_t vf = __builtin_bit_cast(
              bf16x8_t, __builtin_shufflevector(lo[cb][dt], hi[cb][dt], 0, 1, 2, 3, 4, 5, 6, 7));
          o[dt] = mfma32x32x16(vf, pf[kc], o[dt]);
        }
        if (kc + 1 < KC) {
#pragma unroll
          for (int dt = 0; dt < 4; ++dt) {
            asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                         : "=v"(lo[nx][dt]) : "v"(va[dt]), "i"((kc + 1) * 16 * 256));
            asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                         : "=v"(hi[nx][dt]) : "v"(va[dt]), "i"((kc + 1) * 16 * 256 + 8 * 256));
          }
          if constexpr (kPipe) {
            if (kc + 2 < KC) softmax_chunk(kc + 2, pf[kc + 2]);
          }
        }
        if constexpr (!kPipe) {
          __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);  // the chunk's MFMAs ...
          __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);  // ... then the next chunk's reads
        }
      }
      lsum = fmaf(lsum, alpha, rs);
      ++ncomp;
      __builtin_amdgcn_s_setprio(0);
    }
  };

  // End of a phase: LDS writes done (and, with full, this wave's page copies landed), then the
  // workgroup barrier. The compiler barriers keep LDS accesses on their side of it.
  auto end_phase = [&](bool full) __attribute__((always_inline)) {
    if (full)
      __builtin_amdgcn_s_waitcnt(kVmcntLgkm0);
    else
      __builtin_amdgcn_s_waitcnt(kLgkm0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // Page kk, its buffers BUF: QK, fetch page kk+1 into the other buffers, barrier, PV, barrier.
  auto page = [&](int kk, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    if constexpr (PERSIST) {
      if (kk == cnt - 1 && threadIdx.x == 0 && qtried < kNumXcd) {
        k_next = atomicAdd(&P.a.queue[qx * 32], 1u);
        have_next = true;
      }
    }
    pre = raw_entry(kk + 3);
    if constexpr (PAGED) tbl_nxt2 = table_of(nxt2);
    qk_half(bufc);
    if (kk + 1 < cnt && (!MASKED || listed(nxt))) {
      constexpr auto NWH = std::integral_constant<int, WPH>{};
      if constexpr (HPW == 1) {
        copy_block(std::true_type{}, NWH, nxt, tbl_nxt, BUF ? k_lds0 : k_lds1, wl);
        copy_block(std::false_type{}, NWH, nxt, tbl_nxt, BUF ? v_lds0 : v_lds1, wl);
      } else if (hw == 0) {
        copy_block(std::true_type{}, NWH, nxt, tbl_nxt, BUF ? k_lds0 : k_lds1, wl);
      } else {
        copy_block(std::false_type{}, NWH, nxt, tbl_nxt, BUF ? v_lds0 : v_lds1, wl);
      }
    }
    end_phase(false);
    pv_half(kk, bufc);
    end_phase(true);
    cur = nxt;
    nxt = nxt2;
    nxt2 = __builtin_amdgcn_readfirstlane(pre);
    tbl_nxt = tbl_nxt2;
  };

  if (HPW == 2 && hw == 1) end_phase(false);  // head slot 1 runs one phase behind
  for (int kk = 0; kk < cnt; kk += 2) {
    page(kk, std::integral_constant<int, 0>{});
    if (kk + 1 < cnt) page(kk + 1, std::integral_constant<int, 1>{});
  }
  if (HPW == 2 && hw == 0) end_phase(false);  // same barrier count for both head slots

  lsum = half_sum(lsum);
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
  if constexpr (!PERSIST) break;
  }  // tiles of a persistent workgroup
}

template <int BLOCK, int HPW, int WALK, int PG>
void launch_t(const AttnParams& P, int G, hipStream_t stream) {
  using Cfg = TileCfg<BLOCK, HPW>;
  const int slots = (P.n_units + kNumXcd - 1) / kNumXcd * kNumXcd * (G / HPW);
  if constexpr (WALK == kWalkList) {
    if (P.a.queue != nullptr) {
      // One workgroup per CU (the LDS footprint admits one), fed by the work queues.
      int dev = 0, cus = 0;
      if (hipGetDevice(&dev) != hipSuccess ||
          hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
          cus < 1)
        cus = 256;
      hipLaunchKernelGGL(queue_reset, dim3(1), dim3(64), 0, stream, P.a.queue);
      hipLaunchKernelGGL((attention_kernel<BLOCK, HPW, WALK, PG, true>),
                         dim3(cus < slots ? cus : slots), dim3(Cfg::kThreads), 0, stream, P);
      return;
    }
  }
  hipLaunchKernelGGL((attention_kernel<BLOCK, HPW, WALK, PG, false>), dim3(slots),
                     dim3(Cfg::kThreads), 0, stream, P);
}

template <int WALK, int PG>
void launch_shape(const Shape& sh, const AttnParams& P, hipStream_t stream) {
  const bool pair = (sh.G % 2) == 0;
  if (sh.b == 128) {
    if (pair) launch_t<128, 2, WALK, PG>(P, sh.G, stream);
    else launch_t<128, 1, WALK, PG>(P, sh.G, stream);
  } else {
    if (pair) launch_t<64, 2, WALK, PG>(P, sh.G, stream);
    else launch_t<64, 1, WALK, PG>(P, sh.G, stream);
  }
}

template <int WALK>
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
  if constexpr (WALK == kWalkList) {
    if (a.pg.table == nullptr) launch_shape<kWalkList, kPgNone>(sh, P, stream);
    else if ((1 << a.pg.log2_page) >= sh.b) launch_shape<kWalkList, kPgWhole>(sh, P, stream);
    else launch_shape<kWalkList, kPgSplit>(sh, P, stream);
  } else {
    launch_shape<WALK, kPgNone>(sh, P, stream);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_osk_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream) {
  return launch<kWalkList>(sh, a, stream);
}

hipError_t launch_dense_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream) {
  return launch<kWalkDense>(sh, a, stream);
}

hipError_t launch_masked_attention(const Shape& sh, const AttnArgs& a, hipStream_t stream) {
  return launch<kWalkMask>(sh, a, stream);
}

}  // namespace cosa
