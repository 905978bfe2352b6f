// Internal declarations shared by the C ABI (pask_api.cpp) and the gfx950
// kernels (pask_append.hip, pask_attn.hip).  Not part of the public interface.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "pask.h"

namespace pask {

enum Store { kHi = 0, kLo = 1 };
enum Counter { kCntHi = 0, kCntLo = 1, kCntPos = 2, kCntDrop = 3, kCntForced = 4, kCntLost = 5,
               kCntBudget = 6 };   // int64 remaining budget R in words 6, 7
constexpr int kCounterStride = 8;
constexpr int kPage = 16;          // tokens per page
constexpr int kQGroup = 32;        // elements per fp16 scale of a RETAIN-LOW vector
// Range an attention worker on an odd-numbered XCD takes, in sixteenths of
// an even-XCD worker's: measured per-XCD finish times show the odd XCDs
// streaming pages about 10% slower (two boxes, every call).  With four
// workers per workgroup 15 and 14 tie on the batch-64 Qwen3-4B call, 15 is
// 2% faster on the int4-heavy prompt-side call and 0.4% slower on the
// Qwen3-32B-shaped one; 13 is slower on all.  Equal ranges (16) measured
// 1.8% slower on the batch-64 call (202.6 against 198.9 us, interleaved in
// one process), and so did ranges left to chunks taken at run time from a
// counter (2/16 of the work: 208.7 us; 4/16: 218.0 us).
#ifndef PASK_ODD_WEIGHT
#define PASK_ODD_WEIGHT 15
#endif
// Stream-K workers (single waves) per workgroup of the attention kernel for
// calls with more than 64 segments: 2,048 single-wave workgroups took 4.5 us
// to dispatch; four waves per workgroup measured 0.7% faster at batch 64.
#ifndef PASK_ATTN_WPB
#define PASK_ATTN_WPB 4
#endif
// Calls with at most 64 (sequence, KV head) segments take ranges of at least
// 1/PASK_SMALL_PIECES of the longest segment, so no segment is cut into more
// than PASK_SMALL_PIECES + 1 pieces (the ranges grow instead).  Interleaved in one
// process, per call at Qwen3-4B geometry with prompts U{1024..8192} against
// no cap (pieces of 4 pages): 2 sequences 25.0 -> 20.7 us, 3: 26.5 -> 21.2,
// 4: 30.2 -> 25.4, 6: 33.5 -> 29.4, 8: 38.3 -> 36.9, one sequence 17.5 ->
// 16.1 us and one 2.3k-entry sequence unchanged (13.8 / 13.9 us); caps of 16,
// 24 and 48 were each slower somewhere.  Fewer, longer workers carry less of
// the per-worker fixed cost (plan, q loads, block tables, partial rows) and
// leave fewer partials to merge.
#ifndef PASK_SMALL_PIECES
#define PASK_SMALL_PIECES 32
#endif
#ifndef PASK_UNIT_TOKENS
#define PASK_UNIT_TOKENS 128
#endif
constexpr int kUnitTokens = PASK_UNIT_TOKENS;   // slots per attention work unit (multiple of 16)
constexpr uint32_t kKeepAll = 1u;

// The online controller's inputs (Alg. 2; Eq. 9-10), one copy per cache.
// `loaded` holds kBudgetLoaded once pask_budget_init has written the rest.
constexpr uint32_t kBudgetLoaded = 0x42554447u;
struct BudgetTable {
  uint32_t loaded;
  uint32_t n_tags, n_groups, n_states, n_sink;
  uint32_t pad[3];
  int64_t m[PASK_MAX_GROUPS][3];      // bytes a token persists in group c under action a
  int64_t gamma[PASK_MAX_STATES];     // reserve Gamma(s), bytes (Eq. 9)
  uint8_t crit[PASK_MAX_STATES];      // critical or lookahead-critical state
  uint8_t action[PASK_MAX_TAGS][PASK_MAX_GROUPS];
  uint8_t floor_[PASK_MAX_TAGS][PASK_MAX_GROUPS];
  float rho_up[PASK_MAX_TAGS][PASK_MAX_GROUPS][2];   // Eq. 7: R->L, L->H
};
static_assert(sizeof(BudgetTable) % 16 == 0, "BudgetTable is copied in 16-byte words");

// Device-side view of one cache buffer.
struct CacheView {
  uint32_t* status;       // [0] status word, [2] HI cursor, [3] LO cursor
  int32_t* counters;      // [max_batch][n_layers][8]
  int32_t* block_table;   // [max_batch][n_layers][2][max_pages]
  int32_t* index_list;    // [max_batch][n_layers][2][max_tokens]
  int32_t* staging;       // [max_batch][staging_stride]
  BudgetTable* budget;
  uint8_t* ring_act;      // [max_batch][n_layers][window]: action | forced << 2
  uint8_t* hi_pool;       // recent-window pages first, then the HIGH store
  uint8_t* lo_pool;
  int32_t n_layers, n_kv_heads, head_dim, max_tokens, max_pages, lo_pages;
  int32_t hi_pages;       // pool pages including the recent windows
  int32_t hi_base;        // first page of the HIGH store (= recent-window pages)
  int32_t window;         // W
  int32_t ring_pp;        // pages of one (sequence, layer) window: ceil(W / 16)
  int32_t staging_stride; // max_tokens + W + 4: the last four are the append's HIGH and LOW
                          // store counts before it, its first position p0 and n_fit
  uint32_t hi_page_bytes, lo_page_bytes;
};

// Lambda's column for one layer group: selected action a0 and floor a- per tag.
struct TableColumn {
  uint8_t a0[64];
  uint8_t amin[64];
  uint32_t n_tags;
  uint32_t n_sink;
  uint32_t group;           // the layer's group c
};

struct AppendArgs {
  CacheView cv;
  TableColumn tab;
  const int32_t* n_new;     // [batch] or null (all max_new)
  const uint8_t* tags;      // [batch][max_new] or null (KEEP_ALL)
  const uint8_t* states;    // [batch][max_new] parser states, or null (Eq. 10 alone)
  const uint16_t* k;        // bf16 bits [batch][max_new][Hkv][D]
  const uint16_t* v;
  int32_t layer, batch, max_new;
  uint32_t flags;
};

struct AttnArgs {
  CacheView cv;
  const uint16_t* q;        // bf16 bits [batch][Hq][D]
  uint16_t* out;            // bf16 bits [batch][Hq][D]
  float* lse;               // [batch][Hq] or null
  float* ws_o;              // [batch][Hkv][splits][G4 * D], G4 = max(G, 4) heads
  float* ws_ml;             // [batch][Hkv][splits][G4][2]  (max, sum) in log2 units
  // The step's new entry, persisted by the call itself (kFusedMaxBatch
  // sequences at most, no recent window, no parser states): the attention
  // kernel decides it, writes it into its page and attends it; the merge
  // kernel enters it in the counters, lists and block tables.  Null when the
  // call persists nothing or the one-token append kernel ran before it.
  const uint8_t* tags_new;  // [batch]
  const uint16_t* k_new;    // bf16 bits [batch][Hkv][D]
  const uint16_t* v_new;
  int32_t* ws_seq;          // [batch][8]: the merge's page counts and the entry's outcome
  TableColumn tab;          // Lambda's column of the layer (with tags_new)
  float scale_log2;         // softmax_scale * log2(e)
  int32_t layer, batch, n_q_heads, splits;   // splits: partials per (b, g) the workspace holds
  int32_t attn_blocks;      // stream-K workers (waves) of the attention kernel, set at launch
  int32_t min_pages;        // fewest pages a worker takes (HIGH-page weight), set at launch
};

// Calls with at most kSmallSegments (sequence, KV head) segments cut them
// finer (pieces down to kSmallMinPages pages, the workspace holding up to
// kSmallPartials partials in all) and merge each segment's pieces with
// several thread groups at once.
constexpr int kSmallSegments = 64;
constexpr int kSmallPartials = 4096;
// Calls that persist their step's entry themselves: every worker decides the
// entries of all sequences, 64 at a time (one per lane of its wave), and
// keeps their counts and outcomes in LDS.
constexpr int kFusedMaxBatch = 256;

// The library-owned scratch of pask_decode_attn_noalloc: a device array of
// kScratchBytes in pask_attn.hip, one copy per GPU.  scratch_workspace gives
// the current device's address of it (hipGetSymbolAddress, taken once per
// device with that device current, then cached).
constexpr size_t kScratchBytes = PASK_NOALLOC_SCRATCH_BYTES;
hipError_t scratch_workspace(void** ptr);

// Launchers (pask_append.hip: reset, budget init, append; pask_attn.hip:
// attention, distortion).  Return hipSuccess or the launch error.
hipError_t launch_reset(const CacheView& cv, int32_t max_batch, hipStream_t s);
hipError_t launch_append(const AppendArgs& a, hipStream_t s);        // chooses the windowed kernels when W > 0
hipError_t launch_append_step(const AppendArgs& a, hipStream_t s);
hipError_t launch_budget_init(const CacheView& cv, int32_t batch, int64_t r0, hipStream_t s);
hipError_t launch_attention(const AttnArgs& a, int group_size, hipStream_t s);
// Attention over two caches with the same queries (partials in ref.ws_* and itv.ws_*), then
// dist[b] += max over heads of the squared distance of the two outputs (Eq. 4).
hipError_t launch_distortion(const AttnArgs& ref, const AttnArgs& itv, int group_size, const uint8_t* in_s,
                             float* dist, hipStream_t s);

}  // namespace pask
