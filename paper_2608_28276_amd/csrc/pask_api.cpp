// Host side of the PASK C ABI: policy parsing and validation, cache layout,
// argument checks, launch planning and cache accounting.  Every check runs
// before the first HIP call of an entry point.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <vector>

#include <hip/hip_runtime_api.h>

#include "pask_internal.h"

namespace {

using pask::CacheView;

constexpr uint64_t kAlignSmall = 256;
constexpr uint64_t kAlignPool = 4096;

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

bool valid_geom(const pask_geom* g) {
  if (!g) return false;
  if (g->max_batch < 1 || g->max_batch > 65535) return false;
  if (g->n_layers < 1 || g->n_layers > PASK_MAX_LAYERS) return false;
  if (g->n_kv_heads < 1 || g->n_kv_heads > 8 || g->n_q_heads < g->n_kv_heads) return false;
  if (g->n_q_heads % g->n_kv_heads != 0) return false;
  const int gs = g->n_q_heads / g->n_kv_heads;
  if (gs != 1 && gs != 2 && gs != 4 && gs != 8) return false;
  if (g->head_dim != 64 && g->head_dim != 128) return false;
  if (g->page_tokens != PASK_PAGE_TOKENS) return false;
  if (g->max_tokens_per_seq < 1 || g->max_tokens_per_seq > (1 << 28)) return false;
  if (g->hi_pages < 0 || g->lo_pages < 0) return false;
  if (g->recent_window < 0 || g->recent_window > g->max_tokens_per_seq) return false;
  const int64_t ring = (int64_t)g->max_batch * g->n_layers * ((g->recent_window + PASK_PAGE_TOKENS - 1) / PASK_PAGE_TOKENS);
  if (ring + g->hi_pages > INT32_MAX) return false;
  return true;
}

// Layout of a cache buffer; false when the geometry is unsupported.
bool layout_of(const pask_geom* g, pask_cache_layout* L) {
  if (!valid_geom(g)) return false;
  memset(L, 0, sizeof(*L));
  const uint64_t B = (uint64_t)g->max_batch, NL = (uint64_t)g->n_layers;
  const uint64_t D = (uint64_t)g->head_dim, H = (uint64_t)g->n_kv_heads;
  const uint64_t T = (uint64_t)g->max_tokens_per_seq;
  const uint64_t W = (uint64_t)g->recent_window;
  L->max_pages = (int32_t)((T + PASK_PAGE_TOKENS - 1) / PASK_PAGE_TOKENS);
  L->counter_stride = pask::kCounterStride;
  L->ring_pages = (int32_t)(B * NL * ((W + PASK_PAGE_TOKENS - 1) / PASK_PAGE_TOKENS));
  L->staging_stride = (int32_t)(T + W + 4);
  L->hi_page_bytes = H * 2 * PASK_PAGE_TOKENS * D * 2;
  L->lo_page_bytes = H * 2 * (PASK_PAGE_TOKENS * (D / 2) + PASK_PAGE_TOKENS * (D / PASK_QGROUP) * 2);
  uint64_t off = 0;
  L->status_off = off;
  off = align_up(off + 16, kAlignSmall);
  L->counters_off = off;
  off = align_up(off + B * NL * pask::kCounterStride * 4, kAlignSmall);
  L->block_table_off = off;
  off = align_up(off + B * NL * 2 * (uint64_t)L->max_pages * 4, kAlignSmall);
  L->index_list_off = off;
  off = align_up(off + B * NL * 2 * T * 4, kAlignSmall);
  L->staging_off = off;
  off = align_up(off + B * (uint64_t)L->staging_stride * 4, kAlignSmall);
  L->budget_off = off;
  off = align_up(off + sizeof(pask::BudgetTable), kAlignSmall);
  L->ring_act_off = off;
  off = align_up(off + B * NL * W, kAlignPool);
  L->hi_pool_off = off;
  off = align_up(off + ((uint64_t)L->ring_pages + g->hi_pages) * L->hi_page_bytes, kAlignPool);
  L->lo_pool_off = off;
  off = align_up(off + (uint64_t)g->lo_pages * L->lo_page_bytes, kAlignPool);
  L->total_bytes = off;
  return true;
}

CacheView view_of(const pask_cache* c) {
  pask_cache_layout L;
  layout_of(&c->geom, &L);
  uint8_t* base = static_cast<uint8_t*>(c->base);
  CacheView v;
  v.status = reinterpret_cast<uint32_t*>(base + L.status_off);
  v.counters = reinterpret_cast<int32_t*>(base + L.counters_off);
  v.block_table = reinterpret_cast<int32_t*>(base + L.block_table_off);
  v.index_list = reinterpret_cast<int32_t*>(base + L.index_list_off);
  v.staging = reinterpret_cast<int32_t*>(base + L.staging_off);
  v.budget = reinterpret_cast<pask::BudgetTable*>(base + L.budget_off);
  v.ring_act = base + L.ring_act_off;
  v.hi_pool = base + L.hi_pool_off;
  v.lo_pool = base + L.lo_pool_off;
  v.n_layers = c->geom.n_layers;
  v.n_kv_heads = c->geom.n_kv_heads;
  v.head_dim = c->geom.head_dim;
  v.max_tokens = c->geom.max_tokens_per_seq;
  v.max_pages = L.max_pages;
  v.hi_pages = L.ring_pages + c->geom.hi_pages;
  v.hi_base = L.ring_pages;
  v.window = c->geom.recent_window;
  v.ring_pp = (c->geom.recent_window + PASK_PAGE_TOKENS - 1) / PASK_PAGE_TOKENS;
  v.staging_stride = L.staging_stride;
  v.lo_pages = c->geom.lo_pages;
  v.hi_page_bytes = (uint32_t)L.hi_page_bytes;
  v.lo_page_bytes = (uint32_t)L.lo_page_bytes;
  return v;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// PASK_DEBUG set to anything but "" or "0" when the library is first used
// turns on a check after every entry point that launches kernels: it waits for
// the stream, turns a launch or execution error into PASK_E_HIP, and writes to
// stderr the entry point with the HIP error, or with the cache's device status
// flags when they differ from the last ones reported.  A failure is then named
// by the call that caused it, not by a later synchronisation.  Calls on a
// stream that is being captured into a graph are not checked.  Off by default:
// each check costs a host round trip.
bool debug_on() {
  static const bool on = [] {
    const char* e = getenv("PASK_DEBUG");
    return e && e[0] && strcmp(e, "0") != 0;
  }();
  return on;
}

int debug_check(const char* where, int st, const pask_cache* const* caches, int n_caches, hipStream_t stream) {
  if (st != PASK_OK || !debug_on()) return st;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cs);
  if (e == hipSuccess && cs != hipStreamCaptureStatusNone) return st;
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) {
    fprintf(stderr, "pask: %s: %s\n", where, hipGetErrorString(e));
    return PASK_E_HIP;
  }
  static std::atomic<uint32_t> reported{0};
  for (int i = 0; i < n_caches; ++i) {
    pask_cache_layout L;
    layout_of(&caches[i]->geom, &L);
    uint32_t word = 0;
    const uint8_t* status = static_cast<const uint8_t*>(caches[i]->base) + L.status_off;
    if (hipMemcpyAsync(&word, status, sizeof(word), hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess) {
      fprintf(stderr, "pask: %s: status word not readable\n", where);
      return PASK_E_HIP;
    }
    if (word != 0 && reported.exchange(word) != word)
      fprintf(stderr, "pask: %s: device status flags 0x%x\n", where, word);
  }
  return st;
}

int debug_check(const char* where, int st, const pask_cache* cache, hipStream_t stream) {
  return debug_check(where, st, &cache, 1, stream);
}

int check_cache(const pask_cache* c) {
  if (!c || !c->base) return PASK_E_ARG;
  if (!valid_geom(&c->geom)) return PASK_E_SHAPE;
  if (!aligned(c->base, 256)) return PASK_E_ARG;
  pask_cache_layout L;
  layout_of(&c->geom, &L);
  if (c->bytes < L.total_bytes) return PASK_E_CAPACITY;
  return PASK_OK;
}

int check_policy(const pask_policy* p, const pask_cache* c) {
  if (!p) return PASK_E_ARG;
  if (p->n_tags < 1 || p->n_tags > PASK_MAX_TAGS || p->n_groups < 1 || p->n_groups > PASK_MAX_GROUPS)
    return PASK_E_POLICY;
  if ((int32_t)p->n_layers != c->geom.n_layers) return PASK_E_SHAPE;
  if ((int32_t)p->recent_window != c->geom.recent_window) return PASK_E_SHAPE;
  for (uint32_t l = 0; l < p->n_layers; ++l)
    if (p->group_of_layer[l] >= p->n_groups) return PASK_E_POLICY;
  if (p->n_states > PASK_MAX_STATES) return PASK_E_POLICY;
  return PASK_OK;
}

// Bytes one token persists in the layers of group c under action a (the
// accounting of Eq. 1): the group's layer count times one entry's bytes.
void group_costs(const pask_policy* p, const pask_geom& g, int64_t m[PASK_MAX_GROUPS][3]) {
  const int64_t H = g.n_kv_heads, D = g.head_dim;
  const int64_t entry[3] = {0, 2 * H * (D / 2 + 2 * (D / PASK_QGROUP)), 2 * H * D * 2};
  int64_t layers[PASK_MAX_GROUPS] = {};
  for (uint32_t l = 0; l < p->n_layers; ++l) ++layers[p->group_of_layer[l]];
  for (int c = 0; c < PASK_MAX_GROUPS; ++c)
    for (int a = 0; a < 3; ++a) m[c][a] = layers[c] * entry[a];
}

pask::TableColumn column_of(const pask_policy* p, int layer) {
  pask::TableColumn t;
  memset(&t, 0, sizeof(t));
  const int c = p->group_of_layer[layer];
  for (uint32_t z = 0; z < p->n_tags; ++z) {
    t.a0[z] = p->action[z][c];
    t.amin[z] = p->floor_[z][c];
  }
  t.n_tags = p->n_tags;
  t.n_sink = p->n_sink;
  t.group = (uint32_t)c;
  return t;
}

uint32_t fnv1a32(const uint8_t* d, size_t n) {
  uint32_t h = 0x811C9DC5u;
  for (size_t i = 0; i < n; ++i) {
    h ^= d[i];
    h *= 0x01000193u;
  }
  return h;
}

template <typename T>
T rd(const uint8_t* p) {
  T v;
  memcpy(&v, p, sizeof(T));
  return v;
}

// Partials one (sequence, KV head) may be cut into: the attention kernel picks
// its pages-per-block so that this bound holds for any counts; the hint only
// sizes the workspace.  Pieces of kUnitTokens tokens; for calls with few
// segments, pieces down to one page while the call holds at most
// kSmallPartials partials.
int splits_for(int32_t max_ctx_hint, int64_t segments) {
  const int coarse = (max_ctx_hint + pask::kUnitTokens - 1) / pask::kUnitTokens + 2;
  if (segments > pask::kSmallSegments) return coarse;
  const int fine = (max_ctx_hint + pask::kPage - 1) / pask::kPage + 2;
  return std::max(coarse, std::min(fine, (int)(pask::kSmallPartials / std::max<int64_t>(segments, 1))));
}


struct WsLayout {
  uint64_t o_off, ml_off, seq_off, total;
};

// Partials of the attention pieces: per (sequence, KV head, piece) a block of
// G4 = max(G, 4) query-head rows of head_dim fp32 values, and G4 (max, sum)
// pairs; then 8 int32 per sequence for a call that persists its step's
// entries (the counts its attention planned with and each entry's outcome).
WsLayout ws_layout(const pask_geom* g, int32_t batch, int splits) {
  WsLayout w;
  const uint64_t group = (uint64_t)std::max(4, g->n_q_heads / g->n_kv_heads);
  const uint64_t blocks = (uint64_t)batch * g->n_kv_heads * splits;
  w.o_off = 0;
  w.ml_off = align_up(blocks * group * g->head_dim * 4, kAlignSmall);
  w.seq_off = align_up(w.ml_off + blocks * group * 2 * 4, kAlignSmall);
  w.total = align_up(w.seq_off + (uint64_t)batch * 8 * 4, kAlignSmall);
  return w;
}

// One decode step of one layer (pask_decode_attn): validation, then the
// optional one-token append and the attention launches.  use_scratch: the
// partials go to this device's library-owned scratch (kScratchBytes) instead
// of the caller's workspace, with as many pieces per (sequence, KV head) as
// fit there (at least two; fewer pieces only make the per-worker page ranges
// longer, the results are the same).
int decode_attn(const pask_policy* policy, pask_cache* cache, int32_t layer, int32_t batch, const void* q_dev,
                void* out_dev, float* lse_dev, const uint8_t* tags_new_dev, const uint8_t* states_new_dev,
                const void* k_new_dev, const void* v_new_dev, float softmax_scale, int32_t max_ctx_hint,
                void* ws_dev, size_t ws_bytes, bool use_scratch, hipStream_t stream) {
  int st = check_cache(cache);
  if (st != PASK_OK) return st;
  st = check_policy(policy, cache);
  if (st != PASK_OK) return st;
  const pask_geom& g = cache->geom;
  if (layer < 0 || layer >= g.n_layers) return PASK_E_SHAPE;
  if (batch < 1 || batch > g.max_batch) return PASK_E_SHAPE;
  if (!q_dev || !out_dev || !aligned(q_dev, 16) || !aligned(out_dev, 16)) return PASK_E_ARG;
  if (lse_dev && !aligned(lse_dev, 4)) return PASK_E_ARG;
  if (tags_new_dev && (!k_new_dev || !v_new_dev || !aligned(k_new_dev, 16) || !aligned(v_new_dev, 16)))
    return PASK_E_ARG;
  if (tags_new_dev && states_new_dev && policy->n_states == 0) return PASK_E_POLICY;
  if (!isfinite(softmax_scale)) return PASK_E_ARG;
  if (max_ctx_hint < 1) max_ctx_hint = g.max_tokens_per_seq;
  int splits = splits_for(std::min(max_ctx_hint, g.max_tokens_per_seq), (int64_t)batch * g.n_kv_heads);
  if (use_scratch) {
    while (splits > 2 && ws_layout(&g, batch, splits).total > pask::kScratchBytes) --splits;
    if (ws_layout(&g, batch, splits).total > pask::kScratchBytes) return PASK_E_CAPACITY;
  }
  const WsLayout w = ws_layout(&g, batch, splits);
  if (!use_scratch) {
    if (!ws_dev || !aligned(ws_dev, 256)) return PASK_E_ARG;
    if (ws_bytes < w.total) return PASK_E_CAPACITY;
  } else if (pask::scratch_workspace(&ws_dev) != hipSuccess) {   // first HIP call of the scratch path
    return PASK_E_HIP;
  }

  // The step's entries are persisted by the attention call itself (no
  // one-token append kernel) for at most kFusedMaxBatch sequences without a
  // recent window or parser states; otherwise by the append kernel first.
  const bool fused = tags_new_dev && !states_new_dev && g.recent_window == 0 && batch <= pask::kFusedMaxBatch;
  if (tags_new_dev && !fused) {
    pask::AppendArgs a;
    a.cv = view_of(cache);
    a.tab = column_of(policy, layer);
    a.n_new = nullptr;
    a.tags = tags_new_dev;
    a.states = states_new_dev;
    a.k = static_cast<const uint16_t*>(k_new_dev);
    a.v = static_cast<const uint16_t*>(v_new_dev);
    a.layer = layer;
    a.batch = batch;
    a.max_new = 1;
    a.flags = 0;
    if (pask::launch_append_step(a, stream) != hipSuccess) return PASK_E_HIP;
  }
  pask::AttnArgs a;
  a.cv = view_of(cache);
  a.q = static_cast<const uint16_t*>(q_dev);
  a.out = static_cast<uint16_t*>(out_dev);
  a.lse = lse_dev;
  a.ws_o = reinterpret_cast<float*>(static_cast<uint8_t*>(ws_dev) + w.o_off);
  a.ws_ml = reinterpret_cast<float*>(static_cast<uint8_t*>(ws_dev) + w.ml_off);
  a.scale_log2 = (float)((double)softmax_scale * 1.4426950408889634);
  a.layer = layer;
  a.batch = batch;
  a.n_q_heads = g.n_q_heads;
  a.splits = splits;
  a.tags_new = fused ? tags_new_dev : nullptr;
  a.k_new = fused ? static_cast<const uint16_t*>(k_new_dev) : nullptr;
  a.v_new = fused ? static_cast<const uint16_t*>(v_new_dev) : nullptr;
  a.ws_seq = reinterpret_cast<int32_t*>(static_cast<uint8_t*>(ws_dev) + w.seq_off);
  a.tab = column_of(policy, layer);
  return debug_check(use_scratch ? "pask_decode_attn_noalloc" : "pask_decode_attn",
                     pask::launch_attention(a, g.n_q_heads / g.n_kv_heads, stream) == hipSuccess ? PASK_OK : PASK_E_HIP,
                     cache, stream);
}

}  // namespace

extern "C" {

const char* pask_status_string(int s) {
  switch (s) {
    case PASK_OK: return "ok";
    case PASK_E_ARG: return "invalid argument";
    case PASK_E_POLICY: return "malformed policy";
    case PASK_E_SHAPE: return "unsupported or mismatched shape";
    case PASK_E_CAPACITY: return "buffer too small";
    case PASK_E_HIP: return "HIP error";
    case PASK_E_DEVICE_FLAG: return "device status flag set";
    case PASK_E_UNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

int pask_policy_load(const void* blob, size_t nbytes, const pask_geom* geom, pask_policy* out) {
  if (!blob || !out) return PASK_E_ARG;
  if (geom && !valid_geom(geom)) return PASK_E_SHAPE;
  const uint8_t* b = static_cast<const uint8_t*>(blob);
  if (nbytes < 36) return PASK_E_POLICY;
  if (memcmp(b, "PASK", 4) != 0) return PASK_E_POLICY;
  const uint16_t version = rd<uint16_t>(b + 4);
  if ((version != 1 && version != 2) || rd<uint16_t>(b + 6) != 32) return PASK_E_POLICY;
  const uint32_t T = rd<uint32_t>(b + 8), C = rd<uint32_t>(b + 12), NL = rd<uint32_t>(b + 16);
  const uint32_t n_sink = rd<uint32_t>(b + 20), window = rd<uint32_t>(b + 24);
  const uint32_t body = rd<uint32_t>(b + 28);
  if (T < 1 || T > PASK_MAX_TAGS || C < 1 || C > PASK_MAX_GROUPS || NL < 1 || NL > PASK_MAX_LAYERS)
    return PASK_E_POLICY;
  const uint64_t bytes_u8 = (uint64_t)NL + 2ull * T * C;
  const uint64_t table_body = align_up(bytes_u8, 4) + 8ull * T * C;
  // Version 2: the controller section follows the table.
  uint32_t S = 0;
  if (version == 2) {
    if (body < table_body + 8 || nbytes < 32 + table_body + 8) return PASK_E_POLICY;
    S = rd<uint32_t>(b + 32 + table_body);
    if (S < 1 || S > PASK_MAX_STATES) return PASK_E_POLICY;
  }
  const uint64_t want_body = version == 2 ? table_body + 8 + 4ull * S + align_up(S, 4) : table_body;
  if (body != want_body || nbytes != 32 + (uint64_t)body + 4) return PASK_E_POLICY;
  if (rd<uint32_t>(b + 32 + body) != fnv1a32(b, 32 + body)) return PASK_E_POLICY;
  const uint8_t* gol = b + 32;
  const uint8_t* act = gol + NL;
  const uint8_t* flo = act + T * C;
  const uint8_t* rho = b + 32 + align_up(bytes_u8, 4);
  for (uint64_t i = bytes_u8; i < align_up(bytes_u8, 4); ++i)
    if (b[32 + i] != 0) return PASK_E_POLICY;
  const uint8_t* ctl = b + 32 + table_body;   // version 2: n_states, beta_q, reserve_q[S], crit[S]
  if (version == 2) {
    for (uint32_t i = 0; i < S; ++i)
      if (ctl[8 + 4 * S + i] > 1) return PASK_E_POLICY;
    for (uint64_t i = S; i < align_up(S, 4); ++i)
      if (ctl[8 + 4 * S + i] != 0) return PASK_E_POLICY;
  }
  for (uint32_t l = 0; l < NL; ++l)
    if (gol[l] >= C) return PASK_E_POLICY;
  for (uint32_t i = 0; i < T * C; ++i)
    if (act[i] > PASK_RETAIN_HIGH || flo[i] > PASK_RETAIN_HIGH) return PASK_E_POLICY;
  for (uint32_t i = 0; i < 2 * T * C; ++i) {
    const float r = rd<float>(rho + 4 * i);
    if (!(r >= 0.0f) || isinf(r)) return PASK_E_POLICY;
  }
  if (geom && ((int32_t)NL != geom->n_layers || (int64_t)window != (int64_t)geom->recent_window))
    return PASK_E_SHAPE;

  pask_policy p;
  memset(&p, 0, sizeof(p));
  p.n_tags = T;
  p.n_groups = C;
  p.n_layers = NL;
  p.n_sink = n_sink;
  p.recent_window = window;
  memcpy(p.group_of_layer, gol, NL);
  for (uint32_t z = 0; z < T; ++z)
    for (uint32_t c = 0; c < C; ++c) {
      p.action[z][c] = act[z * C + c];
      p.floor_[z][c] = flo[z * C + c];
      p.rho_up[z][c][0] = rd<float>(rho + 4 * (2 * (z * C + c)));
      p.rho_up[z][c][1] = rd<float>(rho + 4 * (2 * (z * C + c) + 1));
    }
  if (version == 2) {
    p.n_states = S;
    p.beta_q = rd<uint32_t>(ctl + 4);
    for (uint32_t i = 0; i < S; ++i) {
      p.reserve_q[i] = rd<uint32_t>(ctl + 8 + 4 * i);
      p.crit[i] = ctl[8 + 4 * S + i];
    }
  }
  if (geom) {
    const uint64_t H = (uint64_t)geom->n_kv_heads, D = (uint64_t)geom->head_dim;
    p.entry_bytes[PASK_DROP] = 0;
    p.entry_bytes[PASK_RETAIN_LOW] = 2 * H * (D / 2 + 2 * (D / PASK_QGROUP));
    p.entry_bytes[PASK_RETAIN_HIGH] = 2 * H * D * 2;
  }
  *out = p;
  return PASK_OK;
}

int pask_cache_layout_query(const pask_geom* geom, pask_cache_layout* out) {
  if (!geom || !out) return PASK_E_ARG;
  return layout_of(geom, out) ? PASK_OK : PASK_E_SHAPE;
}

size_t pask_cache_bytes(const pask_geom* geom) {
  pask_cache_layout L;
  if (!layout_of(geom, &L)) return 0;
  return (size_t)L.total_bytes;
}

int pask_cache_reset(pask_cache* cache, hipStream_t stream) {
  const int st = check_cache(cache);
  if (st != PASK_OK) return st;
  const CacheView v = view_of(cache);
  return debug_check("pask_cache_reset",
                     pask::launch_reset(v, cache->geom.max_batch, stream) == hipSuccess ? PASK_OK : PASK_E_HIP, cache,
                     stream);
}

int pask_cache_init(pask_cache* cache, const pask_geom* geom, void* base, size_t bytes, hipStream_t stream) {
  if (!cache || !geom || !base) return PASK_E_ARG;
  if (!valid_geom(geom)) return PASK_E_SHAPE;
  if (!aligned(base, 256)) return PASK_E_ARG;
  if (bytes < pask_cache_bytes(geom)) return PASK_E_CAPACITY;
  cache->geom = *geom;
  cache->base = base;
  cache->bytes = bytes;
  return pask_cache_reset(cache, stream);
}

int pask_kv_append(const pask_policy* policy, pask_cache* cache, int32_t layer, int32_t batch,
                   const int32_t* n_new_dev, int32_t max_new, const uint8_t* tags_dev,
                   const uint8_t* states_dev, const void* k_dev, const void* v_dev, uint32_t flags,
                   hipStream_t stream) {
  int st = check_cache(cache);
  if (st != PASK_OK) return st;
  st = check_policy(policy, cache);
  if (st != PASK_OK) return st;
  const pask_geom& g = cache->geom;
  if (layer < 0 || layer >= g.n_layers) return PASK_E_SHAPE;
  if (batch < 1 || batch > g.max_batch) return PASK_E_SHAPE;
  if (max_new < 0 || max_new > g.max_tokens_per_seq) return PASK_E_SHAPE;
  if (flags & ~(uint32_t)PASK_APPEND_KEEP_ALL) return PASK_E_ARG;
  if (!k_dev || !v_dev || !aligned(k_dev, 16) || !aligned(v_dev, 16)) return PASK_E_ARG;
  if (!tags_dev && !(flags & PASK_APPEND_KEEP_ALL)) return PASK_E_ARG;
  if (n_new_dev && !aligned(n_new_dev, 4)) return PASK_E_ARG;
  const bool keep_all = (flags & PASK_APPEND_KEEP_ALL) != 0u;
  if (states_dev && !keep_all && policy->n_states == 0) return PASK_E_POLICY;
  if (max_new == 0) return PASK_OK;
  pask::AppendArgs a;
  a.cv = view_of(cache);
  a.tab = column_of(policy, layer);
  a.n_new = n_new_dev;
  a.tags = tags_dev;
  a.states = keep_all ? nullptr : states_dev;   // a keep-all append bypasses the controller
  a.k = static_cast<const uint16_t*>(k_dev);
  a.v = static_cast<const uint16_t*>(v_dev);
  a.layer = layer;
  a.batch = batch;
  a.max_new = max_new;
  a.flags = flags;
  return debug_check("pask_kv_append", pask::launch_append(a, stream) == hipSuccess ? PASK_OK : PASK_E_HIP, cache,
                     stream);
}

int pask_budget_init(const pask_policy* policy, pask_cache* cache, int32_t batch, int32_t t_max,
                     hipStream_t stream) {
  int st = check_cache(cache);
  if (st != PASK_OK) return st;
  st = check_policy(policy, cache);
  if (st != PASK_OK) return st;
  const pask_geom& g = cache->geom;
  if (batch < 1 || batch > g.max_batch) return PASK_E_SHAPE;
  if (t_max < 0) return PASK_E_ARG;
  if (policy->n_states == 0) return PASK_E_POLICY;
  for (uint32_t z = 0; z < policy->n_tags; ++z)
    for (uint32_t c = 0; c < policy->n_groups; ++c)
      if (policy->action[z][c] > PASK_RETAIN_HIGH || policy->floor_[z][c] > PASK_RETAIN_HIGH) return PASK_E_POLICY;
  pask::BudgetTable t;
  memset(&t, 0, sizeof(t));
  t.loaded = pask::kBudgetLoaded;
  t.n_tags = policy->n_tags;
  t.n_groups = policy->n_groups;
  t.n_states = policy->n_states;
  t.n_sink = policy->n_sink;
  group_costs(policy, g, t.m);
  int64_t full = 0;   // bytes of one token kept HIGH in every layer
  for (uint32_t c = 0; c < policy->n_groups; ++c) full += t.m[c][PASK_RETAIN_HIGH];
  const unsigned __int128 r0 = (unsigned __int128)policy->beta_q * (uint64_t)t_max * (uint64_t)full / 65536u;
  if (r0 >= ((unsigned __int128)1 << 62)) return PASK_E_ARG;
  for (uint32_t s = 0; s < policy->n_states; ++s) {
    t.gamma[s] = (int64_t)(((unsigned __int128)policy->reserve_q[s] * (uint64_t)full) / 16u);
    t.crit[s] = policy->crit[s] ? 1 : 0;
  }
  memcpy(t.action, policy->action, sizeof(t.action));
  memcpy(t.floor_, policy->floor_, sizeof(t.floor_));
  memcpy(t.rho_up, policy->rho_up, sizeof(t.rho_up));
  const CacheView v = view_of(cache);
  if (hipMemcpyAsync(v.budget, &t, sizeof(t), hipMemcpyHostToDevice, stream) != hipSuccess) return PASK_E_HIP;
  const bool launched = pask::launch_budget_init(v, batch, (int64_t)r0, stream) == hipSuccess;
  // `t` lives on this frame: the copy must be done before returning.
  const bool synced = hipStreamSynchronize(stream) == hipSuccess;
  return debug_check("pask_budget_init", launched && synced ? PASK_OK : PASK_E_HIP, cache, stream);
}

size_t pask_workspace_bytes(const pask_geom* geom, int32_t batch, int32_t max_ctx_hint) {
  if (!valid_geom(geom) || batch < 1 || batch > geom->max_batch) return 0;
  // no sequence holds more than max_tokens_per_seq entries: a larger hint sizes nothing more
  if (max_ctx_hint < 1 || max_ctx_hint > geom->max_tokens_per_seq) max_ctx_hint = geom->max_tokens_per_seq;
  return (size_t)ws_layout(geom, batch, splits_for(max_ctx_hint, (int64_t)batch * geom->n_kv_heads)).total;
}

int pask_decode_attn(const pask_policy* policy, pask_cache* cache, int32_t layer, int32_t batch,
                     const void* q_dev, void* out_dev, float* lse_dev, const uint8_t* tags_new_dev,
                     const uint8_t* states_new_dev, const void* k_new_dev, const void* v_new_dev,
                     float softmax_scale,
                     int32_t max_ctx_hint, void* ws_dev, size_t ws_bytes, hipStream_t stream) {
  return decode_attn(policy, cache, layer, batch, q_dev, out_dev, lse_dev, tags_new_dev, states_new_dev, k_new_dev,
                     v_new_dev, softmax_scale, max_ctx_hint, ws_dev, ws_bytes, false, stream);
}

int pask_decode_attn_noalloc(const pask_policy* policy, pask_cache* cache, int32_t layer, int32_t batch,
                             const void* q_dev, void* out_dev, float* lse_dev, const uint8_t* tags_new_dev,
                             const uint8_t* states_new_dev, const void* k_new_dev, const void* v_new_dev,
                             float softmax_scale, int32_t max_ctx_hint, hipStream_t stream) {
  return decode_attn(policy, cache, layer, batch, q_dev, out_dev, lse_dev, tags_new_dev, states_new_dev, k_new_dev,
                     v_new_dev, softmax_scale, max_ctx_hint, nullptr, 0, true, stream);
}

int pask_attn_distortion(pask_cache* ref, pask_cache* intervened, int32_t layer, int32_t batch, const void* q_dev,
                         const uint8_t* in_s_dev, float softmax_scale, int32_t max_ctx_hint, void* ws_dev,
                         size_t ws_bytes, float* dist_dev, hipStream_t stream) {
  int st = check_cache(ref);
  if (st != PASK_OK) return st;
  st = check_cache(intervened);
  if (st != PASK_OK) return st;
  const pask_geom& g = ref->geom;
  const pask_geom& h = intervened->geom;
  if (g.n_layers != h.n_layers || g.n_q_heads != h.n_q_heads || g.n_kv_heads != h.n_kv_heads ||
      g.head_dim != h.head_dim || g.recent_window != h.recent_window)
    return PASK_E_SHAPE;
  if (layer < 0 || layer >= g.n_layers) return PASK_E_SHAPE;
  if (batch < 1 || batch > g.max_batch || batch > h.max_batch) return PASK_E_SHAPE;
  if (!q_dev || !aligned(q_dev, 16) || !dist_dev || !aligned(dist_dev, 4)) return PASK_E_ARG;
  if (!isfinite(softmax_scale)) return PASK_E_ARG;
  if (max_ctx_hint < 1) max_ctx_hint = g.max_tokens_per_seq;
  const int splits = splits_for(std::min(max_ctx_hint, g.max_tokens_per_seq), (int64_t)batch * g.n_kv_heads);
  const WsLayout w = ws_layout(&g, batch, splits);
  if (!ws_dev || !aligned(ws_dev, 256)) return PASK_E_ARG;
  if (ws_bytes < 2 * w.total) return PASK_E_CAPACITY;

  pask::AttnArgs a[2];
  pask_cache* caches[2] = {ref, intervened};
  for (int i = 0; i < 2; ++i) {
    uint8_t* base = static_cast<uint8_t*>(ws_dev) + i * w.total;
    a[i].cv = view_of(caches[i]);
    a[i].q = static_cast<const uint16_t*>(q_dev);
    a[i].out = nullptr;
    a[i].lse = nullptr;
    a[i].ws_o = reinterpret_cast<float*>(base + w.o_off);
    a[i].ws_ml = reinterpret_cast<float*>(base + w.ml_off);
    a[i].scale_log2 = (float)((double)softmax_scale * 1.4426950408889634);
    a[i].layer = layer;
    a[i].batch = batch;
    a[i].n_q_heads = g.n_q_heads;
    a[i].splits = splits;
    a[i].tags_new = nullptr;
    a[i].k_new = a[i].v_new = nullptr;
    a[i].ws_seq = reinterpret_cast<int32_t*>(base + w.seq_off);
    a[i].tab = pask::TableColumn{};
  }
  const int launched =
      pask::launch_distortion(a[0], a[1], g.n_q_heads / g.n_kv_heads, in_s_dev, dist_dev, stream) == hipSuccess
          ? PASK_OK
          : PASK_E_HIP;
  const pask_cache* both[2] = {ref, intervened};
  return debug_check("pask_attn_distortion", launched, both, 2, stream);
}

int pask_cache_stats(const pask_policy* policy, const pask_cache* cache, int32_t batch, pask_stats* out,
                     int64_t* per_seq_group_head, hipStream_t stream) {
  int st = check_cache(cache);
  if (st != PASK_OK) return st;
  st = check_policy(policy, cache);
  if (st != PASK_OK) return st;
  if (!out) return PASK_E_ARG;
  const pask_geom& g = cache->geom;
  if (batch < 1 || batch > g.max_batch) return PASK_E_SHAPE;
  pask_cache_layout L;
  layout_of(&g, &L);
  uint32_t status[4];
  std::vector<int32_t> cnt((size_t)batch * g.n_layers * pask::kCounterStride);
  const uint8_t* base = static_cast<const uint8_t*>(cache->base);
  if (hipMemcpyAsync(status, base + L.status_off, sizeof(status), hipMemcpyDeviceToHost, stream) != hipSuccess)
    return PASK_E_HIP;
  if (hipMemcpyAsync(cnt.data(), base + L.counters_off, cnt.size() * 4, hipMemcpyDeviceToHost, stream) !=
      hipSuccess)
    return PASK_E_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return PASK_E_HIP;

  const int64_t mH = (int64_t)(2 * g.n_kv_heads * g.head_dim * 2);
  const int64_t mL = (int64_t)(2 * g.n_kv_heads * (g.head_dim / 2 + 2 * (g.head_dim / PASK_QGROUP)));
  pask_stats s;
  memset(&s, 0, sizeof(s));
  const int C = (int)policy->n_groups;
  if (per_seq_group_head)
    memset(per_seq_group_head, 0, sizeof(int64_t) * (size_t)batch * C * g.n_kv_heads * 3);
  for (int b = 0; b < batch; ++b)
    for (int l = 0; l < g.n_layers; ++l) {
      const int32_t* c = &cnt[((size_t)b * g.n_layers + l) * pask::kCounterStride];
      s.n_entries += c[pask::kCntPos];
      s.n_window += std::min<int64_t>(c[pask::kCntPos], g.recent_window);
      s.n_high += c[pask::kCntHi];
      s.n_low += c[pask::kCntLo];
      s.n_drop += c[pask::kCntDrop];
      s.n_forced_high += c[pask::kCntForced];
      s.n_lost += c[pask::kCntLost];
      if (per_seq_group_head) {
        const int grp = policy->group_of_layer[l];
        for (int h = 0; h < g.n_kv_heads; ++h) {
          int64_t* o = per_seq_group_head + (((size_t)b * C + grp) * g.n_kv_heads + h) * 3;
          o[PASK_DROP] += c[pask::kCntDrop];
          o[PASK_RETAIN_LOW] += c[pask::kCntLo];
          o[PASK_RETAIN_HIGH] += c[pask::kCntHi];
        }
      }
    }
  s.bytes_high = s.n_high * mH;
  s.bytes_low = s.n_low * mL;
  {
    pask_cache_layout L2;
    layout_of(&g, &L2);
    s.hi_pages_used = std::min<int64_t>(status[2], (int64_t)L2.ring_pages + g.hi_pages) - L2.ring_pages;
  }
  s.lo_pages_used = std::min<int64_t>(status[3], g.lo_pages);
  const int64_t gov_high = s.n_high - s.n_forced_high;
  const int64_t gov = gov_high + s.n_low + s.n_drop;
  s.c_kv_governed = gov > 0 ? (double)(gov_high * mH + s.n_low * mL) / (double)(gov * mH) : NAN;
  const int64_t all = s.n_high + s.n_low + s.n_drop;
  s.c_kv_all = all > 0 ? (double)(s.bytes_high + s.bytes_low) / (double)(all * mH) : NAN;
  s.device_flags = status[0];
  *out = s;
  return status[0] ? PASK_E_DEVICE_FLAG : PASK_OK;
}

}  // extern "C"
