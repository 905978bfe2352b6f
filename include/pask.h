/*
 * pask.h - C ABI of the PASK decode hot path on MI355X (gfx950).
 *
 * PASK (parser-aware structural KV persistence) gives every generated token a
 * structural tag z_t from the accepted parser transition (Section 3.2, Eq. 3).
 * The pair (z_t, layer group c) indexes a frozen table Lambda that stores, per
 * bucket, a selected action a0, a protection floor a- and adjacent upgrade
 * scores (Section 3.3, end of the offline calibration).  Online, the action
 * is max(a0, a-) under the order DROP < RETAIN-LOW < RETAIN-HIGH (Eq. 10; the
 * lookup and max steps of Alg. 2), and the token's KV in that group's layers
 * is persisted accordingly (the Persist step of Alg. 2): DROP releases it from
 * future attention, RETAIN-LOW keeps it at low precision, RETAIN-HIGH keeps it
 * at full precision (Section 3.1).  Decode attention then reads only the
 * persisted history.  The normalised KV cost C_KV is that of Eq. 1.  Given
 * the parser state of each token, the online controller of Alg. 2 adjusts
 * those actions to a running byte budget with a per-state reserve (Eq. 9-10).
 *
 * Formats chosen here where the paper is silent:
 *   RETAIN-HIGH  bf16 K and V.
 *   RETAIN-LOW   int4, symmetric: per 32 consecutive head_dim elements of one
 *                (token, layer, KV head, K or V) vector, s = RNE_fp16(absmax/7)
 *                saturated at 65504; code q_i = clamp(RNE(x_i / s), -7, 7),
 *                all 0 when s == 0; dequantised value q_i * s.  Stored form:
 *                each code as the offset-binary nibble q_i + 8 (1..15), in the
 *                attention kernel's operand order (pask_cache_layout,
 *                lo_page_bytes), with the fp16 scales beside the codes; the
 *                stored nibble n dequantises as (n - 8) * s.
 *   Protected recent window (Section 3.1): the last W positions of every
 *                (sequence, layer) stay visible at bf16 whatever their action;
 *                a token's action (decided, and charged by the controller,
 *                when it is appended) takes effect when it leaves the window.
 *                W = 0: actions take effect at once.
 *
 * Conventions for every entry point:
 *   - Return an int status: PASK_OK (0) or a negative PASK_E_* code.  No
 *     exception crosses the ABI.
 *   - Host-side validation happens before any HIP call; a call that fails it
 *     returns an error and touches neither the cache nor the stream.
 *   - Device pointers are HIP device memory owned by the caller; the library
 *     never allocates or frees device memory and keeps no pointer after a call
 *     returns.  Its only device memory of its own is the static scratch array
 *     of pask_decode_attn_noalloc (PASK_NOALLOC_SCRATCH_BYTES per GPU).  Work is enqueued on the caller's stream and is asynchronous
 *     except where stated (pask_cache_stats synchronises its stream).
 *   - Calls on one cache must be ordered on one stream (append before the
 *     attention that must see it).  Distinct caches may run concurrently.
 *   - Device-side anomalies do not fail a launch: they set sticky bits in the
 *     cache's status word (PASK_FLAG_*), reported by pask_cache_stats.
 *   - Debug mode: with the environment variable PASK_DEBUG set to anything
 *     but "" or "0" when the library is first used, every entry point that
 *     launches kernels waits for its stream before returning, returns
 *     PASK_E_HIP if a launch or a kernel failed, and writes to stderr the
 *     entry point with the HIP error, or with the cache's status flags when
 *     they differ from the last ones written.  Return codes are otherwise
 *     unchanged (flags are still reported by pask_cache_stats), and calls on
 *     a stream being captured into a graph are not checked.
 */
#ifndef PASK_H
#define PASK_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
enum {
  PASK_OK = 0,
  PASK_E_ARG = -1,          /* null pointer, misaligned pointer, bad scalar  */
  PASK_E_POLICY = -2,       /* malformed or inconsistent policy blob         */
  PASK_E_SHAPE = -3,        /* geometry / shape not supported or mismatched  */
  PASK_E_CAPACITY = -4,     /* buffer smaller than required                  */
  PASK_E_HIP = -5,          /* a HIP runtime call or launch failed           */
  PASK_E_DEVICE_FLAG = -6,  /* stats read fine, device status word non-zero  */
  PASK_E_UNSUPPORTED = -7   /* valid per the paper, not supported here       */
};

/* ---- actions, ordered R < L < H (Section 3.1) --------------------------- */
enum { PASK_DROP = 0, PASK_RETAIN_LOW = 1, PASK_RETAIN_HIGH = 2 };

/* ---- device status-word bits (sticky until pask_cache_reset) ----------- */
enum {
  PASK_FLAG_BAD_TAG = 1u << 0,          /* tag >= n_tags: token kept HIGH      */
  PASK_FLAG_HI_POOL_EXHAUSTED = 1u << 1,/* no HIGH page: token not stored      */
  PASK_FLAG_LO_POOL_EXHAUSTED = 1u << 2,/* no LOW page: token not stored       */
  PASK_FLAG_SEQ_CAPACITY = 1u << 3,     /* position >= max_tokens_per_seq      */
  PASK_FLAG_BAD_COUNT = 1u << 4,        /* n_new[b] outside [0, max_new]       */
  PASK_FLAG_BAD_STATE = 1u << 5,        /* parser state >= n_states: decided
                                           with Gamma = 0, not critical        */
  PASK_FLAG_NO_BUDGET = 1u << 6,        /* states given but no pask_budget_init
                                           since the last init / reset: token
                                           decided by Eq. 10 alone             */
  PASK_FLAG_WORKSPACE = 1u << 7         /* internal: an attention piece fell
                                           outside the workspace's partials
                                           (never expected); not written, the
                                           call's outputs are undefined        */
};

/* ---- append flags -------------------------------------------------------- */
enum {
  /* Every appended token is RETAIN-HIGH regardless of its tag (prompt KV that
   * the table does not govern).  Counted as "forced". */
  PASK_APPEND_KEEP_ALL = 1u << 0
};

#define PASK_MAX_TAGS 64
#define PASK_MAX_GROUPS 16
#define PASK_MAX_LAYERS 128
#define PASK_PAGE_TOKENS 16
#define PASK_QGROUP 32
#define PASK_MAX_STATES 64
/* Bytes of the library-owned device scratch of pask_decode_attn_noalloc. */
#define PASK_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/* Cache geometry.  Supported: head_dim 64 or 128; n_kv_heads 1..8;
 * n_q_heads / n_kv_heads in {1, 2, 4, 8}; page_tokens 16. */
typedef struct pask_geom {
  int32_t max_batch;           /* sequences the cache holds                      */
  int32_t n_layers;            /* layers the cache holds (== policy n_layers)    */
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t page_tokens;         /* 16                                             */
  int32_t max_tokens_per_seq;  /* positions per (sequence, layer)                */
  int32_t hi_pages;            /* pages in the RETAIN-HIGH pool (all layers)     */
  int32_t lo_pages;            /* pages in the RETAIN-LOW pool (all layers)      */
  int32_t recent_window;       /* W, 0..max_tokens_per_seq (== the policy's W)   */
} pask_geom;

/* The frozen table Lambda after parsing (caller-owned plain data). */
typedef struct pask_policy {
  uint32_t n_tags, n_groups, n_layers, n_sink, recent_window;
  uint8_t group_of_layer[PASK_MAX_LAYERS];
  uint8_t action[PASK_MAX_TAGS][PASK_MAX_GROUPS];   /* selected action a0     */
  uint8_t floor_[PASK_MAX_TAGS][PASK_MAX_GROUPS];   /* protection floor a-    */
  float rho_up[PASK_MAX_TAGS][PASK_MAX_GROUPS][2];  /* Eq. 7: R->L, L->H      */
  uint64_t entry_bytes[3];  /* m(a) per (token, layer): DROP, LOW, HIGH       */
  /* Online budget controller (Alg. 2; Eq. 9-10); absent when n_states == 0. */
  uint32_t n_states;                    /* parser states the table knows         */
  uint32_t beta_q;                      /* budget fraction beta, in 1/65536      */
  uint32_t reserve_q[PASK_MAX_STATES];  /* Gamma(s), in 1/16 of the bytes of one
                                           token kept HIGH in every layer        */
  uint8_t crit[PASK_MAX_STATES];        /* 1: critical or lookahead-critical     */
} pask_policy;

/* A cache: geometry plus one caller-owned device buffer of
 * pask_cache_bytes(&geom) bytes, 256-byte aligned. */
typedef struct pask_cache {
  pask_geom geom;
  void* base;
  uint64_t bytes;
} pask_cache;

/* Byte offsets of the regions inside a cache buffer (for inspection). */
typedef struct pask_cache_layout {
  uint64_t status_off;       /* u32 status word; u32 HI and LO page cursors at +8, +12 */
  uint64_t counters_off;     /* i32 [max_batch][n_layers][8]: n_hi, n_lo, n_pos,
                                n_drop, n_forced, n_lost, then the remaining
                                budget R (int64, bytes; online controller)       */
  uint64_t block_table_off;  /* i32 [max_batch][n_layers][2][max_pages]: page ids,
                                store 0 = HIGH, 1 = LOW                            */
  uint64_t index_list_off;   /* i32 [max_batch][n_layers][2][max_tokens_per_seq]:
                                position of each slot of each store               */
  uint64_t staging_off;      /* i32 [max_batch][staging_stride]: append plan       */
  uint64_t budget_off;       /* the online controller's tables (pask_budget_init)  */
  uint64_t ring_act_off;     /* u8 [max_batch][n_layers][W]: decided action | forced
                                << 2 of the token in each recent-window slot       */
  uint64_t hi_pool_off;      /* ring_pages + hi_pages pages of hi_page_bytes: the
                                recent windows first (sequence b, layer l owns
                                pages (b*n_layers + l)*ceil(W/16) + k; position p
                                sits in window slot p mod W, i.e. page slot
                                (p mod W) % 16 of its k = (p mod W) / 16), then
                                the RETAIN-HIGH store pages                        */
  uint64_t lo_pool_off;      /* lo_pages pages of lo_page_bytes                    */
  uint64_t total_bytes;
  /* In both pools KV head g of page P sits in head slot h = (g + P) mod
     n_kv_heads; the offsets below are those of head slot h. */
  uint64_t hi_page_bytes;    /* head slot h at h * 64*D: K tile then V tile, 16*D bf16
                                each; K element (t, d), d = 32i + 8q + j, at
                                (i*64 + q*16 + t)*8 + j; V element (t, d),
                                d = 16m + e, at (((m/2)*64 + t/4*16 + e)*2 + m%2)*4
                                + t%4 (the bf16 MFMA operand order)              */
  uint64_t lo_page_bytes;    /* head slot h at h * (16*D + 64*D/32); every code c
                                is stored as the nibble c + 8.  K codes (8*D
                                bytes: element (t, d), d = 32i + 8q + j, is in
                                byte ((q*16 + t)*D/32 + i)*4 + j%4, low nibble for
                                j < 4, high nibble for j >= 4), K scales
                                [16][D/32] fp16, V codes (8*D bytes: byte
                                ((t/4*16 + e)*D/32 + i)*4 + t%4 holds dims 32i + e
                                (low nibble) and 32i + 16 + e (high) of slot t,
                                e < 16), V scales [16][D/32] fp16               */
  int32_t max_pages;         /* ceil(max_tokens_per_seq / 16)                      */
  int32_t counter_stride;    /* 8                                                  */
  int32_t ring_pages;        /* max_batch * n_layers * ceil(W / 16)                */
  int32_t staging_stride;    /* i32 per sequence in the staging region:
                                max_tokens_per_seq + recent_window + 4             */
} pask_cache_layout;

/* Accounting of what a cache holds (Eq. 1).  Entry = one (token, layer). */
typedef struct pask_stats {
  int64_t n_entries;       /* positions appended, summed over sequences, layers */
  int64_t n_high, n_low, n_drop, n_lost;
  int64_t n_forced_high;   /* HIGH entries not governed by the table           */
  int64_t bytes_high, bytes_low;
  int64_t hi_pages_used, lo_pages_used;
  double c_kv_governed;    /* Eq. 1 over table-governed entries                */
  double c_kv_all;         /* stored bytes / bf16 bytes over all entries       */
  uint32_t device_flags;
  uint32_t reserved;
  int64_t n_window;        /* entries inside the recent windows (not persisted) */
} pask_stats;

/* Parse and validate a policy blob (the frozen table of the offline
 * calibration, Section 3.3) against a geometry.
 *
 * Blob, little-endian: "PASK", u16 version (1 or 2), u16 header bytes = 32,
 * u32 n_tags, n_groups, n_layers, n_sink, recent_window, payload bytes;
 * payload: u8 group_of_layer[n_layers], u8 action[n_tags][n_groups],
 * u8 floor[n_tags][n_groups], zero pad to 4, f32 rho_up[n_tags][n_groups][2];
 * version 2 appends the online controller (Alg. 2): u32 n_states (1..64),
 * u32 beta_q, u32 reserve_q[n_states] (the reserve Gamma(s) of Eq. 9, in
 * sixteenths of one token's bytes at HIGH in every layer), u8
 * crit[n_states] (0 or 1), zero pad to 4; then u32 FNV-1a hash of all
 * preceding bytes.  A version-1 table loads with n_states = 0.
 *
 * Errors: PASK_E_ARG (null pointers), PASK_E_POLICY (bad magic, version,
 * sizes, hash, action or floor > 2, group id >= n_groups, rho not finite or
 * negative, n_tags/n_groups/n_layers/n_states out of range, crit > 1),
 * PASK_E_SHAPE (n_layers or recent_window != the geometry's, or the geometry
 * itself invalid).  Host only: no HIP call. */
int pask_policy_load(const void* blob, size_t nbytes, const pask_geom* geom, pask_policy* out);

/* Region offsets of a cache of this geometry.  PASK_E_SHAPE if unsupported. */
int pask_cache_layout_query(const pask_geom* geom, pask_cache_layout* out);

/* Bytes a cache of this geometry needs; 0 if the geometry is unsupported. */
size_t pask_cache_bytes(const pask_geom* geom);

/* Bind a caller-owned device buffer (>= pask_cache_bytes, 256-byte aligned) to
 * a cache and reset it.  Errors: PASK_E_ARG, PASK_E_SHAPE, PASK_E_CAPACITY,
 * PASK_E_HIP. */
int pask_cache_init(pask_cache* cache, const pask_geom* geom, void* base, size_t bytes,
                    hipStream_t stream);

/* Empty every sequence: zero counters (the remaining budgets included), page
 * cursors and the status word, and forget the controller tables (page
 * contents are left as they are). */
int pask_cache_reset(pask_cache* cache, hipStream_t stream);

/* Persist new tokens (the Persist step of Alg. 2) for one layer.
 *
 * For sequence b < batch, the next n_new[b] tokens (n_new_dev may be NULL:
 * every sequence appends max_new) with tags tags_dev[b][0..n_new[b]) and
 * bf16 K, V at k_dev / v_dev [batch][max_new][n_kv_heads][head_dim] get the
 * action max(action[z][c], floor[z][c]) of the layer's group c (Eq. 10);
 * positions below n_sink, tokens of a KEEP_ALL call (tags_dev may be NULL) and
 * tags >= n_tags get RETAIN-HIGH.  Surviving tokens receive the next slots of
 * their store in position order; DROP tokens get none (release, Section 3.1).
 * With a recent window W > 0, a token enters the window at bf16 and is
 * persisted by its action (taken now) when it leaves it; the tokens leaving
 * during this call are persisted in position order.
 *
 * states_dev (nullable; ignored by a KEEP_ALL call): parser states
 * [batch][max_new] of the tokens.  Given, the online controller of Alg. 2
 * decides instead, token after token in position order, from the sequence's
 * remaining budget R in this layer (pask_budget_init): start from the Eq. 10
 * actions of every group; while their bytes exceed B = max(0, R - Gamma(s))
 * (Eq. 10), demote one step the group above its floor whose last upgrade
 * scores lowest (rho, Eq. 7; lower group on ties); in a critical state, then
 * promote one step the group whose next upgrade scores highest (positive
 * score, fits in B; lower group on ties), repeatedly; R drops by the token's
 * bytes over all groups.  Sinks and tags >= n_tags are RETAIN-HIGH in every
 * group and charged.  This layer keeps its group's action; every layer holds
 * its own copy of R.  Tokens past max_tokens_per_seq are neither persisted
 * nor charged.
 *
 * Errors: PASK_E_ARG (null or misaligned pointers, flags), PASK_E_SHAPE
 * (layer, batch or max_new out of range, policy / geometry mismatch),
 * PASK_E_POLICY (states given to a policy without the controller),
 * PASK_E_HIP. */
int pask_kv_append(const pask_policy* policy, pask_cache* cache, int32_t layer, int32_t batch,
                   const int32_t* n_new_dev, int32_t max_new, const uint8_t* tags_dev,
                   const uint8_t* states_dev, const void* k_dev, const void* v_dev, uint32_t flags,
                   hipStream_t stream);

/* Set up the online controller (Alg. 2) of sequences b < batch: copy the
 * policy's controller tables into the cache, and set the remaining budget of
 * every layer of those sequences to
 *   R_0 = floor(beta_q * t_max * sum_c m(H, c) / 65536) bytes,
 * m(a, c) being the bytes one token persists in the layers of group c under
 * action a (Eq. 1's accounting); Gamma(s) = floor(reserve_q[s] *
 * sum_c m(H, c) / 16).  Call after pask_cache_init / pask_cache_reset (both
 * forget the tables) and before appends that pass parser states; the
 * sequences' counters should be empty.  Synchronises `stream`.
 *
 * Errors: PASK_E_ARG (t_max < 0, R_0 >= 2^62), PASK_E_SHAPE, PASK_E_POLICY
 * (policy without the controller), PASK_E_HIP. */
int pask_budget_init(const pask_policy* policy, pask_cache* cache, int32_t batch, int32_t t_max,
                     hipStream_t stream);

/* Workspace bytes pask_decode_attn needs for `batch` sequences when no
 * sequence holds more than max_ctx_hint persisted entries (a larger count is
 * still correct, only less parallel; a hint below 1 or above
 * max_tokens_per_seq counts as max_tokens_per_seq; 0 for an invalid geometry
 * or batch outside 1..max_batch): batch * n_kv_heads * S partial blocks
 * of max(G, 4) * (head_dim + 2) fp32, S = ceil(hint / 128) + 2, or for
 * batch * n_kv_heads <= 64 the larger of that and min(ceil(hint / 16) + 2,
 * 4096 / (batch * n_kv_heads)); plus 32 bytes per sequence. */
size_t pask_workspace_bytes(const pask_geom* geom, int32_t batch, int32_t max_ctx_hint);

/* One decode step of one layer: the Persist step of Alg. 2 for the token just
 * accepted, then the future long-term attention over the persisted history
 * (Section 3.1: a released entry leaves it, a RETAIN-LOW entry stays in it at
 * low precision).  Optionally persist one new token per sequence
 * (when tags_new_dev != NULL: tags [batch], parser states [batch] (nullable),
 * k_new / v_new bf16 [batch][n_kv_heads][head_dim]; the same rules as
 * pask_kv_append), then
 * grouped-query attention of q_dev bf16 [batch][n_q_heads][head_dim] over the
 * persisted history of the layer (HIGH entries as stored, LOW entries
 * dequantised), query head h reading KV head h / (n_q_heads / n_kv_heads):
 *   out[b][h] = sum_j softmax_j(softmax_scale * q . k_j) v_j   (bf16)
 *   lse_dev[b][h] = natural-log sum-exp of the scaled scores (fp32; nullable)
 * The history is the persisted entries plus the recent window (bf16).  A
 * sequence with no visible entry gives out = 0 and lse = -inf.
 * With a new token, at most 256 sequences, no recent window and no parser
 * states, the attention kernels persist the tokens themselves (one launch
 * fewer): the pages the call opens are then granted in sequence order (where
 * a pool runs out, the lower sequences get its last pages), where the
 * one-token append of pask_kv_append grants them in the order its blocks
 * reach the pool.  Decisions, stored entries, counters and flags follow the
 * same rules either way.
 * ws_dev: device workspace of at least pask_workspace_bytes(geom, batch,
 * max_ctx_hint) bytes, 256-byte aligned.
 *
 * Errors: PASK_E_ARG, PASK_E_SHAPE, PASK_E_CAPACITY (workspace too small),
 * PASK_E_POLICY (states given to a policy without the controller), PASK_E_HIP. */
int pask_decode_attn(const pask_policy* policy, pask_cache* cache, int32_t layer, int32_t batch,
                     const void* q_dev, void* out_dev, float* lse_dev,
                     const uint8_t* tags_new_dev, const uint8_t* states_new_dev, const void* k_new_dev,
                     const void* v_new_dev, float softmax_scale, int32_t max_ctx_hint, void* ws_dev, size_t ws_bytes,
                     hipStream_t stream);

/* pask_decode_attn for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same append and attention, with no caller workspace.  The
 * attention partials go to a device array the library owns,
 * PASK_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU, held from the first call on
 * that GPU until the process ends; the call makes no allocation of any kind.
 * Arguments and results are those of pask_decode_attn without ws_dev /
 * ws_bytes.  A (sequence, KV head) is cut into as many pieces as fit in the
 * scratch (at least two): results agree with pask_decode_attn's within the
 * attention tolerance, and are bit-identical when both use the same number of
 * pieces.  Every call on one GPU shares that GPU's scratch and overwrites it:
 * calls that overlap on one GPU (concurrent streams, or several host threads)
 * race and give undefined results; calls ordered on one stream are safe.
 *
 * Errors: those of pask_decode_attn, and PASK_E_CAPACITY when even two pieces
 * per (sequence, KV head) exceed the scratch: batch * n_kv_heads * 2 *
 * (max(G, 4) * (head_dim + 2) * 4) bytes (plus alignment) above
 * PASK_NOALLOC_SCRATCH_BYTES, e.g. batch above 504 at 8 KV heads, G 8,
 * head_dim 128. */
int pask_decode_attn_noalloc(const pask_policy* policy, pask_cache* cache, int32_t layer, int32_t batch,
                             const void* q_dev, void* out_dev, float* lse_dev, const uint8_t* tags_new_dev,
                             const uint8_t* states_new_dev, const void* k_new_dev, const void* v_new_dev,
                             float softmax_scale, int32_t max_ctx_hint, hipStream_t stream);

/* Attention-output distortion of one layer for one decode step (Eq. 4,
 * Section 3.3).  `ref` and `intervened` are two caches of the same geometry
 * holding the same reference trajectories persisted under two tables: the
 * reference run (every bucket RETAIN-HIGH) and a one-bucket intervention
 * (bucket (z, c) given an action a, every other bucket RETAIN-HIGH).  With
 * the same queries q_dev bf16 [batch][n_q_heads][head_dim], the attention of
 * pask_decode_attn over the persisted history of `layer` in both caches, in
 * fp32 before any rounding to bf16, and for every sequence b whose
 * in_s_dev[b] != 0 (u8 [batch], device; NULL selects every sequence):
 *   dist_dev[b] += max over query heads h of sum_d (o_ref[b][h][d] - o_int[b][h][d])^2
 * (fp32 [batch], device, caller-owned: the caller zeroes it once).  Calling it
 * for every layer of group c at every decode step of S(q) (in_s_dev marks the
 * sequences whose bucket has occurred by that step), then dividing the sum
 * over b by the number of flagged (sequence, step) pairs gives D(q, a).
 * ws_dev: at least 2 * pask_workspace_bytes(&ref->geom, batch, max_ctx_hint)
 * bytes, 256-byte aligned (one set of partials per cache).  No entry is
 * appended and neither cache is modified.
 *
 * Errors: PASK_E_ARG (null or misaligned pointers), PASK_E_SHAPE (the
 * geometries differ, layer or batch out of range), PASK_E_CAPACITY
 * (workspace too small), PASK_E_HIP. */
int pask_attn_distortion(pask_cache* ref, pask_cache* intervened, int32_t layer, int32_t batch, const void* q_dev,
                         const uint8_t* in_s_dev, float softmax_scale, int32_t max_ctx_hint, void* ws_dev,
                         size_t ws_bytes, float* dist_dev, hipStream_t stream);

/* Read the cache's counters (synchronises `stream`) and fill `out`: entry
 * counts per action, stored bytes, realised C_KV (Eq. 1) and the device
 * status word.  per_seq_group_head (nullable, host) receives int64
 * [batch][n_groups][n_kv_heads][3] counts of DROP, LOW, HIGH entries summed
 * over the layers of each group (identical across KV heads: the table has no
 * head axis).  Returns PASK_E_DEVICE_FLAG when the status word is non-zero
 * (after filling `out`). */
int pask_cache_stats(const pask_policy* policy, const pask_cache* cache, int32_t batch,
                     pask_stats* out, int64_t* per_seq_group_head, hipStream_t stream);

/* Static text for a status code. */
const char* pask_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* PASK_H */
