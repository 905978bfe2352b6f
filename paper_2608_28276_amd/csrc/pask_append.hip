// gfx950 kernels of the PASK hot path that persist entries.
//
//   reset        zero the status word, page cursors and per-(sequence, layer)
//                counters of a cache.
//   append_plan  per sequence: the action of every new token (table column in
//                LDS, the higher of selected action and floor, Eq. 10),
//                wavefront ballot + mbcnt prefix sums giving each surviving
//                token its slot in the HIGH or LOW store in position order,
//                page allocation, index lists and counters (the Persist step
//                of Alg. 2).  DROP tokens get no slot (release, Section 3.1).
//   append_pack  copy RETAIN-HIGH K/V (bf16) or quantise-and-pack RETAIN-LOW
//                K/V (int4, one fp16 scale per 32 elements) into the pages.
//   append_step  both of the above for one token per sequence (decode).
//   window       the protected recent window (Section 3.1): its plan, step
//                and fill kernels (the bulk pack is append_pack, reading the
//                entries that leave the window from their ring slots), and
//                the online budget controller (Alg. 2) in the plan and step
//                kernels.
#include <hip/hip_runtime.h>

#include <limits.h>
#include <math.h>

#include <type_traits>

#include "pask_device.h"

namespace pask {
namespace {

constexpr int kPackTokens = 16;   // tokens per block of the recent-window fill kernel

// A 16-byte piece of a page a bulk append writes once (read only by later
// attention calls): non-temporal, so the stream does not displace other lines
// (and, with whole lines written, none is read first: the batch-64 prompt
// append's counter traffic fell from 1.076x to 1.012x its algorithmic bytes).
__device__ __forceinline__ void stream_store16(uint8_t* p, const uint4& v) {
  __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4_t*>(p));
}


// ---------------------------------------------------------------------------
// reset
// ---------------------------------------------------------------------------
__global__ void reset_kernel(CacheView cv, size_t n_counters) {
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i0 < 4) cv.status[i0] = i0 == 2 ? (uint32_t)cv.hi_base : 0u;   // HIGH cursor after the windows
  if (i0 == 0) cv.budget->loaded = 0u;
  for (size_t i = i0; i < n_counters; i += (size_t)gridDim.x * blockDim.x) cv.counters[i] = 0;
}

// R_0 into every layer of sequences b < batch.
__global__ void budget_init_kernel(CacheView cv, int32_t batch, int64_t r0) {
  const size_t n = (size_t)batch * cv.n_layers;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    *reinterpret_cast<int64_t*>(cv.counters + i * kCounterStride + kCntBudget) = r0;
}

// ---------------------------------------------------------------------------
// decisions and slotting
// ---------------------------------------------------------------------------

// The online controller for one token (Alg. 2 after the lookup; Eq. 9-10):
// the token's actions in every group start at max(a0, a-) (Eq. 10); while
// their bytes exceed B = max(0, R - Gamma(s)), the group above its floor whose
// last upgrade scores lowest (rho, Eq. 7) steps down, lower group on ties; in
// a critical state, the group whose next upgrade scores highest (positive,
// fits in B) steps up, lower group on ties, until none fits.  A forced token
// (sink, tag outside the table) is HIGH everywhere.  R drops by the token's
// bytes over all groups; the action of group `group` is returned.  Actions
// are kept two bits per group in one word.  `t` may point to LDS or global
// memory.
__device__ int budget_decide(const BudgetTable* t, int tag, int state, bool forced, int group, int64_t& R,
                             uint32_t& flags) {
  const int C = (int)t->n_groups;
  int64_t cost = 0;
  if (forced) {
    for (int c = 0; c < C; ++c) cost += t->m[c][kHigh];
    R -= cost;
    return kHigh;
  }
  int64_t gamma = 0;
  bool crit = false;
  if ((uint32_t)state < t->n_states) {
    gamma = t->gamma[state];
    crit = t->crit[state] != 0;
  } else {
    flags |= PASK_FLAG_BAD_STATE;
  }
  const uint8_t* a0 = t->action[tag];
  const uint8_t* fl = t->floor_[tag];
  const float(*rho)[2] = t->rho_up[tag];
  uint32_t A = 0u;
  for (int c = 0; c < C; ++c) {
    const int ac = a0[c] > fl[c] ? a0[c] : fl[c];
    A |= (uint32_t)ac << (2 * c);
    cost += t->m[c][ac];
  }
  const int64_t B = R - gamma > 0 ? R - gamma : 0;
  while (cost > B) {                                   // demote
    int best = -1;
    float best_rho = 0.0f;
    for (int c = 0; c < C; ++c) {
      const int ac = (int)((A >> (2 * c)) & 3u);
      if (ac > fl[c]) {
        const float r = rho[c][ac - 1];
        if (best < 0 || r < best_rho) {
          best = c;
          best_rho = r;
        }
      }
    }
    if (best < 0) break;
    const int ac = (int)((A >> (2 * best)) & 3u);
    cost -= t->m[best][ac] - t->m[best][ac - 1];
    A -= 1u << (2 * best);
  }
  while (crit) {                                       // promote
    int best = -1;
    float best_rho = 0.0f;
    int64_t best_extra = 0;
    for (int c = 0; c < C; ++c) {
      const int ac = (int)((A >> (2 * c)) & 3u);
      if (ac < kHigh) {
        const float r = rho[c][ac];
        const int64_t extra = t->m[c][ac + 1] - t->m[c][ac];
        if (r > 0.0f && cost + extra <= B && (best < 0 || r > best_rho)) {
          best = c;
          best_rho = r;
          best_extra = extra;
        }
      }
    }
    if (best < 0) break;
    cost += best_extra;
    A += 1u << (2 * best);
  }
  R -= cost;
  return (int)((A >> (2 * group)) & 3u);
}

__device__ __forceinline__ int64_t* budget_of(int32_t* cnt) {
  return reinterpret_cast<int64_t*>(cnt + kCntBudget);
}

// Exclusive count of `pred` over a 256-thread block in thread order: wavefront
// ballot + popcount of the lanes below (mbcnt), plus the per-wave totals.
// Also returns the block total.  Every thread of the block must call it.
__device__ __forceinline__ int block_exclusive_count(bool pred, int* s_wave, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long mask = __ballot(pred);
  const int below = __popcll(mask & ((1ull << lane) - 1ull));
  if (lane == 0) s_wave[wave] = __popcll(mask);
  __syncthreads();
  int base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int cw = s_wave[w];
    base += (w < wave) ? cw : 0;
    total += cw;
  }
  __syncthreads();
  return base + below;
}

__device__ __forceinline__ void load_table(const TableColumn& tab, uint8_t* s_a0, uint8_t* s_amin) {
  if (threadIdx.x < 64) {
    s_a0[threadIdx.x] = tab.a0[threadIdx.x];
    s_amin[threadIdx.x] = tab.amin[threadIdx.x];
  }
}

__device__ __forceinline__ int clamp_n_new(const AppendArgs& a, int b, uint32_t& flags) {
  int n = a.n_new ? a.n_new[b] : a.max_new;
  if (n < 0 || n > a.max_new) {
    flags |= PASK_FLAG_BAD_COUNT;
    n = n < 0 ? 0 : a.max_new;
  }
  return n;
}

// Exclusive counts of N predicates over a block of kWaves waves in thread
// order (a wavefront ballot and the popcount of the lanes below for each, plus
// the per-wave totals in s_wave), and the block totals: two barriers for all
// N.  Every thread of the block must call it.
template <int N, int kWaves>
__device__ __forceinline__ void block_counts(const bool (&pred)[N], int (*s_wave)[kWaves], int (&excl)[N],
                                             int (&total)[N]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int below[N];
#pragma unroll
  for (int k = 0; k < N; ++k) {
    const unsigned long long mask = __ballot(pred[k]);
    below[k] = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) s_wave[k][wave] = __popcll(mask);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < N; ++k) {
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int cw = s_wave[k][w];
      base += (w < wave) ? cw : 0;
      tot += cw;
    }
    excl[k] = base + below[k];
    total[k] = tot;
  }
  __syncthreads();
}

// One block of kPlanThreads threads per sequence walks the call's tokens in
// chunks of kPlanThreads.  kBudget: the tokens carry parser states and the
// online controller decides (one thread walks each chunk's tokens in position
// order, the table in LDS).
constexpr int kPlanThreads = 1024, kPlanWaves = kPlanThreads / 64;
template <bool kBudget>
__global__ __launch_bounds__(kPlanThreads) void append_plan_kernel(AppendArgs a) {
  __shared__ uint8_t s_a0[64], s_amin[64];
  __shared__ int s_wave[4][kPlanWaves];
  __shared__ unsigned s_page_base[2];
  __shared__ int s_granted[2];
  struct Empty {};
  __shared__ std::conditional_t<kBudget, BudgetTable, Empty> s_bud;
  __shared__ uint8_t s_act[kBudget ? kPlanThreads : 1];
  const CacheView& cv = a.cv;
  const int b = blockIdx.x;
  load_table(a.tab, s_a0, s_amin);
  uint32_t flags = 0;
  const int n = clamp_n_new(a, b, flags);
  int32_t* cnt = counters_of(cv, b, a.layer);
  const int pos0 = cnt[kCntPos];
  bool budget = false;
  int64_t R = 0;
  if constexpr (kBudget) {
    const uint4* src = reinterpret_cast<const uint4*>(cv.budget);
    uint4* dst = reinterpret_cast<uint4*>(&s_bud);
    for (int i = threadIdx.x; i < (int)(sizeof(BudgetTable) / 16); i += kPlanThreads) dst[i] = src[i];
    __syncthreads();
    budget = s_bud.loaded == kBudgetLoaded;
    if (!budget && threadIdx.x == 0) flags |= PASK_FLAG_NO_BUDGET;
    if (budget && threadIdx.x == 0) R = *budget_of(cnt);
  }
  int nst[2] = {cnt[kCntHi], cnt[kCntLo]};
  int n_drop = 0, n_forced = 0, n_lost = 0, n_fit = 0;
  int32_t* bt[2] = {block_table_of(cv, b, a.layer, kHi), block_table_of(cv, b, a.layer, kLo)};
  int32_t* il[2] = {index_list_of(cv, b, a.layer, kHi), index_list_of(cv, b, a.layer, kLo)};
  int32_t* stg = cv.staging + (size_t)b * cv.staging_stride;
  if (threadIdx.x == 0) {                          // for the pack kernel: stores and position before the call
    stg[cv.staging_stride - 4] = nst[0];
    stg[cv.staging_stride - 3] = nst[1];
    stg[cv.staging_stride - 2] = pos0;
  }
  const bool keep_all = (a.flags & kKeepAll) != 0u;
  const unsigned pool[2] = {(unsigned)cv.hi_pages, (unsigned)cv.lo_pages};
  __syncthreads();

  // Every chunk's reads of the shared words (s_page_base, s_granted, s_act)
  // come before the first barrier of the next chunk's counts, which every
  // writer of the next chunk passes first: no barrier at the end of a chunk.
  for (int c0 = 0; c0 < n; c0 += kPlanThreads) {
    const int j = c0 + (int)threadIdx.x;
    const bool valid = j < n;
    const int pos = pos0 + j;
    const bool fits = valid && pos < cv.max_tokens;
    if constexpr (kBudget) {
      if (budget && threadIdx.x == 0) {
        const int j1 = min(min(n, c0 + kPlanThreads), cv.max_tokens - pos0);
        const int group = (int)a.tab.group;
        for (int jj = c0; jj < j1; ++jj) {
          const size_t at = (size_t)b * a.max_new + jj;
          const int tag = (int)a.tags[at];
          const bool forced = (uint32_t)(pos0 + jj) < s_bud.n_sink || (uint32_t)tag >= s_bud.n_tags;
          s_act[jj - c0] = (uint8_t)budget_decide(&s_bud, tag, (int)a.states[at], forced, group, R, flags);
        }
      }
      __syncthreads();
    }
    int act = kDrop;
    bool forced = false, bad = false;
    if (fits) {
      const int tag = a.tags ? (int)a.tags[(size_t)b * a.max_new + j] : 0;
      act = decide(s_a0, s_amin, a.tab.n_tags, a.tab.n_sink, keep_all, tag, pos, forced, bad);
      if constexpr (kBudget) {
        if (budget) act = s_act[threadIdx.x];
      }
    }
    if (bad) flags |= PASK_FLAG_BAD_TAG;
    if (valid && !fits) flags |= PASK_FLAG_SEQ_CAPACITY;
    const int st = act == kHigh ? kHi : kLo;
    const bool keep = fits && act != kDrop;
    int rank[2], tot[2], prank[2], np[2];
    block_counts<2, kPlanWaves>({keep && st == kHi, keep && st == kLo}, s_wave, rank, tot);
    const int slot = keep ? nst[st] + rank[st] : 0;
    const bool new_page = keep && (slot % kPage) == 0;
    block_counts<2, kPlanWaves>({new_page && st == kHi, new_page && st == kLo}, s_wave, prank, np);
    if (threadIdx.x == 0) {
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        unsigned base = 0u;
        int granted = 0;
        if (np[x] > 0) {
          base = atomicAdd(&cv.status[2 + x], (unsigned)np[x]);
          granted = base >= pool[x] ? 0 : (int)min((unsigned)np[x], pool[x] - base);
        }
        s_page_base[x] = base;
        s_granted[x] = granted;
      }
    }
    __syncthreads();
    int pages_before[2];
#pragma unroll
    for (int x = 0; x < 2; ++x) pages_before[x] = (nst[x] + kPage - 1) / kPage;
    bool stored = false;
    if (keep) {
      const int pidx = slot / kPage;
      stored = pidx < pages_before[st] + s_granted[st];
      if (stored) {
        if (new_page) bt[st][pidx] = (int)(s_page_base[st] + (unsigned)prank[st]);
        il[st][slot] = pos;
      } else {
        flags |= st == kHi ? PASK_FLAG_HI_POOL_EXHAUSTED : PASK_FLAG_LO_POOL_EXHAUSTED;
      }
    }
    if (valid) stg[j] = stored ? ((st << 30) | slot) : -1;
    int unused[4], c[4];
    block_counts<4, kPlanWaves>({fits && act == kDrop, stored && forced, valid && !stored && !(fits && act == kDrop),
                                 fits},
                                s_wave, unused, c);
#pragma unroll
    for (int x = 0; x < 2; ++x) nst[x] = min(nst[x] + tot[x], (pages_before[x] + s_granted[x]) * kPage);
    n_drop += c[0];
    n_forced += c[1];
    n_lost += c[2];
    n_fit += c[3];
  }
  if (threadIdx.x == 0) {
    cnt[kCntHi] = nst[0];
    cnt[kCntLo] = nst[1];
    cnt[kCntPos] = pos0 + n_fit;
    cnt[kCntDrop] += n_drop;
    cnt[kCntForced] += n_forced;
    cnt[kCntLost] += n_lost;
    if (budget) *budget_of(cnt) = R;
  }
  if (flags) atomicOr(cv.status, flags);
}

// ---------------------------------------------------------------------------
// RETAIN-HIGH copy and RETAIN-LOW quantise-and-pack of one token
// ---------------------------------------------------------------------------

template <int D>
__device__ __forceinline__ void write_hi(const CacheView& cv, int page, int t, const uint16_t* kin,
                                         const uint16_t* vin) {
  using PL = PageLayout<D>;
  uint8_t* pg = cv.hi_pool + (size_t)page * cv.hi_page_bytes;
  const int nk = cv.n_kv_heads * (D / 8);          // 16-byte K chunks of the token
  for (int x = threadIdx.x; x < nk; x += blockDim.x) {
    const int g = x / (D / 8), c = x % (D / 8);      // dims 8c..8c+7 = 32i + 8q + 0..7
    const int i = c / 4, q = c % 4;
    uint8_t* dst = pg + (size_t)((g + page) % cv.n_kv_heads) * PL::kHiHead + (i * 64 + q * 16 + t) * 16;
    *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(kin + g * D + c * 8);
  }
  const int nv = cv.n_kv_heads * D;
  const int qq = t / 4, jj = t % 4;
  for (int x = threadIdx.x; x < nv; x += blockDim.x) {
    const int g = x / D, d = x % D;
    const int m = d / 16, dd = d % 16;
    uint16_t* dst = reinterpret_cast<uint16_t*>(pg + (size_t)((g + page) % cv.n_kv_heads) * PL::kHiHead + PL::kHiV);
    dst[(((m >> 1) * 64 + qq * 16 + dd) * 2 + (m & 1)) * 4 + jj] = vin[g * D + d];
  }
}

template <int D>
__device__ __forceinline__ void write_lo(const CacheView& cv, int page, int t, const uint16_t* kin,
                                         const uint16_t* vin) {
  using PL = PageLayout<D>;
  const int n_tasks = cv.n_kv_heads * 2 * PL::NG * 8;               // 8 lanes per 32-element group
  uint8_t* pg = cv.lo_pool + (size_t)page * cv.lo_page_bytes;
  const int qq = t / 4, jj = t % 4;
  for (int base = 0; base < n_tasks; base += blockDim.x) {
    const int task = base + (int)threadIdx.x;
    if (task < n_tasks) {  // whole 8-lane groups are active together
      const int gi = task >> 3, lig = task & 7;
      const int i = gi % PL::NG, row = gi / PL::NG, g = row >> 1, kv = row & 1;
      const uint16_t* src = (kv ? vin : kin) + g * D + i * kQGroup + lig * 4;   // dims 32i + 4lig + e
      const uint2 raw = *reinterpret_cast<const uint2*>(src);
      uint32_t packed, sbits;
      quant4(raw.x, raw.y, packed, sbits);
      uint8_t* hb = pg + (size_t)((g + page) % cv.n_kv_heads) * PL::kLoHead;
      if (kv == 0) {
        // Element j = 4*half + e of the lane pair's 8 goes to byte e, nibble `half`.
        const int q = lig / 2, half = lig % 2;
        const uint32_t mine = nibbles_to_bytes(packed) << (4 * half);
        const uint32_t word = mine | __shfl_xor(mine, 1, 8);
        if (half == 0) *reinterpret_cast<uint32_t*>(hb + ((q * 16 + t) * PL::NG + i) * 4) = word;
        if (lig == 0) *reinterpret_cast<uint16_t*>(hb + PL::kLoKS + (t * PL::NG + i) * 2) = (uint16_t)sbits;
      } else {
        const uint32_t partner = __shfl_xor(packed, 4, 8);           // dims 16 higher
        if (lig < 4) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int dd = 4 * lig + e;
            const uint32_t b = ((packed >> (4 * e)) & 0xFu) | (((partner >> (4 * e)) & 0xFu) << 4);
            hb[PL::kLoVC + ((qq * 16 + dd) * (PL::NM / 2) + i) * 4 + jj] = (uint8_t)b;
          }
        }
        if (lig == 0) *reinterpret_cast<uint16_t*>(hb + PL::kLoVS + (t * PL::NG + i) * 2) = (uint16_t)sbits;
      }
    }
  }
}

// Bulk persist by destination page, after the plan kernel has slotted the
// call's tokens: block (k, store, b) fills page k of the pages of sequence b's
// store that this call's slots reach (slots n0..n1-1 of the store, n0 saved by
// the plan kernel, n1 the store's count after it).  Each slot's source token
// comes from the index list: row position - p0 of the call's input, or, with a
// recent window, for an entry from before the call that leaves the window
// now, its ring slot (position mod W).  So every page is written whole
// by one block, in the operand order of the attention kernel, with 16-byte
// stores of consecutive addresses (1 KiB per wave and instruction).
//   1. Every thread issues its loads at once (non-temporal: read once): the
//      page's V rows (16 slots x Hkv x D bf16) in row order, and its K chunks
//      (HIGH: one 16-byte chunk per page-order chunk; LOW: per KV head, the
//      four 8-element chunks of a 32-element group of a slot, one lane each).
//   2. V rows go to LDS ([slot][Hkv][D], rows padded by 16 bytes).
//   3. HIGH: K chunks are stored as loaded; V chunks (4 slots x 2 dims x 8
//      elements each) are gathered from LDS.  LOW: K groups are quantised in
//      registers (absmax over the group's 4 lanes); V groups are gathered from
//      LDS by 16 lanes (dims 32i + e and 32i + 16 + e) and quantised.
// Slots of the page before n0 hold earlier entries and are left as they are
// (a V piece that mixes them with new slots is written element by element);
// slots from n1 on are not yet in use and may be written.
constexpr int kPackThreads = 256;


// The offset-binary codes q + 8 of the 8 bf16 elements of x under scale s
// (inv ~ 1 / s), the rule of quant_code, with code u in the low byte of b[u]
// (bits 4..7 zero, the bits above unspecified).  y = RN(x * inv + 1.5 * 2^23
// + 8) lies in [2^23, 2^24), where floats are spaced by 1, so its low byte is
// rint(x * inv) + 8; r = x * inv - (y - M) is the part rounded away.  As in
// codes8, x * inv rounds like x / s unless x / s lies within 2^-12 of a
// half-integer, so a lane whose largest |r| comes within 1.2e-4 of 1/2 takes
// quant_code for its 8 elements.  plain: s is a normal, unsaturated fp16
// scale of the group's absmax (quant_scale_bf16), so |x / s| <= 7 (1 + 2^-11)
// for every element of the group and the code needs no clamp; a lane without
// it (s subnormal or zero, or saturated at 65504) takes quant_code too.  About
// half the vector instructions of codes8 + k_word, which the bulk pack of
// RETAIN-LOW pages, bound by its vector ALU, spends most of its time on.
__device__ __forceinline__ void code_bytes8(const uint4& x, float s, float inv, bool plain, uint32_t (&b)[8]) {
  const float f[8] = {bf16_lo(x.x), bf16_hi(x.x), bf16_lo(x.y), bf16_hi(x.y),
                      bf16_lo(x.z), bf16_hi(x.z), bf16_lo(x.w), bf16_hi(x.w)};
  constexpr float M = 12582920.0f;                 // 1.5 * 2^23 + 8
  float worst = 0.0f;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const float y = fmaf(f[u], inv, M);
    worst = fmaxf(worst, fabsf(fmaf(f[u], inv, M - y)));
    b[u] = __float_as_uint(y);
  }
  const bool exact = !plain || worst > 0.49988f;
  if (__ballot(exact)) {
    if (exact) {
#pragma unroll
      for (int u = 0; u < 8; ++u) b[u] = (uint32_t)(quant_code(f[u], s, inv) + 8);
    }
  }
}
// Low bytes of w0..w3 as bytes 0..3 of one word.
__device__ __forceinline__ uint32_t low_bytes4(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  return __builtin_amdgcn_perm(w1, w0, 0x0c0c0400u) | __builtin_amdgcn_perm(w3, w2, 0x04000c0cu);
}

// The largest |element| of the 8 bf16 in x, as the bits of its bf16 magnitude
// (the order of non-negative floats is that of their bits): packed 16-bit
// integer maxima of the sign-cleared words.
typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t abs_max_bits8(const uint4& x) {
  const uint32_t m = 0x7FFF7FFFu;
  const u16x2_t a = __builtin_bit_cast(u16x2_t, x.x & m), b = __builtin_bit_cast(u16x2_t, x.y & m);
  const u16x2_t c = __builtin_bit_cast(u16x2_t, x.z & m), d = __builtin_bit_cast(u16x2_t, x.w & m);
  const u16x2_t r = __builtin_elementwise_max(__builtin_elementwise_max(a, b), __builtin_elementwise_max(c, d));
  return r.x > r.y ? (uint32_t)r.x : (uint32_t)r.y;
}

// quant_scale of a bf16 absmax, dividing only where s is an fp16 subnormal:
// from 7 * 2^-14 up, the product with RN(1/7) rounds to the same fp16 as the
// correctly rounded quotient (an exact quotient of a bf16 by 7 has at most 8
// significant bits, an inexact one never comes within 2^-15 of an fp16
// midpoint); below it an exact quotient can be a midpoint between fp16
// subnormals, which the product may miss.  Equal to quant_scale for every
// bf16 absmax (checked over all of them on the CPU).  plain: s is a normal
// fp16 and not saturated (7 * 2^-14 <= absmax <= 7 * 65504).
__device__ __forceinline__ uint16_t quant_scale_bf16(float absmax, float& s, float& inv, bool& plain) {
  float q = absmax * (1.0f / 7.0f);
  const bool small = absmax < 7.0f * 0x1p-14f;
  if (__ballot(small)) {
    if (small) {
      float a = absmax;
      asm volatile("" : "+v"(a));                  // no code: keeps the division on this rare branch
      q = a / 7.0f;
    }
  }
  plain = !small && absmax <= 7.0f * 65504.0f;
  const _Float16 h = (_Float16)fminf(q, 65504.0f);
  s = (float)h;
  inv = __builtin_amdgcn_rcpf(s);
  return __builtin_bit_cast(uint16_t, h);
}

// Lane l's 32-bit value from lane l ^ 1 / l ^ 2 of its group of four (quad
// DPP: a vector move, no LDS round trip).
__device__ __forceinline__ uint32_t quad_xor1(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, true);   // quad_perm [1, 0, 3, 2]
}
__device__ __forceinline__ uint32_t quad_xor2(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, true);   // quad_perm [2, 3, 0, 1]
}

// Row t and column col (of H * D / 8) of the page's 16-byte input chunks
// e = it * kPackThreads + tid, it = 0, 1, ...: one division per thread, then
// carried from one it to the next.
struct ChunkWalk {
  int t, col, R, dt, dc;
  __device__ __forceinline__ explicit ChunkWalk(int r) : R(r) {
    t = (int)threadIdx.x / R;
    col = (int)threadIdx.x - t * R;
    dt = kPackThreads / R;
    dc = kPackThreads - dt * R;
  }
  __device__ __forceinline__ void next() {
    t += dt;
    col += dc;
    if (col >= R) {
      col -= R;
      ++t;
    }
  }
};

// The LDS image of a LOW page keeps each 16-byte piece of a head's K and V
// code regions at its stored index XOR a key of (image head g, quarter q of
// the 32-element group the piece's codes come from).  In stored order the
// lanes of one store instruction (4 heads x 4 quarters x 4 groups for K, 4 x
// 2 x 4 for V, one slot) fall in 4 / 8 of the 32 LDS banks; with the keys the
// K words spread over all 32 (two lanes a bank) and the V bytes over 32.  The
// XOR keeps q (and the slot quad of V) in place, so the copy-out finds each
// piece from its stored index.
template <int D>
struct LowImage {
  using PL = PageLayout<D>;
  static constexpr int NG = PL::NG;
  static constexpr int kKMask = (4 * NG < 8 ? 4 * NG : 8) - 1;   // K pieces per quarter: 4 NG
  static constexpr int kVMask = (2 * NG < 8 ? 2 * NG : 8) - 1;   // V pieces per quarter of a slot quad: 2 NG
  __device__ __forceinline__ static int k_key(int g, int q) { return (g * 4 + q) & kKMask; }
  __device__ __forceinline__ static int v_key(int g, int q) { return (g * 2 + q) & kVMask; }
  // Image index of stored 16-byte piece p of image head g.
  __device__ __forceinline__ static int piece(int g, int p) {
    if (p < PL::kLoKS / 16) return p ^ k_key(g, p / (4 * NG));
    if (p >= PL::kLoVC / 16 && p < PL::kLoVS / 16) {
      const int r = p - PL::kLoVC / 16;
      return PL::kLoVC / 16 + (r ^ v_key(g, (r % (4 * NG)) / (2 * NG)));
    }
    return p;
  }
};

// The page image of a LOW page from the call's K and V rows (kx, vx: 16-byte
// chunks in row order, chunk e of the page's rows at e = it * threads + tid,
// so the four chunks of a 32-element group sit in four adjacent lanes):
// every lane quantises its 8 elements (the group's absmax over the 4 lanes),
// the codes and scales go to the LDS image of the page (LowImage), which is
// then copied out in stored order with 16-byte stores (whole pages), or byte
// by byte for the new slots only when the page holds earlier slots.
template <int D, int kIt>
__device__ __forceinline__ void low_page(const AppendArgs& a, const CacheView& cv, int page, int tl0, int th0,
                                         const uint4 (&kx)[kIt], const uint4 (&vx)[kIt], int n_chunks,
                                         uint8_t* s_img) {
  using PL = PageLayout<D>;
  using Img = LowImage<D>;
  constexpr int NG = PL::NG, kRowChunks = D / 8;
  const int H = cv.n_kv_heads, tid = (int)threadIdx.x;
  ChunkWalk w(H * kRowChunks);
#pragma unroll
  for (int it = 0; it < kIt; ++it, w.next()) {
    const int e = it * kPackThreads + tid;
    const bool valid = e < n_chunks;
    const uint32_t t = (uint32_t)w.t, col = (uint32_t)w.col;
    const uint32_t g = col / kRowChunks, c = col % kRowChunks, i = c / 4, q = c % 4;
    uint8_t* hd = s_img + g * PL::kLoHead;
#pragma unroll
    for (int kv = 0; kv < 2; ++kv) {
      const uint4 x = kv ? vx[it] : kx[it];
      uint32_t mb = abs_max_bits8(x);
      mb = max(mb, quad_xor1(mb));                 // the group's four lanes
      mb = max(mb, quad_xor2(mb));
      float s, inv;
      bool plain;
      const uint16_t sbits = quant_scale_bf16(__uint_as_float(mb << 16), s, inv, plain);
      uint32_t cb[8];
      code_bytes8(x, s, inv, plain, cb);
      if (kv == 0) {
        if (valid) {
          // byte e: element e in the low nibble, element 4 + e in the high one
          const uint32_t o = ((q * 16u + t) * NG + i) * 4u;
          *reinterpret_cast<uint32_t*>(hd + (((o >> 4) ^ (uint32_t)Img::k_key(g, q)) << 4) + (o & 15u)) =
              low_bytes4((cb[4] << 4) | cb[0], (cb[5] << 4) | cb[1], (cb[6] << 4) | cb[2], (cb[7] << 4) | cb[3]);
          if (q == 0) *reinterpret_cast<uint16_t*>(hd + PL::kLoKS + (t * NG + i) * 2u) = sbits;
        }
      } else {
        // lanes q and q ^ 2 hold dims 32i + dd and 32i + 16 + dd: one byte per dd
        const uint32_t lo = low_bytes4(cb[0], cb[1], cb[2], cb[3]), hi = low_bytes4(cb[4], cb[5], cb[6], cb[7]);
        const uint32_t blo = lo | (quad_xor2(lo) << 4), bhi = hi | (quad_xor2(hi) << 4);
        if (valid && q < 2) {
          const uint32_t key = (uint32_t)Img::v_key(g, q);
          if constexpr (NG == 4) {
            // byte dd = 8q + u sits in piece (t / 4) * 16 + 8q + (u ^ key).  The
            // image is 128-byte aligned and every other term of the offset is a
            // multiple of 128 or below 16, so bits 4..6 of vo are the key and
            // piece 8q + (u ^ key) is at vo ^ (u << 4).
            static_assert(PL::kLoHead % 128 == 0 && PL::kLoVC % 128 == 0, "V offsets of the LOW image");
            const uint32_t vo = g * PL::kLoHead + PL::kLoVC + ((t / 4u) * 16u + 8u * q) * 16u + 4u * i + t % 4u +
                                key * 16u;
#pragma unroll
            for (int u = 0; u < 8; ++u) s_img[vo ^ (uint32_t)(u << 4)] = (uint8_t)((u < 4 ? blo : bhi) >> (8 * (u % 4)));
          } else {
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const uint32_t b = ((t / 4u) * 16u * NG + i) * 4u + t % 4u + (8u * q + u) * NG * 4u;
              hd[PL::kLoVC + (((b >> 4) ^ key) << 4) + (b & 15u)] = (uint8_t)((u < 4 ? blo : bhi) >> (8 * (u % 4)));
            }
          }
        }
        if (valid && q == 0) *reinterpret_cast<uint16_t*>(hd + PL::kLoVS + (t * NG + i) * 2u) = sbits;
      }
    }
  }
  __syncthreads();
  uint8_t* pg = cv.lo_pool + (size_t)page * cv.lo_page_bytes;
  constexpr int kHeadChunks = PL::kLoHead / 16;
  const int pm = page % H;                         // image head g is stored at (g + page) % H
  if (tl0 == 0) {                                  // no earlier slot: whole 16-byte pieces
    for (int k = tid; k < H * kHeadChunks; k += kPackThreads) {
      const int g = k / kHeadChunks, off = k % kHeadChunks;
      const int hg = g + pm < H ? g + pm : g + pm - H;
      stream_store16(pg + (size_t)hg * PL::kLoHead + off * 16,
                     *reinterpret_cast<const uint4*>(s_img + g * PL::kLoHead + Img::piece(g, off) * 16));
    }
    return;
  }
  for (int x = tid; x < H * PL::kLoHead; x += kPackThreads) {   // the new slots' bytes only
    const int g = x / PL::kLoHead, y = x % PL::kLoHead;
    int t;
    if (y < PL::kLoKS) t = (y / 4 / NG) % 16;                             // K word (q*16 + t)*NG + i
    else if (y < PL::kLoVC) t = (y - PL::kLoKS) / 2 / NG;                 // K scale t*NG + i
    else if (y < PL::kLoVS) t = ((y - PL::kLoVC) / 4 / NG / 16) * 4 + (y - PL::kLoVC) % 4;   // V byte
    else t = (y - PL::kLoVS) / 2 / NG;                                    // V scale
    const int hg = g + pm < H ? g + pm : g + pm - H;
    if (t >= tl0 && t < th0)
      pg[(size_t)hg * PL::kLoHead + y] = s_img[g * PL::kLoHead + Img::piece(g, y >> 4) * 16 + (y & 15)];
  }
}
// A window entry that leaves the recent window in a bulk append: its bf16 K
// and V sit in its window slot ws = pos mod W, slot ws % 16 of a HIGH-layout
// page of the (sequence, layer)'s window ring.  ring_head: KV head g of that
// page; ring_k_chunk / ring_v_chunk: the 16-byte chunk c (dims 8c .. 8c + 7)
// of slot t, as a row of the call's input holds it.
template <int D>
__device__ __forceinline__ const uint8_t* ring_head(const CacheView& cv, int b, int layer, int ws, int g) {
  const int page = (b * cv.n_layers + layer) * cv.ring_pp + ws / kPage;
  return cv.hi_pool + (size_t)page * cv.hi_page_bytes + (size_t)((g + page) % cv.n_kv_heads) * PageLayout<D>::kHiHead;
}
__device__ __forceinline__ uint4 ring_k_chunk(const uint8_t* head, int t, int c) {   // d = 32i + 8q + j, c = 4i + q
  return *reinterpret_cast<const uint4*>(head + ((c / 4) * 64 + (c % 4) * 16 + t) * 16);
}
template <int D>
__device__ __forceinline__ uint4 ring_v_chunk(const uint8_t* head, int t, int c) {
  const uint16_t* v = reinterpret_cast<const uint16_t*>(head + PageLayout<D>::kHiV);
  auto at = [&](int d) -> uint32_t {             // element (t, d = 16m + e) of the V tile
    const int m = d / 16, e = d % 16;
    return v[(((m >> 1) * 64 + (t / 4) * 16 + e) * 2 + (m & 1)) * 4 + t % 4];
  };
  uint32_t w[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) w[u] = at(8 * c + 2 * u) | (at(8 * c + 2 * u + 1) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

constexpr int kLdsRowPad = 16;                     // bytes after each staged V row (bank spread)

template <int D>
__global__ __launch_bounds__(kPackThreads) void append_pack_page_kernel(AppendArgs a) {
  using PL = PageLayout<D>;
  constexpr int NG = PL::NG;
  constexpr int kRowChunks = D / 8;                // 16-byte chunks per head row
  constexpr int kMaxChunks = kPage * 8 * kRowChunks;   // a page's K (or V) chunks at Hkv 8
  constexpr int kIt = kMaxChunks / kPackThreads;
  constexpr int kLdsRow = 8 * D * 2 + kLdsRowPad;
  __shared__ __align__(128) uint8_t s_v[kPage * kLdsRow];   // 128: the LOW image's V offsets (low_page)
  __shared__ int s_src[kPage];                     // per slot: input row, -2 - ring slot, or -1 (no new entry)
  const CacheView& cv = a.cv;
  const int b = blockIdx.z, st = blockIdx.y;
  const int H = cv.n_kv_heads;
  const int32_t* stg = cv.staging + (size_t)b * cv.staging_stride;
  const int n0 = stg[cv.staging_stride - 4 + st];
  const int p0 = stg[cv.staging_stride - 2];
  const int n1 = counters_of(cv, b, a.layer)[st];
  const int pidx = n0 / kPage + (int)blockIdx.x;
  const int tl0 = max(n0 - pidx * kPage, 0);       // first new slot of the page
  const int th0 = min(n1 - pidx * kPage, kPage);   // past the last new slot
  if (tl0 >= th0) return;                          // block-uniform: no new slot here
  const int page = block_table_of(cv, b, a.layer, st)[pidx];
  if (threadIdx.x < kPage) {
    const int t = (int)threadIdx.x;
    int j = -1;
    if (t >= tl0 && t < th0) {
      const int pos = index_list_of(cv, b, a.layer, st)[pidx * kPage + t];
      const int r = pos - p0;
      if (r >= 0 && r < a.max_new) j = r;          // row r of the call's input
      else if (r < 0 && r >= -cv.window) j = -2 - pos % cv.window;   // leaving the window: its ring slot
    }
    s_src[t] = j;
  }
  __syncthreads();
  const int tid = (int)threadIdx.x;
  const size_t row = (size_t)H * D;                // bf16 per K (or V) row of a token
  const int n_chunks = kPage * H * kRowChunks;     // the page's V chunks (as many K chunks)
  const uint16_t* vbase = a.v + (size_t)b * a.max_new * row;
  const uint16_t* kbase = a.k + (size_t)b * a.max_new * row;
  const bool is_hi = st == kHi;
  // 1. loads
  uint4 vx[kIt], kx[kIt];
  ChunkWalk w0(H * kRowChunks);
#pragma unroll
  for (int it = 0; it < kIt; ++it, w0.next()) {
    const int e = it * kPackThreads + tid;
    vx[it] = make_uint4(0u, 0u, 0u, 0u);
    kx[it] = make_uint4(0u, 0u, 0u, 0u);
    if (e < n_chunks) {
      const int t = w0.t, col = w0.col;
      const int j = s_src[t];
      if (j >= 0) vx[it] = stream_load16(reinterpret_cast<const uint8_t*>(vbase + (size_t)j * row + col * 8));
      else if (j <= -2)
        vx[it] = ring_v_chunk<D>(ring_head<D>(cv, b, a.layer, -2 - j, col / kRowChunks), (-2 - j) % kPage,
                                 col % kRowChunks);
    }
  }
  if (is_hi) {
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int e = it * kPackThreads + tid;       // page order: (g, i) = e / 64, q = lane / 16, t = lane % 16
      if (e < n_chunks) {
        const int gi = e >> 6, q = (e >> 4) & 3, t = e & 15;
        const int g = gi / NG, i = gi % NG;
        const int j = s_src[t];
        if (j >= 0)
          kx[it] = stream_load16(reinterpret_cast<const uint8_t*>(kbase + (size_t)j * row + g * D + (4 * i + q) * 8));
        else if (j <= -2)
          kx[it] = ring_k_chunk(ring_head<D>(cv, b, a.layer, -2 - j, g), (-2 - j) % kPage, 4 * i + q);
      }
    }
  } else {
    ChunkWalk w(H * kRowChunks);
#pragma unroll
    for (int it = 0; it < kIt; ++it, w.next()) {   // LOW K: row order, like V
      const int e = it * kPackThreads + tid;
      if (e < n_chunks) {
        const int t = w.t, col = w.col;
        const int j = s_src[t];
        if (j >= 0) kx[it] = stream_load16(reinterpret_cast<const uint8_t*>(kbase + (size_t)j * row + col * 8));
        else if (j <= -2)
          kx[it] = ring_k_chunk(ring_head<D>(cv, b, a.layer, -2 - j, col / kRowChunks), (-2 - j) % kPage,
                                col % kRowChunks);
      }
    }
  }
  if (!is_hi) {
    low_page<D>(a, cv, page, tl0, th0, kx, vx, n_chunks, s_v);
    return;
  }
  // 2. HIGH: V rows into LDS
  ChunkWalk w1(H * kRowChunks);
#pragma unroll
  for (int it = 0; it < kIt; ++it, w1.next()) {
    const int e = it * kPackThreads + tid;
    if (e < n_chunks) {
      const int t = w1.t, col = w1.col;
      *reinterpret_cast<uint4*>(s_v + t * kLdsRow + col * 16) = vx[it];
    }
  }
  __syncthreads();
  auto v_at = [&](int t, int g, int d) -> uint32_t {   // bf16 bits of V[t][g][d]
    return *reinterpret_cast<const uint16_t*>(s_v + t * kLdsRow + (g * D + d) * 2);
  };
  {                                                // HIGH page
    uint8_t* pg = cv.hi_pool + (size_t)page * cv.hi_page_bytes;
    // K chunks as loaded: chunk (g, i, q, t) at (i*64 + q*16 + t) * 16 of head slot (g + page) % H
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int e = it * kPackThreads + tid;
      if (e < n_chunks) {
        const int gi = e >> 6, t = e & 15;
        const int g = gi / NG, i = gi % NG;
        if (s_src[t] != -1)                        // a new entry (input row or ring slot)
          stream_store16(pg + (size_t)((g + page) % H) * PL::kHiHead + (size_t)(i * 64 + (e & 63)) * 16, kx[it]);
      }
    }
    // V chunk o = M*64 + T4*16 + e of a head: elements (slot 4*T4 + r, dim 16*(2M + h) + e), h-major
    constexpr int kPerHead = 2 * D;                // 16-byte chunks of one head's V tile
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int c = it * kPackThreads + tid;
      if (c < n_chunks) {
        const int g = c / kPerHead, o = c % kPerHead;
        const int M = o >> 6, T4 = (o >> 4) & 3, e = o & 15;
        if (4 * T4 + 3 < tl0 || 4 * T4 >= th0) continue;   // no new slot in the group
        uint32_t w[4];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int r2 = 0; r2 < 2; ++r2)
            w[2 * h + r2] = v_at(4 * T4 + 2 * r2, g, 16 * (2 * M + h) + e) |
                            (v_at(4 * T4 + 2 * r2 + 1, g, 16 * (2 * M + h) + e) << 16);
        uint8_t* dst = pg + (size_t)((g + page) % H) * PL::kHiHead + PL::kHiV + (size_t)o * 16;
        if (4 * T4 >= tl0) {
          stream_store16(dst, make_uint4(w[0], w[1], w[2], w[3]));
        } else {                                   // the group holds earlier slots: new ones only
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (4 * T4 + r >= tl0 && 4 * T4 + r < th0)
                reinterpret_cast<uint16_t*>(dst)[4 * h + r] = (uint16_t)(w[2 * h + r / 2] >> (16 * (r % 2)));
        }
      }
    }
  }
}

// One token of sequence b (thread 0 of the block): its action (Eq. 10, or
// the online controller when parser states are given).
__device__ __forceinline__ int decide_one(const AppendArgs& a, const uint8_t* s_a0, const uint8_t* s_amin, int b,
                                          int32_t* cnt, int pos, bool& forced, uint32_t& flags) {
  const CacheView& cv = a.cv;
  const int tag = a.tags ? (int)a.tags[(size_t)b * a.max_new] : 0;
  bool bad;
  int act = decide(s_a0, s_amin, a.tab.n_tags, a.tab.n_sink, (a.flags & kKeepAll) != 0u, tag, pos, forced, bad);
  if (bad) flags |= PASK_FLAG_BAD_TAG;
  if (a.states) {
    if (cv.budget->loaded == kBudgetLoaded) {
      int64_t* r = budget_of(cnt);
      int64_t R = *r;
      act = budget_decide(cv.budget, tag, (int)a.states[(size_t)b * a.max_new], forced, (int)a.tab.group, R, flags);
      *r = R;
    } else {
      flags |= PASK_FLAG_NO_BUDGET;
    }
  }
  return act;
}

// Persist step of one entry at position pos (thread 0): DROP is counted; a
// kept entry takes the next slot of its store (a new page when the slot
// starts one) and its index-list entry.  Returns the store code (store << 30
// | slot) and the page, or -1 when the entry is not stored.
__device__ __forceinline__ int slot_one(const CacheView& cv, int b, int layer, int32_t* cnt, int act, bool forced,
                                        int pos, int& page, uint32_t& flags) {
  if (act == kDrop) {
    cnt[kCntDrop] += 1;
    return -1;
  }
  const int st = act == kHigh ? kHi : kLo;
  const int slot = cnt[st];
  int32_t* bt = block_table_of(cv, b, layer, st);
  if (slot % kPage == 0) {
    const unsigned pid = atomicAdd(&cv.status[2 + st], 1u);
    const unsigned pool = st == kHi ? (unsigned)cv.hi_pages : (unsigned)cv.lo_pages;
    if (pid >= pool) {
      flags |= st == kHi ? PASK_FLAG_HI_POOL_EXHAUSTED : PASK_FLAG_LO_POOL_EXHAUSTED;
      cnt[kCntLost] += 1;
      return -1;
    }
    bt[slot / kPage] = (int)pid;
  }
  page = bt[slot / kPage];
  index_list_of(cv, b, layer, st)[slot] = pos;
  cnt[st] = slot + 1;
  if (forced) cnt[kCntForced] += 1;
  return (st << 30) | slot;
}

// One token per sequence: thread 0 decides and slots it, then the block
// writes it.
template <int D>
__global__ __launch_bounds__(256) void append_step_kernel(AppendArgs a) {
  __shared__ uint8_t s_a0[64], s_amin[64];
  __shared__ int s_code, s_page;
  const CacheView& cv = a.cv;
  const int b = blockIdx.x;
  load_table(a.tab, s_a0, s_amin);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t flags = 0;
    const int n = clamp_n_new(a, b, flags);
    int code = -1, page = -1;
    if (n > 0) {
      int32_t* cnt = counters_of(cv, b, a.layer);
      const int pos = cnt[kCntPos];
      if (pos >= cv.max_tokens) {
        flags |= PASK_FLAG_SEQ_CAPACITY;
        cnt[kCntLost] += 1;
      } else {
        bool forced;
        const int act = decide_one(a, s_a0, s_amin, b, cnt, pos, forced, flags);
        code = slot_one(cv, b, a.layer, cnt, act, forced, pos, page, flags);
        cnt[kCntPos] = pos + 1;
      }
    }
    if (flags) atomicOr(cv.status, flags);
    s_code = code;
    s_page = page;
  }
  __syncthreads();
  const int code = s_code;
  if (code < 0) return;
  const size_t row = (size_t)cv.n_kv_heads * D;
  const uint16_t* kin = a.k + (size_t)b * a.max_new * row;
  const uint16_t* vin = a.v + (size_t)b * a.max_new * row;
  const int slot = code & 0x3FFFFFFF;
  if ((code >> 30) == kHi) write_hi<D>(cv, s_page, slot % kPage, kin, vin);
  else write_lo<D>(cv, s_page, slot % kPage, kin, vin);
}

// ---------------------------------------------------------------------------
// the protected recent window (Section 3.1)
// ---------------------------------------------------------------------------
// With W > 0 a token is decided when it is appended (its action and forced
// flag go to ring_act, the controller charges it then) and enters the window
// of its (sequence, layer): window slot p mod W, held in HIGH page layout in
// pages of the HIGH pool reserved for the windows.  It is persisted by its
// action when position p + W is appended.

__device__ __forceinline__ int ring_page(const CacheView& cv, int b, int layer, int k) {
  return (b * cv.n_layers + layer) * cv.ring_pp + k;
}
__device__ __forceinline__ uint8_t* ring_act_of(const CacheView& cv, int b, int layer) {
  return cv.ring_act + ((size_t)b * cv.n_layers + layer) * cv.window;
}

// The bf16 K and V rows [Hkv][D] of slot t of a HIGH-layout page (the
// inverse of write_hi), into kout / vout, by the whole block.
template <int D>
__device__ __forceinline__ void read_hi_token(const CacheView& cv, int page, int t, uint16_t* kout, uint16_t* vout) {
  using PL = PageLayout<D>;
  const uint8_t* pg = cv.hi_pool + (size_t)page * cv.hi_page_bytes;
  const int nk = cv.n_kv_heads * (D / 8);
  for (int x = threadIdx.x; x < nk; x += blockDim.x) {
    const int g = x / (D / 8), c = x % (D / 8);
    const int i = c / 4, q = c % 4;
    const uint8_t* src = pg + (size_t)((g + page) % cv.n_kv_heads) * PL::kHiHead + (i * 64 + q * 16 + t) * 16;
    *reinterpret_cast<uint4*>(kout + g * D + c * 8) = *reinterpret_cast<const uint4*>(src);
  }
  const int nv = cv.n_kv_heads * D;
  const int qq = t / 4, jj = t % 4;
  for (int x = threadIdx.x; x < nv; x += blockDim.x) {
    const int g = x / D, d = x % D;
    const int m = d / 16, dd = d % 16;
    const uint16_t* src =
        reinterpret_cast<const uint16_t*>(pg + (size_t)((g + page) % cv.n_kv_heads) * PL::kHiHead + PL::kHiV);
    vout[g * D + d] = src[(((m >> 1) * 64 + qq * 16 + dd) * 2 + (m & 1)) * 4 + jj];
  }
}

// Bulk append with a window.  The call's combined index x covers positions
// q = e0 + x, e0 = max(0, p0 - W): first the window's tokens from before the
// call (x < nr = p0 - e0; their decisions in ring_act), then the new tokens
// (j = x - nr).  Positions below e1 = max(e0, p0 + n_fit - W) leave the window
// now and are slotted into the stores in position order as in
// append_plan_kernel; the new tokens from e1 on enter the window and their
// decisions go to ring_act (after every read of ring_act in the chunk: the
// W positions of the window after the call have distinct slots, so no slot
// still in the window is overwritten).  staging[x] gets the store code of x
// or -1; the sequence's last four staging words keep the stores' counts
// before the call, p0 and n_fit for the pack (append_pack_page_kernel, which
// reads a leaving window entry from its ring slot) and window-fill kernels.
template <bool kBudget>
__global__ __launch_bounds__(256) void append_plan_window_kernel(AppendArgs a) {
  __shared__ uint8_t s_a0[64], s_amin[64];
  __shared__ int s_wave[4];
  __shared__ unsigned s_page_base[2];
  __shared__ int s_granted[2];
  struct Empty {};
  __shared__ std::conditional_t<kBudget, BudgetTable, Empty> s_bud;
  __shared__ uint8_t s_act[kBudget ? 256 : 1];
  const CacheView& cv = a.cv;
  const int b = blockIdx.x;
  const int W = cv.window;
  load_table(a.tab, s_a0, s_amin);
  uint32_t flags = 0;
  const int n = clamp_n_new(a, b, flags);
  int32_t* cnt = counters_of(cv, b, a.layer);
  const int p0 = cnt[kCntPos];
  const int n_fit = max(0, min(n, cv.max_tokens - p0));
  if (n_fit < n) flags |= PASK_FLAG_SEQ_CAPACITY;
  const int e0 = max(0, p0 - W), nr = p0 - e0;
  const int n_out = max(e0, p0 + n_fit - W) - e0;    // entries leaving the window now
  const int n_x = nr + n_fit;
  uint8_t* ract = ring_act_of(cv, b, a.layer);
  bool budget = false;
  int64_t R = 0;
  if constexpr (kBudget) {
    const uint4* src = reinterpret_cast<const uint4*>(cv.budget);
    uint4* dst = reinterpret_cast<uint4*>(&s_bud);
    for (int i = threadIdx.x; i < (int)(sizeof(BudgetTable) / 16); i += 256) dst[i] = src[i];
    __syncthreads();
    budget = s_bud.loaded == kBudgetLoaded;
    if (!budget && threadIdx.x == 0) flags |= PASK_FLAG_NO_BUDGET;
    if (budget && threadIdx.x == 0) R = *budget_of(cnt);
  }
  int nst[2] = {cnt[kCntHi], cnt[kCntLo]};
  int n_drop = 0, n_forced = 0, n_lost = 0;
  int32_t* bt[2] = {block_table_of(cv, b, a.layer, kHi), block_table_of(cv, b, a.layer, kLo)};
  int32_t* il[2] = {index_list_of(cv, b, a.layer, kHi), index_list_of(cv, b, a.layer, kLo)};
  int32_t* stg = cv.staging + (size_t)b * cv.staging_stride;
  if (threadIdx.x == 0) {                          // for the pack kernel: the stores' counts before the call
    stg[cv.staging_stride - 4] = nst[0];
    stg[cv.staging_stride - 3] = nst[1];
  }
  const bool keep_all = (a.flags & kKeepAll) != 0u;
  const unsigned pool[2] = {(unsigned)cv.hi_pages, (unsigned)cv.lo_pages};
  __syncthreads();

  for (int c0 = 0; c0 < n_x; c0 += 256) {
    const int x = c0 + (int)threadIdx.x;
    const bool valid = x < n_x;
    const bool is_new = valid && x >= nr;
    const int j = x - nr;
    const int q = e0 + x;
    if constexpr (kBudget) {
      if (budget && threadIdx.x == 0) {              // the chunk's new tokens, in position order
        const int j1 = min(n_fit, c0 + 256 - nr);
        for (int jj = max(0, c0 - nr); jj < j1; ++jj) {
          const size_t at = (size_t)b * a.max_new + jj;
          const int tag = (int)a.tags[at];
          const bool forced = (uint32_t)(p0 + jj) < s_bud.n_sink || (uint32_t)tag >= s_bud.n_tags;
          s_act[jj + nr - c0] =
              (uint8_t)budget_decide(&s_bud, tag, (int)a.states[at], forced, (int)a.tab.group, R, flags);
        }
      }
      __syncthreads();
    }
    int act = kDrop;
    bool forced = false, bad = false;
    if (is_new) {
      const int tag = a.tags ? (int)a.tags[(size_t)b * a.max_new + j] : 0;
      act = decide(s_a0, s_amin, a.tab.n_tags, a.tab.n_sink, keep_all, tag, q, forced, bad);
      if constexpr (kBudget) {
        if (budget) act = s_act[threadIdx.x];
      }
    } else if (valid) {
      const uint8_t byte = ract[q % W];
      act = byte & 3;
      forced = ((byte >> 2) & 1) != 0;
    }
    if (bad) flags |= PASK_FLAG_BAD_TAG;
    const bool leaving = valid && x < n_out;
    const int st = act == kHigh ? kHi : kLo;
    const bool keep = leaving && act != kDrop;
    int tot_hi, tot_lo, np_hi, np_lo;
    const int r_hi = block_exclusive_count(keep && st == kHi, s_wave, tot_hi);
    const int r_lo = block_exclusive_count(keep && st == kLo, s_wave, tot_lo);
    const int slot = keep ? nst[st] + (st == kHi ? r_hi : r_lo) : 0;
    const bool new_page = keep && (slot % kPage) == 0;
    const int pr_hi = block_exclusive_count(new_page && st == kHi, s_wave, np_hi);
    const int pr_lo = block_exclusive_count(new_page && st == kLo, s_wave, np_lo);
    if (threadIdx.x == 0) {
      const int np[2] = {np_hi, np_lo};
#pragma unroll
      for (int y = 0; y < 2; ++y) {
        unsigned base = 0u;
        int granted = 0;
        if (np[y] > 0) {
          base = atomicAdd(&cv.status[2 + y], (unsigned)np[y]);
          granted = base >= pool[y] ? 0 : (int)min((unsigned)np[y], pool[y] - base);
        }
        s_page_base[y] = base;
        s_granted[y] = granted;
      }
    }
    __syncthreads();                                 // also: every read of ract in this chunk is done
    int pages_before[2];
#pragma unroll
    for (int y = 0; y < 2; ++y) pages_before[y] = (nst[y] + kPage - 1) / kPage;
    bool stored = false;
    if (keep) {
      const int pidx = slot / kPage;
      stored = pidx < pages_before[st] + s_granted[st];
      if (stored) {
        if (new_page) bt[st][pidx] = (int)(s_page_base[st] + (unsigned)(st == kHi ? pr_hi : pr_lo));
        il[st][slot] = q;
      } else {
        flags |= st == kHi ? PASK_FLAG_HI_POOL_EXHAUSTED : PASK_FLAG_LO_POOL_EXHAUSTED;
      }
    }
    if (valid) stg[x] = stored ? ((st << 30) | slot) : -1;
    if (is_new && !leaving) ract[q % W] = (uint8_t)(act | (forced ? 4 : 0));
    int c_drop, c_forced, c_lost;
    block_exclusive_count(leaving && act == kDrop, s_wave, c_drop);
    block_exclusive_count(stored && forced, s_wave, c_forced);
    block_exclusive_count(keep && !stored, s_wave, c_lost);
    const int tot[2] = {tot_hi, tot_lo};
#pragma unroll
    for (int y = 0; y < 2; ++y) nst[y] = min(nst[y] + tot[y], (pages_before[y] + s_granted[y]) * kPage);
    n_drop += c_drop;
    n_forced += c_forced;
    n_lost += c_lost;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    cnt[kCntHi] = nst[0];
    cnt[kCntLo] = nst[1];
    cnt[kCntPos] = p0 + n_fit;
    cnt[kCntDrop] += n_drop;
    cnt[kCntForced] += n_forced;
    cnt[kCntLost] += n_lost + (n - n_fit);
    if (budget) *budget_of(cnt) = R;
    stg[cv.staging_stride - 2] = p0;
    stg[cv.staging_stride - 1] = n_fit;
  }
  if (flags) atomicOr(cv.status, flags);
}

// The new tokens that stay in the window (the last min(n_fit, W) of the
// call) into their window slots; after the pack kernel has read the slots
// they replace.
template <int D>
__global__ __launch_bounds__(256) void append_window_fill_kernel(AppendArgs a) {
  const CacheView& cv = a.cv;
  const int b = blockIdx.y;
  const int W = cv.window;
  const int32_t* stg = cv.staging + (size_t)b * cv.staging_stride;
  const int p0 = stg[cv.staging_stride - 2], n_fit = stg[cv.staging_stride - 1];
  const int j0 = max(0, n_fit - W);
  const size_t row = (size_t)cv.n_kv_heads * D;
  for (int kk = 0; kk < kPackTokens; ++kk) {
    const int j = j0 + (int)blockIdx.x * kPackTokens + kk;
    if (j >= n_fit) break;
    const int ws = (p0 + j) % W;
    write_hi<D>(cv, ring_page(cv, b, a.layer, ws / kPage), ws % kPage, a.k + ((size_t)b * a.max_new + j) * row,
                a.v + ((size_t)b * a.max_new + j) * row);
  }
}

// One token per sequence with a window: thread 0 decides the new token and,
// when position pos - W leaves the window, slots that entry by its recorded
// action; the block then reads the leaving entry from its window slot into
// LDS, writes the new token into that slot, and persists the leaving entry.
template <int D>
__global__ __launch_bounds__(256) void append_step_window_kernel(AppendArgs a) {
  __shared__ uint8_t s_a0[64], s_amin[64];
  __shared__ int s_code, s_page, s_ws;
  __shared__ __align__(16) uint16_t s_kv[2][8 * D];
  const CacheView& cv = a.cv;
  const int b = blockIdx.x;
  const int W = cv.window;
  load_table(a.tab, s_a0, s_amin);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t flags = 0;
    const int n = clamp_n_new(a, b, flags);
    int code = -1, page = -1, ws = -1;
    if (n > 0) {
      int32_t* cnt = counters_of(cv, b, a.layer);
      const int pos = cnt[kCntPos];
      if (pos >= cv.max_tokens) {
        flags |= PASK_FLAG_SEQ_CAPACITY;
        cnt[kCntLost] += 1;
      } else {
        bool forced;
        const int act = decide_one(a, s_a0, s_amin, b, cnt, pos, forced, flags);
        uint8_t* ract = ring_act_of(cv, b, a.layer);
        ws = pos % W;
        if (pos >= W) {                              // position pos - W leaves the window
          const uint8_t old = ract[ws];
          code = slot_one(cv, b, a.layer, cnt, old & 3, ((old >> 2) & 1) != 0, pos - W, page, flags);
        }
        ract[ws] = (uint8_t)(act | (forced ? 4 : 0));
        cnt[kCntPos] = pos + 1;
      }
    }
    if (flags) atomicOr(cv.status, flags);
    s_code = code;
    s_page = page;
    s_ws = ws;
  }
  __syncthreads();
  const int code = s_code, ws = s_ws;
  if (ws < 0) return;
  const int rpage = ring_page(cv, b, a.layer, ws / kPage);
  if (code >= 0) read_hi_token<D>(cv, rpage, ws % kPage, s_kv[0], s_kv[1]);
  __syncthreads();                                   // the leaving entry is read before its slot is reused
  const size_t row = (size_t)cv.n_kv_heads * D;
  write_hi<D>(cv, rpage, ws % kPage, a.k + (size_t)b * a.max_new * row, a.v + (size_t)b * a.max_new * row);
  if (code >= 0) {
    const int slot = code & 0x3FFFFFFF;
    if ((code >> 30) == kHi) write_hi<D>(cv, s_page, slot % kPage, s_kv[0], s_kv[1]);
    else write_lo<D>(cv, s_page, slot % kPage, s_kv[0], s_kv[1]);
  }
}

}  // namespace

hipError_t launch_reset(const CacheView& cv, int32_t max_batch, hipStream_t s) {
  const size_t n = (size_t)max_batch * cv.n_layers * kCounterStride;
  const size_t blocks = std::min<size_t>((n + 255) / 256 + 1, 4096);
  reset_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(cv, n);
  return hipGetLastError();
}

hipError_t launch_budget_init(const CacheView& cv, int32_t batch, int64_t r0, hipStream_t s) {
  const size_t n = (size_t)batch * cv.n_layers;
  const size_t blocks = std::min<size_t>((n + 255) / 256, 4096);
  budget_init_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(cv, batch, r0);
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, hipStream_t s) {
  if (a.max_new == 1 && a.n_new == nullptr) return launch_append_step(a, s);
  if (a.cv.window > 0) {
    if (a.states) append_plan_window_kernel<true><<<dim3(a.batch), dim3(256), 0, s>>>(a);
    else append_plan_window_kernel<false><<<dim3(a.batch), dim3(256), 0, s>>>(a);
    // pages of a store this call's leaving entries (at most max_new + W) can reach
    const dim3 gp((a.max_new + a.cv.window + kPage - 1) / kPage + 1, 2, a.batch);
    const dim3 gf((std::min(a.max_new, a.cv.window) + kPackTokens - 1) / kPackTokens, a.batch);
    if (a.cv.head_dim == 64) {
      append_pack_page_kernel<64><<<gp, dim3(kPackThreads), 0, s>>>(a);
      append_window_fill_kernel<64><<<gf, dim3(256), 0, s>>>(a);
    } else {
      append_pack_page_kernel<128><<<gp, dim3(kPackThreads), 0, s>>>(a);
      append_window_fill_kernel<128><<<gf, dim3(256), 0, s>>>(a);
    }
    return hipGetLastError();
  }
  if (a.states) append_plan_kernel<true><<<dim3(a.batch), dim3(kPlanThreads), 0, s>>>(a);
  else append_plan_kernel<false><<<dim3(a.batch), dim3(kPlanThreads), 0, s>>>(a);
  // pages of a store one sequence's slots of this call can reach: ceil(max_new / 16) + 1
  const dim3 grid((a.max_new + kPage - 1) / kPage + 1, 2, a.batch);
  if (a.cv.head_dim == 64) append_pack_page_kernel<64><<<grid, dim3(kPackThreads), 0, s>>>(a);
  else append_pack_page_kernel<128><<<grid, dim3(kPackThreads), 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_append_step(const AppendArgs& a, hipStream_t s) {
  if (a.cv.window > 0) {
    if (a.cv.head_dim == 64) append_step_window_kernel<64><<<dim3(a.batch), dim3(256), 0, s>>>(a);
    else append_step_window_kernel<128><<<dim3(a.batch), dim3(256), 0, s>>>(a);
    return hipGetLastError();
  }
  if (a.cv.head_dim == 64) append_step_kernel<64><<<dim3(a.batch), dim3(256), 0, s>>>(a);
  else append_step_kernel<128><<<dim3(a.batch), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace pask
