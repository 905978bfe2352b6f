// gfx950 kernels of the PASK decode hot path.
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
//   attn         grouped-query flash-decode over one (sequence, KV head) and a
//                set of 256-slot work units of the HIGH and LOW stores: query
//                slice in registers, bf16 dot2 for q.k, int4 codes widened
//                exactly in registers, online softmax in base 2, next page
//                prefetched into registers.
//   attn_merge   merge the split partials (max, sum, weighted values).
#include <hip/hip_runtime.h>

#include <math.h>

#include <type_traits>

#include "pask_internal.h"

namespace pask {
namespace {

constexpr int kDrop = 0, kLow = 1, kHigh = 2;
constexpr int kPackTokens = 16;   // tokens per append_pack block

__device__ __forceinline__ size_t sl_index(const CacheView& cv, int b, int layer) {
  return (size_t)b * cv.n_layers + layer;
}
__device__ __forceinline__ int32_t* counters_of(const CacheView& cv, int b, int layer) {
  return cv.counters + sl_index(cv, b, layer) * kCounterStride;
}
__device__ __forceinline__ int32_t* block_table_of(const CacheView& cv, int b, int layer, int st) {
  return cv.block_table + (sl_index(cv, b, layer) * 2 + st) * (size_t)cv.max_pages;
}
__device__ __forceinline__ int32_t* index_list_of(const CacheView& cv, int b, int layer, int st) {
  return cv.index_list + (sl_index(cv, b, layer) * 2 + st) * (size_t)cv.max_tokens;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// acc + a.lo * b.lo + a.hi * b.hi over packed bf16 pairs (v_dot2c_f32_bf16).
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), acc, false);
}

// ---------------------------------------------------------------------------
// reset
// ---------------------------------------------------------------------------
__global__ void reset_kernel(CacheView cv, size_t n_counters) {
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i0 < 4) cv.status[i0] = 0u;
  for (size_t i = i0; i < n_counters; i += (size_t)gridDim.x * blockDim.x) cv.counters[i] = 0;
}

// ---------------------------------------------------------------------------
// decisions and slotting
// ---------------------------------------------------------------------------

// Action of one token (Eq. 10): the higher of the selected action and the
// floor of its (tag, group) bucket.  Sinks, keep-all tokens and tags outside
// the table are RETAIN-HIGH (the latter also flagged).
__device__ __forceinline__ int decide(const uint8_t* s_a0, const uint8_t* s_amin, uint32_t n_tags,
                                      uint32_t n_sink, bool keep_all, int tag, int pos,
                                      bool& forced, bool& bad) {
  bad = (uint32_t)tag >= n_tags;
  if (keep_all || (uint32_t)pos < n_sink || bad) {
    forced = true;
    return kHigh;
  }
  forced = false;
  const int a0 = s_a0[tag], am = s_amin[tag];
  return a0 > am ? a0 : am;
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

__global__ __launch_bounds__(256) void append_plan_kernel(AppendArgs a) {
  __shared__ uint8_t s_a0[64], s_amin[64];
  __shared__ int s_wave[4];
  __shared__ unsigned s_page_base[2];
  __shared__ int s_granted[2];
  const CacheView& cv = a.cv;
  const int b = blockIdx.x;
  load_table(a.tab, s_a0, s_amin);
  uint32_t flags = 0;
  const int n = clamp_n_new(a, b, flags);
  int32_t* cnt = counters_of(cv, b, a.layer);
  const int pos0 = cnt[kCntPos];
  int nst[2] = {cnt[kCntHi], cnt[kCntLo]};
  int n_drop = 0, n_forced = 0, n_lost = 0, n_fit = 0;
  int32_t* bt[2] = {block_table_of(cv, b, a.layer, kHi), block_table_of(cv, b, a.layer, kLo)};
  int32_t* il[2] = {index_list_of(cv, b, a.layer, kHi), index_list_of(cv, b, a.layer, kLo)};
  int32_t* stg = cv.staging + (size_t)b * cv.max_tokens;
  const bool keep_all = (a.flags & kKeepAll) != 0u;
  const unsigned pool[2] = {(unsigned)cv.hi_pages, (unsigned)cv.lo_pages};
  __syncthreads();

  for (int c0 = 0; c0 < n; c0 += 256) {
    const int j = c0 + (int)threadIdx.x;
    const bool valid = j < n;
    const int pos = pos0 + j;
    const bool fits = valid && pos < cv.max_tokens;
    int act = kDrop;
    bool forced = false, bad = false;
    if (fits) {
      const int tag = a.tags ? (int)a.tags[(size_t)b * a.max_new + j] : 0;
      act = decide(s_a0, s_amin, a.tab.n_tags, a.tab.n_sink, keep_all, tag, pos, forced, bad);
    }
    if (bad) flags |= PASK_FLAG_BAD_TAG;
    if (valid && !fits) flags |= PASK_FLAG_SEQ_CAPACITY;
    const int st = act == kHigh ? kHi : kLo;
    const bool keep = fits && act != kDrop;
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
        if (new_page) bt[st][pidx] = (int)(s_page_base[st] + (unsigned)(st == kHi ? pr_hi : pr_lo));
        il[st][slot] = pos;
      } else {
        flags |= st == kHi ? PASK_FLAG_HI_POOL_EXHAUSTED : PASK_FLAG_LO_POOL_EXHAUSTED;
      }
    }
    if (valid) stg[j] = stored ? ((st << 30) | slot) : -1;
    int c_drop, c_forced, c_lost, c_fit;
    block_exclusive_count(fits && act == kDrop, s_wave, c_drop);
    block_exclusive_count(stored && forced, s_wave, c_forced);
    block_exclusive_count(valid && !stored && !(fits && act == kDrop), s_wave, c_lost);
    block_exclusive_count(fits, s_wave, c_fit);
    const int tot[2] = {tot_hi, tot_lo};
#pragma unroll
    for (int x = 0; x < 2; ++x) nst[x] = min(nst[x] + tot[x], (pages_before[x] + s_granted[x]) * kPage);
    n_drop += c_drop;
    n_forced += c_forced;
    n_lost += c_lost;
    n_fit += c_fit;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    cnt[kCntHi] = nst[0];
    cnt[kCntLo] = nst[1];
    cnt[kCntPos] = pos0 + n_fit;
    cnt[kCntDrop] += n_drop;
    cnt[kCntForced] += n_forced;
    cnt[kCntLost] += n_lost;
  }
  if (flags) atomicOr(cv.status, flags);
}

// ---------------------------------------------------------------------------
// RETAIN-HIGH copy and RETAIN-LOW quantise-and-pack of one token
// ---------------------------------------------------------------------------

// Quantise 4 consecutive elements of a 32-element group held by 8 adjacent
// lanes: s = fp16(absmax / 7) (correctly rounded division, saturated at 65504,
// round-to-nearest-even conversion), q = clamp(rint(x / s), -7, 7).  Returns
// the 4 codes as nibbles (element i in bits 4i..4i+3) and the scale bits.
__device__ __forceinline__ void quant4(uint32_t x01, uint32_t x23, uint32_t& packed, uint32_t& sbits) {
  float f[4] = {bf16_lo(x01), bf16_hi(x01), bf16_lo(x23), bf16_hi(x23)};
  float am = fmaxf(fmaxf(fabsf(f[0]), fabsf(f[1])), fmaxf(fabsf(f[2]), fabsf(f[3])));
  am = fmaxf(am, __shfl_xor(am, 1, 8));
  am = fmaxf(am, __shfl_xor(am, 2, 8));
  am = fmaxf(am, __shfl_xor(am, 4, 8));
  const float s32 = fminf(am / 7.0f, 65504.0f);
  const _Float16 h = (_Float16)s32;
  const float s = (float)h;
  sbits = (uint32_t)__builtin_bit_cast(uint16_t, h);
  uint32_t p = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int q = 0;
    if (s != 0.0f) q = (int)fminf(fmaxf(rintf(f[i] / s), -7.0f), 7.0f);
    p |= ((uint32_t)q & 0xFu) << (4 * i);
  }
  packed = p;
}

template <int D>
__device__ __forceinline__ void write_hi(const CacheView& cv, int page, int s16, const uint16_t* kin,
                                         const uint16_t* vin) {
  constexpr int kChunks = D / 8;  // 16-byte chunks per row
  const int n = cv.n_kv_heads * 2 * kChunks;
  uint8_t* pg = cv.hi_pool + (size_t)page * cv.hi_page_bytes;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int row = i / kChunks, col = i % kChunks;
    const int g = row >> 1, kv = row & 1;
    const uint16_t* src = (kv ? vin : kin) + g * D + col * 8;
    uint8_t* dst = pg + (size_t)g * (2 * kPage * D * 2) + kv * (kPage * D * 2) + s16 * (D * 2) + col * 16;
    *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
  }
}

template <int D>
__device__ __forceinline__ void write_lo(const CacheView& cv, int page, int s16, const uint16_t* kin,
                                         const uint16_t* vin) {
  constexpr int kGpr = D / kQGroup;                                 // groups per row
  constexpr int kHalf = kPage * (D / 2) + kPage * kGpr * 2;         // K (or V) bytes per head
  const int n_tasks = cv.n_kv_heads * 2 * kGpr * 8;                 // 8 lanes per group
  uint8_t* pg = cv.lo_pool + (size_t)page * cv.lo_page_bytes;
  for (int base = 0; base < n_tasks; base += blockDim.x) {
    const int task = base + (int)threadIdx.x;
    if (task < n_tasks) {  // whole 8-lane groups are active together
      const int gi = task >> 3, lig = task & 7;
      const int grp = gi % kGpr, row = gi / kGpr, g = row >> 1, kv = row & 1;
      const uint16_t* src = (kv ? vin : kin) + g * D + grp * kQGroup + lig * 4;
      const uint2 raw = *reinterpret_cast<const uint2*>(src);
      uint32_t packed, sbits;
      quant4(raw.x, raw.y, packed, sbits);
      uint8_t* codes = pg + (size_t)g * (2 * kHalf) + kv * kHalf;
      uint8_t* scales = codes + kPage * (D / 2);
      *reinterpret_cast<uint16_t*>(codes + s16 * (D / 2) + grp * 16 + lig * 2) = (uint16_t)packed;
      if (lig == 0) *reinterpret_cast<uint16_t*>(scales + (s16 * kGpr + grp) * 2) = (uint16_t)sbits;
    }
  }
}

template <int D>
__global__ __launch_bounds__(256) void append_pack_kernel(AppendArgs a) {
  const CacheView& cv = a.cv;
  const int b = blockIdx.y;
  uint32_t unused = 0;
  const int n = clamp_n_new(a, b, unused);
  const int32_t* stg = cv.staging + (size_t)b * cv.max_tokens;
  const size_t row = (size_t)cv.n_kv_heads * D;
  for (int jj = 0; jj < kPackTokens; ++jj) {
    const int j = (int)blockIdx.x * kPackTokens + jj;
    if (j >= n) break;
    const int code = stg[j];
    if (code < 0) continue;
    const int st = code >> 30, slot = code & 0x3FFFFFFF;
    const int page = block_table_of(cv, b, a.layer, st)[slot / kPage];
    const uint16_t* kin = a.k + ((size_t)b * a.max_new + j) * row;
    const uint16_t* vin = a.v + ((size_t)b * a.max_new + j) * row;
    if (st == kHi) write_hi<D>(cv, page, slot % kPage, kin, vin);
    else write_lo<D>(cv, page, slot % kPage, kin, vin);
  }
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
        const int tag = a.tags ? (int)a.tags[(size_t)b * a.max_new] : 0;
        bool forced, bad;
        const int act = decide(s_a0, s_amin, a.tab.n_tags, a.tab.n_sink, (a.flags & kKeepAll) != 0u,
                               tag, pos, forced, bad);
        if (bad) flags |= PASK_FLAG_BAD_TAG;
        if (act == kDrop) {
          cnt[kCntDrop] += 1;
        } else {
          const int st = act == kHigh ? kHi : kLo;
          const int slot = cnt[st];
          int32_t* bt = block_table_of(cv, b, a.layer, st);
          bool ok = true;
          if (slot % kPage == 0) {
            const unsigned pid = atomicAdd(&cv.status[2 + st], 1u);
            const unsigned pool = st == kHi ? (unsigned)cv.hi_pages : (unsigned)cv.lo_pages;
            if (pid >= pool) {
              ok = false;
              flags |= st == kHi ? PASK_FLAG_HI_POOL_EXHAUSTED : PASK_FLAG_LO_POOL_EXHAUSTED;
            } else {
              bt[slot / kPage] = (int)pid;
            }
          }
          if (ok) {
            page = bt[slot / kPage];
            index_list_of(cv, b, a.layer, st)[slot] = pos;
            cnt[st] = slot + 1;
            if (forced) cnt[kCntForced] += 1;
            code = (st << 30) | slot;
          } else {
            cnt[kCntLost] += 1;
          }
        }
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
// decode attention
// ---------------------------------------------------------------------------
//
// One wavefront per (split, KV head g, sequence b).  A split walks 256-slot
// work units, HIGH units first, then LOW units; within a unit it streams
// 16-slot pages and loads page p+1 while it computes page p.  Two lane maps
// of a page:
//   K map  lane = 4t + s: slot t, head_dim slice s (D/4 contiguous dims);
//          q . k over the slice, then summed over the 4 lanes of a quad.
//   V map  lane = (D/8) r + c: slots r + (64/(D/8)) i, dims 8c..8c+7; every
//          lane accumulates 8 dims of the G heads' outputs.
// Probabilities move from the K map to the V map through LDS.  Each split
// leaves a partial (max, sum, unnormalised o); attn_merge combines them.

template <int D, int G>
struct Tile {
  static constexpr int KS = D / 4;       // dims per lane, K map
  static constexpr int KP = KS / 2;      // bf16 pairs per lane
  static constexpr int KQ = KS / 8;      // 16-byte K chunks per lane (HIGH)
  static constexpr int VL = D / 8;       // lanes per slot, V map
  static constexpr int VT = 64 / VL;     // slots per V load
  static constexpr int VI = kPage / VT;  // V loads per page
  static constexpr int KW = KS / 8;      // 32-bit words of K codes per lane (LOW)
};

template <int D, int G>
struct RawHi {
  uint4 k[Tile<D, G>::KQ];
  uint4 v[Tile<D, G>::VI];
};

template <int D, int G>
struct RawLo {
  uint32_t k[Tile<D, G>::KW];
  uint32_t ks;
  uint32_t v[Tile<D, G>::VI];
  uint32_t vs[Tile<D, G>::VI];
};

template <int D, int G>
__device__ __forceinline__ RawHi<D, G> load_hi(const uint8_t* head, int t, int s, int r, int c) {
  using T = Tile<D, G>;
  RawHi<D, G> x;
  const uint4* kp = reinterpret_cast<const uint4*>(head + t * (D * 2) + s * (T::KS * 2));
#pragma unroll
  for (int i = 0; i < T::KQ; ++i) x.k[i] = kp[i];
  const uint8_t* vb = head + kPage * D * 2;
#pragma unroll
  for (int i = 0; i < T::VI; ++i)
    x.v[i] = *reinterpret_cast<const uint4*>(vb + (i * T::VT + r) * (D * 2) + c * 16);
  return x;
}

template <int D, int G>
__device__ __forceinline__ RawLo<D, G> load_lo(const uint8_t* head, int t, int s, int r, int c) {
  using T = Tile<D, G>;
  constexpr int kGpr = D / kQGroup;
  const uint8_t* kcodes = head;
  const uint8_t* kscales = head + kPage * (D / 2);
  const uint8_t* vcodes = kscales + kPage * kGpr * 2;
  const uint8_t* vscales = vcodes + kPage * (D / 2);
  RawLo<D, G> x;
  if constexpr (T::KW == 4) {
    const uint4 w = *reinterpret_cast<const uint4*>(kcodes + t * (D / 2) + s * (T::KS / 2));
    x.k[0] = w.x; x.k[1] = w.y; x.k[2] = w.z; x.k[3] = w.w;
  } else {
    const uint2 w = *reinterpret_cast<const uint2*>(kcodes + t * (D / 2) + s * (T::KS / 2));
    x.k[0] = w.x; x.k[1] = w.y;
  }
  x.ks = *reinterpret_cast<const uint16_t*>(kscales + (t * kGpr + (s * T::KS) / kQGroup) * 2);
#pragma unroll
  for (int i = 0; i < T::VI; ++i) {
    const int tv = i * T::VT + r;
    x.v[i] = *reinterpret_cast<const uint32_t*>(vcodes + tv * (D / 2) + c * 4);
    x.vs[i] = *reinterpret_cast<const uint16_t*>(vscales + (tv * kGpr + c / 4) * 2);
  }
  return x;
}

// Order LDS traffic between the lanes of this (single-wave) workgroup without
// waiting for outstanding global loads: wavefront-scope fences around a wave
// barrier.  __syncthreads() would also drain the prefetch of the next page.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// int4 codes of 8 elements (one 32-bit word) as 4 exact bf16 pairs.
__device__ __forceinline__ void codes_to_bf16_pairs(uint32_t w, uint32_t (&out)[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int lo = ((int)(w << (28 - 8 * e))) >> 28;
    const int hi = ((int)(w << (24 - 8 * e))) >> 28;
    out[e] = (__float_as_uint((float)lo) >> 16) | (__float_as_uint((float)hi) & 0xFFFF0000u);
  }
}

// Scores of this lane's slot for the G heads, in log2 units (-inf if invalid).
template <int D, int G>
__device__ __forceinline__ void scores_hi(const RawHi<D, G>& x, const uint32_t (&qp)[G][Tile<D, G>::KP],
                                          bool valid, float scale_log2, float (&sc)[G]) {
  using T = Tile<D, G>;
  uint32_t kw[T::KP];
#pragma unroll
  for (int i = 0; i < T::KQ; ++i) {
    kw[4 * i] = x.k[i].x; kw[4 * i + 1] = x.k[i].y; kw[4 * i + 2] = x.k[i].z; kw[4 * i + 3] = x.k[i].w;
  }
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float d = 0.0f;
#pragma unroll
    for (int p = 0; p < T::KP; ++p) d = dot2_bf16(qp[h][p], kw[p], d);
    d += __shfl_xor(d, 1);
    d += __shfl_xor(d, 2);
    sc[h] = valid ? d * scale_log2 : -INFINITY;
  }
}

template <int D, int G>
__device__ __forceinline__ void scores_lo(const RawLo<D, G>& x, const uint32_t (&qp)[G][Tile<D, G>::KP],
                                          bool valid, float scale_log2, float (&sc)[G]) {
  using T = Tile<D, G>;
  uint32_t pairs[T::KP];
#pragma unroll
  for (int wi = 0; wi < T::KW; ++wi) {
    uint32_t p4[4];
    codes_to_bf16_pairs(x.k[wi], p4);
#pragma unroll
    for (int e = 0; e < 4; ++e) pairs[4 * wi + e] = p4[e];
  }
  const float ks = half_bits_to_float(x.ks);
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float d = 0.0f;
#pragma unroll
    for (int p = 0; p < T::KP; ++p) d = dot2_bf16(qp[h][p], pairs[p], d);
    d *= ks;
    d += __shfl_xor(d, 1);
    d += __shfl_xor(d, 2);
    sc[h] = valid ? d * scale_log2 : -INFINITY;
  }
}

// Online-softmax update for one page; leaves this page's probabilities in s_p.
template <int G>
__device__ __forceinline__ void softmax_page(const float (&sc)[G], float (&m)[G], float (&l)[G],
                                             float (&acc)[G][8], float (*s_p)[G], int t, int s) {
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float mx = sc[h];
    mx = fmaxf(mx, __shfl_xor(mx, 4));
    mx = fmaxf(mx, __shfl_xor(mx, 8));
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mn = fmaxf(m[h], mx);
    const float p = exp2f(sc[h] - mn);
    if (mn > m[h]) {
      const float alpha = exp2f(m[h] - mn);
      l[h] *= alpha;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] *= alpha;
      m[h] = mn;
    }
    l[h] += p;
    if ((h & 3) == s) s_p[t][h] = p;
  }
}

template <int D, int G>
__device__ __forceinline__ void pv_hi(const RawHi<D, G>& x, int r, int nvalid, float (*s_p)[G],
                                      float (&acc)[G][8]) {
  using T = Tile<D, G>;
#pragma unroll
  for (int i = 0; i < T::VI; ++i) {
    const int tv = i * T::VT + r;
    const bool ok = tv < nvalid;
    const uint32_t w[4] = {x.v[i].x, x.v[i].y, x.v[i].z, x.v[i].w};
    float vf[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      vf[2 * e] = ok ? bf16_lo(w[e]) : 0.0f;
      vf[2 * e + 1] = ok ? bf16_hi(w[e]) : 0.0f;
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ph = s_p[tv][h];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(ph, vf[e], acc[h][e]);
    }
  }
}

template <int D, int G>
__device__ __forceinline__ void pv_lo(const RawLo<D, G>& x, int r, int nvalid, float (*s_p)[G],
                                      float (&acc)[G][8]) {
  using T = Tile<D, G>;
#pragma unroll
  for (int i = 0; i < T::VI; ++i) {
    const int tv = i * T::VT + r;
    const bool ok = tv < nvalid;
    const float vs = half_bits_to_float(x.vs[i]);
    float vf[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int q = ((int)(x.v[i] << (28 - 4 * e))) >> 28;
      vf[e] = ok ? (float)q * vs : 0.0f;
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ph = s_p[tv][h];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(ph, vf[e], acc[h][e]);
    }
  }
}

// Stream the pages of one unit, loading page p+1 while computing page p.
template <int D, int G, bool kIsHi>
__device__ __forceinline__ void run_unit(const uint8_t* pool, size_t page_bytes, size_t head_off,
                                         const int32_t* bt, int slot0, int slot_end,
                                         const uint32_t (&qp)[G][Tile<D, G>::KP], float scale_log2,
                                         float (&m)[G], float (&l)[G], float (&acc)[G][8],
                                         float (*s_p)[G], int t, int s, int r, int c) {
  using Raw = typename std::conditional<kIsHi, RawHi<D, G>, RawLo<D, G>>::type;
  auto load = [&](int p) -> Raw {
    const uint8_t* head = pool + (size_t)bt[p / kPage] * page_bytes + head_off;
    if constexpr (kIsHi) return load_hi<D, G>(head, t, s, r, c);
    else return load_lo<D, G>(head, t, s, r, c);
  };
  // The prefetch is unconditional (the last page of the unit is loaded again,
  // an L2 hit) so that the loop body is straight-line code and the compiler
  // waits only for the current page's loads, not for the prefetch.
  const int last = slot_end - 1;
  Raw cur = load(slot0);
  for (int p = slot0; p < slot_end; p += kPage) {
    const Raw nxt = load(min(p + kPage, last));
    const int nvalid = min(kPage, slot_end - p);
    float sc[G];
    if constexpr (kIsHi) scores_hi<D, G>(cur, qp, t < nvalid, scale_log2, sc);
    else scores_lo<D, G>(cur, qp, t < nvalid, scale_log2, sc);
    softmax_page<G>(sc, m, l, acc, s_p, t, s);
    wave_lds_sync();
    if constexpr (kIsHi) pv_hi<D, G>(cur, r, nvalid, s_p, acc);
    else pv_lo<D, G>(cur, r, nvalid, s_p, acc);
    wave_lds_sync();
    cur = nxt;
  }
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

template <int D, int G>
__global__ __launch_bounds__(64) void attn_kernel(AttnArgs a) {
  using T = Tile<D, G>;
  __shared__ float s_p[kPage][G];
  const CacheView& cv = a.cv;
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int S = gridDim.x;
  const int lane = threadIdx.x;
  const int32_t* cnt = counters_of(cv, b, a.layer);
  const int n_hi = cnt[kCntHi], n_lo = cnt[kCntLo];
  const int u_hi = (n_hi + kUnitTokens - 1) / kUnitTokens;
  const int u_all = u_hi + (n_lo + kUnitTokens - 1) / kUnitTokens;
  const size_t bh0 = (size_t)b * a.n_q_heads + (size_t)g * G;   // first query head of this group
  constexpr int E = D / 64;                                       // output dims per lane in the merge
  if (u_all == 0) {                                               // nothing persisted: o = 0, lse = -inf
    if (split == 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
#pragma unroll
        for (int e = 0; e < E; ++e) a.out[(bh0 + h) * D + lane * E + e] = 0;
        if (a.lse && lane == 0) a.lse[bh0 + h] = -INFINITY;
      }
    }
    return;
  }
  if (split >= u_all) return;
  const int nparts = min(u_all, S);

  const int t = lane >> 2, s = lane & 3;
  const int r = lane / T::VL, c = lane % T::VL;
  uint32_t qp[G][T::KP];
  const uint16_t* qb = a.q + bh0 * D + s * T::KS;
#pragma unroll
  for (int h = 0; h < G; ++h) {
#pragma unroll
    for (int i = 0; i < T::KP / 4; ++i) {
      const uint4 w = *reinterpret_cast<const uint4*>(qb + h * D + i * 8);
      qp[h][4 * i] = w.x; qp[h][4 * i + 1] = w.y; qp[h][4 * i + 2] = w.z; qp[h][4 * i + 3] = w.w;
    }
  }
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  }
  const size_t hi_head = (size_t)g * (2 * kPage * D * 2);
  const size_t lo_head = (size_t)g * 2 * (kPage * (D / 2) + kPage * (D / kQGroup) * 2);
  const int32_t* bt_hi = block_table_of(cv, b, a.layer, kHi);
  const int32_t* bt_lo = block_table_of(cv, b, a.layer, kLo);

  for (int u = split; u < u_all; u += S) {
    if (u < u_hi) {
      const int slot0 = u * kUnitTokens;
      run_unit<D, G, true>(cv.hi_pool, cv.hi_page_bytes, hi_head, bt_hi, slot0,
                           min(n_hi, slot0 + kUnitTokens), qp, a.scale_log2, m, l, acc, s_p, t, s, r, c);
    } else {
      const int slot0 = (u - u_hi) * kUnitTokens;
      run_unit<D, G, false>(cv.lo_pool, cv.lo_page_bytes, lo_head, bt_lo, slot0,
                            min(n_lo, slot0 + kUnitTokens), qp, a.scale_log2, m, l, acc, s_p, t, s, r, c);
    }
  }

  // Sum l over slots (lanes with equal s) and acc over V-map rows.
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float lh = l[h];
    lh += __shfl_xor(lh, 4);
    lh += __shfl_xor(lh, 8);
    lh += __shfl_xor(lh, 16);
    lh += __shfl_xor(lh, 32);
    l[h] = lh;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v = acc[h][e];
#pragma unroll
      for (int off = T::VL; off < 64; off <<= 1) v += __shfl_xor(v, off);
      acc[h][e] = v;
    }
  }

  if (nparts == 1) {                       // the only split: write the output directly
    if (r == 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float inv = 1.0f / l[h];
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = (uint32_t)f32_to_bf16_rne(acc[h][2 * e] * inv) |
                 ((uint32_t)f32_to_bf16_rne(acc[h][2 * e + 1] * inv) << 16);
        *reinterpret_cast<uint4*>(a.out + (bh0 + h) * D + c * 8) = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
    if (a.lse && lane < G) {
      float mh = m[0], lh = l[0];
#pragma unroll
      for (int h = 1; h < G; ++h)
        if (lane == h) { mh = m[h]; lh = l[h]; }
      a.lse[bh0 + lane] = (mh + log2f(lh)) * 0.69314718055994530942f;
    }
    return;
  }

  // Publish this split's partial: o (unnormalised), running max, sum.
  if (r == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float* o = a.ws_o + ((bh0 + h) * S + split) * D + c * 8;
      reinterpret_cast<float4*>(o)[0] = make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
      reinterpret_cast<float4*>(o)[1] = make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
    }
  }
  if (lane < G) {
    float mh = m[0], lh = l[0];
#pragma unroll
    for (int h = 1; h < G; ++h)
      if (lane == h) { mh = m[h]; lh = l[h]; }
    *reinterpret_cast<float2*>(a.ws_ml + ((bh0 + lane) * S + split) * 2) = make_float2(mh, lh);
  }
}

// Merge the split partials of one (sequence, query head) when there are two or
// more: lane p holds split p's (max, sum) for the global max and the weights;
// the weighted values are summed with all loads of a batch of splits in
// flight at once.  (One split writes its output itself.)
template <int D>
__global__ __launch_bounds__(64) void attn_merge_kernel(AttnArgs a) {
  constexpr int E = D / 64;           // dims per lane
  constexpr int kBatch = 8;           // splits whose loads are issued together
  const CacheView& cv = a.cv;
  const int b = blockIdx.x / a.n_q_heads;
  const size_t bh = blockIdx.x;
  const int32_t* cnt = counters_of(cv, b, a.layer);
  const int u_all = (cnt[kCntHi] + kUnitTokens - 1) / kUnitTokens + (cnt[kCntLo] + kUnitTokens - 1) / kUnitTokens;
  const int S = a.splits;
  const int nparts = min(u_all, S);
  if (nparts <= 1) return;
  const int lane = threadIdx.x;
  const float2* ml = reinterpret_cast<const float2*>(a.ws_ml + bh * S * 2);
  const float* o = a.ws_o + bh * S * D + lane * E;
  float M = -INFINITY, L = 0.0f, acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0f;
  for (int p0 = 0; p0 < nparts; p0 += 64) {           // nparts <= 64 in every supported shape but one pass each
    const int p = p0 + lane;
    const float2 x = p < nparts ? ml[p] : make_float2(-INFINITY, 0.0f);
    float mx = x.x;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    const float Mn = fmaxf(M, mx);
    const float alpha = exp2f(M - Mn);                   // rescale what earlier passes summed
    const float w = p < nparts ? exp2f(x.x - Mn) : 0.0f;
    float lw = w * x.y;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) lw += __shfl_xor(lw, off);
    L = L * alpha + lw;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= alpha;
    M = Mn;
    const int n = min(64, nparts - p0);
    for (int q0 = 0; q0 < n; q0 += kBatch) {
      float v[kBatch][E], wq[kBatch];
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const int q = min(q0 + k, n - 1);
        wq[k] = q0 + k < n ? __shfl(w, q) : 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) v[k][e] = o[(size_t)(p0 + q) * D + e];
      }
#pragma unroll
      for (int k = 0; k < kBatch; ++k)
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(wq[k], v[k][e], acc[e]);
    }
  }
  const float inv = 1.0f / L;
#pragma unroll
  for (int e = 0; e < E; ++e) a.out[bh * D + lane * E + e] = f32_to_bf16_rne(acc[e] * inv);
  if (a.lse && lane == 0) a.lse[bh] = (M + log2f(L)) * 0.69314718055994530942f;
}

}  // namespace

hipError_t launch_reset(const CacheView& cv, int32_t max_batch, hipStream_t s) {
  const size_t n = (size_t)max_batch * cv.n_layers * kCounterStride;
  const size_t blocks = std::min<size_t>((n + 255) / 256 + 1, 4096);
  reset_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(cv, n);
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, hipStream_t s) {
  if (a.max_new == 1 && a.n_new == nullptr) return launch_append_step(a, s);
  append_plan_kernel<<<dim3(a.batch), dim3(256), 0, s>>>(a);
  const dim3 grid((a.max_new + kPackTokens - 1) / kPackTokens, a.batch);
  if (a.cv.head_dim == 64) append_pack_kernel<64><<<grid, dim3(256), 0, s>>>(a);
  else append_pack_kernel<128><<<grid, dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_append_step(const AppendArgs& a, hipStream_t s) {
  if (a.cv.head_dim == 64) append_step_kernel<64><<<dim3(a.batch), dim3(256), 0, s>>>(a);
  else append_step_kernel<128><<<dim3(a.batch), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, int group_size, hipStream_t s) {
  const int D = a.cv.head_dim;
  const dim3 grid(a.splits, a.cv.n_kv_heads, a.batch);
  const dim3 block(64);
#define PASK_CASE(DD, GG)                                                        \
  if (D == DD && group_size == GG) {                                             \
    attn_kernel<DD, GG><<<grid, block, 0, s>>>(a);                               \
    attn_merge_kernel<DD><<<dim3(a.batch * a.n_q_heads), dim3(64), 0, s>>>(a);   \
    return hipGetLastError();                                                    \
  }
  PASK_CASE(64, 1) PASK_CASE(64, 2) PASK_CASE(64, 4) PASK_CASE(64, 8)
  PASK_CASE(128, 1) PASK_CASE(128, 2) PASK_CASE(128, 4) PASK_CASE(128, 8)
#undef PASK_CASE
  return hipErrorInvalidValue;
}

}  // namespace pask
