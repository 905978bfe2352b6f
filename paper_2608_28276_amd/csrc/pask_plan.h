// Work split of the attention call (stream-K): pure arithmetic on the page
// counts of a call, shared by the attention, merge and distortion kernels
// (pask_attn.hip) and callable on the host, where tests/native/plan_check.hip
// checks its invariants over many shapes.  The work of a call is counted in
// units: kUnit per page of a (sequence, KV head) segment.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

namespace pask {

__host__ __device__ __forceinline__ int cdiv(int x, int y) { return (x + y - 1) / y; }

// a / b for 0 <= a, 0 < b: 32-bit division when both fit, as they do for any
// call below 2^32 units; the 64-bit expansion otherwise.
__host__ __device__ __forceinline__ long long udiv(long long a, long long b) {
  if ((((unsigned long long)a | (unsigned long long)b) >> 32) == 0) return (long long)((uint32_t)a / (uint32_t)b);
  return a / b;
}

// Pages of one sequence in a layer: the HIGH store, the recent window (HIGH
// layout, min(n_pos, W) slots), the LOW store and, when the call itself
// persists the step's entry, one page holding just that entry (n_x = 1), in
// that order.  Every page weighs kUnit work units (with the memory system
// saturated a page iteration costs about the same time whatever its size;
// weighting LOW pages by their bytes measured slower), so every page starts
// at a multiple of kUnit.
constexpr int kUnit = 32;
// The page of the step's own entry weighs four pages: the worker that writes
// and attends it does more than stream a page (its K / V rows are quantised,
// stored and attended from registers).  Interleaved in one process against a
// weight of one page: one Qwen3-4B-shaped sequence 13.3 / 13.3 us per call,
// four sequences 28.1 against 29.3, the batch-64 call 203.5 against 204.8
// (two pages: 13.3, 28.9, 203.7).
#ifndef PASK_ENTRY_UNITS
#define PASK_ENTRY_UNITS 128
#endif
constexpr int kEntryUnits = PASK_ENTRY_UNITS;
struct SeqPages {
  int n_hi, n_win, n_lo;   // slots of the HIGH store, the window, the LOW store
  int np_hi, np_w, np_l;   // pages: HIGH store, + window (HIGH layout), + LOW store
  int np;                  // all pages: np_l + n_x
  int len;                 // units
};
__host__ __device__ __forceinline__ int len_of(int n_hi, int n_win, int n_lo, int n_x = 0) {
  return kUnit * (cdiv(n_hi, 16) + cdiv(n_win, 16) + cdiv(n_lo, 16)) + kEntryUnits * n_x;
}
__host__ __device__ __forceinline__ SeqPages make_pages(int n_hi, int n_win, int n_lo, int n_x = 0) {
  SeqPages s;
  s.n_hi = n_hi;
  s.n_win = n_win;
  s.n_lo = n_lo;
  s.np_hi = cdiv(n_hi, 16);
  s.np_w = s.np_hi + cdiv(n_win, 16);
  s.np_l = s.np_w + cdiv(n_lo, 16);
  s.np = s.np_l + n_x;
  s.len = len_of(n_hi, n_win, n_lo, n_x);
  return s;
}
// Unit offset of page j inside its segment.
__host__ __device__ __forceinline__ int page_start(const SeqPages&, int j) { return kUnit * j; }
// First page whose unit offset is >= u (s.np when there is none).
__host__ __device__ __forceinline__ int first_page_at(const SeqPages& s, int u) {
  const int j = cdiv(u, kUnit);
  return j < s.np ? j : s.np;
}

// Calls with more than 64 (sequence, KV head) segments.  The work list is
// the segments (sequence b, KV head g) in that nesting order, each the units
// of its pages.  Worker w (a wave; kWpb of them per workgroup) takes the
// pages that start in its contiguous range [start_of(w), end_of(w)), of
// weight(w) x step units.  Workgroups are dealt to the 8 XCDs in turn, and
// the waves of the odd-numbered XCDs were measured streaming about 10%
// slower, so a worker there weighs `odd` sixteenths against 16 on an even XCD
// (16 when the ranges are at their minimum size: a latency-bound call).
// Every range is at least lo units, at least one page (pages start at
// multiples of kUnit), so each range between the first and the last of a
// segment holds a page of it, and no segment is cut into more than `splits`
// pieces (lo >= mx / (splits - 1)).
template <int kWpb>
struct StreamPlan {
  long long total;   // units
  int step;          // units per sixteenth of weight
  int odd;           // weight of a worker on an odd XCD, in sixteenths
  __host__ __device__ __forceinline__ int octet() const { return kWpb * (4 * 16 + 4 * odd); }   // 8 workgroups
  __host__ __device__ __forceinline__ int weight(int w) const { return ((w / kWpb) & 1) ? odd : 16; }
  // Sixteenths of weight of workers 0..w-1.
  __host__ __device__ __forceinline__ long long weight_before(int w) const {
    const int wg = w / kWpb, j = wg & 7;
    return (long long)(wg >> 3) * octet() + kWpb * ((j + 1) / 2 * 16 + (j / 2) * odd) + (w % kWpb) * weight(w);
  }
  __host__ __device__ __forceinline__ long long start_of(int w) const {
    return odd == 16 ? (long long)w * (16 * step) : weight_before(w) * step;
  }
  __host__ __device__ __forceinline__ long long end_of(int w) const {
    const long long e = start_of(w) + (long long)weight(w) * step;
    return e < total ? e : total;
  }
  // Worker whose range holds unit u.
  __host__ __device__ __forceinline__ long long block_of(long long u) const {
    if (odd == 16) return udiv(u, 16LL * step);
    const long long wu = udiv(u, step);            // sixteenths of weight before u
    const long long o = udiv(wu, octet());
    int r = (int)(wu - o * octet()), j = 0;
    while (r >= kWpb * weight(j * kWpb)) {
      r -= kWpb * weight(j * kWpb);
      ++j;
    }
    return o * 8 * kWpb + j * kWpb + r / weight(j * kWpb);
  }
};

// total: units of the call; mx: units of its longest segment; splits: pieces
// the workspace holds per segment (>= 2); min_pages: the fewest pages a range
// takes; n: workers; odd: the odd-XCD weight in sixteenths (1..16).
template <int kWpb>
__host__ __device__ __forceinline__ StreamPlan<kWpb> stream_plan_of(long long total, int mx, int splits,
                                                                    int min_pages, int n, int odd) {
  StreamPlan<kWpb> p;
  p.total = total;
  const long long lo0 = (long long)kUnit * min_pages, lo1 = cdiv(mx, splits - 1);
  const long long lo = lo0 > lo1 ? lo0 : lo1;
  p.odd = odd;
  long long step = udiv(total + p.weight_before(n) - 1, p.weight_before(n));
  if (step * odd < lo) {                           // ranges at their minimum: equal ones
    p.odd = 16;
    const long long even = udiv(total + p.weight_before(n) - 1, p.weight_before(n));
    step = even > (lo + 15) / 16 ? even : (lo + 15) / 16;
  }
  p.step = (int)(step < 0x7FFFFFFF / 16 ? step : 0x7FFFFFFF / 16);
  return p;
}

// The same split with equal ranges of U units, for calls with at most 64
// segments (latency-bound: a few pages per worker).
struct EvenPlan {
  long long total;   // units
  int U;             // units per worker
  __host__ __device__ __forceinline__ long long start_of(int w) const { return (long long)w * U; }
  __host__ __device__ __forceinline__ long long end_of(int w) const {
    const long long e = (long long)(w + 1) * U;
    return e < total ? e : total;
  }
  __host__ __device__ __forceinline__ long long block_of(long long u) const { return u / U; }
};
__host__ __device__ __forceinline__ EvenPlan even_plan_of(long long total, int mx, int splits, int min_pages, int n) {
  EvenPlan p;
  p.total = total;
  const long long even = (total + n - 1) / n;
  int U = kUnit * min_pages;
  if (even > U) U = (int)(even < 0x7FFFFFFF ? even : 0x7FFFFFFF);
  const int lo1 = cdiv(mx, splits - 1);
  if (lo1 > U) U = lo1;
  p.U = U;
  return p;
}

// Pieces of the segment starting at unit seg0 with pages sp (sp.np > 0).
template <typename Plan>
__host__ __device__ __forceinline__ int n_pieces(const Plan& plan, const SeqPages& sp, long long seg0) {
  return (int)(plan.block_of(seg0 + page_start(sp, sp.np - 1)) - plan.block_of(seg0)) + 1;
}

}  // namespace pask
