// The attention call's work split (pask_plan.h), checked on the CPU over
// random calls: sequences with random HIGH / window / LOW page counts (empty
// ones included), 1-8 KV heads, the workspace's piece bound of the C ABI for
// a hint at the longest sequence, and worker counts from 1 to 4096.  For the
// per-XCD weighted plan (calls with more than 64 segments; odd-XCD weights
// 12..16, four worker waves per workgroup or one) and the equal plan (at most
// 64), every worker's range is walked the way the attention kernel walks it,
// and:
//   - the ranges tile [0, total): every page is attended exactly once;
//   - the ranges tile [0, total) in worker order and block_of(u) is the
//     worker whose range holds u, for every page start u;
//   - every piece a worker writes has index w - block_of(seg0) in
//     [0, n_pieces) and n_pieces <= splits, and every index in [0, n_pieces)
//     of every segment is written once (the merge reads exactly these).
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <vector>

#include "pask_plan.h"

using namespace pask;

namespace {
uint64_t g_s = 88172645463325252ull;
uint32_t rnd(uint32_t n) {
  g_s ^= g_s << 13;
  g_s ^= g_s >> 7;
  g_s ^= g_s << 17;
  return (uint32_t)(g_s % n);
}

int splits_for(int hint, long long segments) {   // as the C ABI sizes the workspace
  const int coarse = (hint + 127) / 128 + 2;
  if (segments > 64) return coarse;
  const int fine = (hint + 15) / 16 + 2;
  return std::max(coarse, std::min(fine, (int)(4096 / std::max<long long>(segments, 1))));
}

struct Call {
  int H;
  std::vector<SeqPages> seqs;
  std::vector<long long> excl;   // units of the sequences before b (one KV head)
  long long total;
  int mx;
};

template <typename Plan>
int check(const Call& c, const Plan& plan, int n_workers_all, int splits, const char* what) {
  // pieces[seg] -> which indices were written
  const int B = (int)c.seqs.size(), H = c.H;
  std::vector<std::vector<int>> written(B * H);
  std::vector<uint8_t> seen;   // per page of the call, in order
  long long pages_total = 0;
  for (auto& s : c.seqs) pages_total += (long long)s.np * H;
  seen.assign(pages_total, 0);
  std::vector<long long> page_base(B * H + 1, 0);
  for (int b = 0; b < B; ++b)
    for (int g = 0; g < H; ++g) page_base[b * H + g + 1] = page_base[b * H + g] + c.seqs[b].np;
  for (int w = 0; w < n_workers_all; ++w) {
    const long long start = plan.start_of(w), end = plan.end_of(w);
    if (start >= end) continue;
    if (plan.block_of(start) != w) { printf("%s: block_of(start_of(%d)) = %lld\n", what, w, plan.block_of(start)); return 1; }
    // locate
    int b = (int)(std::upper_bound(c.excl.begin(), c.excl.end(), start / H) - c.excl.begin()) - 1;
    while (b < B && (c.seqs[b].len == 0 || (long long)(c.excl[b] + c.seqs[b].len) * H <= start)) ++b;
    if (b >= B) continue;
    long long excl = c.excl[b];
    SeqPages sp = c.seqs[b];
    const long long rel = start - excl * H;
    int g = (int)(rel / sp.len);
    int j0 = first_page_at(sp, (int)(rel - (long long)g * sp.len));
    while (true) {
      const long long seg0 = excl * H + (long long)g * sp.len;
      if (seg0 >= end) break;
      const int j1 = end - seg0 >= sp.len ? sp.np : first_page_at(sp, (int)(end - seg0));
      if (j0 < j1) {
        const long long slot = w - plan.block_of(seg0);
        const int np = n_pieces(plan, sp, seg0);
        if (np > splits || slot < 0 || slot >= np) {
          printf("%s: worker %d seg (%d,%d) slot %lld pieces %d splits %d\n", what, w, b, g, slot, np, splits);
          return 1;
        }
        written[b * H + g].push_back((int)slot);
        for (int j = j0; j < j1; ++j) {
          const long long pg = page_base[b * H + g] + j;
          if (seen[pg]++) { printf("%s: page attended twice\n", what); return 1; }
          if (plan.block_of(seg0 + page_start(sp, j)) != w) { printf("%s: block_of(page) != worker\n", what); return 1; }
        }
      }
      if (j1 < sp.np) break;
      j0 = 0;
      if (++g == H) {
        g = 0;
        excl += sp.len;
        do {
          if (++b >= B) break;
          sp = c.seqs[b];
        } while (sp.len == 0);
        if (b >= B) break;
      }
    }
  }
  for (long long i = 0; i < pages_total; ++i)
    if (!seen[i]) { printf("%s: page %lld never attended\n", what, i); return 1; }
  for (int b = 0; b < B; ++b)
    for (int g = 0; g < H; ++g) {
      if (c.seqs[b].np == 0) continue;
      auto v = written[b * H + g];
      std::sort(v.begin(), v.end());
      const int np = n_pieces(plan, c.seqs[b], c.excl[b] * H + (long long)g * c.seqs[b].len);
      if ((int)v.size() != np) { printf("%s: segment (%d,%d) %zu pieces written, %d expected\n", what, b, g, v.size(), np); return 1; }
      for (int k = 0; k < np; ++k)
        if (v[k] != k) { printf("%s: piece index %d missing\n", what, k); return 1; }
    }
  return 0;
}
}  // namespace

int main(int argc, char** argv) {
  const int rounds = argc > 1 ? atoi(argv[1]) : 400;
  int bad = 0;
  long long calls = 0;
  for (int r = 0; r < rounds && !bad; ++r) {
    Call c;
    const int kind = rnd(4);
    const int B = kind == 0 ? 1 + rnd(8) : (kind == 1 ? 1 + rnd(64) : 1 + rnd(300));
    c.H = 1 + rnd(8);
    int mx_tok = 0;
    long long acc = 0;
    for (int b = 0; b < B; ++b) {
      const int shape = rnd(6);
      int hi = shape == 0 ? 0 : rnd(shape == 1 ? 40 : 9000), win = rnd(3) ? 0 : rnd(70), lo = rnd(2) ? rnd(3000) : 0;
      if (shape == 5) hi = 20000 + rnd(20000);
      SeqPages s = make_pages(hi, win, lo, rnd(3) == 0 ? 1 : 0);   // with or without the step's own entry
      c.excl.push_back(acc);
      acc += s.len;
      c.seqs.push_back(s);
      mx_tok = std::max(mx_tok, hi + win + lo + 1);
    }
    c.total = acc * c.H;
    c.mx = 0;
    for (auto& s : c.seqs) c.mx = std::max(c.mx, s.len);
    if (c.total == 0) continue;
    const long long segs = (long long)B * c.H;
    const int hint = std::max(1, mx_tok + (int)rnd(500));
    const int splits = splits_for(hint, segs);
    static const int workers[] = {1, 7, 64, 100, 256, 512, 1000, 2048, 2047, 4096};
    const int n = workers[rnd(sizeof(workers) / sizeof(workers[0]))];
    ++calls;
    if (segs > 64) {
      const int n4 = (n + 3) / 4 * 4;                // whole workgroups of four worker waves
      for (int odd = 12; odd <= 16 && !bad; ++odd) {
        const StreamPlan<4> p4 = stream_plan_of<4>(c.total, c.mx, splits, 8, n4, odd);
        bad |= check(c, p4, n4, splits, "weighted, 4 waves");
        const StreamPlan<1> p1 = stream_plan_of<1>(c.total, c.mx, splits, 8, n, odd);
        bad |= check(c, p1, n, splits, "weighted, 1 wave");
      }
    } else {
      const EvenPlan p = even_plan_of(c.total, c.mx, splits, 4, n);
      bad |= check(c, p, (int)((c.total + p.U - 1) / p.U), splits, "even");
      const int capped = std::min(splits, 33);     // the attention's ranges of >= 1/32 of the longest segment
      const EvenPlan pc = even_plan_of(c.total, c.mx, capped, 4, n);
      bad |= check(c, pc, (int)((pc.total + pc.U - 1) / pc.U), capped, "even, ranges >= 1/32 of the longest segment");
    }
  }
  printf("%s: %lld calls\n", bad ? "FAIL" : "ok", calls);
  return bad;
}
