// gfx950 kernels of the PASK hot path that read the cache.
//
//   attn         grouped-query flash-decode, stream-K: one worker wave per
//                resident wave slot, each streaming a contiguous range of the
//                (sequence, KV head, page) list over the HIGH and LOW stores
//                (pask_plan.h); q.k on bf16 MFMA (query heads as columns), int4
//                K codes widened exactly to bf16 in registers with the offset
//                removed in the accumulator, the K scale applied per 32-dim
//                group; p.v on bf16 MFMA for HIGH pages and on fp16 MFMA with
//                exact fp16 V codes and the V scale folded into p for LOW
//                pages; online softmax in base 2, next pages prefetched into
//                registers.
//   attn_merge   per (sequence, KV head): combine the partials of its pieces
//                (max, sum, values) into bf16 outputs; zero for empty histories.
//                Calls with few (sequence, KV head) segments cut them into
//                pieces of at least 4 pages and 1/32 of the longest segment
//                and spread each segment's merge over several single-wave
//                blocks (attn_merge_sliced).
//   distortion   the attention-output distortion of Eq. 4: the partials of a
//                reference and an intervened cache merged in fp32, the squared
//                distance of the outputs maximised over query heads.
#include <hip/hip_runtime.h>

#include <limits.h>
#include <math.h>

#include <mutex>
#include <type_traits>

#include "pask_device.h"
#include "pask_plan.h"

namespace pask {
namespace {

// ---------------------------------------------------------------------------
// decode attention
// ---------------------------------------------------------------------------
//
// Stream-K: the work is the list of (sequence b, KV head g, page) triples,
// HIGH and window pages of a (b, g) before its LOW pages, each page weighing
// 32 units.  The grid holds one worker wave per resident wave slot of the
// chip, and worker w takes the w-th of contiguous unit ranges, so every
// worker starts at launch.  Calls with more than 64 (b, g) segments run four
// workers per workgroup, and the workers of workgroups on the odd-numbered
// XCDs (odd workgroup index: workgroups are dealt to the 8 XCDs in turn)
// take PASK_ODD_WEIGHT/16 of an even one's range: their waves stream pages
// about 10% slower, so with equal ranges the even XCDs idle through the last
// ~15 us of the call.  Calls with at most 64 segments run single-wave
// workgroups with equal ranges.  A range crossing a (b, g) boundary closes
// that segment with a partial block; every range is at least what keeps every
// (b, g) within as many pieces as the workspace holds partials.
//
// Per page (16 slots x all G query heads of KV head g), one wave:
//   scores  S^T = K Q^T on v_mfma_f32_16x16x32_bf16: rows = slots, columns
//           = query heads, so lane (q, n) holds the scores of head n for
//           slots 4q..4q+3; a LOW code c becomes the bf16 value 136 + c
//           (exact), the accumulation starts at -136 * sum(q) of the 32-dim
//           group, and the K scale multiplies the group's result;
//   softmax online in base 2, per head, rescaling only when a max grows
//           (LOW pages two at a time under one max and rescale);
//   values  HIGH: O += P V on v_mfma_f32_16x16x16_bf16 with P (split into
//           bf16 high and low parts, so p keeps ~16 bits) as the A operand
//           exactly as the score tile lies; LOW: the weights p x (V scale)
//           rounded to fp16 times the codes as exact fp16 values on
//           v_mfma_f32_16x16x16_f16, into the same accumulators.
// The next page's operands (four pages ahead for LOW pages, whose scales
// take one register) are loaded while the current one is computed.
// Each segment leaves (max, sum, unnormalised o) per head; attn_merge
// combines the partials of a (b, g).

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// D[16x16] += A[16x32] B[32x16], bf16 operands: lane l holds A[l%16][8(l/16)..+8],
// B[8(l/16)..+8][l%16], D[4(l/16)..+4][l%16].
__device__ __forceinline__ f32x4_t mfma_k32(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                 c, 0, 0, 0);
}
// D[16x16] += A[16x16] B[16x16]: lane l holds A[l%16][4(l/16)..+4], B[4(l/16)..+4][l%16].
__device__ __forceinline__ f32x4_t mfma_k16(uint2 a, uint2 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(short4_t, a), __builtin_bit_cast(short4_t, b),
                                                   c, 0, 0, 0);
}

template <int N>
__device__ __forceinline__ void load_words(const uint8_t* p, uint32_t (&w)[N]) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int k = 0; k < N / 4; ++k) {
      const uint4 x = stream_load16(p + 16 * k);
      w[4 * k] = x.x; w[4 * k + 1] = x.y; w[4 * k + 2] = x.z; w[4 * k + 3] = x.w;
    }
  } else if constexpr (N % 2 == 0) {
#pragma unroll
    for (int k = 0; k < N / 2; ++k) {
      const u32x2_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p) + k);
      w[2 * k] = x[0]; w[2 * k + 1] = x[1];
    }
  } else {
#pragma unroll
    for (int k = 0; k < N; ++k) w[k] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p) + k);
  }
}

// Raw operands of one page for one lane.
template <int D>
struct HiRaw {
  uint32_t k[4 * PageLayout<D>::NG];   // QK A operands: NG x 8 bf16
  uint32_t v[2 * PageLayout<D>::NM];   // PV B operands: NM x 4 bf16
};
template <int D>
struct LoRaw {
  uint32_t kc[PageLayout<D>::NG];      // NG x 8 int4 codes
  uint32_t vc[PageLayout<D>::NM / 2];  // 4 slots x NM/2 bytes of V code pairs
  uint32_t sc;                         // word n of the row's scales (load_lo)
};

template <int D>
__device__ __forceinline__ HiRaw<D> load_hi(const uint8_t* head, int q, int n) {
  using PL = PageLayout<D>;
  HiRaw<D> x;
  const int l = q * 16 + n;
#pragma unroll
  for (int i = 0; i < PL::NG; ++i) {
    const uint4 w = stream_load16(head + (i * 64 + l) * 16);
    x.k[4 * i] = w.x; x.k[4 * i + 1] = w.y; x.k[4 * i + 2] = w.z; x.k[4 * i + 3] = w.w;
  }
#pragma unroll
  for (int i = 0; i < PL::NM / 2; ++i) {
    const uint4 w = stream_load16(head + PL::kHiV + (i * 64 + l) * 16);
    x.v[4 * i] = w.x; x.v[4 * i + 1] = w.y; x.v[4 * i + 2] = w.z; x.v[4 * i + 3] = w.w;
  }
  return x;
}

template <int D>
__device__ __forceinline__ LoRaw<D> load_lo(const uint8_t* head, int q, int n) {
  using PL = PageLayout<D>;
  LoRaw<D> x;
  constexpr int KW = 2 * PL::NG;                 // scale words of 4 slots
  load_words(head + (q * 16 + n) * PL::NG * 4, x.kc);
  load_words(head + PL::kLoVC + (q * 16 + n) * (PL::NM / 2) * 4, x.vc);
  // Row q (slots 4q..4q+3) needs KW words of K scales and KW of V scales,
  // the same for its 16 lanes: lane n loads one of them (n < KW: K word n,
  // then V word n - KW; spare lanes repeat K word 0) and attend_page shares
  // them across the row, so a page's scales cost one 4-byte load per lane
  // and one register instead of 2 x KW per lane.
  const int off = n < KW ? PL::kLoKS + 4 * (q * KW + n)
                         : (n < 2 * KW ? PL::kLoVS + 4 * (q * KW + n - KW) : PL::kLoKS + 4 * q * KW);
  x.sc = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(head + off));
  return x;
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}
// x = hi + lo with hi = bf16(x) and lo = bf16(x - hi): 16 significant bits,
// so the weights of the p.v MFMA carry fp32-like precision (two products).
__device__ __forceinline__ void split_bf16x4(const float (&x)[4], uint2& hi, uint2& lo) {
  float r[4];
  hi = make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
  r[0] = x[0] - bf16_lo(hi.x);
  r[1] = x[1] - bf16_hi(hi.x);
  r[2] = x[2] - bf16_lo(hi.y);
  r[3] = x[3] - bf16_hi(hi.y);
  lo = make_uint2(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]));
}
// K codes widened to bf16 with an offset: the pages hold a code c as the
// offset-binary nibble c + 8, and the bf16 bit pattern 0x4300 | (c + 8) is
// the exact value 128 + c + 8 = 136 + c (bf16 spacing is 1 on [128, 256)).
// A K word holds elements 0..3 in the low nibbles of its bytes and 4..7 in
// the high nibbles, so after one mask per nibble plane each pair of elements
// is one byte permute that also inserts the 0x43 bytes; the offset is removed
// by starting the q.k accumulation at -136 * (sum of q over the group).
constexpr float kCodeOffset = 136.0f;
// bf16 pair of the nibbles in bytes e and e + 1 of a nibble plane (one
// nibble per byte); v_perm_b32 selector bytes 0-3 pick bytes of the second
// source, 4-7 bytes of the first (the constant).
template <int e>
__device__ __forceinline__ uint32_t kcodes_pair(uint32_t plane) {
  return __builtin_amdgcn_perm(0x43434343u, plane, 0x04000400u | ((e + 1) << 16) | e);
}
// V codes as exact fp16 values: the fp16 bit pattern 0x6400 | (c + 8) is
// 1024 + c + 8 (fp16 spacing is 1 on [1024, 2048)), and one packed fp16
// subtraction of 1032 leaves c exactly.  Nibbles in bytes j0 and j1 of n4
// (one per byte) as an fp16 pair; the 0x64 bytes come from the constant
// first source.
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));
template <int j0, int j1>
__device__ __forceinline__ uint32_t vcodes_pair(uint32_t n4) {
  const uint32_t w = __builtin_amdgcn_perm(0x64646464u, n4, 0x04000400u | (j1 << 16) | j0);
  const f16x2_t c = __builtin_bit_cast(f16x2_t, w) - f16x2_t{(_Float16)1032.0f, (_Float16)1032.0f};
  return __builtin_bit_cast(uint32_t, c);
}

// Per-wave attention state.  The score tile is S^T (MFMA row = slot 4q + r,
// column = query head n), so lane (q, n) holds p of head n for slots
// 4q..4q+3: the A operand of the p.v MFMA as it stands, with no transpose.
// The output tile has row = query head 4q + r and column = dim 16m + n.
template <int D, int G>
struct AttnState {
  uint32_t qa[4 * PageLayout<D>::NG];   // QK B operands: q of head n, dims 32i + 8q + 0..7
  f32x4_t acc[PageLayout<D>::NM];        // unnormalised outputs
  float m, l;                            // head n: running max (log2 units), lane-partial sum
  float kq[PageLayout<D>::NG];           // head n: -(K code offset) x sum of q over 32-dim group i
};

// Max / sum over the 64 lanes' copies of one head (lanes n, n+16, n+32,
// n+48) with gfx950's row swaps, on the VALU instead of through LDS.  With
// both operands x, v_permlane16_swap yields rows (0, 0, 2, 2) and (1, 1, 3, 3)
// of x, v_permlane32_swap rows (0, 1, 0, 1) and (2, 3, 2, 3); combining the
// pair after each swap reduces lanes l and l ^ 16, then l and l ^ 32.
__device__ __forceinline__ float head_max(float x) {
  const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
  const auto t = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
}
__device__ __forceinline__ float head_sum(float x) {
  const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(s[0]) + __uint_as_float(s[1]);
  const auto t = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(t[0]) + __uint_as_float(t[1]);
}

// Word j of the row, for every lane of the row: DPP row_newbcast:j copies
// lane j of each 16-lane row to the whole row.
template <int J>
__device__ __forceinline__ uint32_t row_word(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x150 + J, 0xF, 0xF, false);
}
// Words OFF..OFF+KW-1 of the row (DPP row_newbcast from lanes OFF..).
template <int KW, int OFF, int J = 0>
__device__ __forceinline__ void row_words(uint32_t x, uint32_t (&w)[KW]) {
  if constexpr (J < KW) {
    w[J] = row_word<OFF + J>(x);
    row_words<KW, OFF, J + 1>(x, w);
  }
}

// Scores of one page in log2 units (-inf for slots past nvalid when kMasked):
// lane (q, n) gets head n at slots 4q..4q+3.
template <int D, int G, bool kIsHi, bool kMasked, typename Raw>
__device__ __forceinline__ f32x4_t page_scores(const Raw& x, const AttnState<D, G>& st, int nvalid,
                                               float scale_log2, int q) {
  using PL = PageLayout<D>;
  f32x4_t sc = {0.0f, 0.0f, 0.0f, 0.0f};
  if constexpr (kIsHi) {
#pragma unroll
    for (int i = 0; i < PL::NG; ++i)
      sc = mfma_k32(make_uint4(x.k[4 * i], x.k[4 * i + 1], x.k[4 * i + 2], x.k[4 * i + 3]),
                    make_uint4(st.qa[4 * i], st.qa[4 * i + 1], st.qa[4 * i + 2], st.qa[4 * i + 3]), sc);
  } else {
    uint32_t ks[2 * PL::NG];                        // the row's K scale words
    row_words<2 * PL::NG, 0>(x.sc, ks);
    f32x4_t c[PL::NG];
#pragma unroll
    for (int i = 0; i < PL::NG; ++i) {
      const uint32_t lo4 = x.kc[i] & 0x0F0F0F0Fu, hi4 = (x.kc[i] >> 4) & 0x0F0F0F0Fu;   // elements 0-3, 4-7
      const f32x4_t off = {st.kq[i], st.kq[i], st.kq[i], st.kq[i]};   // removes the code offset
      c[i] = mfma_k32(make_uint4(kcodes_pair<0>(lo4), kcodes_pair<2>(lo4), kcodes_pair<0>(hi4),
                                 kcodes_pair<2>(hi4)),
                      make_uint4(st.qa[4 * i], st.qa[4 * i + 1], st.qa[4 * i + 2], st.qa[4 * i + 3]), off);
    }
#pragma unroll
    for (int i = 0; i < PL::NG; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {                 // K scale of slot 4q + r, group i
        const int hidx = r * PL::NG + i;
        sc[r] = fmaf(half_bits_to_float(ks[hidx / 2] >> (16 * (hidx % 2))), c[i][r], sc[r]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) sc[r] = (!kMasked || 4 * q + r < nvalid) ? sc[r] * scale_log2 : -INFINITY;
  return sc;
}

// Online softmax for head n given the lane's max of new scores: rescale the
// outputs and the sum only when some head's max grew.
template <int D, int G>
__device__ __forceinline__ void softmax_step(AttnState<D, G>& st, float mx, int q) {
  using PL = PageLayout<D>;
  const float mn = fmaxf(st.m, head_max(mx));
  if (__ballot(mn > st.m)) {
    const float alpha = __builtin_amdgcn_exp2f(st.m - mn);
    st.l *= alpha;
    st.m = mn;
#pragma unroll
    for (int r = 0; r < 4; ++r) {                   // output row 4q + r takes head 4q + r's factor
      const float ar = __shfl(alpha, 4 * q + r);
#pragma unroll
      for (int k = 0; k < PL::NM; ++k) st.acc[k][r] *= ar;
    }
  }
}

// fp16 pair (p0 x half H of s0, p1 x half H of s1), each product rounded
// once to fp16 (the compiler makes a v_fma_mixlo_f16 / v_fma_mixhi_f16 pair
// of the fma with a zero addend).
template <int H>
__device__ __forceinline__ uint32_t mix_pair(float p0, float p1, uint32_t s0, uint32_t s1) {
  const float a = half_bits_to_float(s0 >> (16 * H)), b = half_bits_to_float(s1 >> (16 * H));
  const f16x2_t r = {(_Float16)__builtin_fmaf(p0, a, 0.0f), (_Float16)__builtin_fmaf(p1, b, 0.0f)};
  return __builtin_bit_cast(uint32_t, r);
}

// Weights p = exp2(score - max) of one page (summed into l) and O += P V.
template <int D, int G, bool kIsHi, bool kMasked, typename Raw>
__device__ __forceinline__ void page_values(const Raw& x, AttnState<D, G>& st, const f32x4_t& sc, int nvalid,
                                            int q) {
  using PL = PageLayout<D>;
  // exp2 on v_exp_f32 directly: arguments are <= 0, and results that would
  // be fp32 subnormals (weights below 2^-126 of the running max) become 0.
  float pr[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    pr[r] = __builtin_amdgcn_exp2f(sc[r] - st.m);
    st.l += pr[r];
  }
  if constexpr (kIsHi) {
    uint2 pa_hi, pa_lo;
    split_bf16x4(pr, pa_hi, pa_lo);
#pragma unroll
    for (int mm = 0; mm < PL::NM; ++mm) {
      uint32_t v0 = x.v[2 * mm], v1 = x.v[2 * mm + 1];
      if constexpr (kMasked) {   // zero V of slots past the end (their memory is not written)
        const int t0 = 4 * q;
        v0 = (t0 + 1 < nvalid) ? v0 : (t0 < nvalid ? (v0 & 0xFFFFu) : 0u);
        v1 = (t0 + 3 < nvalid) ? v1 : (t0 + 2 < nvalid ? (v1 & 0xFFFFu) : 0u);
      }
      st.acc[mm] = mfma_k16(pa_hi, make_uint2(v0, v1), st.acc[mm]);
      st.acc[mm] = mfma_k16(pa_lo, make_uint2(v0, v1), st.acc[mm]);
    }
  } else {
    // V: the weights p x (V scale of the slot's group), rounded once to
    // fp16 (11 significant bits), times the exact fp16 codes on the fp16
    // MFMA.  Slots past the end get scale 0, so weight 0 (their scales are
    // not written); their codes are finite by construction.
    uint32_t vs[2 * PL::NG];                        // the row's V scale words: slot 4q + jj at jj*NG/2..
    row_words<2 * PL::NG, 2 * PL::NG>(x.sc, vs);
    if constexpr (kMasked) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int e = 0; e < PL::NG / 2; ++e)
          vs[jj * (PL::NG / 2) + e] = 4 * q + jj < nvalid ? vs[jj * (PL::NG / 2) + e] : 0u;
    }
#pragma unroll
    for (int i = 0; i < PL::NG; ++i) {
      // slot 4q + jj, group i: half i % 2 of word jj * NG/2 + i/2
      const int w0 = i / 2;
      const uint32_t wlo = (i & 1) ? mix_pair<1>(pr[0], pr[1], vs[w0], vs[PL::NG / 2 + w0])
                                   : mix_pair<0>(pr[0], pr[1], vs[w0], vs[PL::NG / 2 + w0]);
      const uint32_t whi = (i & 1) ? mix_pair<1>(pr[2], pr[3], vs[PL::NG + w0], vs[3 * PL::NG / 2 + w0])
                                   : mix_pair<0>(pr[2], pr[3], vs[PL::NG + w0], vs[3 * PL::NG / 2 + w0]);
      const f16x4_t wa = __builtin_bit_cast(f16x4_t, make_uint2(wlo, whi));
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        // byte jj of vc[i]: slot 4q + jj, dim 32i + n (low nibble) and 32i + 16 + n (high)
        const uint32_t n4 = (hh ? x.vc[i] >> 4 : x.vc[i]) & 0x0F0F0F0Fu;
        const f16x4_t vb = __builtin_bit_cast(f16x4_t, make_uint2(vcodes_pair<0, 1>(n4), vcodes_pair<2, 3>(n4)));
        st.acc[2 * i + hh] = __builtin_amdgcn_mfma_f32_16x16x16f16(wa, vb, st.acc[2 * i + hh], 0, 0, 0);
      }
    }
  }
}

__device__ __forceinline__ float max4(const f32x4_t& v) { return fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])); }

// One page of HIGH (kIsHi) or LOW slots; kMasked when fewer than 16 are valid.
template <int D, int G, bool kIsHi, bool kMasked, typename Raw>
__device__ __forceinline__ void attend_page(const Raw& x, AttnState<D, G>& st, int nvalid, float scale_log2, int q) {
  const f32x4_t sc = page_scores<D, G, kIsHi, kMasked>(x, st, nvalid, scale_log2, q);
  softmax_step(st, max4(sc), q);
  page_values<D, G, kIsHi, kMasked>(x, st, sc, nvalid, q);
}

// Two pages under one softmax step (one max reduction and at most one
// rescale for both): page a is full, page b holds nvb valid slots.
template <int D, int G, bool kIsHi, bool kMaskedB, typename Raw>
__device__ __forceinline__ void attend_pair(const Raw& xa, const Raw& xb, AttnState<D, G>& st, int nvb,
                                            float scale_log2, int q) {
  const f32x4_t sa = page_scores<D, G, kIsHi, false>(xa, st, kPage, scale_log2, q);
  const f32x4_t sb = page_scores<D, G, kIsHi, kMaskedB>(xb, st, nvb, scale_log2, q);
  softmax_step(st, fmaxf(max4(sa), max4(sb)), q);
  page_values<D, G, kIsHi, false>(xa, st, sa, kPage, q);
  page_values<D, G, kIsHi, kMaskedB>(xb, st, sb, nvb, q);
}

// A value the whole wave holds alike, moved to a scalar register so the
// compiler treats what depends on it as uniform.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ int wave_sum(int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}
__device__ __forceinline__ int wave_max(int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = max(x, __shfl_xor(x, off));
  return x;
}
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

__device__ __forceinline__ int window_slots(const AttnArgs& a, int n_pos) { return min(n_pos, a.cv.window); }

// Store counts of sequence `lane` for the first 64 sequences, read once per
// block: the plan, the search for a block's first sequence and the walk to
// the next sequence take them from registers instead of memory.
// A call that persists its step's entries plans with counts that differ
// from the counters: those of every sequence (n_hi, n_win, n_lo, n_x as four
// ints) are then at more[b * stride], for the sequences beyond the first 64.
struct FirstCounts {
  int n_hi, n_lo, n_win;   // 0 past the batch
  int n_x;                 // 1 when the call persists and attends an entry of the sequence
  const int32_t* more;     // null: the counters
  int stride;
};
__device__ __forceinline__ FirstCounts first_counts(const AttnArgs& a) {
  const int lane = threadIdx.x & 63;
  const int32_t* c = counters_of(a.cv, lane < a.batch ? lane : 0, a.layer);
  const int hi = c[kCntHi], lo = c[kCntLo], pos = c[kCntPos];
  FirstCounts f;
  f.n_hi = lane < a.batch ? hi : 0;
  f.n_lo = lane < a.batch ? lo : 0;
  f.n_win = lane < a.batch ? window_slots(a, pos) : 0;
  f.n_x = 0;
  f.more = nullptr;
  f.stride = 0;
  return f;
}

// ---------------------------------------------------------------------------
// the step's new entry, persisted by the attention call itself
// ---------------------------------------------------------------------------
// Outcome of the one-token append of a sequence.  word: action (bits 0-1),
// stored (bit 2), forced (3), opens a page (4), past the sequence capacity
// (5), status flags (bits 8 on); page: the page granted when the entry opens
// one, else -1.
struct EntryRecord {
  int word, slot, page, pos;
};
constexpr int kEntStored = 4, kEntForced = 8, kEntOpens = 16, kEntCapacity = 32;

// The one-token append's rules (decide, then the next slot of the entry's
// store, a new page when that slot opens one), with the pages a call opens
// granted in sequence order from the pool cursors rather than by atomics, so
// that every worker computes the same outcome for every sequence from the
// cache as it stands when the call starts.  Lane l takes sequence b = c0 + l
// of a chunk of 64 (n_hi, n_lo, pos: its counters; opened_*: the pages the
// sequences of earlier chunks open, advanced past this chunk's); s_a0 /
// s_amin: Lambda's column.
__device__ __forceinline__ EntryRecord predict_entry(const AttnArgs& a, const uint8_t* s_a0, const uint8_t* s_amin,
                                                     int b, int n_hi, int n_lo, int pos, uint32_t& opened_hi,
                                                     uint32_t& opened_lo) {
  const CacheView& cv = a.cv;
  const bool live = b < a.batch;
  const int tag = live ? (int)a.tags_new[b] : 0;
  uint32_t flags = 0u;
  bool forced = false, bad = false, opens = false, stored = false;
  int act = kDrop, store = kHi, slot = 0, page = -1;
  const bool cap = pos >= cv.max_tokens;
  if (cap) {
    flags |= PASK_FLAG_SEQ_CAPACITY;
  } else {
    act = decide(s_a0, s_amin, a.tab.n_tags, a.tab.n_sink, false, tag, pos, forced, bad);
    if (bad) flags |= PASK_FLAG_BAD_TAG;
    if (act != kDrop) {
      store = act == kHigh ? kHi : kLo;
      slot = store == kHi ? n_hi : n_lo;
      opens = slot % kPage == 0;
      stored = !opens;
    }
  }
  const unsigned long long open_hi = __ballot(live && opens && store == kHi);
  const unsigned long long open_lo = __ballot(live && opens && store == kLo);
  if (live && opens) {
    const unsigned long long m = store == kHi ? open_hi : open_lo;
    const uint32_t before = (store == kHi ? opened_hi : opened_lo) +
                            __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    const uint32_t pid = cv.status[2 + store] + before;
    const uint32_t pool = store == kHi ? (uint32_t)cv.hi_pages : (uint32_t)cv.lo_pages;
    if (pid < pool) {
      page = (int)pid;
      stored = true;
    } else {
      flags |= store == kHi ? PASK_FLAG_HI_POOL_EXHAUSTED : PASK_FLAG_LO_POOL_EXHAUSTED;
    }
  }
  opened_hi += (uint32_t)__popcll(open_hi);       // the lower sequences' page openings, in later chunks
  opened_lo += (uint32_t)__popcll(open_lo);
  EntryRecord r;
  r.word = act | (stored ? kEntStored : 0) | (forced ? kEntForced : 0) | (opens ? kEntOpens : 0) |
           (cap ? kEntCapacity : 0) | (int)(flags << 8);
  r.slot = slot;
  r.page = page;
  r.pos = pos;
  return r;
}

// First counts of a call that persists its step's entries (at most
// kFusedMaxBatch sequences, no recent window): the stores as they stand, plus
// the entry of each sequence that gets stored (n_x).  Every sequence's counts
// go to cnt[b] and its entry's outcome to ent[b]; the first 64 also stay in
// registers.
template <int kSeq>                                // the sequences ent and cnt hold (>= batch)
__device__ __forceinline__ FirstCounts first_counts_entry(const AttnArgs& a, const uint8_t* s_a0,
                                                          const uint8_t* s_amin, EntryRecord* ent, int4* cnt) {
  const int lane = threadIdx.x & 63;
  uint32_t opened_hi = 0u, opened_lo = 0u;
  FirstCounts f;
#pragma unroll
  for (int c0 = 0; c0 < kSeq; c0 += 64) {
    if (c0 > 0 && c0 >= a.batch) break;
    const int b = c0 + lane;
    const int32_t* c = counters_of(a.cv, b < a.batch ? b : 0, a.layer);
    const int hi = c[kCntHi], lo = c[kCntLo], pos = c[kCntPos];
    const EntryRecord r = predict_entry(a, s_a0, s_amin, b, hi, lo, pos, opened_hi, opened_lo);
    const bool live = b < a.batch;
    const int4 k = live ? make_int4(hi, 0, lo, (r.word & kEntStored) ? 1 : 0) : make_int4(0, 0, 0, 0);
    ent[b] = r;
    cnt[b] = k;
    if (c0 == 0) {
      f.n_hi = k.x;
      f.n_win = 0;
      f.n_lo = k.z;
      f.n_x = k.w;
    }
  }
  f.more = reinterpret_cast<const int32_t*>(cnt);
  f.stride = 4;
  return f;
}
// The merge kernels of such a call take the counts the attention kernel
// planned with from the workspace (the counters change under them: the
// merge kernel also enters the entries).
__device__ __forceinline__ FirstCounts planned_counts(const AttnArgs& a) {
  if (!a.tags_new) return first_counts(a);
  const int lane = threadIdx.x & 63;
  const int4 r = lane < a.batch ? *reinterpret_cast<const int4*>(a.ws_seq + lane * 8) : make_int4(0, 0, 0, 0);
  FirstCounts f;
  f.n_hi = r.x;
  f.n_win = r.y;
  f.n_lo = r.z;
  f.n_x = r.w;
  f.more = a.ws_seq;
  f.stride = 8;
  return f;
}

// Pages of sequence b (wave-uniform, < batch).
__device__ __forceinline__ SeqPages seq_pages(const AttnArgs& a, const FirstCounts& f, int b) {
  if (b < 64)
    return make_pages(__builtin_amdgcn_readlane(f.n_hi, b), __builtin_amdgcn_readlane(f.n_win, b),
                      __builtin_amdgcn_readlane(f.n_lo, b), __builtin_amdgcn_readlane(f.n_x, b));
  if (f.more) {
    const int4 c = *reinterpret_cast<const int4*>(f.more + (size_t)b * f.stride);
    return make_pages(uni(c.x), uni(c.y), uni(c.z), uni(c.w));
  }
  const int32_t* c = counters_of(a.cv, b, a.layer);
  return make_pages(uni(c[kCntHi]), uni(window_slots(a, c[kCntPos])), uni(c[kCntLo]));
}
// The same from a wave's copy of the counts in LDS (sequence b's at c[b] for
// b < n_lds), so that the walk over sequences keeps no registers for them.
__device__ __forceinline__ SeqPages seq_pages(const AttnArgs& a, const int4* c_lds, int n_lds, int b) {
  if (b < n_lds) {
    const int4 c = c_lds[b];
    return make_pages(uni(c.x), uni(c.y), uni(c.z), uni(c.w));
  }
  const int32_t* c = counters_of(a.cv, b, a.layer);
  return make_pages(uni(c[kCntHi]), uni(window_slots(a, c[kCntPos])), uni(c[kCntLo]));
}
// Length in units of sequence c0 + lane (c0 wave-uniform; 0 past `limit`).
__device__ __forceinline__ int lane_len(const AttnArgs& a, const FirstCounts& f, int c0, int limit) {
  const int b = c0 + (int)(threadIdx.x & 63);
  if (c0 == 0) return b < limit ? len_of(f.n_hi, f.n_win, f.n_lo, f.n_x) : 0;
  if (f.more) {
    const int4 r = b < limit ? *reinterpret_cast<const int4*>(f.more + (size_t)b * f.stride) : make_int4(0, 0, 0, 0);
    return len_of(r.x, r.y, r.z, r.w);
  }
  const int32_t* c = counters_of(a.cv, b < a.batch ? b : 0, a.layer);
  const int len = len_of(c[kCntHi], window_slots(a, c[kCntPos]), c[kCntLo]);
  return b < limit ? len : 0;
}
// The work split of a call (pask_plan.h) from its counts: every block of the
// attention, merge and distortion kernels computes the same plan.
constexpr int kWpb = PASK_ATTN_WPB;   // workers (waves) per workgroup of the weighted attention kernel
using WeightedPlan = StreamPlan<kWpb>;
constexpr int kMinPagesPerBlock = kUnitTokens / kPage;   // 8 pages: the workspace's piece size
// Calls with few segments: workers of at least 4 pages (8 and 12 measured
// slower at one Qwen3-4B-shaped sequence of 2.3k entries, 2 slower too), and
// of at least 1/PASK_SMALL_PIECES of the longest segment.
constexpr int kSmallMinPages = 4;
static_assert(PASK_SMALL_PIECES >= 1, "pieces per segment");
static_assert(PASK_ODD_WEIGHT >= 1 && PASK_ODD_WEIGHT <= 16, "odd-XCD worker weight out of range");

__device__ __forceinline__ void call_totals(const AttnArgs& a, const FirstCounts& f, long long& total, int& mx) {
  int t = 0, m = 0;
  for (int c0 = 0; c0 < a.batch; c0 += 64) {
    const int len = lane_len(a, f, c0, a.batch);
    t += uni(wave_sum(len));
    m = max(m, uni(wave_max(len)));
  }
  total = (long long)t * a.cv.n_kv_heads;
  mx = m;
}
__device__ __forceinline__ WeightedPlan stream_plan(const AttnArgs& a, const FirstCounts& f, int n_blocks) {
  long long total;
  int mx;
  call_totals(a, f, total, mx);
  return stream_plan_of<kWpb>(total, mx, a.splits, a.min_pages, n_blocks, PASK_ODD_WEIGHT);
}
__device__ __forceinline__ EvenPlan even_plan(const AttnArgs& a, const FirstCounts& f, int n_blocks) {
  long long total;
  int mx;
  call_totals(a, f, total, mx);
  return even_plan_of(total, mx, min(a.splits, PASK_SMALL_PIECES + 1), a.min_pages, n_blocks);
}
template <typename Plan>
__device__ __forceinline__ Plan make_plan(const AttnArgs& a, const FirstCounts& f, int n_blocks) {
  if constexpr (std::is_same<Plan, EvenPlan>::value) return even_plan(a, f, n_blocks);
  else return stream_plan(a, f, n_blocks);
}

// Sequence whose segments hold unit P, and the units of the sequences before it.
__device__ __forceinline__ void locate(const AttnArgs& a, const FirstCounts& f, long long P, int& b_out,
                                       int& excl_out) {
  const long long H = a.cv.n_kv_heads;
  int base = 0;
  b_out = -1;
  excl_out = 0;
  for (int c0 = 0; c0 < a.batch; c0 += 64) {
    const int len = lane_len(a, f, c0, a.batch);
    const int incl = wave_inclusive_scan(len) + base;
    const int excl = incl - len;
    const bool hit = len > 0 && (long long)excl * H <= P && P < (long long)incl * H;
    const unsigned long long m = __ballot(hit);
    if (m) {
      const int src = __ffsll((long long)m) - 1;
      b_out = uni(c0 + src);
      excl_out = uni(__shfl(excl, src));
      return;
    }
    base = uni(__shfl(incl, 63));
  }
}

// Stream pages [p0, p1) of one store of (b, g), loading page p+1 while
// computing page p.  The page ids come from the block table kIdChunk at a time, one per
// lane, and are read with readlane, so a page's loads depend on no other
// memory access.  The prefetches are unconditional (past the end they read
// the pool's first head slot, which every worker reads there, so they hit in
// the caches; the non-temporal page loads would not hit on a re-read of the
// run's last page): the loop body is straight-line code and the compiler
// waits only for the current page's loads.  KV head g of a page
// sits in head slot (g + page) mod n_kv_heads, which spreads one head's data
// over DRAM channels.
constexpr int kIdChunk = 128;

// kWindow: the pages are a recent window, consecutive pool pages from id0 on
// (bt unused).
// `prologue` runs once, after the first block-table loads are issued and
// before the first page is loaded, so work that waits for earlier loads (the
// LOW code offsets wait for q) overlaps the block-table latency.
struct NoPrologue {
  __device__ __forceinline__ void operator()() const {}
};
template <int D, int G, bool kIsHi, bool kWindow = false, typename Prologue = NoPrologue>
__device__ __forceinline__ void run_pages(const uint8_t* pool, size_t page_bytes, int head_bytes, int n_heads,
                                          const int32_t* bt, int id0, int p0, int p1, int n_slots, int g,
                                          AttnState<D, G>& st, float scale_log2, int q, int n,
                                          Prologue prologue = Prologue()) {
  using Raw = typename std::conditional<kIsHi, HiRaw<D>, LoRaw<D>>::type;
  const int lane = threadIdx.x & 63;
  auto load = [&](int page, bool real) -> Raw {
    const uint8_t* head = pool + (size_t)page * page_bytes + (size_t)((g + page) % n_heads) * head_bytes;
    head = real ? head : pool;   // past the end: the pool's first head slot, read by every worker
    if constexpr (kIsHi) return load_hi<D>(head, q, n);
    else return load_lo<D>(head, q, n);
  };
  auto attend = [&](const Raw& r, int p) {
    const int nvalid = min(kPage, n_slots - p * kPage);
    if (nvalid == kPage) attend_page<D, G, kIsHi, false>(r, st, nvalid, scale_log2, q);
    else attend_page<D, G, kIsHi, true>(r, st, nvalid, scale_log2, q);
  };
  for (int c = p0; c < p1; c += kIdChunk) {
    const int cn = min(kIdChunk, p1 - c);
    const int ids0 = kWindow ? id0 + c + min(lane, cn - 1) : bt[c + min(lane, cn - 1)];
    const int ids1 = kWindow ? id0 + c + min(64 + lane, cn - 1) : bt[c + min(64 + lane, cn - 1)];
    if (c == p0) prologue();
    auto id = [&](int i) -> int {   // i: wave-uniform, < cn
      return i < 64 ? __builtin_amdgcn_readlane(ids0, i) : __builtin_amdgcn_readlane(ids1, i - 64);
    };
    auto ld = [&](int i) -> Raw { return load(id(min(i, cn - 1)), i < cn); };
    if constexpr (kIsHi) {
      // Two page buffers used in turn (unrolled by two), so no buffer is
      // copied while its loads are in flight.
      Raw x0 = ld(0);
      for (int i = 0; i < cn; i += 2) {
        const Raw x1 = ld(i + 1);
        attend(x0, c + i);
        x0 = ld(i + 2);
        if (i + 1 < cn) attend(x1, c + i + 1);
      }
    } else {
      // LOW pages (2 + 2 KiB of codes and 2 x 128 B of scales per head at
      // D 128) in pairs under one softmax step; six buffers in turn keep
      // four pages in flight while a pair is computed.
      auto pair = [&](const Raw& xa, const Raw& xb, int i) {   // pages c+i and c+i+1 (when < cn)
        if (i + 1 < cn) {                          // page c+i is then not the store's last: full
          const int nvb = min(kPage, n_slots - (c + i + 1) * kPage);
          if (nvb == kPage) attend_pair<D, G, false, false>(xa, xb, st, nvb, scale_log2, q);
          else attend_pair<D, G, false, true>(xa, xb, st, nvb, scale_log2, q);
        } else {
          attend(xa, c + i);
        }
      };
      Raw x0 = ld(0), x1 = ld(1), x2 = ld(2), x3 = ld(3);
      for (int i = 0; i < cn; i += 6) {
        const Raw x4 = ld(i + 4), x5 = ld(i + 5);
        pair(x0, x1, i);
        x0 = ld(i + 6);
        x1 = ld(i + 7);
        if (i + 2 < cn) pair(x2, x3, i + 2);
        x2 = ld(i + 8);
        x3 = ld(i + 9);
        if (i + 4 < cn) pair(x4, x5, i + 4);
      }
    }
  }
}

// The step's entry's K and V rows, fetched at the start of its segment as
// D/64 words per lane (the rows' 4D bytes spread over the wave: lane l holds
// words l D/64 .. of [K; V]), so that only D/64 registers stay live while the
// pages stream; read back by lane shuffles.
template <int D>
struct EntryRows {
  static constexpr int kW = D / 64;            // words per lane
  uint32_t w[kW];
  // Word j (< D) of [K; V] (two bf16 per word), for any lane's j.
  __device__ __forceinline__ uint32_t word(int j) const {
    if constexpr (kW == 1) {
      return (uint32_t)__shfl((int)w[0], j);
    } else {
      const uint32_t a0 = (uint32_t)__shfl((int)w[0], j / kW), a1 = (uint32_t)__shfl((int)w[1], j / kW);
      return (j % kW) ? a1 : a0;
    }
  }
  // bf16 bits of element e (< 2D) of [K; V].
  __device__ __forceinline__ uint32_t elem(int e) const { return (word(e >> 1) >> (16 * (e & 1))) & 0xFFFFu; }
};

// The step's entry of (b, g), stored per record r: KV head g of it is
// written into slot r.slot of its page, exactly as the one-token append
// writes it (bf16 for HIGH; for LOW the same codes and scales: the group's
// absmax, quant_scale, and the code rule, here through codes8, which is
// quant_code wherever it counts).  A LOW entry's operands, as slot 0 of a
// page in the attention's layout, are left in x.
template <int D>
__device__ __forceinline__ void prepare_entry(const AttnArgs& a, int b, int g, const EntryRecord& r, int q, int n,
                                              LoRaw<D>& x, const EntryRows<D>& rows) {
  using PL = PageLayout<D>;
  const CacheView& cv = a.cv;
  const int H = cv.n_kv_heads, lane = threadIdx.x & 63;
  const int act = r.word & 3;
  const int store = act == kHigh ? kHi : kLo;
  const int t = r.slot % kPage, qq = t / 4, jj = t % 4;
  const int page = r.page >= 0 ? r.page : block_table_of(cv, b, a.layer, store)[r.slot / kPage];
  if (act == kHigh) {
    uint8_t* hd = cv.hi_pool + (size_t)page * cv.hi_page_bytes + (size_t)((g + page) % H) * PL::kHiHead;
#pragma unroll
    for (int i = 0; i < PL::NG; ++i) {           // K chunk (i, q) of the slot: dims 32i + 8q .. +8
      const int w0 = 16 * i + 4 * q;
      const uint4 c = make_uint4(rows.word(w0), rows.word(w0 + 1), rows.word(w0 + 2), rows.word(w0 + 3));
      if (n == t) *reinterpret_cast<uint4*>(hd + (size_t)(i * 64 + q * 16 + t) * 16) = c;
    }
    uint16_t* vd = reinterpret_cast<uint16_t*>(hd + PL::kHiV);
#pragma unroll
    for (int k = 0; k < D / 64; ++k) {           // V dim d = 16m + dd
      const int d = lane + 64 * k, m = d / 16, dd = d % 16;
      vd[(((m >> 1) * 64 + qq * 16 + dd) * 2 + (m & 1)) * 4 + jj] = (uint16_t)rows.elem(D + d);
    }
    return;
  }
  uint8_t* hb = cv.lo_pool + (size_t)page * cv.lo_page_bytes + (size_t)((g + page) % H) * PL::kLoHead;
  constexpr int NG = PL::NG;
  uint32_t sk[NG], sv[NG];
#pragma unroll
  for (int i = 0; i < NG; ++i) {                 // K group i: lane (q, n) holds elements 8q .. 8q + 7
    const int w0 = 16 * i + 4 * q;
    const uint4 w = make_uint4(rows.word(w0), rows.word(w0 + 1), rows.word(w0 + 2), rows.word(w0 + 3));
    const float f[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                        bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
    float am = fabsf(f[0]);
#pragma unroll
    for (int u = 1; u < 8; ++u) am = fmaxf(am, fabsf(f[u]));
    am = fmaxf(am, __shfl_xor(am, 16));          // the group's absmax over its four lanes
    am = fmaxf(am, __shfl_xor(am, 32));
    float sc, inv;
    sk[i] = quant_scale(am, sc, inv);
    const uint32_t kw = k_word(codes8(w, sc, inv));
    if (n == t) *reinterpret_cast<uint32_t*>(hb + ((q * 16 + t) * NG + i) * 4) = kw;
    x.kc[i] = n == 0 ? kw : 0x88888888u;         // other slots: code 0 (masked)
  }
#pragma unroll
  for (int i = 0; i < NG; ++i) {                 // V group i: lane (q, n) holds dims n, n + 16
    const float v0 = __uint_as_float(rows.elem(D + 32 * i + n) << 16);
    const float v1 = __uint_as_float(rows.elem(D + 32 * i + 16 + n) << 16);
    float am = fmaxf(fabsf(v0), fabsf(v1));
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) am = fmaxf(am, __shfl_xor(am, off));
    float sc, inv;
    sv[i] = quant_scale(am, sc, inv);
    const uint32_t byte = (uint32_t)(quant_code(v0, sc, inv) + 8) | ((uint32_t)(quant_code(v1, sc, inv) + 8) << 4);
    if (q == 0) hb[PL::kLoVC + ((qq * 16 + n) * (PL::NM / 2) + i) * 4 + jj] = (uint8_t)byte;
    x.vc[i] = q == 0 ? (0x88888800u | byte) : 0x88888888u;
  }
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      *reinterpret_cast<uint16_t*>(hb + PL::kLoKS + (t * NG + i) * 2) = (uint16_t)sk[i];
      *reinterpret_cast<uint16_t*>(hb + PL::kLoVS + (t * NG + i) * 2) = (uint16_t)sv[i];
    }
  }
  // The row's scale words as load_lo hands them out: lane n < KW holds K word
  // n, KW <= n < 2 KW V word n - KW; word w holds halves 2w, 2w + 1 of the
  // row's [4 slots][NG] scales, and only slot 0 of row 0 is the entry.
  constexpr int KW = 2 * NG;
  const bool is_v = n >= KW && n < 2 * KW;
  const int wd = n < KW ? n : (is_v ? n - KW : 0);
  uint32_t lo16 = 0u, hi16 = 0u;
#pragma unroll
  for (int i = 0; i < NG; ++i) {
    const uint32_t v = is_v ? sv[i] : sk[i];
    if (2 * wd == i) lo16 = v;
    if (2 * wd + 1 == i) hi16 = v;
  }
  x.sc = q == 0 ? (lo16 | (hi16 << 16)) : 0u;
}

// The entry attended as a page holding just that slot (slot 0): HIGH from
// its bf16 rows, LOW from the operands prepare_entry made; `offsets`
// computes the LOW code offsets of q.
template <int D, int G, typename Offsets>
__device__ __forceinline__ void attend_entry(const AttnArgs& a, const EntryRecord& r, AttnState<D, G>& st, int q,
                                             int n, Offsets offsets, const LoRaw<D>& xl, const EntryRows<D>& rows) {
  using PL = PageLayout<D>;
  if ((r.word & 3) == kHigh) {
    HiRaw<D> x;
#pragma unroll
    for (int i = 0; i < PL::NG; ++i) {           // K dims 32i + 8q .. +8 of slot 0: lanes (q, 0)
      const int w0 = 16 * i + 4 * q;
      const uint4 w = make_uint4(rows.word(w0), rows.word(w0 + 1), rows.word(w0 + 2), rows.word(w0 + 3));
      x.k[4 * i] = n == 0 ? w.x : 0u;
      x.k[4 * i + 1] = n == 0 ? w.y : 0u;
      x.k[4 * i + 2] = n == 0 ? w.z : 0u;
      x.k[4 * i + 3] = n == 0 ? w.w : 0u;
    }
#pragma unroll
    for (int m = 0; m < PL::NM; ++m) {           // V dim 16m + n of slot 0: lanes (0, n)
      const uint32_t e = rows.elem(D + 16 * m + n);
      x.v[2 * m] = q == 0 ? e : 0u;
      x.v[2 * m + 1] = 0u;
    }
    attend_page<D, G, true, true>(x, st, 1, a.scale_log2, q);
    return;
  }
  offsets();
  attend_page<D, G, false, true>(xl, st, 1, a.scale_log2, q);
}

// Pages [j0, j1) of (b, g) (HIGH store, recent window, LOW store): this
// piece's partial of (b, g), combined with the others by attn_merge.
template <int D, int G, typename Plan>
__device__ __forceinline__ void attend_segment(const AttnArgs& a, int w, int b, int g, int j0, int j1, const SeqPages& sp,
                                               long long seg0, const Plan& plan, int q, int n,
                                               const EntryRecord* ent) {
  using PL = PageLayout<D>;
  const CacheView& cv = a.cv;
  const int H = cv.n_kv_heads;
  EntryRows<D> rows;                               // the step's entry, attended last: its rows now
  if (j1 > sp.np_l) {
    const uint32_t* src = reinterpret_cast<const uint32_t*>(
        ((threadIdx.x & 63) < 32 ? a.k_new : a.v_new) + ((size_t)b * H + g) * D);
    const int l = threadIdx.x & 31;                // [K; V]: lanes 0-31 K, 32-63 V
#pragma unroll
    for (int k = 0; k < EntryRows<D>::kW; ++k) rows.w[k] = src[l * EntryRows<D>::kW + k];
  }
  const size_t bh0 = (size_t)b * a.n_q_heads + (size_t)g * G;
  AttnState<D, G> st;
  // Columns n >= G repeat head G-1 (finite scores; their results are unused).
  const uint16_t* qh = a.q + (bh0 + min(n, G - 1)) * D + 8 * q;
#pragma unroll
  for (int i = 0; i < PL::NG; ++i) {
    const uint4 w = *reinterpret_cast<const uint4*>(qh + 32 * i);
    st.qa[4 * i] = w.x; st.qa[4 * i + 1] = w.y; st.qa[4 * i + 2] = w.z; st.qa[4 * i + 3] = w.w;
  }
#pragma unroll
  for (int k = 0; k < PL::NM; ++k) st.acc[k] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  st.m = -INFINITY;
  st.l = 0.0f;
  // -offset x sum of q over group i (head n), for LOW pages only: computed in
  // the LOW run's prologue, after its block-table loads are issued.
  auto code_offsets = [&]() {
#pragma unroll
    for (int i = 0; i < PL::NG; ++i) {
      float part = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) part += bf16_lo(st.qa[4 * i + e]) + bf16_hi(st.qa[4 * i + e]);
      st.kq[i] = -kCodeOffset * head_sum(part);
    }
  };
  if (j0 < sp.np_hi)
    run_pages<D, G, true>(cv.hi_pool, cv.hi_page_bytes, PL::kHiHead, H, block_table_of(cv, b, a.layer, kHi), 0, j0,
                          min(j1, sp.np_hi), sp.n_hi, g, st, a.scale_log2, q, n);
  if (j0 < sp.np_w && j1 > sp.np_hi)             // the recent window's pages
    run_pages<D, G, true, true>(cv.hi_pool, cv.hi_page_bytes, PL::kHiHead, H, nullptr,
                                (b * cv.n_layers + a.layer) * cv.ring_pp, max(j0, sp.np_hi) - sp.np_hi,
                                min(j1, sp.np_w) - sp.np_hi, sp.n_win, g, st, a.scale_log2, q, n);
  const int l0 = max(j0, sp.np_w), l1 = min(j1, sp.np_l);   // the LOW store's pages of the range
  if (l0 < l1)
    run_pages<D, G, false>(cv.lo_pool, cv.lo_page_bytes, PL::kLoHead, H, block_table_of(cv, b, a.layer, kLo), 0,
                           l0 - sp.np_w, l1 - sp.np_w, sp.n_lo, g, st, a.scale_log2, q, n, code_offsets);
  if (j1 > sp.np_l) {                            // the step's entry (only when the call persists it)
    const EntryRecord er = ent[b];
    LoRaw<D> xl;
    prepare_entry<D>(a, b, g, er, q, n, xl, rows);
    attend_entry<D, G>(a, er, st, q, n, code_offsets, xl, rows);
  }
  // Partial of piece `slot` of (b, g): rows of G4 = max(G, 4) query heads,
  // stored as float4s of 4 heads at one dim (index ((q*NM + k)*16 + n)*4 + r
  // for head 4q + r, dim 16k + n): each store instruction writes 256
  // contiguous bytes, and the (max, sum) pairs of the G4 heads sit together.
  // Rows past G hold finite values that are never read into an output.
  constexpr int G4 = G > 4 ? G : 4;
  const float l_n = head_sum(st.l);              // head n, over all slots
  const int slot = (int)(w - plan.block_of(seg0));   // < a.splits by the choice of range sizes
  if (slot < 0 || slot >= a.splits) {            // never expected: report it, write nothing
    if ((threadIdx.x & 63) == 0) atomicOr(a.cv.status, (uint32_t)PASK_FLAG_WORKSPACE);
    return;
  }
  const size_t blk = ((size_t)b * H + g) * a.splits + slot;
  if (4 * q < G4) {
    float* o = a.ws_o + blk * (G4 * D);
#pragma unroll
    for (int k = 0; k < PL::NM; ++k)
      *reinterpret_cast<float4*>(o + ((q * PL::NM + k) * 16 + n) * 4) =
          make_float4(st.acc[k][0], st.acc[k][1], st.acc[k][2], st.acc[k][3]);
  }
  if (q == 0 && n < G4) *reinterpret_cast<float2*>(a.ws_ml + (blk * G4 + n) * 2) = make_float2(st.m, l_n);
}

// kWeighted: workgroups of kWpb worker waves with the per-XCD weighted
// ranges (StreamPlan); else one single-wave workgroup per worker with equal
// ranges (EvenPlan).
template <int D, int G, bool kWeighted>
__global__ __launch_bounds__(64 * (kWeighted ? kWpb : 1), 2) void attn_kernel(AttnArgs a) {
  using Plan = typename std::conditional<kWeighted, WeightedPlan, EvenPlan>::type;
  constexpr int kWaves = kWeighted ? kWpb : 1;   // workers per workgroup
  const int lane = threadIdx.x & 63;
  const int w = uni(blockIdx.x * kWaves + (int)(threadIdx.x >> 6));
  const int q = lane >> 4, n = lane & 15;
  const int H = a.cv.n_kv_heads;
  // A call that persists its step's entry: Lambda's column and every
  // sequence's entry outcome, one copy per wave (no barrier).
  constexpr int kSeq = kWeighted ? kFusedMaxBatch : 64;   // the equal-range plan takes at most 64 segments
  __shared__ uint8_t s_tab[kWaves][128];
  __shared__ EntryRecord s_ent[kWaves][kSeq];
  __shared__ int4 s_cnt[kWaves][kSeq];
  const int wv = (int)(threadIdx.x >> 6);
  FirstCounts f;
  if (a.tags_new) {
    s_tab[wv][lane] = a.tab.a0[lane];
    s_tab[wv][64 + lane] = a.tab.amin[lane];
    f = first_counts_entry<kSeq>(a, &s_tab[wv][0], &s_tab[wv][64], &s_ent[wv][0], &s_cnt[wv][0]);
    if (w == 0) {                                // the merge kernel's copy
      for (int b = lane; b < a.batch; b += 64) {
        int4* rec = reinterpret_cast<int4*>(a.ws_seq + b * 8);
        const EntryRecord r = s_ent[wv][b];
        rec[0] = s_cnt[wv][b];
        rec[1] = make_int4(r.word, r.slot, r.page, r.pos);
      }
    }
  } else {
    f = first_counts(a);
    s_cnt[wv][lane] = make_int4(f.n_hi, f.n_win, f.n_lo, 0);
  }
  const int n_lds = a.tags_new ? a.batch : 64;   // sequences whose counts the wave holds in LDS
  const Plan plan = make_plan<Plan>(a, f, a.attn_blocks);
  const long long start = plan.start_of(w);
  if (start >= plan.total) return;
  const long long end = plan.end_of(w);
  int b, excl;
  locate(a, f, start, b, excl);
  if (b < 0) return;
  SeqPages sp = seq_pages(a, &s_cnt[wv][0], n_lds, b);
  const long long rel = start - (long long)excl * H;
  int g = (int)udiv(rel, sp.len);
  int j0 = first_page_at(sp, (int)(rel - (long long)g * sp.len));
  while (true) {
    const long long seg0 = (long long)excl * H + (long long)g * sp.len;
    if (seg0 >= end) return;
    const int j1 = end - seg0 >= sp.len ? sp.np : first_page_at(sp, (int)(end - seg0));
    if (j0 < j1) attend_segment<D, G, Plan>(a, w, b, g, j0, j1, sp, seg0, plan, q, n, &s_ent[wv][0]);
    if (j1 < sp.np) return;
    j0 = 0;
    if (++g == H) {                              // next sequence that holds any page
      g = 0;
      excl += sp.len;
      do {
        if (++b >= a.batch) return;
        sp = seq_pages(a, &s_cnt[wv][0], n_lds, b);
      } while (sp.len == 0);
    }
  }
}

// Online merge of the partials of one (sequence, KV head) by thread t of a
// merge block: float4 position t of the partial rows, i.e. heads 4q..4q+3 at
// one dim, with the running (max, sum) of those 4 heads.
template <int D, int G>
constexpr int merge_threads() { return (G > 4 ? G : 4) * D / 4; }

template <int D, int G, int kB = 8>
struct PieceMerge {
  static constexpr int G4 = G > 4 ? G : 4;
  static constexpr int kBatch = kB;              // pieces whose loads are issued together
  float4 v[kBatch], mla[kBatch], mlb[kBatch];
  float acc[4], M[4], L[4];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      acc[r] = 0.0f;
      M[r] = -INFINITY;
      L[r] = 0.0f;
    }
  }
  // Loads pieces p0, p0 + stride, ... of the (b, g) whose first partial
  // block is blk0; past `last` the last piece is repeated (fold skips it).
  __device__ __forceinline__ void load(const AttnArgs& a, size_t blk0, int t, int q, int p0, int last,
                                       int stride = 1) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const size_t pb = blk0 + min(p0 + stride * u, last);
      const float* ml = a.ws_ml + pb * G4 * 2 + 8 * q;
      v[u] = *reinterpret_cast<const float4*>(a.ws_o + pb * (G4 * D) + t * 4);
      mla[u] = *reinterpret_cast<const float4*>(ml);       // (m, l) of heads 4q, 4q+1
      mlb[u] = *reinterpret_cast<const float4*>(ml + 4);   // (m, l) of heads 4q+2, 4q+3
    }
  }
  // Merges the first n (<= kBatch) loaded pieces.
  __device__ __forceinline__ void fold(int n) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (u < n) {
        const float vv[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
        const float mlv[8] = {mla[u].x, mla[u].y, mla[u].z, mla[u].w, mlb[u].x, mlb[u].y, mlb[u].z, mlb[u].w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float mp = mlv[2 * r], lp = mlv[2 * r + 1];
          const float mn = fmaxf(M[r], mp);
          const float alpha = exp2f(M[r] - mn), wgt = exp2f(mp - mn);
          L[r] = L[r] * alpha + wgt * lp;
          acc[r] = acc[r] * alpha + wgt * vv[r];
          M[r] = mn;
        }
      }
    }
  }
};

// Pieces of segment (b, g) in the stream-K decomposition (sp: pages of b,
// excl: units of the sequences before b; sp.np > 0).
template <typename Plan>
__device__ __forceinline__ int pieces_of(const Plan& plan, const SeqPages& sp, int excl, int g, int H) {
  return n_pieces(plan, sp, (long long)excl * H + (long long)g * sp.len);
}
// Units of the sequences before b (wave-uniform).
__device__ __forceinline__ int units_before(const AttnArgs& a, const FirstCounts& f, int b) {
  int excl = 0;
  for (int c0 = 0; c0 < b; c0 += 64) excl += uni(wave_sum(lane_len(a, f, c0, b)));
  return excl;
}

// The step's entries of a call that persists them, entered into the cache
// after the attention kernel has planned, written and attended them (one
// wave, lane b = sequence b): counters, index lists, the block table entry
// of an opened page, the pool cursors (one page per opening entry, granted or
// not, as the one-token append counts them) and the status flags.
__device__ __forceinline__ void enter_entries(const AttnArgs& a) {
  const CacheView& cv = a.cv;
  const int lane = threadIdx.x & 63;
  uint32_t flags = 0u, opened_hi = 0u, opened_lo = 0u;
  for (int c0 = 0; c0 < a.batch; c0 += 64) {
    const int b = c0 + lane;
    const bool live = b < a.batch;
    const int4 r = live ? *reinterpret_cast<const int4*>(a.ws_seq + b * 8 + 4) : make_int4(0, 0, 0, 0);
    const int word = r.x, slot = r.y, page = r.z, pos = r.w;
    const int act = word & 3, store = act == kHigh ? kHi : kLo;
    const bool opens = (word & kEntOpens) != 0;
    if (live) {
      int32_t* cnt = counters_of(cv, b, a.layer);
      if (word & kEntCapacity) {
        cnt[kCntLost] += 1;
      } else {
        if (act == kDrop) {
          cnt[kCntDrop] += 1;
        } else if (!(word & kEntStored)) {       // no page left in its pool
          cnt[kCntLost] += 1;
        } else {
          if (opens) block_table_of(cv, b, a.layer, store)[slot / kPage] = page;
          index_list_of(cv, b, a.layer, store)[slot] = pos;
          cnt[store] = slot + 1;
          if (word & kEntForced) cnt[kCntForced] += 1;
        }
        cnt[kCntPos] = pos + 1;
      }
      flags |= (uint32_t)word >> 8;
    }
    opened_hi += (uint32_t)__popcll(__ballot(live && opens && store == kHi));
    opened_lo += (uint32_t)__popcll(__ballot(live && opens && store == kLo));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) flags |= (uint32_t)__shfl_xor((int)flags, off);
  if (lane == 0) {
    if (opened_hi) atomicAdd(&cv.status[2], opened_hi);
    if (opened_lo) atomicAdd(&cv.status[3], opened_lo);
    if (flags) atomicOr(cv.status, flags);
  }
}

// One (sequence, KV head): combine the partials of its pieces (one or more)
// into the bf16 outputs and log-sum-exps of its G query heads; zero output
// and -inf for an empty history.  Thread t merges float4 position t of the
// partial rows; the normalised rows are staged in LDS and written as
// contiguous 16-byte pieces.
template <int D, int G>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {   // merge_threads <= 256
  constexpr int NM = D / 16;
  static_assert(merge_threads<D, G>() % 64 == 0 && merge_threads<D, G>() <= 256, "merge block size");
  __shared__ __align__(16) uint16_t s_out[G][D];
  const int t = threadIdx.x;
  const int H = a.cv.n_kv_heads;
  if (a.tags_new && blockIdx.x == gridDim.x - 1) {   // the extra block: the step's entries
    if (t < 64) enter_entries(a);
    return;
  }
  const int b = uni(blockIdx.x / H), g = uni(blockIdx.x % H);
  const size_t row0 = (size_t)b * a.n_q_heads + (size_t)g * G;   // first query head row
  const size_t blk0 = ((size_t)b * H + g) * a.splits;
  const int q = t / (NM * 16), k = (t / 16) % NM, n = t % 16;
  PieceMerge<D, G> pm;
  // The first pieces are loaded before the piece count is known (slots
  // below `splits` are in bounds; those past the count are skipped), so their
  // latency overlaps that of the counters the count comes from.
  pm.load(a, blk0, t, q, 0, a.splits - 1);
  const FirstCounts f = planned_counts(a);
  const SeqPages sp = seq_pages(a, f, b);
  if (sp.np == 0) {
    for (int i = t; i < G * D; i += merge_threads<D, G>()) a.out[row0 * D + i] = 0;
    if (a.lse && t < G) a.lse[row0 + t] = -INFINITY;
    return;
  }
  const WeightedPlan plan = stream_plan(a, f, a.attn_blocks);
  const int nparts = pieces_of(plan, sp, units_before(a, f, b), g, H);
  pm.init();
  for (int p0 = 0; p0 < nparts; p0 += PieceMerge<D, G>::kBatch) {
    if (p0 > 0) pm.load(a, blk0, t, q, p0, nparts - 1);
    pm.fold(nparts - p0);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int h = 4 * q + r;
    if (h < G) {
      s_out[h][16 * k + n] = f32_to_bf16_rne_dev(pm.acc[r] / pm.L[r]);
      if (a.lse && k == 0 && n == 0) a.lse[row0 + h] = (pm.M[r] + log2f(pm.L[r])) * 0.69314718055994530942f;
    }
  }
  __syncthreads();
  // G rows of D bf16 are contiguous in the output: 16-byte pieces.
  const uint4* src = reinterpret_cast<const uint4*>(&s_out[0][0]);
  uint4* dst = reinterpret_cast<uint4*>(a.out + row0 * D);
  for (int i = t; i < G * D / 8; i += merge_threads<D, G>()) dst[i] = src[i];
}

// The same merge for calls with few segments, whose segments hold many
// pieces: the merge of one segment is spread over NM * G4 / 4 single-wave
// blocks (one per 16 float4 positions of the partial rows: query heads
// 4q..4q+3 at dims 16k..16k+15), so the pieces' bytes are read by many CUs.
// Lane 16j + n merges position n of the block over the pieces p = j (mod 4);
// the four lane groups are then combined across lanes.
constexpr int kSlicedBatch = 12;                 // pieces per lane group and round
template <int D, int G>
__global__ __launch_bounds__(64) void attn_merge_sliced_kernel(AttnArgs a) {
  constexpr int NM = D / 16, X = merge_threads<D, G>() / 16;
  const int lane = threadIdx.x, j = lane >> 4, n = lane & 15;
  const int H = a.cv.n_kv_heads;
  if (a.tags_new && blockIdx.x == gridDim.x - 1) {   // the extra block: the step's entries
    enter_entries(a);
    return;
  }
  const int seg = uni(blockIdx.x / X), x = uni(blockIdx.x % X);
  const int b = seg / H, g = seg % H;
  const int q = x / NM, k = x % NM, t = 16 * x + n;
  const size_t row0 = (size_t)b * a.n_q_heads + (size_t)g * G;
  const size_t blk0 = (size_t)seg * a.splits;
  PieceMerge<D, G, kSlicedBatch> pm;
  constexpr int kB = kSlicedBatch;
  // Before the piece count is known: slots up to the most a segment can have
  // (the ranges' 1/PASK_SMALL_PIECES floor), not the workspace's last, so the
  // loads past the count re-read one slot instead of stale partials.
  pm.load(a, blk0, t, q, j, min(a.splits, PASK_SMALL_PIECES + 1) - 1, 4);
  const FirstCounts f = planned_counts(a);
  const SeqPages sp = seq_pages(a, f, b);
  if (sp.np == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (j == 0 && 4 * q + r < G) a.out[(row0 + 4 * q + r) * D + 16 * k + n] = 0;
    if (a.lse && j == 0 && k == 0 && n < 4 && 4 * q + n < G) a.lse[row0 + 4 * q + n] = -INFINITY;
    return;
  }
  const EvenPlan plan = even_plan(a, f, a.attn_blocks);
  const int nparts = pieces_of(plan, sp, units_before(a, f, b), g, H);
  pm.init();
  for (int p0 = 0; p0 < nparts; p0 += 4 * kB) {
    const int first = p0 + j;
    if (p0 > 0) pm.load(a, blk0, t, q, first, nparts - 1, 4);
    pm.fold(first < nparts ? (nparts - 1 - first) / 4 + 1 : 0);
  }
#pragma unroll
  for (int off = 16; off <= 32; off *= 2) {      // lanes n, n+16, n+32, n+48
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float m2 = __shfl_xor(pm.M[r], off), l2 = __shfl_xor(pm.L[r], off), v2 = __shfl_xor(pm.acc[r], off);
      if (m2 != -INFINITY) {
        const float mn = fmaxf(pm.M[r], m2);
        const float alpha = exp2f(pm.M[r] - mn), wgt = exp2f(m2 - mn);
        pm.L[r] = pm.L[r] * alpha + wgt * l2;
        pm.acc[r] = pm.acc[r] * alpha + wgt * v2;
        pm.M[r] = mn;
      }
    }
  }
  if (j == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = 4 * q + r;
      if (h < G) {
        a.out[(row0 + h) * D + 16 * k + n] = f32_to_bf16_rne_dev(pm.acc[r] / pm.L[r]);
        if (a.lse && k == 0 && n == 0) a.lse[row0 + h] = (pm.M[r] + log2f(pm.L[r])) * 0.69314718055994530942f;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// attention-output distortion (Eq. 4)
// ---------------------------------------------------------------------------

// Normalised fp32 outputs of heads 4q..4q+3 at thread t's dim for (b, g) in
// the reference (or_) and the intervened (oi) cache: both sets of partials
// loaded before either is merged, so their latencies overlap; 0 for an
// empty history.
template <int D, int G>
__device__ __forceinline__ void merged_pair(const AttnArgs& ref, const WeightedPlan& pr, const SeqPages& sr, int er,
                                            const AttnArgs& itv, const WeightedPlan& pi, const SeqPages& si, int ei,
                                            int b, int g, int t, int q, float (&or_)[4], float (&oi)[4]) {
  constexpr int kB = 4;                          // pieces per batch and cache: both in flight, no spills
  const int H = ref.cv.n_kv_heads;
  const int nr = sr.np ? pieces_of(pr, sr, er, g, H) : 0, ni = si.np ? pieces_of(pi, si, ei, g, H) : 0;
  const size_t blk0 = ((size_t)b * H + g);
  PieceMerge<D, G, kB> mr, mi;
  mr.init();
  mi.init();
  for (int p0 = 0; p0 < max(nr, ni); p0 += kB) {
    if (p0 < nr) mr.load(ref, blk0 * ref.splits, t, q, p0, nr - 1);
    if (p0 < ni) mi.load(itv, blk0 * itv.splits, t, q, p0, ni - 1);
    if (p0 < nr) mr.fold(nr - p0);
    if (p0 < ni) mi.fold(ni - p0);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    or_[r] = nr ? mr.acc[r] / mr.L[r] : 0.0f;
    oi[r] = ni ? mi.acc[r] / mi.L[r] : 0.0f;
  }
}

__device__ __forceinline__ float wave_sum_f(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// KV heads a distortion block handles at once: that many merge groups of
// merge_threads threads, at most 512 threads (256 VGPRs per thread).
template <int D, int G>
constexpr int distortion_heads() { return 512 / merge_threads<D, G>() < 8 ? 512 / merge_threads<D, G>() : 8; }

// One block per sequence b: for every KV head g (distortion_heads of them at
// a time, one merge group each), the outputs of its G query heads over the
// reference cache (partials of `ref`) and the intervened one (`itv`) in fp32,
// the squared L2 distance of each head's rows summed over the D dims, and the
// maximum over all query heads (Eq. 4, inside the expectation), added to
// dist[b] when in_s is null or in_s[b] != 0.
template <int D, int G>
__global__ __launch_bounds__(512) void distortion_kernel(AttnArgs ref, AttnArgs itv, const uint8_t* in_s,
                                                          float* dist) {
  constexpr int NM = D / 16;
  constexpr int G4 = G > 4 ? G : 4;
  constexpr int MT = merge_threads<D, G>();
  constexpr int GP = distortion_heads<D, G>();
  __shared__ float s_d2[GP][G4];
  const int b = uni(blockIdx.x);
  if (in_s && in_s[b] == 0) return;
  const int gl = threadIdx.x / MT, t = threadIdx.x % MT;   // merge group, thread in it
  const int H = ref.cv.n_kv_heads;
  const int q = t / (NM * 16);
  const FirstCounts fr = first_counts(ref), fi = first_counts(itv);
  const WeightedPlan pr = stream_plan(ref, fr, ref.attn_blocks), pi = stream_plan(itv, fi, itv.attn_blocks);
  const SeqPages sr = seq_pages(ref, fr, b), si = seq_pages(itv, fi, b);
  const int er = units_before(ref, fr, b), ei = units_before(itv, fi, b);
  float worst = 0.0f;
  for (int g0 = 0; g0 < H; g0 += GP) {
    if (threadIdx.x < GP * G4) s_d2[threadIdx.x / G4][threadIdx.x % G4] = 0.0f;
    __syncthreads();
    const int g = g0 + gl;
    if (g < H) {                                 // whole merge groups (waves) take this branch alike
      float o_r[4], o_i[4];
      merged_pair<D, G>(ref, pr, sr, er, itv, pi, si, ei, b, g, t, q, o_r, o_i);
#pragma unroll
      for (int r = 0; r < 4; ++r) {              // each wave holds 64 dims of heads 4q..4q+3
        const float e = o_r[r] - o_i[r];
        const float w = wave_sum_f(e * e);
        if ((t & 63) == 0) atomicAdd(&s_d2[gl][4 * q + r], w);
      }
    }
    __syncthreads();
    if (threadIdx.x == 0)
      for (int j = 0; j < GP && g0 + j < H; ++j)
        for (int h = 0; h < G; ++h) worst = fmaxf(worst, s_d2[j][h]);
    __syncthreads();
  }
  if (threadIdx.x == 0) dist[b] += worst;
}

}  // namespace

// Partials of pask_decode_attn_noalloc (which has no caller workspace): a
// device array the library owns, one copy per GPU, kept until the process
// ends.  Host code never passes its name to a kernel (in host code the name
// is a host-side stand-in, not a device address); it passes the address
// scratch_workspace resolved for the current device.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

hipError_t scratch_workspace(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r != hipSuccess) return r;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

// Stream-K workers of attn_kernel<D, G> on the current device: as many waves
// as can be resident at once (occupancy x compute units), so every worker
// starts at launch.  Queried once per device and instance.
template <int D, int G, bool kWeighted>
int attn_grid() {
  constexpr int kWaves = kWeighted ? kWpb : 1;
  constexpr int kMaxDevices = 64;
  static int cached[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  if (cached[dev] == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_kernel<D, G, kWeighted>, 64 * kWaves, 0) !=
            hipSuccess ||
        per_cu <= 0)
      return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return 0;
    cached[dev] = per_cu * cus * kWaves;
  }
  return cached[dev];
}

hipError_t launch_attention(const AttnArgs& args, int group_size, hipStream_t s) {
  const int D = args.cv.head_dim;
  AttnArgs a = args;
  const int segs = a.batch * a.cv.n_kv_heads;
  const bool small = segs <= kSmallSegments;
  if (a.tags_new && (a.batch > kFusedMaxBatch || a.cv.window != 0 || a.ws_seq == nullptr)) return hipErrorInvalidValue;
  const int extra = a.tags_new ? 1 : 0;           // the merge block that enters the step's entries
#define PASK_CASE(DD, GG)                                                        \
  if (D == DD && group_size == GG) {                                             \
    a.attn_blocks = small ? attn_grid<DD, GG, false>() : attn_grid<DD, GG, true>(); \
    if (a.attn_blocks <= 0) return hipErrorInvalidDeviceFunction;                \
    a.min_pages = small ? kSmallMinPages : kMinPagesPerBlock;                    \
    if (small) {                                                                 \
      attn_kernel<DD, GG, false><<<dim3(a.attn_blocks), dim3(64), 0, s>>>(a);    \
      attn_merge_sliced_kernel<DD, GG><<<dim3(segs * (merge_threads<DD, GG>() / 16) + extra), dim3(64), 0, s>>>(a); \
    } else {                                                                     \
      attn_kernel<DD, GG, true><<<dim3(a.attn_blocks / kWpb), dim3(64 * kWpb), 0, s>>>(a); \
      attn_merge_kernel<DD, GG><<<dim3(segs + extra), dim3(merge_threads<DD, GG>()), 0, s>>>(a); \
    }                                                                            \
    return hipGetLastError();                                                    \
  }
  PASK_CASE(64, 1) PASK_CASE(64, 2) PASK_CASE(64, 4) PASK_CASE(64, 8)
  PASK_CASE(128, 1) PASK_CASE(128, 2) PASK_CASE(128, 4) PASK_CASE(128, 8)
#undef PASK_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_distortion(const AttnArgs& ref_args, const AttnArgs& itv_args, int group_size,
                             const uint8_t* in_s, float* dist, hipStream_t s) {
  const int D = ref_args.cv.head_dim;
  AttnArgs ref = ref_args, itv = itv_args;
  const dim3 block(64 * kWpb);
#define PASK_CASE(DD, GG)                                                        \
  if (D == DD && group_size == GG) {                                             \
    ref.attn_blocks = itv.attn_blocks = attn_grid<DD, GG, true>();               \
    ref.tags_new = itv.tags_new = nullptr;                                       \
    ref.min_pages = itv.min_pages = kMinPagesPerBlock;                           \
    if (ref.attn_blocks <= 0) return hipErrorInvalidDeviceFunction;              \
    attn_kernel<DD, GG, true><<<dim3(ref.attn_blocks / kWpb), block, 0, s>>>(ref); \
    attn_kernel<DD, GG, true><<<dim3(itv.attn_blocks / kWpb), block, 0, s>>>(itv); \
    distortion_kernel<DD, GG><<<dim3(ref.batch), dim3(merge_threads<DD, GG>() * distortion_heads<DD, GG>()), 0, s>>>(ref, itv, in_s, dist); \
    return hipGetLastError();                                                    \
  }
  PASK_CASE(64, 1) PASK_CASE(64, 2) PASK_CASE(64, 4) PASK_CASE(64, 8)
  PASK_CASE(128, 1) PASK_CASE(128, 2) PASK_CASE(128, 4) PASK_CASE(128, 8)
#undef PASK_CASE
  return hipErrorInvalidValue;
}

}  // namespace pask
