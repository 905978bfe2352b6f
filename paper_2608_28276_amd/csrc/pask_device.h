// Device-side helpers shared by the append kernels (pask_append.hip) and the
// attention kernels (pask_attn.hip): addresses of a cache's counters, block
// tables and index lists, bf16 helpers, the RETAIN-LOW quantiser, the
// decision rule (Eq. 10), non-temporal loads and the page layout.  Included
// by those two files only.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "pask_internal.h"

namespace pask {
namespace {

constexpr int kDrop = 0, kHigh = 2;   // RETAIN-LOW is 1 (R < L < H)

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

// fp32 -> bf16, round to nearest even: gfx950's v_cvt_pk_bf16_f32.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}
__device__ __forceinline__ uint16_t f32_to_bf16_rne_dev(float f) {
  return (uint16_t)pack_bf16x2(f, 0.0f);
}


// The RETAIN-LOW code of x under scale s: clamp(RNE(x / s), -7, 7), 0 when
// s == 0, without a division.  c = rint(x * inv) is within one of RNE(x / s)
// whenever inv is 1 / s to a few ulp (|x / s| < 8 here); the residual
// e = x - c*s is exact (c*s has at most 15 significant bits and |e| < 2s), so
// comparing it with s/2 moves c to the nearest integer of x / s, ties to
// even.  Host-callable so that the rule can be checked exhaustively on the CPU.
__host__ __device__ inline int quant_code(float x, float s, float inv) {
  float c = rintf(x * inv);
  const float e = fmaf(-c, s, x);
  const float h = 0.5f * s;
  const bool odd = ((int)c & 1) != 0;
  c += (e > h || (e == h && odd)) ? 1.0f : ((e < -h || (e == -h && odd)) ? -1.0f : 0.0f);
  return s != 0.0f ? (int)fminf(fmaxf(c, -7.0f), 7.0f) : 0;
}

// The scale of a RETAIN-LOW group from its absmax: s = fp16(absmax / 7) with
// a correctly rounded fp32 division, saturated at 65504, rounded to nearest
// even; returns its fp16 bits, s as fp32 and an approximation of 1 / s.
__device__ __forceinline__ uint16_t quant_scale(float absmax, float& s, float& inv) {
  const _Float16 h = (_Float16)fminf(absmax / 7.0f, 65504.0f);
  s = (float)h;
  inv = __builtin_amdgcn_rcpf(s);
  return __builtin_bit_cast(uint16_t, h);
}
// Quantise 4 consecutive elements of a 32-element group held by 8 adjacent
// lanes (quant_scale of the group's absmax, quant_code of each element).
// Returns the 4 codes as offset-binary nibbles q + 8 (element i in bits
// 4i..4i+3; the pages hold codes in this form) and the scale bits.
__device__ __forceinline__ void quant4(uint32_t x01, uint32_t x23, uint32_t& packed, uint32_t& sbits) {
  float f[4] = {bf16_lo(x01), bf16_hi(x01), bf16_lo(x23), bf16_hi(x23)};
  float am = fmaxf(fmaxf(fabsf(f[0]), fabsf(f[1])), fmaxf(fabsf(f[2]), fabsf(f[3])));
  am = fmaxf(am, __shfl_xor(am, 1, 8));
  am = fmaxf(am, __shfl_xor(am, 2, 8));
  am = fmaxf(am, __shfl_xor(am, 4, 8));
  float s, inv;
  sbits = quant_scale(am, s, inv);
  uint32_t p = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) p |= (uint32_t)(quant_code(f[i], s, inv) + 8) << (4 * i);
  packed = p;
}
// The 8 codes of the bf16 elements of x (element u in bits 4u..4u+3, offset
// binary) under scale s, inv ~ 1/s.  rint(x * inv) is the nearest integer of
// x / s whenever x / s is not within 2^-12 of a half-integer: for a bf16 x
// and an fp16 s no quotient other than an exact tie comes that close, and
// x * inv is within 2^-19 of x / s.  Lanes holding an element near a tie take
// the exact rule (quant_code) for their 8 elements.
__device__ __forceinline__ uint32_t codes8(const uint4& x, float s, float inv) {
  const float f[8] = {bf16_lo(x.x), bf16_hi(x.x), bf16_lo(x.y), bf16_hi(x.y),
                      bf16_lo(x.z), bf16_hi(x.z), bf16_lo(x.w), bf16_hi(x.w)};
  uint32_t p = 0u;
  bool near_tie = false;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const float y = f[u] * inv;
    const float c = rintf(y);
    near_tie |= fabsf(y - c) > 0.49988f;
    p |= (uint32_t)(fminf(fmaxf(c, -7.0f), 7.0f) + 8.0f) << (4 * u);
  }
  if (__ballot(near_tie)) {
    if (near_tie) {
      p = 0u;
#pragma unroll
      for (int u = 0; u < 8; ++u) p |= (uint32_t)(quant_code(f[u], s, inv) + 8) << (4 * u);
    }
  }
  return s != 0.0f ? p : 0x88888888u;
}
// Nibbles 0..3 of p moved to the low nibbles of bytes 0..3.
__device__ __forceinline__ uint32_t nibbles_to_bytes(uint32_t p) {
  p &= 0xFFFFu;
  p = (p | (p << 8)) & 0x00FF00FFu;
  return (p | (p << 4)) & 0x0F0F0F0Fu;
}
// A K word in page order from 8 codes in element order: element e (< 4) in
// the low nibble of byte e, element 4 + e in its high nibble.
__device__ __forceinline__ uint32_t k_word(uint32_t packed) {
  return nibbles_to_bytes(packed) | (nibbles_to_bytes(packed >> 16) << 4);
}

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

// Data read once per call (pages in the attention, a bulk append's input
// rows): non-temporal loads, so the streamed lines do not displace others in
// the L2 and the last-level cache (the attention call on the 64-sequence
// Qwen3-4B workload measured 10% faster than with plain loads).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint4 stream_load16(const uint8_t* p) {
  const u32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(x[0], x[1], x[2], x[3]);
}

// Page layout, per KV head, chosen so that the MFMA operands of the attention
// kernel arrive by fully coalesced loads: load instruction i of lane l = 16q + n
// reads bytes 1024 i + 16 l of a HIGH tile, so each instruction of the wave
// covers 1 KiB contiguously.
//   HIGH  K tile: element (t, d), d = 32i + 8q + j  at ((i*64 + q*16 + t)*8 + j)   (bf16)
//         V tile: element (t, d), d = 16m + dd      at (((m/2)*64 + t/4*16 + dd)*2 + m%2)*4 + t%4
//   LOW   codes are offset-binary nibbles c + 8 (c in [-7, 7]).
//         K codes: word (q*16 + t)*NG + i holds d = 32i + 8q + j, j = 0..7: element
//                  j < 4 in the low nibble of byte j, element 4 + j' in the high
//                  nibble of byte j'; K scales [t][NG] fp16;
//         V codes: byte ((t/4*16 + dd)*(NM/2) + i)*4 + t%4 holds dims 32i+dd (low
//                  nibble) and 32i+16+dd (high nibble) of slot t; V scales [t][NG].
// NG = D/32 scale groups, NM = D/16.  Every byte belongs to a single slot, so
// appends of different slots never share a byte.  KV head g of page P is kept
// in head slot (g + P) mod n_kv_heads of the page.
template <int D>
struct PageLayout {
  static constexpr int NG = D / 32, NM = D / 16;
  static constexpr int kHiHead = 64 * D, kHiV = 32 * D;
  static constexpr int kLoKS = 8 * D, kLoVC = 8 * D + 32 * NG, kLoVS = 16 * D + 32 * NG;
  static constexpr int kLoHead = 16 * D + 64 * NG;
};

}  // namespace
}  // namespace pask
