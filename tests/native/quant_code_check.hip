// The division-free RETAIN-LOW code rule of the append kernels (quant_code in
// pask_device.h), checked on the CPU against RNE(x / s) computed in fp64 (exact
// here: a tie x / s = k + 1/2 is exact in fp64, and any other quotient lies at
// least 2^-12 from a tie), clamped to [-7, 7].  Every positive fp16 scale s,
// every bf16 x with s/8 <= |x| <= 9s (11s for a subnormal s, where a group's
// |x / s| reaches 10.5: s = 2^-24 from absmax / 7 just above 2^-25; both
// signs), and an approximate
// reciprocal 1/s moved by up to 4 ulp either way (the device takes it from
// v_rcp_f32, accurate to 1 ulp); then every bf16 x below s/8 at the exact
// reciprocal, and s = 0.  Over the same x, s and reciprocals, the two fast
// paths give the exact code wherever they do not defer to quant_code: codes8
// (the decode call's entry: rint(x * 1/s) unless within kNearTie of a tie) and
// code_bytes8 (the bulk pack: the low byte of RN(x * 1/s + 1.5 * 2^23 + 8),
// unless the part rounded away is within kNearTie of 1/2; only for a normal
// s, and there every element of a group has |x| < 7 s (1 + 2^-11), so no
// clamp: an absmax with fp16(absmax / 7) = s is below 7 (s + ulp(s) / 2)).
// Last, the bulk pack's division-free scale against fp16(absmax / 7) for
// every bf16 absmax.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "pask_device.h"

static float bf16_value(uint32_t bits) {
  const uint32_t w = bits << 16;
  float f;
  memcpy(&f, &w, 4);
  return f;
}

static int want(float x, float s) {
  if (s == 0.0f) return 0;
  const double q = nearbyint((double)x / (double)s);
  return (int)fmin(fmax(q, -7.0), 7.0);
}

// The near-tie threshold of both fast paths.
constexpr float kNearTie = 0.49988f;
constexpr float kM = 12582920.0f;                    // 1.5 * 2^23 + 8

// code_bytes8's fast code of x under a normal scale s, or 100 when it
// defers to quant_code (or x lies outside what a group with scale s holds);
// its low byte must hold the code + 8 with bits 4..7 zero (else -100).
static int fast_byte_code(float x, float s, float inv) {
  if (!(s >= 0x1p-14f) || !(fabsf(x) < 7.0f * s * (1.0f + 0x1p-11f))) return 100;
  const float y = fmaf(x, inv, kM);
  if (fabsf(fmaf(x, inv, kM - y)) > kNearTie) return 100;
  uint32_t bits;
  memcpy(&bits, &y, 4);
  return ((bits & 0xF0u) || (bits & 0xFFu) == 0 || (bits & 0xFFu) > 15) ? -100 : (int)(bits & 0xFFu) - 8;
}

int main() {
  long n = 0, bad = 0;
  for (uint32_t hs = 1; hs < 0x7C00; ++hs) {        // every positive finite fp16 scale
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)hs);
    for (int du = -4; du <= 4; ++du) {
      float inv = 1.0f / s;
      for (int k = 0; k < (du < 0 ? -du : du); ++k) inv = nextafterf(inv, du < 0 ? 0.0f : INFINITY);
      for (uint32_t bx = 0; bx < 0x7F80; ++bx) {
        const float x = bf16_value(bx);
        if (x < s / 8) continue;
        if (x > (hs < 0x400 ? 11 : 9) * s) break;
        for (int sg = 0; sg < 2; ++sg) {
          const float xs = sg ? -x : x;
          const int got = pask::quant_code(xs, s, inv);
          ++n;
          if (got != want(xs, s)) {
            if (++bad <= 10) printf("mismatch: x=%a s=%a inv=%a got %d want %d\n", xs, s, inv, got, want(xs, s));
          }
          // codes8: rint(x * inv) clamped, unless |x * inv - rint(x * inv)| >
          // kNearTie sends the lane to quant_code.  Wherever a fast path keeps
          // its code, that code must be the exact one.
          const float y = xs * inv, c = rintf(y);
          if (!(fabsf(y - c) > kNearTie)) {
            const int fast = (int)fminf(fmaxf(c, -7.0f), 7.0f);
            if (fast != want(xs, s) && ++bad <= 10)
              printf("fast-path mismatch: x=%a s=%a inv=%a got %d want %d\n", xs, s, inv, fast, want(xs, s));
          }
          const int fb = fast_byte_code(xs, s, inv);
          if (fb != 100 && fb != want(xs, s) && ++bad <= 10)
            printf("byte fast-path mismatch: x=%a s=%a inv=%a got %d want %d\n", xs, s, inv, fb, want(xs, s));
        }
      }
      if (du == 0) {
        for (uint32_t bx = 0; bx < 0x7F80; ++bx) {  // small x (codes 0 and +-1) at the exact reciprocal
          const float x = bf16_value(bx);
          if (x >= s / 8) break;
          for (int sg = 0; sg < 2; ++sg) {
            const float xs = sg ? -x : x;
            ++n;
            if (pask::quant_code(xs, s, inv) != want(xs, s) && ++bad <= 10) printf("mismatch (small): x=%a s=%a\n", xs, s);
            const int fb = fast_byte_code(xs, s, inv);
            if (fb != 100 && fb != want(xs, s) && ++bad <= 10) printf("byte fast-path mismatch (small): x=%a s=%a\n", xs, s);
          }
        }
      }
    }
  }
  for (uint32_t bx = 0; bx < 0x7F80; bx += 7) {      // s == 0: every code 0
    ++n;
    if (pask::quant_code(bf16_value(bx), 0.0f, INFINITY) != 0 && ++bad <= 10) printf("s = 0 gives a code\n");
  }
  // The bulk pack's scale (quant_scale_bf16 in pask_append.hip): absmax times
  // RN(1/7), divided instead below 7 * 2^-14, rounds to the fp16 of the
  // correctly rounded absmax / 7 (quant_scale) for every finite bf16 absmax.
  for (uint32_t bx = 0; bx < 0x7F80; ++bx) {
    const float am = bf16_value(bx);
    float q = am * (1.0f / 7.0f);
    if (am < 7.0f * 0x1p-14f) q = am / 7.0f;
    const _Float16 want_s = (_Float16)fminf(am / 7.0f, 65504.0f), got_s = (_Float16)fminf(q, 65504.0f);
    ++n;
    if (__builtin_bit_cast(uint16_t, want_s) != __builtin_bit_cast(uint16_t, got_s) && ++bad <= 10)
      printf("scale mismatch: absmax=%a\n", am);
    // plain (7 * 2^-14 <= absmax <= 7 * 65504): s is normal and every element
    // of the group has |x| <= absmax < 7 s (1 + 2^-11), the premise of
    // code_bytes8's clamp-free fast path (fast_byte_code above).
    const float sv = (float)want_s;
    if (am >= 7.0f * 0x1p-14f && am <= 7.0f * 65504.0f && !(sv >= 0x1p-14f && am < 7.0f * sv * (1.0f + 0x1p-11f)) &&
        ++bad <= 10)
      printf("plain scale premise fails: absmax=%a s=%a\n", am, sv);
  }
  printf("%s: %ld cases, %ld mismatches\n", bad ? "FAIL" : "ok", n, bad);
  return bad ? 1 : 0;
}
