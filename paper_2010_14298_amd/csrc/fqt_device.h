// Device helpers shared by the FQT kernels: Philox4x32-7, stochastic
// rounding, the scalars of a block Householder group.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fqt {

// ---------------------------------------------------------------------------
// Philox4x32 (Salmon et al., SC'11): four 32-bit words from a 128-bit
// counter under a 64-bit key; the key is advanced by the two Weyl increments
// between rounds.  The stochastic-rounding stream takes seven rounds (the
// family's count from which its authors' test batteries pass; ten is their
// safety margin).
// ---------------------------------------------------------------------------
struct u32x4 {
  uint32_t x, y, z, w;
};

constexpr int PHILOX_ROUNDS = 7;
constexpr uint32_t PHILOX_M0 = 0xD2511F53u, PHILOX_M1 = 0xCD9E8D57u;  // round multipliers
constexpr uint32_t PHILOX_W0 = 0x9E3779B9u, PHILOX_W1 = 0xBB67AE85u;  // key increments

// n rounds from counter (c0, c1, c2, c3) under key (k0, k1).
__device__ __forceinline__ u32x4 philox_rounds(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                               uint32_t k1, int n) {
#pragma unroll
  for (int r = 0; r < n; ++r) {
    const uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
    const uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
    // three-way xors in one gfx950 bitop3 each (truth table 0x96)
    const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
    const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += PHILOX_W0;
    k1 += PHILOX_W1;
  }
  return u32x4{c0, c1, c2, c3};
}

// The block with counter (blk low word, blk high word, stream, 0) under key
// seed.  The first two rounds are written out: the stream and zero counter
// words make round one's second product, and round two's second counter
// word, the same in every lane, so those xors combine the uniform operands
// first (one scalar op) and leave one vector op per word.
__device__ __forceinline__ u32x4 philox_of_block(uint64_t blk, uint64_t seed, uint32_t stream) {
  uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const uint64_t p0 = (uint64_t)PHILOX_M0 * (uint32_t)blk;
  const uint64_t p1 = (uint64_t)PHILOX_M1 * stream;
  uint32_t c0 = (uint32_t)(blk >> 32) ^ ((uint32_t)(p1 >> 32) ^ k0);
  uint32_t c1 = (uint32_t)p1;
  uint32_t c2 = (uint32_t)(p0 >> 32) ^ k1;  // counter word 3 is zero
  uint32_t c3 = (uint32_t)p0;
  k0 += PHILOX_W0;
  k1 += PHILOX_W1;
  const uint64_t q0 = (uint64_t)PHILOX_M0 * c0;
  const uint64_t q1 = (uint64_t)PHILOX_M1 * c2;
  const uint32_t n0 = (uint32_t)(q1 >> 32) ^ (c1 ^ k0);
  const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(q0 >> 32), c3, k1, 0x96);
  c1 = (uint32_t)q1;
  c3 = (uint32_t)q0;
  k0 += PHILOX_W0;
  k1 += PHILOX_W1;
  return philox_rounds(n0, c1, n2, c3, k0, k1, PHILOX_ROUNDS - 2);
}
__device__ __forceinline__ u32x4 philox_block(uint64_t e, uint64_t seed, uint32_t stream) {
  return philox_of_block(e >> 2, seed, stream);
}

__device__ __forceinline__ uint32_t philox_word(const u32x4& o, int i) {
  return i == 0 ? o.x : (i == 1 ? o.y : (i == 2 ? o.z : o.w));
}

// ---------------------------------------------------------------------------
// Stochastic rounding with a 24-bit uniform (Sec. 3.3), the low 24 bits of
// the Philox word:
//   fl = floor(y); frac = y - fl; round up iff float(word & 0xFFFFFF) < frac * 2^24;
//   code clamped to [0, B].
// fl is clamped to [-1, B] first, which leaves the clamped code unchanged and
// keeps the integer conversion in range.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int sr_code(float y, uint32_t word, int B) {
  float fl = floorf(y);
  const float frac = y - fl;
  const float thr = frac * 16777216.0f;
  const float u = (float)(word & 0xFFFFFFu);
  fl = fminf(fmaxf(fl, -1.0f), (float)B);
  int c = (int)fl + (u < thr ? 1 : 0);
  return min(max(c, 0), B);
}

// Deterministic round-half-to-even, clamped to [0, B] (Q_f, Q_theta).
__device__ __forceinline__ int rne_code(float y, int B) {
  float r = rintf(y);
  r = fminf(fmaxf(r, 0.0f), (float)B);
  return (int)r;
}

// ---------------------------------------------------------------------------
// The same two rounding rules in 8.24 fixed point, for the bulk quantizers.
// Both return a word whose top byte is the offset code (code - half) as int8
// (hoff = half << 24), so that four results pack into one word with byte
// permutes and sum with one 4-way int8 dot product.
//
// sr_top: with yc = clamp(y, 0, B) (clamping first leaves the clamped code
// of sr_code unchanged), T = ceil(yc * 2^24) = floor(yc) * 2^24 + ceil(frac
// * 2^24) (the scaling is exact and floor(yc) * 2^24 is an integer), u =
// word & 0xFFFFFF and u' = 2^24 - 1 - u = ~word & 0xFFFFFF, the sum T + u'
// carries into bit 24 exactly when u < ceil(frac * 2^24), i.e. when u <
// frac * 2^24: the rounding-up decision of sr_code.  T + u' < 2^32 since
// yc <= 255 and at yc = B the fraction is 0.  -hoff only has top-byte bits
// and u' only low ones, so u' - hoff is one three-input logic operation.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int32_t sr_top(float y, uint32_t word, float Bf, uint32_t hoff) {
  const float yc = __builtin_amdgcn_fmed3f(y, 0.0f, Bf);
  const uint32_t t = (uint32_t)ceilf(yc * 16777216.0f);
  // (~word & 0xFFFFFF) | -hoff in one bitop3 (table 0xAE: ~S0 & S1 | S2)
  return (int32_t)(t + __builtin_amdgcn_bitop3_b32(word, 0xFFFFFFu, 0u - hoff, 0xAE));  // T + u' - hoff
}
__device__ __forceinline__ int32_t rne_top(float y, float Bf, uint32_t hoff) {
  const float r = rintf(__builtin_amdgcn_fmed3f(y, 0.0f, Bf));
  return (int32_t)(((uint32_t)(int)r << 24) - hoff);
}
// The offset code in the top byte of t shifted left by sh (the caller keeps
// the result inside int8); the low 24 bits are dropped.
__device__ __forceinline__ int32_t shift_top(int32_t t, int sh) {
  return (int32_t)(((uint32_t)t & 0xFF000000u) << sh);
}
// Top bytes of a, b, c, d as bytes 0..3 of one word.
__device__ __forceinline__ uint32_t pack_top4(int32_t a, int32_t b, int32_t c, int32_t d) {
  const uint32_t lo = __builtin_amdgcn_perm((uint32_t)b, (uint32_t)a, 0x0c0c0703u);
  const uint32_t hi = __builtin_amdgcn_perm((uint32_t)d, (uint32_t)c, 0x07030c0cu);
  return lo | hi;
}
// w with byte b replaced by the top byte of v (b is a constant after unrolling).
__device__ __forceinline__ uint32_t insert_top(uint32_t w, int32_t v, int b) {
  const uint32_t sel = b == 0 ? 0x03020107u : (b == 1 ? 0x03020700u : (b == 2 ? 0x03070100u : 0x07020100u));
  return __builtin_amdgcn_perm((uint32_t)v, w, sel);
}
// Sum of the four signed bytes of w, added to acc.
__device__ __forceinline__ int32_t sum4_i8(uint32_t w, int32_t acc) {
  return __builtin_amdgcn_sdot4((int)w, 0x01010101, acc, false);
}

constexpr float FLT_MAX_F = 3.402823466e+38f;

// s = B / R (one correctly rounded float32 division); R = 0 gives 1;
// overflow saturates at FLT_MAX.
__device__ __forceinline__ float scale_from_range(float R, int B) {
  if (!(R > 0.0f)) return 1.0f;
  float s = __fdiv_rn((float)B, R);
  return (s > FLT_MAX_F) ? FLT_MAX_F : s;
}

// ---------------------------------------------------------------------------
// Scalars of a block Householder group (App. C.4).
// ---------------------------------------------------------------------------

// Correctly rounded float32 cube root of a positive finite float: a float64
// estimate, then exact comparisons of x with the cubes of the midpoints to
// the float32 neighbours.  mid^2 is exact in float64 (25-bit mid); mid^3 =
// p + e exactly with p = fl(mid^2 mid), e = fma(mid^2, mid, -p); p - x is
// exact (Sterbenz), so mid^3 > x iff (p - x) > -e.
__device__ inline bool cube_gt(double mid, double x) {
  const double m2 = mid * mid;
  const double p = m2 * mid;
  const double e = fma(m2, mid, -p);
  return (p - x) > -e;
}
__device__ inline bool cube_lt(double mid, double x) {
  const double m2 = mid * mid;
  const double p = m2 * mid;
  const double e = fma(m2, mid, -p);
  return (p - x) < -e;
}
__device__ inline float cbrt_rn(float x) {
  if (!(x > 0.0f)) return 0.0f;
  float r = (float)cbrt((double)x);
  const double xd = (double)x;
  for (int it = 0; it < 8; ++it) {
    const uint32_t b = __float_as_uint(r);
    const float up = __uint_as_float(b + 1);
    const float dn = __uint_as_float(b - 1);
    const double mid_up = 0.5 * ((double)r + (double)up);
    const double mid_dn = 0.5 * ((double)r + (double)dn);
    if (cube_lt(mid_up, xd)) {
      r = up;
    } else if (cube_gt(mid_dn, xd)) {
      r = dn;
    } else {
      break;
    }
  }
  return r;
}

__device__ __forceinline__ float to_f32_sat(double v) {
  float f = (float)v;
  return (f > FLT_MAX_F) ? FLT_MAX_F : f;
}

// s1, s2 of a group of k >= 2 rows: s1 = B sqrt(k) / (a (a^2 + c^2 k)),
// s2 = B sqrt(k) / (c (a^2 + c^2 k)) with a = cbrt(lambda1), c =
// cbrt(lambda2) (App. C.4 multiplied through by k^(1/3)), float64 in this
// operation order, rounded once to float32.  lambda1 = 0 takes lambda2;
// lambda2 = 0 gives s1 = s2 = B sqrt(k) / lambda1; both zero give 1.  The
// cube roots come in precomputed (ca = cbrt_rn(lambda1), cc =
// cbrt_rn(lambda2)); sk = sqrt(k) in float64.
__device__ __forceinline__ void group_scales(float lam1, float lam2, float ca, float cc, int64_t k, double sk, int B,
                                             float& s1, float& s2) {
  if (lam1 == 0.0f) {
    lam1 = lam2;
    ca = cc;
  }
  if (lam1 == 0.0f && lam2 == 0.0f) {
    s1 = s2 = 1.0f;
  } else if (lam2 == 0.0f) {
    s1 = s2 = to_f32_sat(((double)B * sk) / (double)lam1);
  } else {
    const double a = (double)ca;
    const double c = (double)cc;
    const double t = a * a + (c * c) * (double)k;
    const double num = (double)B * sk;
    s1 = to_f32_sat(num / (a * t));
    s2 = to_f32_sat(num / (c * t));
  }
}

// A group's share of |S^-1|_F^2 (Eq. matrix-quantizer-variance):
// 1/s1^2 + (k - 1)/s2^2, a one-row group 1/s^2, float64.
__device__ __forceinline__ double group_term(float s1, float s2, int64_t k) {
  double t = 1.0 / ((double)s1 * (double)s1);
  if (k > 1) t = t + (double)(k - 1) * (1.0 / ((double)s2 * (double)s2));
  return t;
}

// Status word bits (first word of every workspace).
constexpr uint32_t STATUS_NONFINITE = 1u;
constexpr int STATUS_WORDS = 4;  // one per statistics segment; the workspace header reserves 64

}  // namespace fqt
