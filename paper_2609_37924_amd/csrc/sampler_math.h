// Sampling contract arithmetic shared by the standalone sampler and the sampling
// epilogue of the vocabulary projection: Philox4x32-10, the uniform map, the own
// float32 log / exp, the exact Gumbel score and the screening score.
//
// Every function that decides a token or a confidence uses individually rounded
// float32 +, -, *, / only: a translation unit that includes this header must be
// compiled with -ffp-contract=off and -fhip-fp32-correctly-rounded-divide-sqrt.
#pragma once
#include "common.h"

#pragma clang fp contract(off)

namespace tadm {
namespace {

constexpr int SAMPLE_GROUP = 64;  // vocabulary entries per normaliser group

__device__ __forceinline__ float bits_f(uint32_t b) { return __uint_as_float(b); }

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    // one 32x32->64 multiply per product (v_mad_u64_u32) gives both halves
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0], p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0, n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = (uint32_t)p1;
    c[2] = n2;
    c[3] = (uint32_t)p0;
  }
}

// (2 (x >> 9) + 1) 2^-24: the float 1 + (x >> 9) 2^-23 minus 1 - 2^-24, a subtraction
// that is exact (Sterbenz: the operands are within a factor of two)
__device__ __forceinline__ float uniform01(uint32_t x) {
  return __uint_as_float((x >> 9) | 0x3F800000u) - bits_f(0x3F7FFFFFu);
}

// log(x) for positive normal x (within 1 ulp): x = 2^e m, m in [sqrt(1/2), sqrt(2)),
// f = m - 1 (exact), s = f / (2 + f), log(1 + f) = 2 atanh(s) = 2 s + s R(s^2) with R
// the atanh series; taken as f - (f^2/2 - s (f^2/2 + R)) so that the exact f leads (the
// arrangement of Sun's fdlibm logarithm), e ln 2 added in two parts (Cody-Waite).
__device__ __forceinline__ float own_log(float x) {
  const float LN2_HI = bits_f(0x3F317200u), LN2_LO = bits_f(0x35BFBE8Eu);
  const uint32_t bits = __float_as_uint(x);
  int e = (int)(bits >> 23) - 127;
  uint32_t mb = (bits & 0x007FFFFFu) | 0x3F800000u;
  if (mb > 0x3FB504F3u) {  // m above sqrt(2): halve it
    mb -= 0x00800000u;
    e += 1;
  }
  const float m = __uint_as_float(mb);
  const float f = m - 1.0f;
  const float s = f / (2.0f + f);
  const float z = s * s;
  float c = bits_f(0x3E3A2E8Cu);       // 2/11
  c = c * z + bits_f(0x3E638E39u);     // 2/9
  c = c * z + bits_f(0x3E924925u);     // 2/7
  c = c * z + bits_f(0x3ECCCCCDu);     // 2/5
  c = c * z + bits_f(0x3F2AAAABu);     // 2/3
  const float R = z * c;
  const float hfsq = 0.5f * f * f;
  const float ef = (float)e;
  return ef * LN2_HI - ((hfsq - (s * (hfsq + R) + ef * LN2_LO)) - f);
}

// e^r = 1 + r + r^2 c(r) with c the Taylor series to r^5/7!, r = y - k ln 2 (Cody-Waite:
// rh = y - k ln2_hi exact, r = rh - k ln2_lo), summed as 1 + (rh + (r^2 c - k ln2_lo)) so
// that the rounding of r does not enter the linear term (within 1 ulp for y in [-30, 0]).
__device__ __forceinline__ float own_exp_core(float y, int bias) {
  const float LN2_HI = bits_f(0x3F317200u), LN2_LO = bits_f(0x35BFBE8Eu);
  const float k = rintf(y * bits_f(0x3FB8AA3Bu));
  const float rh = y - k * LN2_HI;
  const float kl = k * LN2_LO;
  const float r = rh - kl;
  float c = bits_f(0x39500D01u);       // 1/5040
  c = c * r + bits_f(0x3AB60B61u);     // 1/720
  c = c * r + bits_f(0x3C088889u);     // 1/120
  c = c * r + bits_f(0x3D2AAAABu);     // 1/24
  c = c * r + bits_f(0x3E2AAAABu);     // 1/6
  c = c * r + 0.5f;
  const float q = (r * r) * c;
  const float p = 1.0f + (rh + (q - kl));
  const float scale = __uint_as_float((uint32_t)((int)k + 127 + bias) << 23);
  return p * scale;
}

__device__ __forceinline__ float own_exp(float y) {
  if (y < -30.0f) return 0.0f;
  return own_exp_core(y, 0);
}

// own_exp without a branch: the same rounded operations for y >= -30 (and NaN), and 0 below,
// selected rather than branched on, for loops that unroll many exponentials.
__device__ __forceinline__ float own_exp_sel(float y) {
  const bool under = y < -30.0f;
  const float e = own_exp(under ? -30.0f : y);
  return under ? 0.0f : e;
}

// own_exp_sel(y) * 2^40 with the power of two folded into the exponent: the same value,
// since both scalings by powers of two are exact in the normal range own_exp reaches
// (its results lie in [e^-30, e^0.35] or are 0).
__device__ __forceinline__ float own_exp_sel_2p40(float y) {
  const bool under = y < -30.0f;
  const float e = own_exp_core(under ? -30.0f : y, 40);
  return under ? 0.0f : e;
}

struct Best {
  float score;
  int v;
};
__device__ __forceinline__ Best better(Best a, Best b) {
  return (b.score > a.score || (b.score == a.score && b.v < a.v)) ? b : a;
}

// Exact contract score of an entry from its scaled logit l' and uniform u:
// l' + G with G = -log(-log u).
__device__ __forceinline__ float exact_score_of(float lp, float u) {
  const float E = -own_log(u);
  return lp + (-own_log(E));
}

// Screening score a_v = l'_v - ln2 * log2(-log2 u_v) = (l'_v + G_v) - ln(ln 2) up to the
// hardware log2's error: it ranks entries and never decides a token.
__device__ __forceinline__ float screen_score(float lp, float u) {
  return lp - 0.6931471805599453f * __builtin_amdgcn_logf(-__builtin_amdgcn_logf(u));
}

// A thread's two best screening scores and the entry of the best.
struct Top2 {
  float a1 = -INFINITY, a2 = -INFINITY;
  int v1 = 0x7FFFFFFF;
  __device__ __forceinline__ void add(float a, int v) {  // by selects: no divergent branches
    const bool t = a > a1;
    a2 = t ? a1 : fmaxf(a2, a);
    v1 = t ? v : v1;
    a1 = t ? a : a1;
  }
};

}  // namespace
}  // namespace tadm
