// qd_device.hpp -- device-side arithmetic of the generation kernels (gfx950).
//
// Counter-based random numbers, the Gaussian sampler and the fp32
// transcendental functions the kernels use.  Every function here is evaluated
// with explicit fused multiply-adds in a fixed order and the library is built
// with -ffp-contract=off, so each result is a fixed function of its inputs,
// independent of launch shape or scheduling.  That makes a generation
// reproducible bit for bit, which the insertion step needs: which elite keeps
// a cell is decided by comparing fp32 objectives.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qd {

// ---------------------------------------------------------------------------
// Philox4x32 with 10 rounds (Salmon et al., SC'11).  Counter words:
// (item, individual, generation, stream tag); key = the 64-bit seed.
// ---------------------------------------------------------------------------
enum : uint32_t { kTagInit = 0, kTagSelect = 1, kTagIso = 2, kTagCentroid = 3, kTagEnv = 4,
                  kTagCvtSample = 5 };

struct Key {
  uint32_t k0, k1;
};

// a ^ b ^ c in one v_bitop3_b32 (truth table 0x96)
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ uint4 philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                        Key key) {
  uint32_t k0 = key.k0, k1 = key.k1;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint64_t m0 = (uint64_t)0xD2511F53u * c0;   // one v_mad_u64_u32 each
    const uint64_t m1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = xor3((uint32_t)(m1 >> 32), c1, k0);
    const uint32_t n2 = xor3((uint32_t)(m0 >> 32), c3, k1);
    c0 = n0;
    c1 = (uint32_t)m1;
    c2 = n2;
    c3 = (uint32_t)m0;
    k0 += 0x9E3779B9u;                                 // Weyl schedule; the key is
    k1 += 0xBB67AE85u;                                 // wave-uniform (scalar unit)
  }
  return make_uint4(c0, c1, c2, c3);
}

__device__ __forceinline__ float unit24(uint32_t x) {        // [0, 1)
  return (float)(x >> 8) * 0x1p-24f;
}
__device__ __forceinline__ float unit24_open0(uint32_t x) {  // (0, 1]
  return (float)((x >> 8) + 1u) * 0x1p-24f;
}

// ---------------------------------------------------------------------------
// fp32 functions from +, -, *, fma, IEEE division and square root.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float fma32(float a, float b, float c) {
  return __builtin_fmaf(a, b, c);
}

constexpr float kLn2Hi = 0x1.62e4p-1f;      // ln 2, 16 leading bits
constexpr float kLn2Lo = 0x1.7f7d1cp-20f;   // remainder of ln 2
constexpr float kPi = 0x1.921fb6p+1f;
constexpr float kHalfPi = 0x1.921fb6p+0f;
constexpr float kLog2e = 0x1.715476p+0f;

// Square root of a positive normal x (or +-0) without the small-input
// scaling: hardware estimate, then the neighbour one unit in the last place
// below or above is taken when the fma residual says the estimate rounded
// the wrong way.  (For x = +-0 both neighbours fail their test, so +-0 comes
// back unchanged.)  On every input the Box-Muller radius can feed it this
// returns the IEEE square root bit for bit; the library checks that over all
// of them (qd_check_fast_arith).
__device__ __forceinline__ float sqrt_normal(float x) {
  const float s = __builtin_amdgcn_sqrtf(x);
  const float dn = __uint_as_float(__float_as_uint(s) - 1u);
  const float up = __uint_as_float(__float_as_uint(s) + 1u);
  const float r = fma32(-dn, s, x) <= 0.0f ? dn : s;
  return fma32(-up, s, x) > 0.0f ? up : r;
}

// ln x for positive normal x.  x = 2^e m, m folded into [sqrt(1/2), sqrt(2));
// ln m = 2 atanh(s) with s = (m - 1)/(m + 1), odd series through s^9.  Used
// to fill the log table of the Gaussian sampler.
__device__ __forceinline__ float log_pos(float x) {
  const uint32_t bits = __float_as_uint(x);
  const uint32_t frac = bits & 0x7fffffu;
  const bool fold = frac > 0x3504f3u;
  const int e = (int)(bits >> 23) - 127 + (fold ? 1 : 0);
  const float m = __uint_as_float((frac | 0x3f800000u) - (fold ? 0x00800000u : 0u));
  const float s = (m - 1.0f) / (m + 1.0f);
  const float s2 = s * s;
  float p = fma32(s2, 2.0f / 9.0f, 2.0f / 7.0f);
  p = fma32(s2, p, 2.0f / 5.0f);
  p = fma32(s2, p, 2.0f / 3.0f);
  const float lnm = fma32(s * s2, p, s + s);
  const float fe = (float)e;
  return fma32(fe, kLn2Hi, fma32(fe, kLn2Lo, lnm));
}

// sin / cos of x, |x| <= pi/4: Taylor polynomials through x^9 and x^10.
__device__ __forceinline__ float sin_small(float x) {
  const float x2 = x * x;
  float p = fma32(x2, 1.0f / 362880.0f, -1.0f / 5040.0f);
  p = fma32(x2, p, 1.0f / 120.0f);
  p = fma32(x2, p, -1.0f / 6.0f);
  return fma32(x * x2, p, x);
}
__device__ __forceinline__ float cos_small(float x) {
  const float x2 = x * x;
  float p = fma32(x2, -1.0f / 3628800.0f, 1.0f / 40320.0f);
  p = fma32(x2, p, -1.0f / 720.0f);
  p = fma32(x2, p, 1.0f / 24.0f);
  p = fma32(x2, p, -0.5f);
  return fma32(x2, p, 1.0f);
}

// (cos, sin) of 2 pi m / 2^24 for a 24-bit m: the nearest quarter turn q
// (halves rounding up) is split off in integers, leaving (pi/2) f with
// f = m / 2^22 - q, |f| <= 1/2, exactly.
__device__ __forceinline__ float2 turn_cos_sin(uint32_t m) {
  const uint32_t t = m + 0x200000u;
  const uint32_t q = t >> 22;
  // f * pi/2 with f = rem 2^-22: the power-of-two factor is exact, so it is
  // folded into the constant and the product still rounds once
  const float x = (float)((int32_t)(t & 0x3fffffu) - 0x200000) * (kHalfPi * 0x1p-22f);
  const float s = sin_small(x), c = cos_small(x);
  // quarter turns q = 0..3 (4 = 0): (c, s), (-s, c), (-c, -s), (s, -c),
  // written as a swap on odd q and sign flips, without branches
  const bool odd = (q & 1u) != 0u;
  const float a = odd ? s : c, b = odd ? c : s;
  const uint32_t flip_cos = ((q + 1u) & 2u) << 30, flip_sin = (q & 2u) << 30;
  return make_float2(__uint_as_float(__float_as_uint(a) ^ flip_cos),
                     __uint_as_float(__float_as_uint(b) ^ flip_sin));
}

// ---------------------------------------------------------------------------
// Table-driven forms for the Gaussian sampler.  Each workgroup builds the two
// small tables in LDS from the functions above, so they hold the same bits
// everywhere:
//   turn[i] = (cos, sin) of 2 pi i / 256 (turn_cos_sin at i << 16)
//   logt[i] = (R_i, L_i) for bin i of m in [1, 2) ([1 + i/128, 1 + (i+1)/128)):
//             R_i = 1 / c_i (IEEE division, c_i the bin's midpoint) and
//             L_i = -ln R_i, or -ln(2 R_i) with a factor 2 moved into the
//             exponent for bins from 53 up (m >= 1.4140625); bin 0 uses R = 1
//             and bin 127 R = 1/2, with L = 0, so logs near 1 do not cancel.
// ---------------------------------------------------------------------------
struct Tables {
  const float2* turn;   // [256]
  const float2* logt;   // [128]
};

__device__ __forceinline__ void build_tables(float2* turn, float2* logt, int tid, int nthreads) {
  for (int i = tid; i < 256; i += nthreads) turn[i] = turn_cos_sin((uint32_t)i << 16);
  for (int i = tid; i < 128; i += nthreads) {
    float r = 1.0f, l = 0.0f;
    if (i == 127) {
      r = 0.5f;
    } else if (i > 0) {
      const float c = 1.0f + ((float)i + 0.5f) / 128.0f;
      r = 1.0f / c;
      l = -log_pos(i >= 53 ? r + r : r);
    }
    logt[i] = make_float2(r, l);
  }
}

// cos and sin of 2 pi m / 2^24 from the turn table and the remainder
// delta = (m & 0xffff) 2 pi 2^-24: sin delta ~ delta - delta^3/6,
// cos delta ~ 1 - delta^2/2 + delta^4/24, angle-addition formulas.
__device__ __forceinline__ float2 turn_tab(uint32_t m, const Tables& tb) {
  const float2 t = tb.turn[m >> 16];
  const float d = (float)(m & 0xffffu) * (kPi * 0x1p-23f);
  const float d2 = d * d;
  const float sd = fma32(d * d2, -1.0f / 6.0f, d);
  const float cd = fma32(d2, fma32(d2, 1.0f / 24.0f, -0.5f), 1.0f);
  return make_float2(fma32(t.x, cd, -(t.y * sd)), fma32(t.y, cd, t.x * sd));
}

// ln(k 2^-24), integer k in [1, 2^24]: k = 2^E m, bin i = top 7 fraction bits
// of m, t = m R_i - 1 in one rounding, ln(m 2^-f) = L_i + t - t^2/2 + t^3/3
// - t^4/4 (f = 1 for bins from 53 up), exponent E - 24 + f.
__device__ __forceinline__ float log_k24(uint32_t k, const Tables& tb) {
  const uint32_t b = __float_as_uint((float)k);
  const uint32_t i = (b >> 16) & 0x7fu;
  const int e = (int)(b >> 23) - (127 + 24) + (i >= 53u ? 1 : 0);
  const float m = __uint_as_float((b & 0x7fffffu) | 0x3f800000u);
  const float2 rl = tb.logt[i];
  const float t = fma32(m, rl.x, -1.0f);
  float q = fma32(t, -0.25f, 1.0f / 3.0f);
  q = fma32(t, q, -0.5f);
  const float lnm = rl.y + fma32(t * t, q, t);
  const float fe = (float)e;
  return fma32(fe, kLn2Hi, fma32(fe, kLn2Lo, lnm));
}

// Box-Muller radius sqrt(-2 ln u1), u1 = ((xa >> 8) + 1) 2^-24: with the IEEE
// square root, and with the short sequence the kernels use.
__device__ __forceinline__ float bm_radius_ieee(uint32_t xa, const Tables& tb) {
  return __builtin_sqrtf(-2.0f * log_k24((xa >> 8) + 1u, tb));
}
__device__ __forceinline__ float bm_radius(uint32_t xa, const Tables& tb) {
  return sqrt_normal(-2.0f * log_k24((xa >> 8) + 1u, tb));
}

// Two standard normals (Box-Muller) from two Philox words.
__device__ __forceinline__ float2 gauss2(uint32_t xa, uint32_t xb, const Tables& tb) {
  const float r = bm_radius(xa, tb);
  const float2 cs = turn_tab(xb >> 8, tb);
  return make_float2(r * cs.x, r * cs.y);
}


// sqrt(20) sin(pi x) up to sign (the sign may differ by (-1)^rint(x)):
// r = x - rint(x) in [-1/2, 1/2] (exact), then r P(r^2), P the Taylor series
// of sqrt(20) sin(pi r) / r in u = r^2 through u^5 by Horner's rule.  Its
// coefficient k, sqrt(20) (-1)^k pi^(2k+1) / (2k+1)!, is worked out in double
// at compile time and rounded once to fp32.
constexpr float rsin_coef(int k) {
  double c = 4.47213595499957939282;   // sqrt(20)
  for (int i = 1; i <= 2 * k + 1; ++i) c *= 3.14159265358979323846 / (double)i;
  return (float)((k & 1) ? -c : c);
}
__device__ __forceinline__ float rsinpi(float x) {
  constexpr float c0 = rsin_coef(0), c1 = rsin_coef(1), c2 = rsin_coef(2);
  constexpr float c3 = rsin_coef(3), c4 = rsin_coef(4), c5 = rsin_coef(5);
  const float r = x - __builtin_rintf(x);
  const float u = r * r;
  float q = fma32(u, c5, c4);
  q = fma32(u, q, c3);
  q = fma32(u, q, c2);
  q = fma32(u, q, c1);
  q = fma32(u, q, c0);
  return r * q;
}

// e^x, input clamped to [-87, 88]: k = rint(x log2 e), r = x - k ln 2 in two
// fma steps, Taylor through r^7, times 2^k assembled in the exponent field.
__device__ __forceinline__ float exp32(float x) {
  const float y = x < -87.0f ? -87.0f : (x > 88.0f ? 88.0f : x);
  const float k = __builtin_rintf(y * kLog2e);
  float r = fma32(-k, kLn2Hi, y);
  r = fma32(-k, kLn2Lo, r);
  float p = fma32(r, 1.0f / 5040.0f, 1.0f / 720.0f);
  p = fma32(r, p, 1.0f / 120.0f);
  p = fma32(r, p, 1.0f / 24.0f);
  p = fma32(r, p, 1.0f / 6.0f);
  p = fma32(r, p, 0.5f);
  p = fma32(r, p, 1.0f);
  p = fma32(r, p, 1.0f);
  const float scale = __uint_as_float((uint32_t)((int32_t)k + 127) << 23);
  const float e = p * scale;
  return x == x ? e : x;
}

// a / b by the hardware reciprocal and one residual correction.  Used where
// the library has checked, over every input the caller can pass, that the
// result equals the IEEE quotient (qd_check_fast_arith).
__device__ __forceinline__ float div_rcp(float a, float b) {
  const float y = __builtin_amdgcn_rcpf(b);
  const float q = a * y;
  const float r = fma32(-q, b, a);
  return fma32(r, y, q);
}

// tanh: odd Taylor polynomial through x^11 for |x| < 0.3,
// else 1 - 2 / (e^{2|x|} + 1); the sign is copied back.  FAST takes the
// quotient from div_rcp (same bits for every fp32 input).
template <bool FAST = true>
__device__ __forceinline__ float tanh32(float x) {
  const float a = __builtin_fabsf(x);
  float r;
  if (a < 0.3f) {
    const float a2 = a * a;
    float p = fma32(a2, -1382.0f / 155925.0f, 62.0f / 2835.0f);
    p = fma32(a2, p, -17.0f / 315.0f);
    p = fma32(a2, p, 2.0f / 15.0f);
    p = fma32(a2, p, -1.0f / 3.0f);
    r = fma32(a * a2, p, a);
  } else {
    const float d = exp32(a + a) + 1.0f;
    r = 1.0f - (FAST ? div_rcp(2.0f, d) : 2.0f / d);
  }
  return __builtin_copysignf(r, x);
}

// 1 / (1 + e^{-x}); FAST as for tanh32 (same bits for |x| <= 1, the range of
// the tanh states it is applied to).
template <bool FAST = true>
__device__ __forceinline__ float sigmoid32(float x) {
  const float d = 1.0f + exp32(-x);
  return FAST ? div_rcp(1.0f, d) : 1.0f / d;
}

// ---------------------------------------------------------------------------
// Wave64 helpers.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Pairwise fold of one value per lane in the fixed tree h = 32, 16, ..., 1
// (the partial of lane l is added to that of lane l + h), without LDS: the
// steps h = 32 and 16 exchange halves and rows with the lane-swap
// instructions, h = 8 .. 1 rotate within rows of 16 lanes (DPP).  Every step
// leaves each lane holding its pair's sum (addition commutes, so both members
// of a pair hold the same bits), and the total ends in every lane.
// DPP within rows of 16 lanes: row_shl<N> gives lane l the value of lane
// l + N (0 past the row's end), row_ror<N> that of lane (l - N) mod 16.
template <int N>
__device__ __forceinline__ float row_shl(float v) {
  return __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x100 + N, 0xf, 0xf, false));
}
template <int N>
__device__ __forceinline__ float row_ror(float v) {
  return __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x120 + N, 0xf, 0xf, false));
}
template <int N>
__device__ __forceinline__ int row_ror(int v) {
  return (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)v, 0x120 + N, 0xf, 0xf, false);
}

// One rotation step of a row-wide minimum of (value, index) pairs, smaller
// index first among equal values.
template <int N>
__device__ __forceinline__ void min_pair_row(float& v, int& idx) {
  const float ov = row_ror<N>(v);
  const int oi = row_ror<N>(idx);
  const bool take = ov < v || (ov == v && oi < idx);
  v = take ? ov : v;
  idx = take ? oi : idx;
}
__device__ __forceinline__ float wave_fold_sum(float v) {
  const auto h32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(h32[0]) + __uint_as_float(h32[1]);
  const auto h16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(h16[0]) + __uint_as_float(h16[1]);
  v = v + row_ror<8>(v);
  v = v + row_ror<4>(v);
  v = v + row_ror<2>(v);
  v = v + row_ror<1>(v);
  return v;
}

// wave_fold_sum for partials that are zero in lanes 32 .. 63 of the wave the
// R64 order describes (at most 128 genes: its h = 32 step adds +0 and changes
// nothing), with two such waves packed into the two halves of this one: the
// h = 16 .. 1 steps stay inside each half, whose every lane ends up with its
// half's sum.
__device__ __forceinline__ float half_fold_sum(float v) {
  const auto h16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(h16[0]) + __uint_as_float(h16[1]);
  v = v + row_ror<8>(v);
  v = v + row_ror<4>(v);
  v = v + row_ror<2>(v);
  v = v + row_ror<1>(v);
  return v;
}

// The same fold for three values at once.  The first two steps pack values
// into halves and rows of one register (a half-swap of a with b leaves lane l
// of the sum holding a_l + a_{l+32} below lane 32 and b's pair sums above;
// the row swap then does the same for rows of 16 lanes), after which the
// rotations finish all three in one register: a ends in lanes 0-15, c in
// 16-31, b in 32-47.  Each value goes through exactly the pairs of
// wave_fold_sum.
__device__ __forceinline__ void wave_fold_sum3(float a, float b, float c, float& sa, float& sb,
                                               float& sc) {
  const auto ab = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  const float pab = __uint_as_float(ab[0]) + __uint_as_float(ab[1]);
  const auto cz = __builtin_amdgcn_permlane32_swap(__float_as_uint(c), 0u, false, false);
  const float pcz = __uint_as_float(cz[0]) + __uint_as_float(cz[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(pab), __float_as_uint(pcz), false, false);
  float v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  v = v + row_ror<8>(v);
  v = v + row_ror<4>(v);
  v = v + row_ror<2>(v);
  v = v + row_ror<1>(v);
  sa = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(v), 0));
  sc = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(v), 16));
  sb = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(v), 32));
}

// Order-preserving map of an fp32 objective to u32 (-0 folded onto +0).
__device__ __forceinline__ uint32_t order_bits(float f) {
  const uint32_t u = __float_as_uint(f == 0.0f ? 0.0f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace qd
