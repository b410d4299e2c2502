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

#include "../../include/qd.h"

namespace qd {

// ---------------------------------------------------------------------------
// Philox4x32 with 10 rounds (Salmon et al., SC'11).  Counter words:
// (item, individual, generation, stream tag); key = the 64-bit seed.
// ---------------------------------------------------------------------------
enum : uint32_t { kTagInit = 0, kTagSelect = 1, kTagIso = 2, kTagCentroid = 3, kTagEnv = 4,
                  kTagCvtSample = 5, kTagInitLevel = 6 };

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

// ---------------------------------------------------------------------------
// fp32 functions from +, -, *, fma and IEEE division.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float fma32(float a, float b, float c) {
  return __builtin_fmaf(a, b, c);
}

constexpr float kLn2Hi = 0x1.62e4p-1f;      // ln 2, 16 leading bits
constexpr float kLn2Lo = 0x1.7f7d1cp-20f;   // remainder of ln 2
constexpr float kLog2e = 0x1.715476p+0f;

// ---------------------------------------------------------------------------
// Gaussian sampler: one standard normal per Philox word x by inversion.
// k = (x & 0xffffff) + 1 (exact in fp32), p = k 2^-24; the magnitude is the
// half-normal quantile Phi^-1(1 - p/2), read from the table of cubics that
// qd_archive_init builds on the host (QD_NORMAL_ROWS rows of (c0, c1, c2,
// c3)): row = binary exponent of k times 16 plus its next four bits, taken
// straight from the fp32 bits of k; u = its remaining 19 bits as an integer;
// z = c0 + u (c1 + u (c2 + u c3)) by fma from the cubic term.  Bit 31 of x
// is the sign (bits 24..30 are not used).  Ten VALU instructions and one
// 16-byte LDS read per normal.  Every workgroup that draws normals stages the
// table in LDS (6160 bytes).
// ---------------------------------------------------------------------------
constexpr int kNormalRows = QD_NORMAL_ROWS;

struct Tables {
  const float4* ntab;   // LDS copy of the table
};

__device__ __forceinline__ void stage_normal_table(float4* dst, const float4* src, int tid,
                                                   int nthreads) {
  for (int i = tid; i < kNormalRows; i += nthreads) dst[i] = src[i];
}

__device__ __forceinline__ float normal(uint32_t x, const Tables& tb) {
  // k = (x & 0xffffff) + 1 as one 24-bit multiply-add (k * 1 + 1)
  uint32_t k;
  asm("v_mad_u32_u24 %0, %1, 1, 1" : "=v"(k) : "v"(x));
  const uint32_t b = __float_as_uint((float)k);
  // row = (b >> 19) - 127 * 16: a bit-field extract (kept as one instruction:
  // the compiler would rewrite it into a shift and a mask), then the scaled
  // index and the bias go into one shift-and-add of the address
  uint32_t e4;
  asm("v_bfe_u32 %0, %1, 19, 12" : "=v"(e4) : "v"(b));
  const float4 c = (tb.ntab - (127 << 4))[e4];
  const float u = (float)(b & 0x7ffffu);
  const float z = fma32(u, fma32(u, fma32(u, c.w, c.z), c.y), c.x);
  return __uint_as_float(__float_as_uint(z) ^ (x & 0x80000000u));   // one v_bitop3
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
