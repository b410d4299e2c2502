/*
 * qd_oracle.c -- plain, slow CPU oracle of massively-parallel MAP-Elites
 * ("Accelerated Quality-Diversity through Massive Parallelism", Lim, Allard,
 * Grillotti, Cully; arXiv 2202.01258).  The per-offspring loops (select,
 * vary, evaluate, map to a cell) may run on several threads through OpenMP:
 * each offspring depends only on the archive before the generation, so the
 * results do not depend on the thread count.  Insertion is Algorithm 1's
 * sequential loop and always runs in one thread.
 *
 * TEST INFRASTRUCTURE ONLY.  It exists so that the HIP library can be checked
 * against something written straight from the paper.  Only the test-suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product path never calls it and shares no code with it.
 *
 * What it computes, and where the paper says so:
 *   - MAP-Elites, Algorithm 1: random first batch, then select -> vary ->
 *     evaluate -> insert per cell, with an offspring entering an empty cell or
 *     replacing an incumbent only on a strictly greater objective.
 *   - Archive as static arrays, filled cells found from the objective array
 *     (Appendix A.1, A.2); selection uniform with replacement over the filled
 *     cells (Appendix A.2).
 *   - Iso+LineDD variation, Algorithm 2 in Appendix A.2.
 *   - Rastrigin and Sphere objectives and the (theta_0, theta_1) descriptor,
 *     Appendix B.2; the policy network shape of Section 5.1 (two hidden tanh
 *     layers, tanh output).
 *   - Insertion: Algorithm 1's sequential loop over the batch (the four masked
 *     steps of Appendix A.4 reach the same archive; a test shows it).
 *   - QD-score (Eq. 1), coverage and best objective (Appendix B.1).
 *
 * Where the paper is silent (random number generator, Gaussian sampler,
 * transcendental functions, reduction order, cell formula, tie-breaks, the
 * synthetic rollout) this file follows one fixed arithmetic contract, written
 * out in the design notes, so that an independently written GPU program can
 * reach bit-identical archives.  Every floating-point step below is fp32 with
 * explicit fmaf() where a fused multiply-add is meant; the file is compiled
 * with -ffp-contract=off so the compiler fuses nothing by itself.
 *
 * Parity pins (tests/test_oracle_*.py) check each function here against
 * closed forms, fp64 library routines, brute force and invariants.
 */
#include "qd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Bits                                                                      */
/* ------------------------------------------------------------------------ */
static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11).  The paper fixes no generator; a counter-based  */
/* one lets every offspring draw its own numbers independently.              */
/* ------------------------------------------------------------------------ */
void or_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { /* Weyl key schedule */
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    uint32_t n1 = (uint32_t)p1;
    uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    uint32_t n3 = (uint32_t)p0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Stream tags (fourth counter word).  Counter = (item, individual, generation, tag). */
enum { TAG_INIT = 0, TAG_SELECT = 1, TAG_ISO = 2, TAG_CENTROID = 3, TAG_ENV = 4,
       TAG_CVT_SAMPLE = 5, TAG_INIT_LEVEL = 6 };

static void draw(const or_state* s, uint32_t item, uint32_t indiv, uint32_t gen,
                 uint32_t tag, uint32_t out[4]);

/* Top 24 bits as a uniform on [0,1) and on (0,1]; both exact in fp32. */
float or_u24(uint32_t x) { return (float)(x >> 8) * 0x1p-24f; }
float or_u24p(uint32_t x) { return (float)((x >> 8) + 1u) * 0x1p-24f; }

/* ------------------------------------------------------------------------ */
/* Own transcendental functions.  Built from +, -, *, fmaf and IEEE / in a   */
/* fixed order, with Taylor coefficients (exact rationals rounded once to    */
/* fp32) and a Cody-Waite split of ln 2.                                     */
/* ------------------------------------------------------------------------ */
static const float kLn2Hi = 0x1.62e4p-1f;       /* ln 2 to 16 significant bits   */
static const float kLn2Lo = 0x1.7f7d1cp-20f;    /* ln 2 - kLn2Hi, rounded        */
static const float kLog2e = 0x1.715476p+0f;     /* 1/ln 2 rounded to fp32        */

/* ------------------------------------------------------------------------ */
/* Gaussian sampler.  Algorithm 2 draws eps1 ~ N(0, I) and eps2 ~ N(0, 1)    */
/* without saying how.  Here each standard normal comes from one Philox word */
/* x by inversion of the half-normal law: with k = (x & 0xffffff) + 1 and    */
/* p = k 2^-24 in (0, 1], the magnitude is z(p) = Phi^-1(1 - p/2), the       */
/* point with P(|Z| >= z) = p, and bit 31 of x is the sign (bits 24..30 are  */
/* not used).  z(p) is read from a table of cubic pieces: p = 2^(E-24) (1 +  */
/* (j + t)/16) with E the binary exponent of k (0..24), j its next four bits */
/* and t in [0, 1) the remaining 19 bits / 2^19; row r = 16 E + j holds the  */
/* monomial coefficients of the cubic in t that interpolates z at the four   */
/* Chebyshev points of [0, 1], worked out in double and rounded once to fp32 */
/* (coefficient i scaled by 2^(-19 i) so that the polynomial is evaluated    */
/* in the integer t 2^19 directly).  Row 384 (k = 2^24, p = 1, z = 0) is     */
/* zero.  Largest magnitude: z(2^-24) = 5.42.                                */
/* ------------------------------------------------------------------------ */
static float g_ntab[OR_NORMAL_ROWS][4];
static int g_ntab_built = 0;

/* z(p) = Phi^-1(1 - p/2) for p in (0, 1): the root of erfc(z / sqrt 2) = p,
 * by 100 bisection steps on [0, 16] (erfc from the C library). */
double or_normal_quantile(double p) {
  const double inv_sqrt2 = 0.70710678118654752440;
  double lo = 0.0, hi = 16.0;
  for (int it = 0; it < 100; ++it) {
    double mid = 0.5 * (lo + hi);
    if (erfc(mid * inv_sqrt2) > p) lo = mid;
    else hi = mid;
  }
  return 0.5 * (lo + hi);
}

static void build_normal_table(void) {
  if (g_ntab_built) return;
  /* Chebyshev points of [0, 1]: (1 -+ cos(pi/8)) / 2, (1 -+ cos(3 pi/8)) / 2 */
  const double r2 = sqrt(2.0);
  const double ca = 0.5 * sqrt(2.0 + r2), cb = 0.5 * sqrt(2.0 - r2);
  const double t[4] = {0.5 * (1.0 - ca), 0.5 * (1.0 - cb), 0.5 * (1.0 + cb), 0.5 * (1.0 + ca)};
  for (int r = 0; r < OR_NORMAL_ROWS - 1; ++r) {
    int E = r >> 4, j = r & 15;
    double f[4];
    for (int i = 0; i < 4; ++i)
      f[i] = or_normal_quantile(ldexp(1.0 + ((double)j + t[i]) / 16.0, E - 24));
    /* Newton divided differences: f[i] becomes z[t_0, ..., t_i] */
    for (int k = 1; k < 4; ++k)
      for (int i = 3; i >= k; --i) f[i] = (f[i] - f[i - 1]) / (t[i] - t[i - k]);
    /* Newton form f0 + (t - t0)(f1 + (t - t1)(f2 + (t - t2) f3)) -> powers of
     * t, innermost factor first: m <- m (t - t_k) + f_k for k = 2, 1, 0 */
    double m[4] = {f[3], 0.0, 0.0, 0.0};
    for (int k = 2; k >= 0; --k) {
      for (int i = 3; i >= 1; --i) m[i] = m[i - 1] - t[k] * m[i];
      m[0] = f[k] - t[k] * m[0];
    }
    for (int i = 0; i < 4; ++i) g_ntab[r][i] = (float)ldexp(m[i], -19 * i);
  }
  for (int i = 0; i < 4; ++i) g_ntab[OR_NORMAL_ROWS - 1][i] = 0.0f;
  g_ntab_built = 1;
}

void or_normal_table(float* out) {
  build_normal_table();
  memcpy(out, g_ntab, sizeof(g_ntab));
}

/* One standard normal from one Philox word (see above): Horner's rule from
 * the cubic term, then the sign of bit 31. */
float or_normal(uint32_t x) {
  build_normal_table();
  uint32_t k = (x & 0xffffffu) + 1u;
  uint32_t b = f2u((float)k);                    /* k <= 2^24: exact           */
  uint32_t r = (b >> 19) - (127u << 4);          /* 16 E + j                   */
  float tf = (float)(b & 0x7ffffu);              /* t 2^19, exact              */
  const float* c = g_ntab[r];
  float z = fmaf(tf, fmaf(tf, fmaf(tf, c[3], c[2]), c[1]), c[0]);
  return (x >> 31) ? -z : z;
}

/* sqrt(20) sin(pi x), up to sign, for the Rastrigin term.  r = x - rint(x)
 * lies in [-1/2, 1/2] (exact); sqrt(20) sin(pi r) = r P(r^2) with P the
 * Taylor series in u = r^2 through u^5, whose coefficient k is
 * sqrt(20) (-1)^k pi^(2k+1) / (2k+1)!, worked out in double and rounded once to
 * fp32; P is evaluated by Horner's rule from the u^5 end.  The sign may differ
 * from that of sin(pi x) by (-1)^rint(x); callers square it. */
static float g_rsin[6];
static int g_rsin_built = 0;

void or_rsin_coef(float out[6]) {
  if (!g_rsin_built) {
    const double pi = 3.14159265358979323846;
    for (int k = 0; k < 6; ++k) {
      double c = sqrt(20.0);
      for (int i = 1; i <= 2 * k + 1; ++i) c *= pi / (double)i;
      g_rsin[k] = (float)((k & 1) ? -c : c);
    }
    g_rsin_built = 1;
  }
  for (int k = 0; k < 6; ++k) out[k] = g_rsin[k];
}

float or_rsinpi(float x) {
  float c[6];
  or_rsin_coef(c);
  float r = x - rintf(x);
  float u = r * r;
  float q = c[5];
  for (int k = 4; k >= 0; --k) q = fmaf(u, q, c[k]);
  return r * q;
}

/* exp(x): k = rint(x log2 e), r = x - k ln 2 (two steps), Taylor to r^7,
 * scaled by 2^k built in the exponent field.  Input clamped to [-87, 88]. */
float or_expf(float x) {
  if (!(x == x)) return x;
  float y = x < -87.0f ? -87.0f : (x > 88.0f ? 88.0f : x);
  float k = rintf(y * kLog2e);
  float r = fmaf(-k, kLn2Hi, y);
  r = fmaf(-k, kLn2Lo, r);
  float p = fmaf(r, 1.0f / 5040.0f, 1.0f / 720.0f);
  p = fmaf(r, p, 1.0f / 120.0f);
  p = fmaf(r, p, 1.0f / 24.0f);
  p = fmaf(r, p, 1.0f / 6.0f);
  p = fmaf(r, p, 0.5f);
  p = fmaf(r, p, 1.0f);
  p = fmaf(r, p, 1.0f);
  float scale = u2f((uint32_t)((int32_t)k + 127) << 23);
  return p * scale;
}

/* tanh(x): odd Taylor series to x^11 below |x| = 0.3, else
 * 1 - 2/(exp(2|x|) + 1); sign restored at the end. */
float or_tanhf(float x) {
  float a = fabsf(x);
  float r;
  if (a < 0.3f) {
    float a2 = a * a;
    float p = fmaf(a2, -1382.0f / 155925.0f, 62.0f / 2835.0f);
    p = fmaf(a2, p, -17.0f / 315.0f);
    p = fmaf(a2, p, 2.0f / 15.0f);
    p = fmaf(a2, p, -1.0f / 3.0f);
    r = fmaf(a * a2, p, a);
  } else {
    float e = or_expf(2.0f * a);
    r = 1.0f - 2.0f / (e + 1.0f);
  }
  return copysignf(r, x);
}

float or_sigmoidf(float x) { return 1.0f / (1.0f + or_expf(-x)); }

/* ------------------------------------------------------------------------ */
/* Fixed reduction order ("R64"): genes are taken in groups of four          */
/* consecutive indices; group q feeds partial sum q mod 64 in ascending      */
/* order; the 64 partials are then folded pairwise, p[l] += p[l+h] for       */
/* h = 32, 16, ..., 1.  The sum runs over the index range [a, b).            */
/* ------------------------------------------------------------------------ */
float or_r64_sum(const float* t, int32_t a, int32_t b) {
  float p[64];
  for (int l = 0; l < 64; ++l) p[l] = 0.0f;
  for (int32_t g = a; g < b; ++g) p[(g >> 2) & 63] = p[(g >> 2) & 63] + t[g];
  for (int h = 32; h >= 1; h >>= 1)
    for (int l = 0; l < h; ++l) p[l] = p[l] + p[l + h];
  return p[0];
}

static float clampf(float x, float lo, float hi) { return fminf(fmaxf(x, lo), hi); }

/* Rastrigin, Sphere (Appendix B.2) and the two-half projection descriptor.
 * Rastrigin uses 10 - 10 cos(2 pi x) = 20 sin^2(pi x), so that every term
 * x^2 + 20 sin^2(pi x) = x^2 + s^2 with s = sqrt(20) sin(pi x) is
 * non-negative and nothing cancels; the objective is the negated R64 sum of
 * the terms. */
void or_eval_testfn(int32_t task, const float* x, int32_t n, const float* lo,
                    const float* hi, float* fit, float* desc) {
  float* t = (float*)calloc((size_t)(n > 0 ? n : 1), sizeof(float));
  for (int32_t g = 0; g < n; ++g) {
    if (task == OR_SPHERE) {
      t[g] = x[g] * x[g];
    } else {
      float sv = or_rsinpi(x[g]);
      t[g] = fmaf(sv, sv, x[g] * x[g]);
    }
  }
  *fit = -or_r64_sum(t, 0, n);
  if (task == OR_RASTRIGIN_PROJ) {
    int32_t half = n / 2;
    for (int32_t g = 0; g < n; ++g)
      t[g] = g < half ? clampf(x[g], lo[0], hi[0]) : clampf(x[g], lo[1], hi[1]);
    desc[0] = or_r64_sum(t, 0, half) / (float)half;
    desc[1] = or_r64_sum(t, half, n) / (float)(n - half);
  } else {
    desc[0] = clampf(x[0], lo[0], hi[0]);
    desc[1] = clampf(x[1], lo[1], hi[1]);
  }
  free(t);
}

/* ------------------------------------------------------------------------ */
/* Descriptor -> cell (Appendix A.1: descriptors are turned into archive     */
/* indexes).  Grid: per-dimension bin floor(t * bins), t = (d-lo)/(hi-lo),   */
/* clamped, row-major with the last dimension fastest.  CVT: index of the    */
/* nearest centroid in the unit box, lowest index on ties.  -1 = invalid.    */
/* ------------------------------------------------------------------------ */
int32_t or_grid_cell(const float* d, int32_t D, const int32_t* grid, const float* lo,
                     const float* hi) {
  int32_t cell = 0;
  for (int32_t k = 0; k < D; ++k) {
    if (!(d[k] == d[k])) return -1;
    float t = (d[k] - lo[k]) / (hi[k] - lo[k]);
    float fb = floorf(t * (float)grid[k]);
    int32_t b;
    if (fb < 0.0f) b = 0;
    else if (fb > (float)(grid[k] - 1)) b = grid[k] - 1;
    else b = (int32_t)fb;
    cell = cell * grid[k] + b;
  }
  return cell;
}

static int32_t nearest_centroid(const float* u, int32_t D, const float* cent, int32_t C);

int32_t or_cvt_cell(const float* d, int32_t D, const float* lo, const float* hi,
                    const float* cent, int32_t C) {
  float u[4];
  for (int32_t k = 0; k < D; ++k) {
    if (!(d[k] == d[k])) return -1;
    u[k] = (d[k] - lo[k]) / (hi[k] - lo[k]);
  }
  return nearest_centroid(u, D, cent, C);
}

/* Brute-force nearest centroid of a point u of [0,1]^D: squared distance as
 * an fma chain over the dimensions from 0, first minimum in index order. */
static int32_t nearest_centroid(const float* u, int32_t D, const float* cent, int32_t C) {
  int32_t best = -1;
  float bestd = 0.0f;
  for (int32_t c = 0; c < C; ++c) {
    float acc = 0.0f;
    for (int32_t k = 0; k < D; ++k) {
      float diff = u[k] - cent[(size_t)c * D + k];
      acc = fmaf(diff, diff, acc);
    }
    if (best < 0 || acc < bestd) {
      best = c;
      bestd = acc;
    }
  }
  return best;
}

/* ------------------------------------------------------------------------ */
/* Policy rollout on synthetic dynamics s' = tanh(A s + B a).  Policy: the    */
/* fully connected net of Section 5.1 with two hidden tanh layers and a tanh */
/* output.  Genotype = [W1 (hid x obs), b1, W2 (hid x hid), b2, W3 (act x    */
/* hid), b3], row-major.  Return = sum_t (s_{t+1}[0] - 0.5 |a_t|^2);          */
/* descriptor k = mean over t = 1..T of sigmoid(s_t[k+1]), k = 0..3.          */
/* Summation order ("dot4"): input k goes to partial sum k mod 4, each an    */
/* fma chain in input order from 0, folded as (p0 + p2) + (p1 + p3).  Hidden  */
/* layers: tanh(dot4 + bias).  The output layer sums 8 contiguous slices of   */
/* hid/8 inputs each (one chain each), folds the 8 partial sums pairwise (s   */
/* with s+4, then s+2, then s+1) and adds the bias.  Dynamics:                */
/* tanh(dot4(A row, s) + (B row . a in order)).                               */
/* ------------------------------------------------------------------------ */
static float dot4(const float* w, const float* x, int32_t n) {
  float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int32_t k = 0; k < n; ++k) p[k & 3] = fmaf(w[k], x[k], p[k & 3]);
  return (p[0] + p[2]) + (p[1] + p[3]);
}

static void dense_tanh(const float* W, const float* bias, const float* in, int32_t nin,
                       int32_t nout, float* out) {
  for (int32_t o = 0; o < nout; ++o) out[o] = or_tanhf(dot4(W + (size_t)o * nin, in, nin) + bias[o]);
}

static void dense_tanh_sliced8(const float* W, const float* bias, const float* in, int32_t nin,
                               int32_t nout, float* out) {
  const int32_t len = nin / 8;
  for (int32_t o = 0; o < nout; ++o) {
    float part[8];
    for (int32_t sl = 0; sl < 8; ++sl) {
      float acc = 0.0f;
      for (int32_t k = sl * len; k < (sl + 1) * len; ++k)
        acc = fmaf(W[(size_t)o * nin + k], in[k], acc);
      part[sl] = acc;
    }
    for (int32_t h = 4; h >= 1; h >>= 1)
      for (int32_t sl = 0; sl < h; ++sl) part[sl] = part[sl] + part[sl + h];
    out[o] = or_tanhf(part[0] + bias[o]);
  }
}

/* Failure (Appendix A.3, A.4 i): with death_mode != 0 the episode stops at
 * the first step whose new state has component 0 below death_below; that step
 * and the rest count for nothing, so the return and the descriptor cover only
 * the states before the failure (a variable-length episode; the descriptor
 * is the mean over those states).  death_mode 2 also discards every failed
 * solution, and an episode with no state before its failure is discarded in
 * both modes: a discarded solution gets a NaN objective, which insertion
 * never accepts (the death flag). */
void or_mlp_rollout(const float* w, int32_t obs, int32_t hid, int32_t act, int32_t T,
                    const float* A, const float* B, const float* s0, int32_t death_mode,
                    float death_below, float* fit, float* desc) {
  const float* W1 = w;
  const float* b1 = W1 + (size_t)hid * obs;
  const float* W2 = b1 + hid;
  const float* b2 = W2 + (size_t)hid * hid;
  const float* W3 = b2 + hid;
  const float* b3 = W3 + (size_t)act * hid;
  float* s = (float*)malloc(sizeof(float) * (size_t)(2 * obs + 2 * hid + act));
  float* sn = s + obs;
  float* h1 = sn + obs;
  float* h2 = h1 + hid;
  float* a = h2 + hid;
  for (int32_t i = 0; i < obs; ++i) s[i] = s0[i];
  float ret = 0.0f;
  float dsum[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  int32_t valid = 0, failed = 0;
  for (int32_t t = 0; t < T; ++t) {
    dense_tanh(W1, b1, s, obs, hid, h1);
    dense_tanh(W2, b2, h1, hid, hid, h2);
    dense_tanh_sliced8(W3, b3, h2, hid, act, a);
    for (int32_t i = 0; i < obs; ++i) {
      const float as = dot4(A + (size_t)i * obs, s, obs);
      float ba = 0.0f;
      for (int32_t k = 0; k < act; ++k) ba = fmaf(B[(size_t)i * act + k], a[k], ba);
      sn[i] = or_tanhf(as + ba);
    }
    if (death_mode != 0 && sn[0] < death_below) {
      failed = 1;
      break;
    }
    float q = 0.0f;
    for (int32_t o = 0; o < act; ++o) q = fmaf(a[o], a[o], q);
    ret = ret + fmaf(-0.5f, q, sn[0]);
    for (int32_t k = 0; k < 4; ++k) dsum[k] = dsum[k] + or_sigmoidf(sn[1 + k]);
    for (int32_t i = 0; i < obs; ++i) s[i] = sn[i];
    valid += 1;
  }
  *fit = ((death_mode == 2 && failed) || valid == 0) ? NAN : ret;
  for (int32_t k = 0; k < 4; ++k) desc[k] = valid > 0 ? dsum[k] / (float)valid : 0.0f;
  free(s);
}

/* ------------------------------------------------------------------------ */
/* Insertion key: order-preserving map of the objective in the high word     */
/* (-0 taken as +0), N_B-1-j in the low word so that equal objectives go to  */
/* the lowest batch index.  An incumbent's low word is all ones, so it keeps */
/* its cell on a tie (Algorithm 1 replaces only on a strictly greater        */
/* return).  The sequential oracle does not need the key; tests use it to    */
/* check that the max over keys equals the sequential loop.                  */
/* ------------------------------------------------------------------------ */
uint64_t or_key(float f, int32_t j, int32_t batch) {
  if (f == 0.0f) f = 0.0f;
  uint32_t u = f2u(f);
  uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  uint32_t low = j < 0 ? 0xffffffffu : (uint32_t)(batch - 1 - j);
  return ((uint64_t)o << 32) | (uint64_t)low;
}

/* ------------------------------------------------------------------------ */
/* State                                                                     */
/* ------------------------------------------------------------------------ */
struct or_state {
  or_config cfg;
  int32_t n;
  float* geno;       /* [C][n]   archive parameters (zeros when empty)        */
  float* fit;        /* [C]      archive objective (NaN when empty)           */
  float* desc;       /* [C][D]                                                */
  uint8_t* occ;      /* [C]      1 = filled                                   */
  float* cent;       /* [C][D]   CVT centroids                                */
  float* env;        /* A, B, s0 of the synthetic dynamics                    */
  int32_t* parents;  /* [N_B][2]                                              */
  float* off_fit;    /* [N_B]                                                 */
  float* off_desc;   /* [N_B][D]                                              */
  int32_t* off_cell; /* [N_B]                                                 */
  uint8_t* off_won;  /* [N_B]                                                 */
  float* off_geno;   /* [N_B][n]                                              */
  int32_t* occ_list; /* [C]                                                   */
};

int32_t or_genotype_len(const or_config* c) {
  if (c->task == OR_MLP)
    return c->hid * c->obs + c->hid + c->hid * c->hid + c->hid + c->act * c->hid + c->act;
  return c->n;
}

int32_t or_env_len(const or_config* c) {
  if (c->task != OR_MLP) return 0;
  return c->obs * c->obs + c->obs * c->act + c->obs;
}

static void draw(const or_state* s, uint32_t item, uint32_t indiv, uint32_t gen,
                 uint32_t tag, uint32_t out[4]) {
  uint32_t ctr[4] = {item, indiv, gen, tag};
  uint32_t key[2] = {(uint32_t)(s->cfg.seed & 0xffffffffu), (uint32_t)(s->cfg.seed >> 32)};
  or_philox(ctr, key, out);
}

or_state* or_new(const or_config* cfg, int32_t keep_offspring) {
  /* the lazily built tables are built here, before any parallel loop reads them */
  float coef[6];
  build_normal_table();
  or_rsin_coef(coef);
  or_state* s = (or_state*)calloc(1, sizeof(or_state));
  s->cfg = *cfg;
  s->n = or_genotype_len(cfg);
  (void)keep_offspring;
  size_t C = (size_t)cfg->C, n = (size_t)s->n, D = (size_t)cfg->D, nb = (size_t)cfg->batch;
  s->geno = (float*)calloc(C * n, sizeof(float));
  s->fit = (float*)malloc(C * sizeof(float));
  for (size_t c = 0; c < C; ++c) s->fit[c] = NAN;
  s->desc = (float*)calloc(C * D, sizeof(float));
  s->occ = (uint8_t*)calloc(C, 1);
  s->cent = (float*)calloc(C * D, sizeof(float));
  s->env = (float*)calloc((size_t)or_env_len(cfg) + 1, sizeof(float));
  s->parents = (int32_t*)calloc(nb * 2, sizeof(int32_t));
  s->off_fit = (float*)calloc(nb, sizeof(float));
  s->off_desc = (float*)calloc(nb * D, sizeof(float));
  s->off_cell = (int32_t*)calloc(nb, sizeof(int32_t));
  s->off_won = (uint8_t*)calloc(nb, 1);
  s->off_geno = NULL; /* allocated by the first whole-batch call */
  s->occ_list = (int32_t*)calloc(C + 1, sizeof(int32_t));
  return s;
}

void or_free(or_state* s) {
  if (!s) return;
  free(s->geno); free(s->fit); free(s->desc); free(s->occ); free(s->cent); free(s->env);
  free(s->parents); free(s->off_fit); free(s->off_desc); free(s->off_cell);
  free(s->off_won); free(s->off_geno); free(s->occ_list);
  free(s);
}

/* Centroids: coordinate k of centroid c is the 24-bit uniform of word k of
 * block (c, 0, 0, CENTROID).  Environment: entry e of [A | B | s0] is 0.1
 * times the normal of word e mod 4 of block (e/4, 0, 0, ENV). */
/* Centroidal Voronoi tessellation by Lloyd's algorithm (the CVT the paper
 * cites for its tessellations): cvt_iters times, every one of cvt_samples
 * uniform points of [0,1]^D (point i, coordinate k = U24 of word k of block
 * (i, 0, 0, CVT_SAMPLE)) goes to its nearest centroid, and every centroid
 * that received points moves to their mean; the others stay.  A point's
 * coordinate is m 2^-24 with an integer m < 2^24, so a centroid's coordinate
 * sum is kept exactly as the sum of the m; the new coordinate is
 * ((double)sum / (double)count) 2^-24 rounded to fp32. */
static void lloyd(or_state* s) {
  const or_config* c = &s->cfg;
  const int32_t C = c->C, D = c->D;
  uint64_t* sum = (uint64_t*)calloc((size_t)C * D, sizeof(uint64_t));
  uint64_t* cnt = (uint64_t*)calloc((size_t)C, sizeof(uint64_t));
  for (int32_t it = 0; it < c->cvt_iters; ++it) {
    memset(sum, 0, (size_t)C * D * sizeof(uint64_t));
    memset(cnt, 0, (size_t)C * sizeof(uint64_t));
    for (int32_t i = 0; i < c->cvt_samples; ++i) {
      uint32_t x[4];
      float u[4];
      draw(s, (uint32_t)i, 0, 0, TAG_CVT_SAMPLE, x);
      for (int32_t k = 0; k < D; ++k) u[k] = or_u24(x[k]);
      const int32_t b = nearest_centroid(u, D, s->cent, C);
      for (int32_t k = 0; k < D; ++k) sum[(size_t)b * D + k] += x[k] >> 8;
      cnt[b] += 1;
    }
    for (int32_t b = 0; b < C; ++b) {
      if (cnt[b] == 0) continue;
      for (int32_t k = 0; k < D; ++k)
        s->cent[(size_t)b * D + k] =
            (float)(((double)sum[(size_t)b * D + k] / (double)cnt[b]) * 0x1p-24);
    }
  }
  free(sum);
  free(cnt);
}

void or_setup(or_state* s) {
  const or_config* c = &s->cfg;
  if (c->tess == OR_CVT) {
    for (int32_t i = 0; i < c->C; ++i) {
      uint32_t x[4];
      draw(s, (uint32_t)i, 0, 0, TAG_CENTROID, x);
      for (int32_t k = 0; k < c->D; ++k) s->cent[(size_t)i * c->D + k] = or_u24(x[k]);
    }
    if (c->cvt_samples > 0) lloyd(s);
  }
  int32_t ne = or_env_len(c);
  for (int32_t e = 0; e < ne; ++e) {
    uint32_t x[4];
    draw(s, (uint32_t)(e / 4), 0, 0, TAG_ENV, x);
    s->env[e] = 0.1f * or_normal(x[e % 4]);
  }
}

/* Random first batch (Algorithm 1, first iteration: random solutions).
 * Test functions: gene i = lo + U * (hi - lo); with init_mode 1 individual j
 * also draws one level per genotype half h (genes [0, n/2) and [n/2, n)),
 * uniform over descriptor dimension h's box, lo_h + U (hi_h - lo_h) from word
 * h of block (0, j, 0, INIT_LEVEL), and adds it to every gene of that half,
 * so that the first batch covers the descriptor box even where a descriptor
 * averages many genes.  Policies: Glorot-uniform weights in
 * [-a, a), a = sqrt(6 / (fan_in + fan_out)), zero biases. */
static void init_genotype(const or_state* s, int32_t j, float* out) {
  const or_config* c = &s->cfg;
  int32_t n = s->n;
  uint32_t x[4] = {0, 0, 0, 0};
  float level[2] = {0.0f, 0.0f};
  if (c->task != OR_MLP && c->init_mode == 1) {
    uint32_t y[4];
    draw(s, 0, (uint32_t)j, 0, TAG_INIT_LEVEL, y);
    for (int h = 0; h < 2; ++h) level[h] = fmaf(or_u24(y[h]), c->hi[h] - c->lo[h], c->lo[h]);
  }
  for (int32_t i = 0; i < n; ++i) {
    if ((i & 3) == 0) draw(s, (uint32_t)(i >> 2), (uint32_t)j, 0, TAG_INIT, x);
    float u = or_u24(x[i & 3]);
    if (c->task != OR_MLP) {
      out[i] = fmaf(u, c->init_hi - c->init_lo, c->init_lo);
      if (c->init_mode == 1) out[i] = level[i < n / 2 ? 0 : 1] + out[i];
    } else {
      int32_t o = c->obs, h = c->hid, a = c->act;
      int32_t e1 = h * o, e2 = e1 + h, e3 = e2 + h * h, e4 = e3 + h, e5 = e4 + a * h;
      float lim;
      if (i < e1) lim = sqrtf(6.0f / (float)(o + h));
      else if (i < e2) lim = 0.0f;
      else if (i < e3) lim = sqrtf(6.0f / (float)(h + h));
      else if (i < e4) lim = 0.0f;
      else if (i < e5) lim = sqrtf(6.0f / (float)(h + a));
      else lim = 0.0f;
      out[i] = lim == 0.0f ? 0.0f : fmaf(u, lim + lim, -lim);
    }
  }
}

static void evaluate(const or_state* s, const float* x, float* fit, float* desc) {
  const or_config* c = &s->cfg;
  if (c->task == OR_MLP) {
    const float* A = s->env;
    const float* B = A + (size_t)c->obs * c->obs;
    const float* s0 = B + (size_t)c->obs * c->act;
    or_mlp_rollout(x, c->obs, c->hid, c->act, c->T, A, B, s0, c->death_mode, c->death_below,
                   fit, desc);
  } else {
    or_eval_testfn(c->task, x, s->n, c->lo, c->hi, fit, desc);
  }
}

static int32_t cell_of(const or_state* s, float fit, const float* desc) {
  const or_config* c = &s->cfg;
  if (!(fit == fit)) return -1;
  if (c->tess == OR_GRID) return or_grid_cell(desc, c->D, c->grid, c->lo, c->hi);
  return or_cvt_cell(desc, c->D, c->lo, c->hi, s->cent, c->C);
}

/* Filled cells in ascending order (Appendix A.2). */
static int32_t build_occ_list(or_state* s) {
  int32_t m = 0;
  for (int32_t c = 0; c < s->cfg.C; ++c)
    if (s->occ[c]) s->occ_list[m++] = c;
  return m;
}

/* Offspring j of generation g >= 1 (Appendix A.2, Algorithm 2):
 * parents drawn uniformly with replacement from the filled cells,
 * theta~ = theta1 + sigma1 eps1 + sigma2 eps2 (theta2 - theta1). */
static void make_offspring(or_state* s, uint32_t g, int32_t j, int32_t nocc, float* out,
                           int32_t* par) {
  const or_config* c = &s->cfg;
  int32_t n = s->n;
  uint32_t x[4];
  draw(s, 0, (uint32_t)j, g, TAG_SELECT, x);
  int32_t p1 = s->occ_list[(uint32_t)(((uint64_t)x[0] * (uint64_t)(uint32_t)nocc) >> 32)];
  int32_t p2 = s->occ_list[(uint32_t)(((uint64_t)x[1] * (uint64_t)(uint32_t)nocc) >> 32)];
  float lambda = c->line_sigma * or_normal(x[2]);
  const float* t1 = s->geno + (size_t)p1 * n;
  const float* t2 = s->geno + (size_t)p2 * n;
  uint32_t y[4] = {0, 0, 0, 0};
  for (int32_t i = 0; i < n; ++i) {
    /* block i/4 holds the words of genes i .. i+3, one normal each */
    if ((i & 3) == 0) draw(s, (uint32_t)(i >> 2), (uint32_t)j, g, TAG_ISO, y);
    float eps1 = or_normal(y[i & 3]);
    out[i] = fmaf(lambda, t2[i] - t1[i], fmaf(c->iso_sigma, eps1, t1[i]));
  }
  par[0] = p1;
  par[1] = p2;
}

/* Algorithm 1's insertion loop, in batch order. */
static void insert_sequential(or_state* s, int32_t nb, const float* fit, const float* desc,
                              const float* geno, const int32_t* cell, uint8_t* won) {
  const or_config* c = &s->cfg;
  int32_t n = s->n, D = c->D;
  int32_t* holder = (int32_t*)malloc(sizeof(int32_t) * (size_t)c->C);
  for (int32_t k = 0; k < c->C; ++k) holder[k] = -1;
  for (int32_t j = 0; j < nb; ++j) {
    won[j] = 0;
    int32_t k = cell[j];
    if (k < 0 || !(fit[j] == fit[j])) continue;       /* discarded (death flag) */
    int take = 0;
    if (!s->occ[k]) take = 1;                          /* empty cell: add        */
    else if (fit[j] > s->fit[k]) take = 1;             /* strictly better        */
    if (!take) continue;
    s->occ[k] = 1;
    s->fit[k] = fit[j];
    for (int32_t d = 0; d < D; ++d) s->desc[(size_t)k * D + d] = desc[(size_t)j * D + d];
    if (geno)
      memcpy(s->geno + (size_t)k * n, geno + (size_t)j * n, sizeof(float) * (size_t)n);
    holder[k] = j;
  }
  for (int32_t k = 0; k < c->C; ++k)
    if (holder[k] >= 0) won[holder[k]] = 1;
  free(holder);
}

/* Whole batches keep every offspring genotype, as the archive copies the
 * winners' rows after the sequential loop. */
static void ensure_offspring_storage(or_state* s) {
  if (!s->off_geno)
    s->off_geno = (float*)calloc((size_t)s->cfg.batch * (size_t)s->n, sizeof(float));
}

int32_t or_init(or_state* s) {
  const or_config* c = &s->cfg;
  or_setup(s);
  int32_t n = s->n, D = c->D, nb = c->batch;
  ensure_offspring_storage(s);
  /* the offspring are independent of one another: evaluated in parallel */
#pragma omp parallel for schedule(dynamic, 8)
  for (int32_t j = 0; j < nb; ++j) {
    float* x = s->off_geno + (size_t)j * n;
    init_genotype(s, j, x);
    evaluate(s, x, &s->off_fit[j], s->off_desc + (size_t)j * D);
    s->off_cell[j] = cell_of(s, s->off_fit[j], s->off_desc + (size_t)j * D);
    s->parents[2 * j] = -1;
    s->parents[2 * j + 1] = -1;
  }
  insert_sequential(s, nb, s->off_fit, s->off_desc, s->off_geno, s->off_cell, s->off_won);
  return 0;
}

int32_t or_generation(or_state* s, uint32_t g) {
  const or_config* c = &s->cfg;
  int32_t n = s->n, D = c->D, nb = c->batch;
  int32_t nocc = build_occ_list(s);
  if (nocc == 0) return -1;
  ensure_offspring_storage(s);
  /* select, vary, evaluate and map each offspring (independent of one
   * another, in parallel); then Algorithm 1's insertion loop in batch order */
#pragma omp parallel for schedule(dynamic, 8)
  for (int32_t j = 0; j < nb; ++j) {
    float* x = s->off_geno + (size_t)j * n;
    make_offspring(s, g, j, nocc, x, s->parents + 2 * j);
    evaluate(s, x, &s->off_fit[j], s->off_desc + (size_t)j * D);
    s->off_cell[j] = cell_of(s, s->off_fit[j], s->off_desc + (size_t)j * D);
  }
  insert_sequential(s, nb, s->off_fit, s->off_desc, s->off_geno, s->off_cell, s->off_won);
  return 0;
}

/* One offspring of generation g computed from the archive as it stands now
 * (g == 0: the random first batch).  Nothing is inserted. */
int32_t or_offspring(or_state* s, uint32_t g, int32_t j, float* geno, float* fit,
                     float* desc, int32_t* parents) {
  int32_t par[2] = {-1, -1};
  if (g == 0) {
    init_genotype(s, j, geno);
  } else {
    int32_t nocc = build_occ_list(s);
    if (nocc == 0) return -1;
    make_offspring(s, g, j, nocc, geno, par);
  }
  evaluate(s, geno, fit, desc);
  if (parents) { parents[0] = par[0]; parents[1] = par[1]; }
  return 0;
}

/* Offspring js[0 .. count) of generation g from the archive as it stands now
 * (g == 0: members of the random first batch): objectives, descriptors (D per
 * offspring) and parent pairs (-1 for the first batch), computed in parallel.
 * Nothing is inserted. */
int32_t or_offspring_many(or_state* s, uint32_t g, const int32_t* js, int32_t count,
                          float* fit, float* desc, int32_t* parents) {
  const int32_t D = s->cfg.D, n = s->n;
  const int32_t nocc = g == 0 ? 0 : build_occ_list(s);
  if (g != 0 && nocc == 0) return -1;
#pragma omp parallel
  {
    float* x = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
    float d4[4];
#pragma omp for schedule(dynamic, 1)
    for (int32_t i = 0; i < count; ++i) {
      if (g == 0) {
        init_genotype(s, js[i], x);
        parents[2 * i] = parents[2 * i + 1] = -1;
      } else {
        make_offspring(s, g, js[i], nocc, x, parents + 2 * i);
      }
      evaluate(s, x, &fit[i], d4);
      for (int32_t k = 0; k < D; ++k) desc[(size_t)i * D + k] = d4[k];
    }
    free(x);
  }
  return 0;
}

int32_t or_set_threads(int32_t n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
  return (int32_t)omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

/* Cell mapping and insertion driven by externally computed objectives and
 * descriptors (and optionally genotypes) of a batch of nb offspring. */
int32_t or_insert_driven(or_state* s, const float* fit, const float* desc,
                         const float* geno, int32_t nb, int32_t* cell, uint8_t* won) {
  for (int32_t j = 0; j < nb; ++j) cell[j] = cell_of(s, fit[j], desc + (size_t)j * s->cfg.D);
  insert_sequential(s, nb, fit, desc, geno, cell, won);
  return 0;
}

/* QD-score (Eq. 1) as sum over filled cells of (f + offset), coverage as the
 * number of filled cells, best objective (Appendix B.1). */
void or_stats(const or_state* s, double offset, double out[3]) {
  double qd = 0.0, best = -INFINITY;
  int64_t cnt = 0;
  for (int32_t c = 0; c < s->cfg.C; ++c) {
    if (!s->occ[c]) continue;
    cnt++;
    qd += (double)s->fit[c] + offset;
    if ((double)s->fit[c] > best) best = (double)s->fit[c];
  }
  out[0] = qd;
  out[1] = (double)cnt;
  out[2] = cnt ? best : NAN;
}

float* or_archive_geno(or_state* s) { return s->geno; }
float* or_archive_fit(or_state* s) { return s->fit; }
float* or_archive_desc(or_state* s) { return s->desc; }
uint8_t* or_archive_occ(or_state* s) { return s->occ; }
float* or_centroids(or_state* s) { return s->cent; }
float* or_env(or_state* s) { return s->env; }
int32_t* or_off_parents(or_state* s) { return s->parents; }
float* or_off_fit(or_state* s) { return s->off_fit; }
float* or_off_desc(or_state* s) { return s->off_desc; }
int32_t* or_off_cell(or_state* s) { return s->off_cell; }
uint8_t* or_off_won(or_state* s) { return s->off_won; }
float* or_off_geno(or_state* s) { return s->off_geno; }

/* ------------------------------------------------------------------------ */
/* Array forms of the primitives, for the pin tests' dense sweeps.           */
/* ------------------------------------------------------------------------ */
void or_map_f32(int32_t fn, const float* in, float* out, int64_t count) {
  for (int64_t i = 0; i < count; ++i) {
    float x = in[i];
    switch (fn) {
      case 1: out[i] = or_rsinpi(x); break;
      case 2: out[i] = or_expf(x); break;
      case 3: out[i] = or_tanhf(x); break;
      case 4: out[i] = or_sigmoidf(x); break;
      default: out[i] = NAN; break;
    }
  }
}

void or_philox_many(const uint32_t* ctr, const uint32_t key[2], uint32_t* out, int64_t count) {
  for (int64_t i = 0; i < count; ++i) or_philox(ctr + 4 * i, key, out + 4 * i);
}

void or_normal_many(const uint32_t* x, float* out, int64_t count) {
  for (int64_t i = 0; i < count; ++i) out[i] = or_normal(x[i]);
}
