// qd_kernels.hpp -- HIP kernels of one MAP-Elites generation for gfx950.
//
// Pipeline of one generation (Algorithm 1 after the first iteration; the
// first iteration runs the same kernels with the random-init genotype):
//   k_vary_eval   a wave takes 4 offspring (1 in batches of at most 2048, 2 in
//                 batches of at most 8192; two at a time, one per half-wave,
//                 for genotypes of at most 128 genes): draws their parents
//                 uniformly from the filled cells (Appendix A.2), runs Iso+LineDD
//                 (Algorithm 2) gene by gene on coalesced float4 rows of both parents with
//                 the objective / descriptor reduction (Appendix B.2) in the
//                 same pass, then finds each offspring's cell (grid bin, or
//                 exact nearest CVT centroid through a bucket grid) and inserts
//                 its packed key with a 64-bit atomicMax that only offspring
//                 beating the cell's current key issue.  Offspring genotypes
//                 are not stored.
//   k_rollout     (policies, qd_rollout.hpp) then k_insert_cvt_lds (a 4-D
//                 CVT of at most 2048 cells, searched from LDS) or k_insert:
//                 the same outputs; keys folded per wave (and per workgroup)
//                 before the atomics.
//   k_regen       a workgroup per few cells: a cell whose key now names an
//                 offspring regenerates that offspring's genotype into the
//                 cell's other genotype bank (the parents' banks were recorded
//                 per offspring, so they stay readable), records objective and
//                 descriptor, then flips its bank and marks the key incumbent.
//                 One more workgroup of this kernel compacts the filled cells
//                 (only when a new cell was filled) into the ascending list the
//                 next selection draws from.
#pragma once

#include "../../include/qd.h"
#include "qd_device.hpp"

namespace qd {

constexpr int kTaskRastrigin = 0, kTaskSphere = 1, kTaskProj = 2, kTaskMlp = 3;
constexpr int kTessGrid = 0, kTessCvt = 1;

struct Params {
  int task, tess, n, nb, D, C, stride;
  int grid[4];
  float lo[4], hi[4], span[4];    // span = hi - lo in fp32
  float iso_sigma, line_sigma, init_lo, init_span;
  int init_mode;                  // first batch: 0 uniform genes, 1 plus a level per half
  int obs, hid, act, T;
  Key key;
  int bucket_res, num_buckets;
  double inv_bucket_res;          // 1 / bucket_res
  uint64_t* arch_key;
  float* arch_fit;
  float* arch_desc;
  uint32_t* arch_slot;
  float* arch_geno;               // [2][C][stride]
  float* cent;                    // [C][D]
  int* bucket_start;              // [num_buckets + 1], then [num_buckets] cursors
  float4* bucket_pts;             // [C]
  int* bucket_idx;                // [C]
  int death_mode;                 // policies: 0 none, 1 truncate, 2 discard failed
  float death_below;              // failure: new state component 0 below this
  int cvt_samples;                // Lloyd points (set-up only)
  unsigned long long* lloyd_acc;  // [C][D + 1]: coordinate numerator sums, count
  int cand_res, cand_buckets;     // D = 2 CVT fine buckets (0: none)
  int* cand_count;                // [cand_buckets]
  float4* cand_pts;               // [cand_buckets][QD_CAND_SLOTS]
  float* env;
  int* occ_list;
  int* counters;                  // [0] filled cells, [1] flags, [3] occupancy changed
  int* off_par;
  float* off_fit;
  float* off_desc;
  int* off_cell;
  uint8_t* off_won;
  uint64_t* off_key;
  uint8_t* off_bank;              // bank of parent 1 | bank of parent 2 << 1
  float* off_geno;                // [N_B][stride] or null
  double* stats;
  const float4* ntab;   // Gaussian sampler table [QD_NORMAL_ROWS]
};

__device__ __forceinline__ float* geno_row(const Params& p, uint32_t bank, int cell) {
  return p.arch_geno + ((size_t)bank * (size_t)p.C + (size_t)cell) * (size_t)p.stride;
}

__device__ __forceinline__ int pick(const int* occ_list, uint32_t x, int nocc) {
  return occ_list[(uint32_t)(((uint64_t)x * (uint32_t)nocc) >> 32)];
}

// Parents and line coefficient of offspring j in generation g >= 1.
struct Pair {
  const float* row1;
  const float* row2;
  float lambda;
  int c1, c2;
  uint32_t banks;
  Tables tb;                      // the workgroup's sampler table (LDS)
};

__device__ __forceinline__ Pair select_pair(const Params& p, uint32_t g, int j, int nocc,
                                            const Tables& tb) {
  const uint4 x = philox(0u, (uint32_t)j, g, kTagSelect, p.key);
  Pair q;
  q.c1 = pick(p.occ_list, x.x, nocc);
  q.c2 = pick(p.occ_list, x.y, nocc);
  q.tb = tb;
  q.lambda = p.line_sigma * normal(x.z, tb);
  const uint32_t b1 = p.arch_slot[q.c1], b2 = p.arch_slot[q.c2];
  q.banks = b1 | (b2 << 1);
  q.row1 = geno_row(p, b1, q.c1);
  q.row2 = geno_row(p, b2, q.c2);
  return q;
}

// The same pair, rebuilt after the generation from what the offspring
// recorded (cells and banks) -- independent of the archive's current state.
__device__ __forceinline__ Pair pair_from_record(const Params& p, uint32_t g, int j, int c1, int c2,
                                                 uint32_t banks, const Tables& tb) {
  const uint4 x = philox(0u, (uint32_t)j, g, kTagSelect, p.key);
  Pair q;
  q.c1 = c1;
  q.c2 = c2;
  q.banks = banks;
  q.tb = tb;
  q.lambda = p.line_sigma * normal(x.z, tb);
  q.row1 = geno_row(p, q.banks & 1u, q.c1);
  q.row2 = geno_row(p, (q.banks >> 1) & 1u, q.c2);
  return q;
}

__device__ __forceinline__ Pair recorded_pair(const Params& p, uint32_t g, int j,
                                              const Tables& tb) {
  return pair_from_record(p, g, j, p.off_par[2 * j], p.off_par[2 * j + 1], p.off_bank[j], tb);
}

// Genes base..base+3 of offspring j (base a multiple of 4).  GEN0: the random
// first batch of a test function, lo + U (hi - lo).  Otherwise Algorithm 2:
// theta1 + sigma1 eps1 + lambda (theta2 - theta1), eps1 from block base/4.
template <bool GEN0>
__device__ __forceinline__ float4 make_genes(const Params& p, const Pair& q, uint32_t g, int j,
                                             int base) {
  if (GEN0) {
    const uint4 x = philox((uint32_t)(base >> 2), (uint32_t)j, 0u, kTagInit, p.key);
    float4 v = make_float4(fma32(unit24(x.x), p.init_span, p.init_lo),
                           fma32(unit24(x.y), p.init_span, p.init_lo),
                           fma32(unit24(x.z), p.init_span, p.init_lo),
                           fma32(unit24(x.w), p.init_span, p.init_lo));
    if (p.init_mode == 1) {
      // spread first batch: a level per genotype half, uniform over that
      // descriptor dimension's box (word h of block (0, j, 0, INIT_LEVEL))
      const uint4 y = philox(0u, (uint32_t)j, 0u, kTagInitLevel, p.key);
      const float l0 = fma32(unit24(y.x), p.span[0], p.lo[0]);
      const float l1 = fma32(unit24(y.y), p.span[1], p.lo[1]);
      const int half = p.n >> 1;
      v.x = (base < half ? l0 : l1) + v.x;
      v.y = (base + 1 < half ? l0 : l1) + v.y;
      v.z = (base + 2 < half ? l0 : l1) + v.z;
      v.w = (base + 3 < half ? l0 : l1) + v.w;
    }
    return v;
  } else {
    // wave-uniform row pointer + 32-bit unsigned byte offset (rows are far
    // below 4 GiB): the address form of a scalar base and a vector offset
    const uint32_t off = 4u * (uint32_t)base;
    const float4 t1 = *reinterpret_cast<const float4*>(reinterpret_cast<const char*>(q.row1) + off);
    const float4 t2 = *reinterpret_cast<const float4*>(reinterpret_cast<const char*>(q.row2) + off);
    const uint4 x = philox((uint32_t)(base >> 2), (uint32_t)j, g, kTagIso, p.key);
    const float e0 = normal(x.x, q.tb), e1 = normal(x.y, q.tb);
    const float e2 = normal(x.z, q.tb), e3 = normal(x.w, q.tb);
    const float s1 = p.iso_sigma, l = q.lambda;
    return make_float4(fma32(l, t2.x - t1.x, fma32(s1, e0, t1.x)),
                       fma32(l, t2.y - t1.y, fma32(s1, e1, t1.y)),
                       fma32(l, t2.z - t1.z, fma32(s1, e2, t1.z)),
                       fma32(l, t2.w - t1.w, fma32(s1, e3, t1.w)));
  }
}

// min(max(x, lo), hi) for lo < hi and x not NaN, in one v_med3_f32.
__device__ __forceinline__ float clip(float x, float lo, float hi) {
  return __builtin_amdgcn_fmed3f(x, lo, hi);
}

template <int TASK>
__device__ __forceinline__ float task_term(float x) {
  if (TASK == kTaskSphere) return x * x;
  const float s = rsinpi(x);   // x^2 + 20 sin^2(pi x) = x^2 + s^2
  return fma32(s, s, x * x);
}

// ---------------------------------------------------------------------------
// Descriptor -> cell.  Every lane of the calling wave holds the same
// descriptor and gets the same answer.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int grid_cell(const Params& p, const float* d) {
  int cell = 0;
  for (int k = 0; k < p.D; ++k) {
    if (!(d[k] == d[k])) return -1;
    const float t = (d[k] - p.lo[k]) / p.span[k];
    const float fb = __builtin_floorf(t * (float)p.grid[k]);
    const int b = fb < 0.0f ? 0 : (fb > (float)(p.grid[k] - 1) ? p.grid[k] - 1 : (int)fb);
    cell = cell * p.grid[k] + b;
  }
  return cell;
}

// Exact nearest centroid of u = (d - lo) / (hi - lo): squared distance as an
// fma chain over dimensions from 0, ties to the lowest centroid index -- the
// brute-force argmin -- found by one thread through a bucket grid of
// bucket_res^D cells over the unit box.  Rings of buckets (Chebyshev distance
// r from the query's bucket) are visited in order until the best distance is
// certainly below the distance to every unvisited bucket (a relative margin of
// 1e-5, far above the fp32 rounding of either side).
template <int D>
__device__ __forceinline__ void visit_range(const Params& p, int s0, int s1, const float* u,
                                            float& best, int& best_idx) {
  for (int s = s0; s < s1; ++s) {
    const float4 c = p.bucket_pts[s];
    const float cc[4] = {c.x, c.y, c.z, c.w};
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < D; ++k) {
      const float diff = u[k] - cc[k];
      acc = fma32(diff, diff, acc);
    }
    const int idx = p.bucket_idx[s];
    if (acc < best || (acc == best && idx < best_idx)) {
      best = acc;
      best_idx = idx;
    }
  }
}

template <int D>
__device__ __forceinline__ void visit_bucket(const Params& p, int bucket, const float* u,
                                             float& best, int& best_idx) {
  visit_range<D>(p, p.bucket_start[bucket], p.bucket_start[bucket + 1], u, best, best_idx);
}

template <int D>
__device__ int cvt_cell(const Params& p, const float* d) {
  const int R = p.bucket_res;
  float u[D];
  int qb[D];
#pragma unroll
  for (int k = 0; k < D; ++k) {
    if (!(d[k] == d[k])) return -1;
    u[k] = (d[k] - p.lo[k]) / p.span[k];
    float fb = __builtin_floorf(u[k] * (float)R);
    fb = fb < 0.0f ? 0.0f : (fb > (float)(R - 1) ? (float)(R - 1) : fb);
    qb[k] = (int)fb;
  }
  float best = __builtin_inff();
  int best_idx = 0x7fffffff;
  int r0 = 0;
  if (D == 2) {
    // rings 0 and 1 together: all 9 bucket ranges, then the first centroid of
    // each bucket, are fetched with independent loads (one round trip each)
    int st[9], en[9];
#pragma unroll
    for (int i = 0; i < 9; ++i) {
      const int b0 = qb[0] + i / 3 - 1, b1 = qb[1] + i % 3 - 1;
      const bool in = b0 >= 0 && b0 < R && b1 >= 0 && b1 < R;
      const int bucket = in ? b0 * R + b1 : 0;
      st[i] = in ? p.bucket_start[bucket] : 0;
      en[i] = in ? p.bucket_start[bucket + 1] : 0;
    }
    float4 first[9];
    int fidx[9];
#pragma unroll
    for (int i = 0; i < 9; ++i) {
      const bool any = st[i] < en[i];
      first[i] = any ? p.bucket_pts[st[i]] : make_float4(0.f, 0.f, 0.f, 0.f);
      fidx[i] = any ? p.bucket_idx[st[i]] : 0;
    }
#pragma unroll
    for (int i = 0; i < 9; ++i) {
      if (st[i] < en[i]) {
        const float d0 = u[0] - first[i].x;
        float acc = fma32(d0, d0, 0.0f);
        const float d1 = u[1] - first[i].y;
        acc = fma32(d1, d1, acc);
        if (acc < best || (acc == best && fidx[i] < best_idx)) {
          best = acc;
          best_idx = fidx[i];
        }
      }
    }
    for (int i = 0; i < 9; ++i)
      if (st[i] + 1 < en[i]) visit_range<D>(p, st[i] + 1, en[i], u, best, best_idx);
    r0 = 1;
  }
  for (int r = r0; r < R; ++r) {
    if (r > r0 || D != 2) {
      // the buckets at Chebyshev distance exactly r that lie in the grid
      if (D == 2) {
      for (int o0 = -r; o0 <= r; ++o0) {
        const int b0 = qb[0] + o0;
        if (b0 < 0 || b0 >= R) continue;
        const int step = (o0 == -r || o0 == r) ? 1 : 2 * r;
        for (int o1 = -r; o1 <= r; o1 += step) {
          const int b1 = qb[1] + o1;
          if (b1 >= 0 && b1 < R) visit_bucket<D>(p, b0 * R + b1, u, best, best_idx);
        }
      }
    } else {
      for (int o0 = -r; o0 <= r; ++o0) {
        const int b0 = qb[0] + o0;
        if (b0 < 0 || b0 >= R) continue;
        for (int o1 = -r; o1 <= r; ++o1) {
          const int b1 = qb[1] + o1;
          if (b1 < 0 || b1 >= R) continue;
          for (int o2 = -r; o2 <= r; ++o2) {
            const int b2 = qb[2] + o2;
            if (b2 < 0 || b2 >= R) continue;
            const bool edge = o0 == -r || o0 == r || o1 == -r || o1 == r || o2 == -r || o2 == r;
            const int step = (edge || r == 0) ? 1 : 2 * r;
            for (int o3 = -r; o3 <= r; o3 += step) {
              const int b3 = qb[3] + o3;
              if (b3 >= 0 && b3 < R)
                visit_bucket<D>(p, ((b0 * R + b1) * R + b2) * R + b3, u, best, best_idx);
            }
          }
        }
      }
    }
    }
    // lower bound on the distance to anything outside the visited box
    double bound = __builtin_inf();
    bool face = false;
#pragma unroll
    for (int k = 0; k < D; ++k) {
      if (qb[k] - r >= 1) {
        const double gap = (double)u[k] - (double)(qb[k] - r) * p.inv_bucket_res - 1e-6;
        bound = fmin(bound, gap > 0.0 ? gap * gap : 0.0);
        face = true;
      }
      if (qb[k] + r + 1 <= R - 1) {
        const double gap = (double)(qb[k] + r + 1) * p.inv_bucket_res - (double)u[k] - 1e-6;
        bound = fmin(bound, gap > 0.0 ? gap * gap : 0.0);
        face = true;
      }
    }
    if (!face) break;
    if (best_idx != 0x7fffffff && (double)best * (1.0 + 1e-5) < bound) break;
  }
  return best_idx;
}

// Nearest centroid for four offspring at once, on a two-dimensional CVT with
// candidate lists: the 16 lanes of row i take the descriptor (d0, d1) held by
// lane i, look up its fine bucket and test one candidate each, then keep the
// smallest (distance, index) pair of the row -- the brute-force argmin with
// ties to the lower index, as the list holds every centroid that can win.
// Lane i gets offspring i's cell: -1 for a NaN descriptor, -2 when its bucket
// lists more than QD_CAND_SLOTS centroids or the descriptor lies outside the
// box (the caller then runs the ring search).  Every lane must call it.
__device__ __forceinline__ int cvt_cell_rows(const Params& p, float d0, float d1, int lane) {
  const int row = lane >> 4, sub = lane & 15;
  const float g0 = __shfl(d0, row, 64), g1 = __shfl(d1, row, 64);
  const bool nan = !(g0 == g0 && g1 == g1);
  const float u0 = (g0 - p.lo[0]) / p.span[0];
  const float u1 = (g1 - p.lo[1]) / p.span[1];
  const bool inside = !nan && u0 >= 0.0f && u0 <= 1.0f && u1 >= 0.0f && u1 <= 1.0f;
  float best = __builtin_inff();
  int best_idx = 0x7fffffff;
  int cnt = 0;
  if (inside) {
    const int R = p.cand_res;
    const int q0 = __builtin_fminf(__builtin_floorf(u0 * (float)R), (float)(R - 1));
    const int q1 = __builtin_fminf(__builtin_floorf(u1 * (float)R), (float)(R - 1));
    const int bucket = q0 * R + q1;
    cnt = p.cand_count[bucket];
    if (cnt <= QD_CAND_SLOTS && sub < cnt) {
      const float4 c = p.cand_pts[(size_t)bucket * QD_CAND_SLOTS + sub];
      const float e0 = u0 - c.x;
      float acc = fma32(e0, e0, 0.0f);
      const float e1 = u1 - c.y;
      acc = fma32(e1, e1, acc);
      best = acc;
      best_idx = __float_as_int(c.z);
    }
  }
  min_pair_row<8>(best, best_idx);
  min_pair_row<4>(best, best_idx);
  min_pair_row<2>(best, best_idx);
  min_pair_row<1>(best, best_idx);
  // an empty list (never built: every bucket lists the centroid that sets its
  // distance bound) would leave best_idx unset; the ring search takes it then
  const int res = nan ? -1
                      : (inside && cnt <= QD_CAND_SLOTS && best_idx != 0x7fffffff ? best_idx : -2);
  return __shfl(res, (lane & 3) * 16, 64);
}

// Insertion key: order-preserving bits of the objective (-0 as +0), then
// N_B-1-j so that equal objectives go to the lowest batch index; 0 = none.
__device__ __forceinline__ uint64_t insert_key(const Params& p, float f, int cell, int j) {
  return cell < 0 ? 0ull
                  : ((uint64_t)order_bits(f) << 32) | (uint64_t)(uint32_t)(p.nb - 1 - j);
}

// Writes the batch outputs of offspring j (called by one lane).
__device__ __forceinline__ void record_offspring(const Params& p, int j, const Pair& q, float f,
                                                 const float* d) {
  p.off_fit[j] = f;
  for (int k = 0; k < p.D; ++k) p.off_desc[(size_t)j * p.D + k] = d[k];
  p.off_par[2 * j] = q.c1;
  p.off_par[2 * j + 1] = q.c2;
  p.off_bank[j] = (uint8_t)q.banks;
  p.off_won[j] = 0;
}

__device__ __forceinline__ void record_empty_archive(const Params& p, int j) {
  p.off_fit[j] = __builtin_nanf("");
  p.off_par[2 * j] = -1;
  p.off_par[2 * j + 1] = -1;
  p.off_bank[j] = 0;
  p.off_cell[j] = -1;
  p.off_key[j] = 0ull;
  p.off_won[j] = 0;
  atomicOr(reinterpret_cast<unsigned int*>(p.counters + 1), 1u);
}

// Inserts one packed key: an atomicMax on the cell's key, skipped when an
// agent-scope read already shows a key at least as large (keys only grow),
// so only offspring that beat everything seen so far reach the atomic unit.
// An atomic that finds an empty cell raises the occupancy-changed flag.
__device__ __forceinline__ void insert_one(const Params& p, int cell, uint64_t key) {
  if (cell < 0) return;
  unsigned long long* slot = (unsigned long long*)&p.arch_key[cell];
  const unsigned long long cur = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (key <= cur) return;
  if (atomicMax(slot, (unsigned long long)key) == 0ull) p.counters[3] = 1;
}

// ---------------------------------------------------------------------------
// Select + vary + evaluate + cell + insert (test functions).  A wave takes
// OPW consecutive offspring: lanes 0 .. OPW-1 draw their parents together,
// then the whole wave runs each offspring's genes in turn (lane l owns genes
// 256c + 4l .. 256c + 4l + 3 of every chunk c, i.e. gene groups q = g/4 with
// q mod 64 = l; its partial sums run in ascending gene order and the wave
// folds them pairwise, h = 32 .. 1); finally lanes 0 .. OPW-1 find their
// offspring's cell and insert its key.  Large batches take four offspring per
// wave (the per-wave set-up -- sampler table, selection -- spread over more
// work); small ones fewer, since there a generation is a chain of dependent
// memory round trips and more waves in flight shorten it: one offspring per
// wave up to kOneOffspringBatch, two up to kTwoOffspringBatch.  Every choice
// gives the same bits (each offspring's arithmetic does not depend on it).
// ---------------------------------------------------------------------------
constexpr int kOffspringPerWave = 4;             // the most a wave takes
constexpr int kOneOffspringBatch = 2048;
constexpr int kTwoOffspringBatch = 8192;

inline int offspring_per_wave(int nb) {
  return nb <= kOneOffspringBatch ? 1 : (nb <= kTwoOffspringBatch ? 2 : kOffspringPerWave);
}

template <int TASK, bool GEN0, bool KEEP, int OPW>
__global__ __launch_bounds__(256) void k_vary_eval(const Params p, uint32_t g) {
  static_assert(OPW == 1 || OPW == 2 || OPW == kOffspringPerWave, "one, two or four offspring");
  __shared__ float4 s_ntab[kNormalRows];
  const Tables tb{s_ntab};
  const int lane = threadIdx.x & 63;
  const int j0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * OPW;
  const int nmine = p.nb - j0 < OPW ? p.nb - j0 : OPW;
  const bool mine = lane < nmine;          // lane i speaks for offspring j0 + i

  // The parents' cells and banks (Appendix A.2) are read while the sampler
  // table is being staged: the chain filled-cell count -> list entry -> bank
  // runs beside the table's loads; the line coefficient, which needs the
  // table, comes after the barrier.
  Pair sel{nullptr, nullptr, 0.0f, -1, -1, 0u};
  int nocc = 0;
  uint32_t sel_z = 0u;
  if (!GEN0) {
    nocc = p.counters[0];
    if (mine && nocc > 0) {
      const uint4 x = philox(0u, (uint32_t)(j0 + lane), g, kTagSelect, p.key);
      sel.c1 = pick(p.occ_list, x.x, nocc);
      sel.c2 = pick(p.occ_list, x.y, nocc);
      sel.banks = p.arch_slot[sel.c1] | (p.arch_slot[sel.c2] << 1);
      sel_z = x.z;
    }
    stage_normal_table(s_ntab, p.ntab, (int)threadIdx.x, 256);
    __syncthreads();
  }
  if (j0 >= p.nb) return;
  if (!GEN0) {
    if (nocc <= 0) {
      if (mine) record_empty_archive(p, j0 + lane);
      return;
    }
    if (mine) {
      sel.lambda = p.line_sigma * normal(sel_z, tb);
      sel.row1 = geno_row(p, sel.banks & 1u, sel.c1);
      sel.row2 = geno_row(p, (sel.banks >> 1) & 1u, sel.c2);
    }
  }

  const int n = p.n;
  const int half = n >> 1;
  float my_f = 0.0f, my_d0 = 0.0f, my_d1 = 0.0f;
  if (TASK != kTaskProj && n <= 128) {
    // Short genotypes: two offspring at a time, one per 32-lane half (lane h
    // of a half owns genes 4h .. 4h + 3, as lane h of a whole wave would, and
    // the fold stays in the half).  With an odd count the spare half repeats
    // its partner and its result is dropped.
    const int hl = lane >> 5, hlane = lane & 31;
    for (int i = 0; i < nmine; i += 2) {
      const int ib = i + 1 < nmine ? i + 1 : i;   // the upper half's offspring slot
      const int j = j0 + (hl ? ib : i);
      Pair q{nullptr, nullptr, 0.0f, -1, -1, 0u, tb};
      if (!GEN0) {
        const int c1a = __builtin_amdgcn_readlane(sel.c1, i), c1b = __builtin_amdgcn_readlane(sel.c1, ib);
        const int c2a = __builtin_amdgcn_readlane(sel.c2, i), c2b = __builtin_amdgcn_readlane(sel.c2, ib);
        const int bka = __builtin_amdgcn_readlane((int)sel.banks, i);
        const int bkb = __builtin_amdgcn_readlane((int)sel.banks, ib);
        const uint32_t lma = __builtin_amdgcn_readlane(__float_as_uint(sel.lambda), i);
        const uint32_t lmb = __builtin_amdgcn_readlane(__float_as_uint(sel.lambda), ib);
        q.c1 = hl ? c1b : c1a;
        q.c2 = hl ? c2b : c2a;
        q.banks = (uint32_t)(hl ? bkb : bka);
        q.lambda = __uint_as_float(hl ? lmb : lma);
        q.row1 = geno_row(p, q.banks & 1u, q.c1);
        q.row2 = geno_row(p, (q.banks >> 1) & 1u, q.c2);
      }
      const int base = 4 * hlane;
      float acc = 0.0f, g0 = 0.0f, g1 = 0.0f;
      if (base < n) {
        const float4 v4 = make_genes<GEN0>(p, q, g, j, base);
        if (KEEP && (hl == 0 || ib != i))
          *reinterpret_cast<float4*>(p.off_geno + (size_t)j * (size_t)p.stride + base) = v4;
        g0 = v4.x;
        g1 = v4.y;
        const float v[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (base + k < n) acc = acc + task_term<TASK>(v[k]);
      }
      const float f = half_fold_sum(acc);
      const float fa = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(f), 0));
      const float fb = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(f), 32));
      const float g0a = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(g0), 0));
      const float g1a = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(g1), 0));
      const float g0b = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(g0), 32));
      const float g1b = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(g1), 32));
      if (lane == i) {
        my_f = -fa;
        my_d0 = clip(g0a, p.lo[0], p.hi[0]);
        my_d1 = clip(g1a, p.lo[1], p.hi[1]);
      } else if (lane == ib) {
        my_f = -fb;
        my_d0 = clip(g0b, p.lo[0], p.hi[0]);
        my_d1 = clip(g1b, p.lo[1], p.hi[1]);
      }
    }
  } else
  for (int i = 0; i < nmine; ++i) {
    const int j = j0 + i;
    Pair q{nullptr, nullptr, 0.0f, -1, -1, 0u, tb};
    if (!GEN0) {
      // lane i's selection, read into scalar registers (i is wave-uniform)
      q.c1 = __builtin_amdgcn_readlane(sel.c1, i);
      q.c2 = __builtin_amdgcn_readlane(sel.c2, i);
      q.banks = (uint32_t)__builtin_amdgcn_readlane((int)sel.banks, i);
      q.lambda = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(sel.lambda), i));
      q.row1 = geno_row(p, q.banks & 1u, q.c1);
      q.row2 = geno_row(p, (q.banks >> 1) & 1u, q.c2);
    }
    float acc = 0.0f, dlo = 0.0f, dhi = 0.0f;
    float g0 = 0.0f, g1 = 0.0f;
    float* keep_row = KEEP ? p.off_geno + (size_t)j * (size_t)p.stride : nullptr;
    const int nchunks = (n + 255) >> 8;
    for (int c = 0; c < nchunks; ++c) {   // a wave-uniform trip count
      const int base = 256 * c + 4 * lane;
      if (base >= n) continue;
      const float4 v4 = make_genes<GEN0>(p, q, g, j, base);
      if (KEEP) *reinterpret_cast<float4*>(keep_row + base) = v4;
      if (base == 0) {
        g0 = v4.x;
        g1 = v4.y;
      }
      if (base + 4 <= n) {
        // whole block: the same additions in the same order, without per-gene tests
        acc = acc + task_term<TASK>(v4.x);
        acc = acc + task_term<TASK>(v4.y);
        acc = acc + task_term<TASK>(v4.z);
        acc = acc + task_term<TASK>(v4.w);
        if (TASK == kTaskProj) {
          if (base + 4 <= half) {
            dlo = dlo + clip(v4.x, p.lo[0], p.hi[0]);
            dlo = dlo + clip(v4.y, p.lo[0], p.hi[0]);
            dlo = dlo + clip(v4.z, p.lo[0], p.hi[0]);
            dlo = dlo + clip(v4.w, p.lo[0], p.hi[0]);
          } else if (base >= half) {
            dhi = dhi + clip(v4.x, p.lo[1], p.hi[1]);
            dhi = dhi + clip(v4.y, p.lo[1], p.hi[1]);
            dhi = dhi + clip(v4.z, p.lo[1], p.hi[1]);
            dhi = dhi + clip(v4.w, p.lo[1], p.hi[1]);
          } else {
            const float v[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              if (base + k < half) dlo = dlo + clip(v[k], p.lo[0], p.hi[0]);
              else dhi = dhi + clip(v[k], p.lo[1], p.hi[1]);
            }
          }
        }
      } else {
        // ragged last block
        const float v[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int gi = base + k;
          if (gi < n) {
            acc = acc + task_term<TASK>(v[k]);
            if (TASK == kTaskProj) {
              if (gi < half) dlo = dlo + clip(v[k], p.lo[0], p.hi[0]);
              else dhi = dhi + clip(v[k], p.lo[1], p.hi[1]);
            }
          }
        }
      }
    }
    // folded sums (wave-uniform); lane i keeps offspring i's, and divides the
    // half sums once after the loop
    float f, d0, d1;
    if (TASK == kTaskProj) {
      wave_fold_sum3(acc, dlo, dhi, f, d0, d1);
    } else {
      f = wave_fold_sum(acc);
      d0 = clip(__uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(g0), 0)), p.lo[0], p.hi[0]);
      d1 = clip(__uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(g1), 0)), p.lo[1], p.hi[1]);
    }
    if (lane == i) {
      my_f = -f;
      my_d0 = d0;
      my_d1 = d1;
    }
  }
  if (TASK == kTaskProj) {
    my_d0 = my_d0 / (float)half;
    my_d1 = my_d1 / (float)(n - half);
  }
  const int listed = p.tess == kTessCvt && p.cand_res > 0 ? cvt_cell_rows(p, my_d0, my_d1, lane) : -2;
  if (mine) {
    const int j = j0 + lane;
    const float d[2] = {my_d0, my_d1};
    int cell = -1;
    if (my_f == my_f) {
      if (p.tess == kTessGrid) cell = grid_cell(p, d);
      else cell = listed != -2 ? listed : cvt_cell<2>(p, d);
    }
    const uint64_t key = insert_key(p, my_f, cell, j);
    record_offspring(p, j, sel, my_f, d);
    p.off_cell[j] = cell;
    p.off_key[j] = key;
    insert_one(p, cell, key);
  }
}

// ---------------------------------------------------------------------------
// Insertion.  One thread per offspring finds its cell and packs its key; keys
// are then folded per wave (lanes sharing a cell) and per workgroup in an LDS
// hash table, so each workgroup issues at most one global 64-bit atomicMax per
// distinct cell it saw -- and none when a plain read of the cell's key already
// shows a key at least as large (keys only grow, so a stale read can only make
// the workgroup do an atomic it did not need).  A batch crowding into a few
// cells therefore does not serialise on them.  An atomic that finds an empty
// cell raises the "occupancy changed" flag read by the compaction.
// ---------------------------------------------------------------------------
constexpr int kInsertBlock = 256, kInsertSlots = 512;

template <int TESS, int D>
__global__ __launch_bounds__(kInsertBlock) void k_insert(const Params p) {
  __shared__ int tag[kInsertSlots];
  __shared__ unsigned long long kmax[kInsertSlots];
  for (int e = threadIdx.x; e < kInsertSlots; e += kInsertBlock) {
    tag[e] = -1;
    kmax[e] = 0ull;
  }
  __syncthreads();
  const int j = blockIdx.x * kInsertBlock + threadIdx.x;
  int cell = -1;
  uint64_t key = 0ull;
  if (j < p.nb) {
    const float f = p.off_fit[j];
    if (f == f) {
      float d[D];
#pragma unroll
      for (int k = 0; k < D; ++k) d[k] = p.off_desc[(size_t)j * D + k];
      cell = TESS == kTessGrid ? grid_cell(p, d) : cvt_cell<D>(p, d);
    }
    key = insert_key(p, f, cell, j);
    p.off_cell[j] = cell;
    p.off_key[j] = key;
  }
  uint64_t todo = __ballot(cell >= 0);
  while (todo) {
    const int leader = __ffsll((unsigned long long)todo) - 1;
    const int c = __shfl(cell, leader, 64);
    const uint64_t same = __ballot(cell == c);
    uint64_t k = cell == c ? key : 0ull;
#pragma unroll
    for (int h = 32; h >= 1; h >>= 1) {
      const uint64_t o = __shfl_xor(k, h, 64);
      k = o > k ? o : k;
    }
    if (lane_id() == leader) {
      int h = (int)(((uint32_t)c * 2654435761u) >> 23) & (kInsertSlots - 1);
      for (;;) {   // at most kInsertBlock distinct cells: a free slot always exists
        const int t = atomicCAS(&tag[h], -1, c);
        if (t == -1 || t == c) {
          atomicMax(&kmax[h], (unsigned long long)k);
          break;
        }
        h = (h + 1) & (kInsertSlots - 1);
      }
    }
    todo &= ~same;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kInsertSlots; e += kInsertBlock) {
    const int c = tag[e];
    if (c < 0) continue;
    const unsigned long long k = kmax[e];
    unsigned long long* slot = (unsigned long long*)&p.arch_key[c];
    if (k <= *slot) continue;
    if (atomicMax(slot, k) == 0ull) p.counters[3] = 1;
  }
}

// Insertion on a four-dimensional CVT small enough for LDS (C <= kCvtLdsCells):
// the workgroup stages every centroid in LDS and takes kInsertLdsOffspring
// offspring, four per wave, 16 lanes per offspring.  Lane s of a row
// measures centroids s, s + 16, ... (the same fma chain as the ring search,
// keeping the first smallest), then the row keeps its smallest (distance,
// index) pair -- the brute-force argmin with ties to the lower index.  Wave 0
// then packs the keys and folds them per cell before the global atomicMax.
constexpr int kCvtLdsCells = 2048, kInsertLdsOffspring = 16;

// Squared distance from u to centroid c: fma chain over the dimensions.
__device__ __forceinline__ float cvt_dist4(const float* u, const float4& c) {
  const float cc[4] = {c.x, c.y, c.z, c.w};
  float acc = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float diff = u[k] - cc[k];
    acc = fma32(diff, diff, acc);
  }
  return acc;
}

__global__ __launch_bounds__(256) void k_insert_cvt_lds(const Params p) {
  constexpr int D = 4;
  __shared__ float4 s_cent[kCvtLdsCells];
  __shared__ int s_cell[kInsertLdsOffspring];
  const float4* cent = reinterpret_cast<const float4*>(p.cent);
  for (int i = threadIdx.x; i < p.C; i += 256) s_cent[i] = cent[i];
  __syncthreads();
  const int lane = lane_id(), wave = threadIdx.x >> 6, row = lane >> 4, sub = lane & 15;
  const int first = blockIdx.x * kInsertLdsOffspring;
#pragma unroll 1
  for (int r = 0; r < kInsertLdsOffspring / 16; ++r) {
    const int t = r * 16 + wave * 4 + row;
    const int j = first + t;
    bool live = false;
    float u[D];
    if (j < p.nb && p.off_fit[j] == p.off_fit[j]) {
      live = true;
#pragma unroll
      for (int k = 0; k < D; ++k) {
        const float d = p.off_desc[(size_t)j * D + k];
        live = live && d == d;
        u[k] = (d - p.lo[k]) / p.span[k];
      }
    }
    float best = __builtin_inff();
    int best_idx = 0x7fffffff;
    if (live) {
      int i = sub;
      for (; i + 48 < p.C; i += 64) {   // four loads in flight, compared in index order
        float4 c4[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) c4[q] = s_cent[i + 16 * q];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float acc = cvt_dist4(u, c4[q]);
          // (distance, index) order, as the ring search: an infinite distance
          // still names a centroid, so a live row always gets a cell < C
          if (acc < best || (acc == best && i + 16 * q < best_idx)) {
            best = acc;
            best_idx = i + 16 * q;
          }
        }
      }
      for (; i < p.C; i += 16) {
        const float acc = cvt_dist4(u, s_cent[i]);
        if (acc < best || (acc == best && i < best_idx)) {
          best = acc;
          best_idx = i;
        }
      }
    }
    min_pair_row<8>(best, best_idx);
    min_pair_row<4>(best, best_idx);
    min_pair_row<2>(best, best_idx);
    min_pair_row<1>(best, best_idx);
    if (sub == 0) s_cell[t] = live ? best_idx : -1;
  }
  __syncthreads();
  if (wave != 0) return;
  // lanes 0 .. kInsertLdsOffspring - 1 of wave 0 take this workgroup's offspring
  static_assert(kInsertLdsOffspring % 16 == 0 && kInsertLdsOffspring <= 64, "one wave folds them");
  const int j = first + lane;
  int cell = -1;
  uint64_t key = 0ull;
  if (lane < kInsertLdsOffspring && j < p.nb) {
    cell = s_cell[lane];
    key = insert_key(p, p.off_fit[j], cell, j);
    p.off_cell[j] = cell;
    p.off_key[j] = key;
  }
  uint64_t todo = __ballot(cell >= 0);
  while (todo) {
    const int leader = __ffsll((unsigned long long)todo) - 1;
    const int c = __shfl(cell, leader, 64);
    const uint64_t same = __ballot(cell == c);
    uint64_t k = cell == c ? key : 0ull;
#pragma unroll
    for (int h = 32; h >= 1; h >>= 1) {
      const uint64_t o = __shfl_xor(k, h, 64);
      k = o > k ? o : k;
    }
    if (lane == leader) insert_one(p, c, k);
    todo &= ~same;
  }
}

// ---------------------------------------------------------------------------
// Compaction of the filled cells into the ascending list the next selection
// draws from (Appendix A.2).  Run by one extra workgroup of the winner kernel,
// only when an insertion filled a new cell (counters[3]); it clears that flag.
// The winner workgroups running beside it change keys only from one non-zero
// value to another, so filled/empty is already final.
// ---------------------------------------------------------------------------
constexpr int kCompactItems = 16;

__device__ void compact_filled(const Params& p) {
  constexpr int kThreads = 256;
  __shared__ int wave_tot[kThreads / 64];
  __shared__ int base_sh;
  if (p.counters[3] == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) base_sh = 0;
  for (int start = 0; start < p.C; start += kThreads * kCompactItems) {
    const int c0 = start + tid * kCompactItems;
    uint64_t keys[kCompactItems];
#pragma unroll
    for (int i = 0; i < kCompactItems; ++i) keys[i] = c0 + i < p.C ? p.arch_key[c0 + i] : 0ull;
    uint32_t filled = 0u;
#pragma unroll
    for (int i = 0; i < kCompactItems; ++i) filled |= (keys[i] != 0ull ? 1u : 0u) << i;
    const int cnt = __popc(filled);
    int incl = cnt;
#pragma unroll
    for (int h = 1; h < 64; h <<= 1) {
      const int o = __shfl_up(incl, h, 64);
      if (lane >= h) incl += o;
    }
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int off = base_sh + incl - cnt;
    for (int w = 0; w < wave; ++w) off += wave_tot[w];
#pragma unroll
    for (int i = 0; i < kCompactItems; ++i)
      if ((filled >> i) & 1u) p.occ_list[off++] = c0 + i;
    __syncthreads();
    if (tid == 0) {
      int tot = 0;
      for (int w = 0; w < kThreads / 64; ++w) tot += wave_tot[w];
      base_sh += tot;
    }
    __syncthreads();
  }
  if (tid == 0) {
    p.counters[0] = base_sh;
    p.counters[3] = 0;
  }
}

// ---------------------------------------------------------------------------
// Winners: a workgroup takes kRegenCells consecutive cells, kRegenCellsPerWave
// to each of its four waves.  For each of its cells whose key names an
// offspring, a wave regenerates that offspring's genotype into the cell's
// other bank from the recorded parents; then the wave's cells record
// objective and descriptor, switch to the new bank, and turn the key into the
// incumbent form (low word all ones: a later offspring must be strictly
// better).  No other wave touches those cells.
// ---------------------------------------------------------------------------
constexpr int kRegenCellsPerWave = 8;
constexpr int kRegenCells = 4 * kRegenCellsPerWave;

__device__ __forceinline__ void finish_winner(const Params& p, int c, int j, uint64_t key) {
  p.arch_fit[c] = p.off_fit[j];
  for (int k = 0; k < p.D; ++k) p.arch_desc[(size_t)c * p.D + k] = p.off_desc[(size_t)j * p.D + k];
  p.off_won[j] = 1;
  p.arch_slot[c] ^= 1u;
  p.arch_key[c] = key | 0xffffffffull;
}

__device__ __forceinline__ bool names_offspring(uint64_t key) {
  return key != 0ull && (uint32_t)key != 0xffffffffu;
}

// Copies the keys of the workgroup's cells first .. first + NCELLS - 1 into
// LDS (0 past the archive's end) and returns whether any names an offspring
// of this batch (the same answer in every thread).  Every thread must call it.
template <int NCELLS>
__device__ __forceinline__ bool stage_keys(const Params& p, int first, uint64_t* s_key) {
  bool won = false;
  if (threadIdx.x < NCELLS) {
    const int c = first + (int)threadIdx.x;
    const uint64_t key = c < p.C ? p.arch_key[c] : 0ull;
    s_key[threadIdx.x] = key;
    won = names_offspring(key);
  }
  return __syncthreads_or(won) != 0;
}

// Workgroups 0 .. ceil(C / cells) - 1 take cells; one more compacts.
inline unsigned regen_blocks(int C, int cells) { return (unsigned)((C + cells - 1) / cells) + 1u; }

template <bool GEN0>
__global__ __launch_bounds__(256) void k_regen(const Params p, uint32_t g) {
  if (blockIdx.x == gridDim.x - 1) {
    compact_filled(p);
    return;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int first = blockIdx.x * kRegenCells;
  __shared__ uint64_t s_key[kRegenCells];
  __shared__ float4 s_ntab[kNormalRows];
  if (!stage_keys<kRegenCells>(p, first, s_key)) return;
  const int wfirst = first + wave * kRegenCellsPerWave;
  const uint64_t* w_key = s_key + wave * kRegenCellsPerWave;
  // lane t < kRegenCellsPerWave reads what its cell's winner recorded (test
  // functions have two descriptor components), in flight with the table's loads
  const uint64_t my_key = lane < kRegenCellsPerWave ? w_key[lane] : 0ull;
  const bool my_won = names_offspring(my_key);
  const int my_j = p.nb - 1 - (int)(uint32_t)my_key;
  int par1 = 0, par2 = 0, banks = 0, slot = 0;
  float fit = 0.0f, desc[2] = {0.0f, 0.0f};
  if (my_won) {
    if (!GEN0) {
      par1 = p.off_par[2 * my_j];
      par2 = p.off_par[2 * my_j + 1];
      banks = p.off_bank[my_j];
    }
    slot = (int)p.arch_slot[wfirst + lane];
    fit = p.off_fit[my_j];
    desc[0] = p.off_desc[2 * (size_t)my_j];
    desc[1] = p.off_desc[2 * (size_t)my_j + 1];
  }
  if (!GEN0) {
    stage_normal_table(s_ntab, p.ntab, (int)threadIdx.x, 256);
    __syncthreads();
  }
  const Tables tb{s_ntab};
  for (int t = 0; t < kRegenCellsPerWave; ++t) {
    const uint64_t key = w_key[t];
    if (!names_offspring(key)) continue;
    const int c = wfirst + t;
    const int j = p.nb - 1 - (int)(uint32_t)key;
    Pair q{nullptr, nullptr, 0.0f, -1, -1, 0u};
    if (!GEN0)
      q = pair_from_record(p, g, j, __builtin_amdgcn_readlane(par1, t),
                           __builtin_amdgcn_readlane(par2, t),
                           (uint32_t)__builtin_amdgcn_readlane(banks, t), tb);
    float* dst = geno_row(p, (uint32_t)__builtin_amdgcn_readlane(slot, t) ^ 1u, c);
    for (int base = 4 * lane; base < p.n; base += 256)
      *reinterpret_cast<float4*>(dst + base) = make_genes<GEN0>(p, q, g, j, base);
  }
  // then lane t finishes its cell: objective, descriptor, bank, incumbent key
  if (my_won) {
    const int c = wfirst + lane;
    p.arch_fit[c] = fit;
    p.arch_desc[2 * (size_t)c] = desc[0];
    p.arch_desc[2 * (size_t)c + 1] = desc[1];
    p.off_won[my_j] = 1;
    p.arch_slot[c] = (uint32_t)slot ^ 1u;
    p.arch_key[c] = my_key | 0xffffffffull;
  }
}

// ---------------------------------------------------------------------------
// Statistics over the archive (fp64 accumulation).  One workgroup; the four
// results go to out[0 .. 3] (the workspace's statistics buffer, or the
// library's own device scratch for callers that cannot allocate).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_stats(const Params p, double offset, double* out) {
  __shared__ double s_sum[16];
  __shared__ double s_best[16];
  __shared__ int s_cnt[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double sum = 0.0, best = -__builtin_inf();
  int cnt = 0;
  for (int c = tid; c < p.C; c += 1024) {
    if (p.arch_key[c] != 0ull) {
      const double f = (double)p.arch_fit[c];
      sum += f + offset;
      best = f > best ? f : best;
      ++cnt;
    }
  }
  for (int h = 32; h >= 1; h >>= 1) {
    sum += __shfl_xor(sum, h, 64);
    const double ob = __shfl_xor(best, h, 64);
    best = ob > best ? ob : best;
    cnt += __shfl_xor(cnt, h, 64);
  }
  if (lane == 0) {
    s_sum[wave] = sum;
    s_best[wave] = best;
    s_cnt[wave] = cnt;
  }
  __syncthreads();
  if (tid == 0) {
    double ts = 0.0, tb = -__builtin_inf();
    int tc = 0;
    for (int w = 0; w < 16; ++w) {
      ts += s_sum[w];
      tb = s_best[w] > tb ? s_best[w] : tb;
      tc += s_cnt[w];
    }
    out[0] = ts;
    out[1] = (double)tc;
    out[2] = tc ? tb : __builtin_nan("");
    out[3] = (double)p.counters[1];
  }
}

// ---------------------------------------------------------------------------
// Set-up kernels (first iteration only).
// ---------------------------------------------------------------------------
__global__ void k_clear_archive(const Params p, int clear_geno) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t nthr = (size_t)gridDim.x * blockDim.x;
  for (size_t c = tid; c < (size_t)p.C; c += nthr) {
    p.arch_key[c] = 0ull;
    p.arch_fit[c] = __builtin_nanf("");
    p.arch_slot[c] = 0u;
    p.occ_list[c] = 0;
    for (int k = 0; k < p.D; ++k) p.arch_desc[c * p.D + k] = 0.0f;
  }
  if (clear_geno) {
    const size_t nv = (size_t)2 * p.C * p.stride / 4;
    float4* gp = reinterpret_cast<float4*>(p.arch_geno);
    for (size_t i = tid; i < nv; i += nthr) gp[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if (tid < 64) p.counters[tid] = 0;
  if (p.lloyd_acc)
    for (size_t b = tid; b < (size_t)p.C * (p.D + 1); b += nthr) p.lloyd_acc[b] = 0ull;
  if (p.num_buckets > 0)
    for (size_t b = tid; b < (size_t)2 * (p.num_buckets + 1); b += nthr) p.bucket_start[b] = 0;
}

__device__ __forceinline__ int centroid_bucket(const Params& p, const float* c) {
  int b = 0;
  for (int k = 0; k < p.D; ++k) {
    int bk = (int)(c[k] * (float)p.bucket_res);
    bk = bk > p.bucket_res - 1 ? p.bucket_res - 1 : bk;
    b = b * p.bucket_res + bk;
  }
  return b;
}

// Centroid i, coordinate k = 24-bit uniform of word k of block (i, 0, 0, CENTROID).
__global__ void k_centroids(const Params p) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= p.C) return;
  const uint4 x = philox((uint32_t)i, 0u, 0u, kTagCentroid, p.key);
  const float c[4] = {unit24(x.x), unit24(x.y), unit24(x.z), unit24(x.w)};
  for (int k = 0; k < p.D; ++k) p.cent[(size_t)i * p.D + k] = c[k];
}

// Centroids per bucket of the ring-search grid (counts at [1 .. num_buckets]).
__global__ void k_bucket_count(const Params p) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= p.C) return;
  float c[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < p.D; ++k) c[k] = p.cent[(size_t)i * p.D + k];
  atomicAdd(&p.bucket_start[centroid_bucket(p, c) + 1], 1);
}

// Lloyd's algorithm for a centroidal Voronoi tessellation, one iteration in
// two kernels.  Assignment: point i (coordinate k = U24 of word k of block
// (i, 0, 0, CVT_SAMPLE)) goes to its nearest centroid by the cell rule (fma
// chain over the dimensions, first minimum in index order); the centroids
// pass through LDS in tiles of kLloydTile, in index order.  Each point adds
// its coordinates' 24-bit numerators and a count to its centroid's
// accumulators -- integer sums, so the order of the atomics does not matter.
constexpr int kLloydBlock = 256;
constexpr int kLloydTile = 1024;

template <int D>
__global__ __launch_bounds__(kLloydBlock) void k_lloyd_assign(const Params p) {
  __shared__ float4 s_c[kLloydTile];
  const int i = blockIdx.x * kLloydBlock + threadIdx.x;
  const bool live = i < p.cvt_samples;
  const uint4 x = philox((uint32_t)i, 0u, 0u, kTagCvtSample, p.key);
  const uint32_t m[4] = {x.x >> 8, x.y >> 8, x.z >> 8, x.w >> 8};
  float u[D];
#pragma unroll
  for (int k = 0; k < D; ++k) u[k] = (float)m[k] * 0x1p-24f;
  float best = __builtin_inff();
  int best_idx = 0;
  for (int t0 = 0; t0 < p.C; t0 += kLloydTile) {
    const int n = p.C - t0 < kLloydTile ? p.C - t0 : kLloydTile;
    __syncthreads();
    for (int t = threadIdx.x; t < n; t += kLloydBlock) {
      const float* c = p.cent + (size_t)(t0 + t) * D;
      float4 v = make_float4(c[0], c[1], 0.0f, 0.0f);
      if (D == 4) {
        v.z = c[2];
        v.w = c[3];
      }
      s_c[t] = v;
    }
    __syncthreads();
    for (int t = 0; t < n; ++t) {
      const float4 c = s_c[t];
      const float e0 = u[0] - c.x;
      float acc = fma32(e0, e0, 0.0f);
      const float e1 = u[1] - c.y;
      acc = fma32(e1, e1, acc);
      if (D == 4) {
        const float e2 = u[D > 2 ? 2 : 0] - c.z;
        acc = fma32(e2, e2, acc);
        const float e3 = u[D > 3 ? 3 : 0] - c.w;
        acc = fma32(e3, e3, acc);
      }
      if (acc < best) {
        best = acc;
        best_idx = t0 + t;
      }
    }
  }
  if (live) {
    unsigned long long* a = p.lloyd_acc + (size_t)best_idx * (D + 1);
#pragma unroll
    for (int k = 0; k < D; ++k) atomicAdd(a + k, (unsigned long long)m[k]);
    atomicAdd(a + D, 1ull);
  }
}

// Update: a centroid that received points moves to their mean,
// ((double)sum / (double)count) 2^-24 rounded to fp32; the accumulators are
// cleared for the next iteration.
__global__ void k_lloyd_update(const Params p) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= p.C) return;
  unsigned long long* a = p.lloyd_acc + (size_t)c * (p.D + 1);
  const unsigned long long cnt = a[p.D];
  if (cnt != 0ull) {
    for (int k = 0; k < p.D; ++k)
      p.cent[(size_t)c * p.D + k] = (float)(((double)a[k] / (double)cnt) * 0x1p-24);
  }
  for (int k = 0; k <= p.D; ++k) a[k] = 0ull;
}

__global__ __launch_bounds__(1024) void k_bucket_scan(const Params p) {
  // inclusive scan of counts stored at [1..NB] -> starts; single workgroup
  __shared__ int carry;
  __shared__ int wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) carry = 0;
  __syncthreads();
  const int NB = p.num_buckets;
  for (int start = 1; start <= NB; start += 1024) {
    const int i = start + tid;
    int v = i <= NB ? p.bucket_start[i] : 0;
    for (int h = 1; h < 64; h <<= 1) {
      const int o = __shfl_up(v, h, 64);
      if (lane >= h) v += o;
    }
    if (lane == 63) wsum[wave] = v;
    __syncthreads();
    int off = carry;
    for (int w = 0; w < wave; ++w) off += wsum[w];
    if (i <= NB) p.bucket_start[i] = v + off;
    __syncthreads();
    if (tid == 0) {
      int t = 0;
      for (int w = 0; w < 16; ++w) t += wsum[w];
      carry += t;
    }
    __syncthreads();
  }
}

__global__ void k_bucket_fill(const Params p) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= p.C) return;
  float c[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < p.D; ++k) c[k] = p.cent[(size_t)i * p.D + k];
  const int b = centroid_bucket(p, c);
  int* cursor = p.bucket_start + (p.num_buckets + 1);
  const int slot = p.bucket_start[b] + atomicAdd(&cursor[b], 1);
  p.bucket_pts[slot] = make_float4(c[0], c[1], c[2], c[3]);
  p.bucket_idx[slot] = i;
}

// Candidate lists of a two-dimensional CVT.  Fine bucket (b0, b1) is the box
// [b0/R, (b0+1)/R] x [b1/R, (b1+1)/R], widened by 1e-6 on every side to cover
// the rounding of the bucket index.  Every point of it lies within
// Dmax = min over centroids of the farthest-corner distance of some centroid,
// so a centroid whose nearest-point distance to the box exceeds Dmax (with a
// relative margin of 1e-5, far above the fp32 error of the distances the
// search compares) is never the argmin for a point of the box.  The rest are
// listed in ascending index; the count keeps counting past QD_CAND_SLOTS.
// kCandGroup lanes per bucket walk the centroids together, staged in LDS
// tiles: at step i lane q of the group takes centroid kCandGroup i + q.  The
// bound is the group's minimum (order-free); the listed centroids are
// appended in q order at each step, i.e. in ascending index.
constexpr int kCandTile = 2048, kCandGroup = 16, kCandBuckets = 256 / kCandGroup;

__global__ __launch_bounds__(256) void k_cand_build(const Params p) {
  constexpr int G = kCandGroup;
  static_assert(G == 4 || G == 8 || G == 16, "a group is a power of two within a row");
  __shared__ float2 s_c[kCandTile];
  const int lane = lane_id(), q = lane & (G - 1);
  const int b = blockIdx.x * kCandBuckets + (int)(threadIdx.x / G);
  const bool live = b < p.cand_buckets;
  const int R = p.cand_res;
  const double w = 1.0 / (double)R, pad = 1e-6;
  const int bb = live ? b : 0;
  const double lo0 = (bb / R) * w - pad, hi0 = (bb / R + 1) * w + pad;
  const double lo1 = (bb % R) * w - pad, hi1 = (bb % R + 1) * w + pad;
  const float2* cent = reinterpret_cast<const float2*>(p.cent);
  double dmax = __builtin_inf();
  for (int t0 = 0; t0 < p.C; t0 += kCandTile) {
    const int tn = p.C - t0 < kCandTile ? p.C - t0 : kCandTile;
    __syncthreads();
    for (int e = threadIdx.x; e < tn; e += 256) s_c[e] = cent[t0 + e];
    __syncthreads();
    for (int e = q; e < tn; e += G) {
      const double x = s_c[e].x, y = s_c[e].y;
      const double fx = fmax(x - lo0, hi0 - x), fy = fmax(y - lo1, hi1 - y);
      dmax = fmin(dmax, fx * fx + fy * fy);
    }
  }
#pragma unroll
  for (int h = 1; h < G; h <<= 1) dmax = fmin(dmax, __shfl_xor(dmax, h, 64));   // group minimum
  const double limit = dmax * (1.0 + 1e-5) + 1e-12;
  int count = 0;
  float4* out = p.cand_pts + (size_t)bb * QD_CAND_SLOTS;
  const int group0 = lane & ~(G - 1);
  const uint32_t gmask = (uint32_t)((1ull << G) - 1ull);
  for (int t0 = 0; t0 < p.C; t0 += kCandTile) {
    const int tn = p.C - t0 < kCandTile ? p.C - t0 : kCandTile;
    __syncthreads();
    for (int e = threadIdx.x; e < tn; e += 256) s_c[e] = cent[t0 + e];
    __syncthreads();
    for (int e0 = 0; e0 < tn; e0 += G) {   // the group's centroids e0 .. e0 + G - 1
      const int e = e0 + q;
      bool hit = false;
      float2 c = make_float2(0.0f, 0.0f);
      if (e < tn) {
        c = s_c[e];
        const double x = c.x, y = c.y;
        const double gx = fmax(0.0, fmax(lo0 - x, x - hi0)), gy = fmax(0.0, fmax(lo1 - y, y - hi1));
        hit = gx * gx + gy * gy <= limit;
      }
      const uint32_t bits = (uint32_t)(__ballot(hit) >> group0) & gmask;
      const int pos = count + __popc(bits & ((1u << q) - 1u));
      if (live && hit && pos < QD_CAND_SLOTS)
        out[pos] = make_float4(c.x, c.y, __int_as_float(t0 + e), 0.0f);
      count += __popc(bits);
    }
  }
  if (live && q == 0) p.cand_count[b] = count;
}

// Entry e of [A | B | s0] = 0.1 * normal (e mod 4) of block (e/4, 0, 0, ENV).
__global__ void k_env(const Params p, int count) {
  __shared__ float4 s_ntab[kNormalRows];
  stage_normal_table(s_ntab, p.ntab, (int)threadIdx.x, (int)blockDim.x);
  __syncthreads();
  const Tables tb{s_ntab};
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (4 * b >= count) return;
  const uint4 x = philox((uint32_t)b, 0u, 0u, kTagEnv, p.key);
  const float z[4] = {normal(x.x, tb), normal(x.y, tb), normal(x.z, tb), normal(x.w, tb)};
  for (int k = 0; k < 4; ++k)
    if (4 * b + k < count) p.env[4 * b + k] = 0.1f * z[k];
}

// The Gaussian sampler's table reaches the workspace as kernel arguments,
// kTableChunk rows per launch, so that writing it needs no host buffer the
// copy engine would have to read.
constexpr int kTableChunk = 128;
struct TableChunk {
  float4 rows[kTableChunk];
};
__global__ void k_put_table(float4* dst, const TableChunk chunk, int first, int count) {
  const int i = (int)threadIdx.x;
  if (i < count) dst[first + i] = chunk.rows[i];
}

// The sampler on caller-given words (a grid-stride loop; i < count bounds
// every access).
__global__ __launch_bounds__(256) void k_sample_normals(const float4* ntab, const uint32_t* x,
                                                        float* z, uint64_t count) {
  __shared__ float4 s_ntab[kNormalRows];
  stage_normal_table(s_ntab, ntab, (int)threadIdx.x, 256);
  __syncthreads();
  const Tables tb{s_ntab};
  const uint64_t stride = (uint64_t)gridDim.x * 256u;
  for (uint64_t i = (uint64_t)blockIdx.x * 256u + threadIdx.x; i < count; i += stride)
    z[i] = normal(x[i], tb);
}

// Self-checks of the short division sequences against the IEEE operations,
// over every input each one can receive: tanh for all 2^32 fp32 bit patterns,
// sigmoid for all fp32 values in [-1, 1].  Counts results that differ (both
// NaN = equal).
__global__ void k_zero_u64(unsigned long long* x) {
  if (threadIdx.x < 2) x[threadIdx.x] = 0ull;
}

__device__ __forceinline__ bool same_bits(float a, float b) {
  return __float_as_uint(a) == __float_as_uint(b) || (a != a && b != b);
}

__global__ __launch_bounds__(256) void k_check_fast(unsigned long long* count) {
  const uint64_t nthr = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t tid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  unsigned long long bad_t = 0, bad_s = 0;
  for (uint64_t k = tid; k < (1ull << 32); k += nthr) {
    const float x = __uint_as_float((uint32_t)k);
    bad_t += same_bits(tanh32<true>(x), tanh32<false>(x)) ? 0 : 1;
    if (__builtin_fabsf(x) <= 1.0f) bad_s += same_bits(sigmoid32<true>(x), sigmoid32<false>(x)) ? 0 : 1;
  }
  if (bad_t) atomicAdd(count, bad_t);
  if (bad_s) atomicAdd(count + 1, bad_s);
}

}  // namespace qd
