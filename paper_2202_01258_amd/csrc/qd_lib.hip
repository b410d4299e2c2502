// qd_lib.hip -- host side of libqd.so: config validation, workspace layout,
// launch sequencing on the caller's stream, per-kernel event timing and error
// mapping.  The C ABI is declared in include/qd.h.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/qd.h"
#include "qd_kernels.hpp"
#include "qd_rollout.hpp"

namespace {

thread_local hipError_t g_last_hip = hipSuccess;

constexpr uint64_t kAlign = 256;
// Candidate lists are built (one thread per fine bucket, each scanning every
// centroid twice) only up to this many cells.
constexpr int kCandMaxCells = 65536;

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

bool is_mlp(const qd_config* c) { return c->task == QD_TASK_MLP_SYNTH; }

int32_t genotype_len(const qd_config* c) {
  if (!is_mlp(c)) return c->genotype_dim;
  const int64_t o = c->mlp_obs, h = c->mlp_hidden, a = c->mlp_act;
  const int64_t n = h * o + h + h * h + h + a * h + a;
  return n > (int64_t)0x7fffffff ? -1 : (int32_t)n;
}

// Largest R with R^D <= C: about one centroid per bucket.
int bucket_res_for(int C, int D) {
  int R = 1;
  for (;;) {
    int64_t p = 1;
    for (int k = 0; k < D; ++k) p *= (R + 1);
    if (p > C) break;
    ++R;
  }
  return R;
}

bool finite(float x) { return std::isfinite(x); }

qd_status validate(const qd_config* c) {
  if (!c) return QD_ERR_INVALID_ARG;
  if (c->abi_version != QD_ABI_VERSION) return QD_ERR_INVALID_ARG;
  if (c->task < QD_TASK_RASTRIGIN || c->task > QD_TASK_MLP_SYNTH) return QD_ERR_INVALID_ARG;
  if (c->tess != QD_TESS_GRID && c->tess != QD_TESS_CVT) return QD_ERR_INVALID_ARG;
  if (c->batch_size < 1) return QD_ERR_INVALID_ARG;
  if (c->num_cells < 1 || c->num_cells > (1 << 28)) return QD_ERR_INVALID_ARG;
  if (c->keep_offspring != 0 && c->keep_offspring != 1) return QD_ERR_INVALID_ARG;
  if (c->cvt_samples < 0 || c->cvt_samples > (1 << 28) || c->cvt_iters < 0 ||
      c->cvt_iters > 10000)
    return QD_ERR_INVALID_ARG;
  if (c->tess == QD_TESS_GRID && (c->cvt_samples != 0 || c->cvt_iters != 0))
    return QD_ERR_INVALID_ARG;
  if (c->death_mode < 0 || c->death_mode > 2 || (c->death_mode != 0 && !is_mlp(c)) ||
      c->death_below != c->death_below)
    return QD_ERR_INVALID_ARG;
  if (c->init_mode < 0 || c->init_mode > 1 || (c->init_mode != 0 && is_mlp(c)))
    return QD_ERR_INVALID_ARG;
  const int D = c->desc_dim;
  if (is_mlp(c)) {
    if (c->genotype_dim != 0 || D != 4) return QD_ERR_INVALID_ARG;
    if (c->mlp_obs < 5 || c->mlp_hidden < 1 || c->mlp_act < 1 || c->episode_len < 1)
      return QD_ERR_INVALID_ARG;
  } else {
    if (c->genotype_dim < 2 || D != 2) return QD_ERR_INVALID_ARG;
    if (!finite(c->init_lo) || !finite(c->init_hi) || !(c->init_lo < c->init_hi))
      return QD_ERR_INVALID_ARG;
  }
  for (int k = 0; k < D; ++k)
    if (!finite(c->desc_lo[k]) || !finite(c->desc_hi[k]) || !(c->desc_lo[k] < c->desc_hi[k]))
      return QD_ERR_INVALID_ARG;
  if (!finite(c->iso_sigma) || !finite(c->line_sigma)) return QD_ERR_INVALID_ARG;
  if (c->tess == QD_TESS_GRID) {
    int64_t prod = 1;
    for (int k = 0; k < D; ++k) {
      if (c->grid_shape[k] < 1) return QD_ERR_INVALID_ARG;
      prod *= c->grid_shape[k];
      if (prod > (int64_t)1 << 31) return QD_ERR_INVALID_ARG;
    }
    if (prod != c->num_cells) return QD_ERR_INVALID_ARG;
  }
  if (genotype_len(c) < 1) return QD_ERR_INVALID_ARG;
  if (is_mlp(c) && !qd::rollout_supported(c->mlp_obs, c->mlp_hidden, c->mlp_act))
    return QD_ERR_UNSUPPORTED;
  return QD_OK;
}

qd_status make_layout(const qd_config* c, qd_layout* L) {
  std::memset(L, 0, sizeof(*L));
  const uint64_t C = (uint64_t)c->num_cells, D = (uint64_t)c->desc_dim,
                 nb = (uint64_t)c->batch_size;
  const int32_t n = genotype_len(c);
  const uint64_t stride = align_up((uint64_t)n, 64);
  if (stride > 0x7fffffffull) return QD_ERR_INVALID_ARG;
  L->genotype_dim = n;
  L->row_stride = (int32_t)stride;
  if (c->tess == QD_TESS_CVT) {
    L->bucket_res = bucket_res_for(c->num_cells, c->desc_dim);
    int64_t nbk = 1;
    for (uint64_t k = 0; k < D; ++k) nbk *= L->bucket_res;
    L->num_buckets = (int32_t)nbk;
    if (c->desc_dim == 2 && c->num_cells <= kCandMaxCells) {
      L->cand_res = bucket_res_for(4 * c->num_cells, 2);
      L->cand_buckets = L->cand_res * L->cand_res;
    }
  }
  const uint64_t env = is_mlp(c) ? (uint64_t)c->mlp_obs * (c->mlp_obs + c->mlp_act + 1) : 0;
  uint64_t bytes[QD_NUM_BUFFERS] = {};
  // overflow guard: every product below stays far under 2^63 for these limits
  if (nb > ((uint64_t)1 << 31) || stride * (nb + 2 * C) > ((uint64_t)1 << 60))
    return QD_ERR_INVALID_ARG;
  bytes[QD_BUF_ARCHIVE_KEY] = 8 * C;
  bytes[QD_BUF_ARCHIVE_FIT] = 4 * C;
  bytes[QD_BUF_ARCHIVE_DESC] = 4 * C * D;
  bytes[QD_BUF_ARCHIVE_SLOT] = 4 * C;
  bytes[QD_BUF_ARCHIVE_GENO] = 4 * 2 * C * stride;
  bytes[QD_BUF_CENTROIDS] = c->tess == QD_TESS_CVT ? 4 * C * D : 0;
  bytes[QD_BUF_BUCKET_START] = c->tess == QD_TESS_CVT ? 4 * 2 * ((uint64_t)L->num_buckets + 1) : 0;
  bytes[QD_BUF_BUCKET_ITEMS] = c->tess == QD_TESS_CVT ? (16 + 4) * C : 0;
  bytes[QD_BUF_CAND_COUNT] = 4 * (uint64_t)L->cand_buckets;
  bytes[QD_BUF_CAND_PTS] = 16 * (uint64_t)QD_CAND_SLOTS * (uint64_t)L->cand_buckets;
  bytes[QD_BUF_LLOYD_ACC] =
      c->tess == QD_TESS_CVT && c->cvt_samples > 0 && c->cvt_iters > 0 ? 8 * C * (D + 1) : 0;
  bytes[QD_BUF_ENV] = 4 * env;
  bytes[QD_BUF_OCC_LIST] = 4 * C;
  bytes[QD_BUF_COUNTERS] = 4 * 64;
  bytes[QD_BUF_OFF_PARENTS] = 4 * 2 * nb;
  bytes[QD_BUF_OFF_FIT] = 4 * nb;
  bytes[QD_BUF_OFF_DESC] = 4 * nb * D;
  bytes[QD_BUF_OFF_CELL] = 4 * nb;
  bytes[QD_BUF_OFF_WON] = nb;
  bytes[QD_BUF_OFF_KEY] = 8 * nb;
  bytes[QD_BUF_OFF_BANK] = nb;
  bytes[QD_BUF_OFF_GENO] = c->keep_offspring ? 4 * nb * stride : 0;
  bytes[QD_BUF_STATS] = 8 * 8;
  bytes[QD_BUF_NORMAL_TAB] = 16 * QD_NORMAL_ROWS;
  uint64_t off = 0;
  for (int b = 0; b < QD_NUM_BUFFERS; ++b) {
    L->offset[b] = off;
    L->bytes[b] = bytes[b];
    off = align_up(off + bytes[b], kAlign);
  }
  L->workspace_bytes = off;
  return QD_OK;
}

// ---------------------------------------------------------------------------
// Gaussian sampler table (host, fp64, no contraction).  A normal's magnitude
// is z(p) = Phi^-1(1 - p/2) at p = k 2^-24; row 16 E + j covers the bin
// p = 2^(E-24) (1 + (j + t)/16), t in [0, 1), with the cubic in t that passes
// through z at the four Chebyshev points of [0, 1]; its coefficient of t^i is
// stored times 2^(-19 i), rounded once to fp32, so the kernels evaluate it in
// the integer t 2^19.  The last row (k = 2^24, z = 0) is zero.
// ---------------------------------------------------------------------------
#pragma clang fp contract(off)
double half_normal_quantile(double p) {
  // erfc(z / sqrt 2) falls from 1 towards 0 on [0, 16]: 100 bisection halvings
  double a = 0.0, b = 16.0;
  for (int it = 0; it < 100; ++it) {
    const double mid = 0.5 * (a + b);
    if (std::erfc(mid * 0.70710678118654752440) > p) a = mid;
    else b = mid;
  }
  return 0.5 * (a + b);
}

using NormalTable = std::array<float, 4 * QD_NORMAL_ROWS>;

NormalTable make_normal_table() {
  NormalTable out{};
  const double s2 = std::sqrt(2.0);
  const double cos1 = 0.5 * std::sqrt(2.0 + s2);   // cos(pi/8)
  const double cos3 = 0.5 * std::sqrt(2.0 - s2);   // cos(3 pi/8)
  const double node[4] = {0.5 * (1.0 - cos1), 0.5 * (1.0 - cos3), 0.5 * (1.0 + cos3),
                          0.5 * (1.0 + cos1)};
  for (int row = 0; row + 1 < QD_NORMAL_ROWS; ++row) {
    const int e = row / 16, j = row % 16;
    double d[4];
    for (int i = 0; i < 4; ++i)
      d[i] = half_normal_quantile(std::ldexp(1.0 + ((double)j + node[i]) / 16.0, e - 24));
    // divided differences over the nodes in order: d[i] = z[node_0 .. node_i]
    for (int order = 1; order <= 3; ++order)
      for (int i = 3; i >= order; --i) d[i] = (d[i] - d[i - 1]) / (node[i] - node[i - order]);
    // Newton form to powers of t: a <- a (t - node_k) + d_k, k = 2, 1, 0
    double a[4] = {d[3], 0.0, 0.0, 0.0};
    for (int k = 2; k >= 0; --k) {
      for (int i = 3; i >= 1; --i) a[i] = a[i - 1] - node[k] * a[i];
      a[0] = d[k] - node[k] * a[0];
    }
    for (int i = 0; i < 4; ++i) out[4 * row + i] = (float)std::ldexp(a[i], -19 * i);
  }
  return out;
}

const NormalTable& normal_table() {
  static const NormalTable tab = make_normal_table();   // built once per process
  return tab;
}

}  // namespace

// Device scratch of qd_archive_stats_noalloc: the statistics kernel's four
// results, staged here instead of in the workspace, for callers that cannot
// allocate.  Every GPU the library runs on holds its own copy until the
// process ends; host code must use the per-device address from
// hipGetSymbolAddress (the array's name is only a host-side stand-in).
constexpr int kScratchDoubles = 32;   // 256 bytes
static __device__ __align__(256) double scratch[kScratchDoubles];


struct qd_archive {
  int device = -1;          // the device current at qd_archive_init
  qd_config cfg;
  qd_layout lay;
  qd::Params p;
  uint32_t timing_mask = 0;
  struct Rec {
    int kernel;
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
};

namespace {

qd_status hip_fail(hipError_t e) {
  g_last_hip = e;
  return QD_ERR_HIP;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_ptr[kMaxDevices] = {};

// Address of `scratch` on device `dev` (which must be current), looked up
// once per device.
qd_status noalloc_scratch(int dev, double** out) {
  if (dev < 0 || dev >= kMaxDevices) return QD_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol);
    g_scratch_ptr[dev] = (double*)ptr;
  }
  *out = g_scratch_ptr[dev];
  return QD_OK;
}


hipEvent_t take_event(qd_archive* h) {
  if (!h->pool.empty()) {
    hipEvent_t e = h->pool.back();
    h->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Launches a kernel on the handle's stream.  When its kernel id is being
// timed the launch goes through hipExtLaunchKernelGGL with a start/stop event
// pair, which the runtime stamps when the dispatch begins and ends (no marker
// packets of their own in the stream).
struct Go {
  qd_archive* h;
  hipStream_t s;
  int kernel_id;
  template <typename K, typename... A>
  void operator()(K kernel, dim3 grid, dim3 block, A... args) const {
    hipEvent_t a = nullptr, b = nullptr;
    if ((h->timing_mask >> kernel_id) & 1u) {
      a = take_event(h);
      b = a ? take_event(h) : nullptr;
      if (a && !b) {
        h->pool.push_back(a);
        a = nullptr;
      }
    }
    if (a) {
      hipExtLaunchKernelGGL(kernel, grid, block, 0, s, a, b, 0u, args...);
      h->recs.push_back({kernel_id, a, b});
    } else {
      hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
    }
  }
};

unsigned blocks_for(uint64_t items, unsigned per_block) {
  return (unsigned)((items + per_block - 1) / per_block);
}

template <int TASK, bool GEN0, int OPW>
void launch_vary_eval_as(const Go& go, dim3 grid, const qd::Params& p, uint32_t g, bool keep) {
  if (keep) go(qd::k_vary_eval<TASK, GEN0, true, OPW>, grid, dim3(256), p, g);
  else go(qd::k_vary_eval<TASK, GEN0, false, OPW>, grid, dim3(256), p, g);
}

template <int TASK, bool GEN0>
void launch_vary_eval_task(const Go& go, const qd::Params& p, uint32_t g, bool keep) {
  const int opw = qd::offspring_per_wave(p.nb);
  const dim3 grid(blocks_for((uint64_t)p.nb, 4u * (unsigned)opw));
  if (opw == 1) launch_vary_eval_as<TASK, GEN0, 1>(go, grid, p, g, keep);
  else if (opw == 2) launch_vary_eval_as<TASK, GEN0, 2>(go, grid, p, g, keep);
  else launch_vary_eval_as<TASK, GEN0, qd::kOffspringPerWave>(go, grid, p, g, keep);
}

template <bool GEN0>
void launch_vary_eval(qd_archive* h, hipStream_t s, uint32_t g) {
  const qd::Params& p = h->p;
  const Go go{h, s, QD_K_VARY_EVAL};
  const bool keep = h->cfg.keep_offspring != 0;
  switch (p.task) {
    case qd::kTaskRastrigin: launch_vary_eval_task<qd::kTaskRastrigin, GEN0>(go, p, g, keep); break;
    case qd::kTaskSphere: launch_vary_eval_task<qd::kTaskSphere, GEN0>(go, p, g, keep); break;
    default: launch_vary_eval_task<qd::kTaskProj, GEN0>(go, p, g, keep); break;
  }
}

void launch_insert(qd_archive* h, hipStream_t s) {
  const qd::Params& p = h->p;
  const Go go{h, s, QD_K_INSERT};
  const dim3 grid(blocks_for((uint64_t)p.nb, qd::kInsertBlock)), block(qd::kInsertBlock);
  if (p.tess == qd::kTessGrid) {
    if (p.D == 2) go(qd::k_insert<qd::kTessGrid, 2>, grid, block, p);
    else go(qd::k_insert<qd::kTessGrid, 4>, grid, block, p);
  } else if (p.D == 4 && p.C <= qd::kCvtLdsCells) {
    go(qd::k_insert_cvt_lds, dim3(blocks_for((uint64_t)p.nb, qd::kInsertLdsOffspring)), dim3(256), p);
  } else {
    if (p.D == 2) go(qd::k_insert<qd::kTessCvt, 2>, grid, block, p);
    else go(qd::k_insert<qd::kTessCvt, 4>, grid, block, p);
  }
}

template <bool GEN0>
void launch_regen(qd_archive* h, hipStream_t s, uint32_t g) {
  const qd::Params& p = h->p;
  const Go go{h, s, QD_K_REGEN};
  if (p.task == qd::kTaskMlp) {
    qd::launch_mlp_regen(p, GEN0, g, go);
  } else {
    const dim3 grid(qd::regen_blocks(p.C, qd::kRegenCells)), block(256);
    go(qd::k_regen<GEN0>, grid, block, p, g);
  }
}

template <bool GEN0>
qd_status enqueue_generation(qd_archive* h, hipStream_t s, uint32_t g) {
  if (h->p.task == qd::kTaskMlp) {
    qd::launch_rollout(h->p, GEN0, g, h->cfg.keep_offspring != 0, Go{h, s, QD_K_ROLLOUT});
    launch_insert(h, s);
  } else {
    launch_vary_eval<GEN0>(h, s, g);   // also finds cells and inserts
  }
  launch_regen<GEN0>(h, s, g);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? QD_OK : hip_fail(e);
}

// k_stats into `dev` (4 doubles of device memory), then to *out; synchronises.
qd_status stats_into(qd_archive* h, double qd_offset, hipStream_t s, double* dev, qd_stats* out) {
  hipLaunchKernelGGL(qd::k_stats, dim3(1), dim3(1024), 0, s, h->p, qd_offset, dev);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e);
  double host[4];
  e = hipMemcpyAsync(host, dev, sizeof(host), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e);
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e);
  out->qd_score = host[0];
  out->num_occupied = (int32_t)host[1];
  out->coverage = host[1] / (double)h->cfg.num_cells;
  out->best_fitness = (float)host[2];
  out->flags = (uint32_t)host[3];
  out->reserved = 0;
  return QD_OK;
}

qd::Params make_params(const qd_config* c, const qd_layout* L, uint8_t* ws) {
  qd::Params p;
  std::memset(&p, 0, sizeof(p));
  p.task = c->task;
  p.tess = c->tess;
  p.n = L->genotype_dim;
  p.nb = c->batch_size;
  p.D = c->desc_dim;
  p.C = c->num_cells;
  p.stride = L->row_stride;
  for (int k = 0; k < 4; ++k) {
    p.grid[k] = c->grid_shape[k];
    p.lo[k] = c->desc_lo[k];
    p.hi[k] = c->desc_hi[k];
    const volatile float hi = c->desc_hi[k], lo = c->desc_lo[k];
    p.span[k] = hi - lo;  // fp32 subtraction, as the descriptor formula defines it
  }
  p.iso_sigma = c->iso_sigma;
  p.line_sigma = c->line_sigma;
  p.init_lo = c->init_lo;
  p.init_mode = c->init_mode;
  {
    const volatile float hi = c->init_hi, lo = c->init_lo;
    p.init_span = hi - lo;
  }
  p.obs = c->mlp_obs;
  p.hid = c->mlp_hidden;
  p.act = c->mlp_act;
  p.T = c->episode_len;
  p.key.k0 = (uint32_t)(c->seed & 0xffffffffull);
  p.key.k1 = (uint32_t)(c->seed >> 32);
  p.bucket_res = L->bucket_res;
  p.inv_bucket_res = L->bucket_res > 0 ? 1.0 / (double)L->bucket_res : 0.0;
  p.num_buckets = L->num_buckets;
  auto at = [&](int b) -> void* { return L->bytes[b] ? ws + L->offset[b] : nullptr; };
  p.arch_key = (uint64_t*)at(QD_BUF_ARCHIVE_KEY);
  p.arch_fit = (float*)at(QD_BUF_ARCHIVE_FIT);
  p.arch_desc = (float*)at(QD_BUF_ARCHIVE_DESC);
  p.arch_slot = (uint32_t*)at(QD_BUF_ARCHIVE_SLOT);
  p.arch_geno = (float*)at(QD_BUF_ARCHIVE_GENO);
  p.cent = (float*)at(QD_BUF_CENTROIDS);
  p.bucket_start = (int*)at(QD_BUF_BUCKET_START);
  if (L->bytes[QD_BUF_BUCKET_ITEMS]) {
    p.bucket_pts = (float4*)(ws + L->offset[QD_BUF_BUCKET_ITEMS]);
    p.bucket_idx = (int*)(ws + L->offset[QD_BUF_BUCKET_ITEMS] + 16ull * c->num_cells);
  }
  p.cand_res = L->cand_res;
  p.cand_buckets = L->cand_buckets;
  p.cand_count = (int*)at(QD_BUF_CAND_COUNT);
  p.cand_pts = (float4*)at(QD_BUF_CAND_PTS);
  p.death_mode = c->death_mode;
  p.death_below = c->death_below;
  p.cvt_samples = c->cvt_samples;
  p.lloyd_acc = (unsigned long long*)at(QD_BUF_LLOYD_ACC);
  p.env = (float*)at(QD_BUF_ENV);
  p.occ_list = (int*)at(QD_BUF_OCC_LIST);
  p.counters = (int*)at(QD_BUF_COUNTERS);
  p.off_par = (int*)at(QD_BUF_OFF_PARENTS);
  p.off_fit = (float*)at(QD_BUF_OFF_FIT);
  p.off_desc = (float*)at(QD_BUF_OFF_DESC);
  p.off_cell = (int*)at(QD_BUF_OFF_CELL);
  p.off_won = (uint8_t*)at(QD_BUF_OFF_WON);
  p.off_key = (uint64_t*)at(QD_BUF_OFF_KEY);
  p.off_bank = (uint8_t*)at(QD_BUF_OFF_BANK);
  p.off_geno = (float*)at(QD_BUF_OFF_GENO);
  p.stats = (double*)at(QD_BUF_STATS);
  p.ntab = (const float4*)at(QD_BUF_NORMAL_TAB);
  return p;
}

}  // namespace

extern "C" {

qd_status qd_layout_query(const qd_config* cfg, qd_layout* out) {
  if (!out) return QD_ERR_INVALID_ARG;
  const qd_status st = validate(cfg);
  if (st != QD_OK) return st;
  return make_layout(cfg, out);
}

qd_status qd_archive_init(const qd_config* cfg, void* d_workspace, uint64_t workspace_bytes,
                          void* stream, qd_archive** out) {
  if (!out || !d_workspace) return QD_ERR_INVALID_ARG;
  *out = nullptr;
  qd_layout L;
  qd_status st = qd_layout_query(cfg, &L);
  if (st != QD_OK) return st;
  if (((uintptr_t)d_workspace % kAlign) != 0) return QD_ERR_INVALID_ARG;
  if (workspace_bytes < L.workspace_bytes) return QD_ERR_WORKSPACE_TOO_SMALL;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return QD_ERR_HIP;
  qd_archive* h = new (std::nothrow) qd_archive();
  if (!h) return QD_ERR_INVALID_ARG;
  h->device = dev;
  {
    // the no-allocation scratch's address on this device, looked up here once
    // (a failure is reported by qd_archive_stats_noalloc, which retries)
    double* scr = nullptr;
    (void)noalloc_scratch(dev, &scr);
    (void)hipGetLastError();
  }
  h->cfg = *cfg;
  h->lay = L;
  h->p = make_params(cfg, &L, (uint8_t*)d_workspace);
  hipStream_t s = (hipStream_t)stream;
  const qd::Params& p = h->p;
  {
    // the sampler's table, as kernel arguments (no host copy to wait on)
    const NormalTable& tab = normal_table();
    for (int first = 0; first < QD_NORMAL_ROWS; first += qd::kTableChunk) {
      const int count = std::min(qd::kTableChunk, QD_NORMAL_ROWS - first);
      qd::TableChunk chunk;
      std::memset(&chunk, 0, sizeof(chunk));
      std::memcpy(&chunk.rows[0], &tab[4 * first], 16 * (size_t)count);
      hipLaunchKernelGGL(qd::k_put_table, dim3(1), dim3(qd::kTableChunk), 0, s,
                         (float4*)p.ntab, chunk, first, count);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
      delete h;
      return hip_fail(e);
    }
  }
  {
    const Go go{h, s, QD_K_SETUP};
    go(qd::k_clear_archive, dim3(1024), dim3(256), p, 1);
    if (p.tess == qd::kTessCvt) {
      go(qd::k_centroids, dim3(blocks_for(p.C, 256)), dim3(256), p);
      if (p.lloyd_acc) {
        for (int it = 0; it < cfg->cvt_iters; ++it) {
          const dim3 grid(blocks_for((uint64_t)p.cvt_samples, qd::kLloydBlock)), block(qd::kLloydBlock);
          if (p.D == 2) go(qd::k_lloyd_assign<2>, grid, block, p);
          else go(qd::k_lloyd_assign<4>, grid, block, p);
          go(qd::k_lloyd_update, dim3(blocks_for(p.C, 256)), dim3(256), p);
        }
      }
      go(qd::k_bucket_count, dim3(blocks_for(p.C, 256)), dim3(256), p);
      go(qd::k_bucket_scan, dim3(1), dim3(1024), p);
      go(qd::k_bucket_fill, dim3(blocks_for(p.C, 256)), dim3(256), p);
      if (p.cand_buckets > 0) go(qd::k_cand_build, dim3(blocks_for(p.cand_buckets, qd::kCandBuckets)), dim3(256), p);
    }
    if (p.task == qd::kTaskMlp) {
      const int count = p.obs * (p.obs + p.act + 1);
      go(qd::k_env, dim3(blocks_for((count + 3) / 4, 256)), dim3(256), p, count);
    }
  }
  st = enqueue_generation<true>(h, s, 0u);
  if (st != QD_OK) {
    delete h;
    return st;
  }
  *out = h;
  return QD_OK;
}

qd_status qd_generation(qd_archive* h, uint32_t gen_index, void* stream) {
  if (!h || gen_index == 0) return QD_ERR_INVALID_ARG;
  return enqueue_generation<false>(h, (hipStream_t)stream, gen_index);
}

qd_status qd_generations(qd_archive* h, uint32_t first_gen, uint32_t count, void* stream) {
  if (!h || first_gen == 0 || (uint64_t)first_gen + count - 1 > UINT32_MAX) return QD_ERR_INVALID_ARG;
  for (uint32_t k = 0; k < count; ++k) {
    const qd_status st = enqueue_generation<false>(h, (hipStream_t)stream, first_gen + k);
    if (st != QD_OK) return st;
  }
  return QD_OK;
}

qd_status qd_archive_stats(qd_archive* h, double qd_offset, void* stream, qd_stats* out) {
  if (!h || !out) return QD_ERR_INVALID_ARG;
  return stats_into(h, qd_offset, (hipStream_t)stream, h->p.stats, out);
}

qd_status qd_archive_stats_noalloc(qd_archive* h, double qd_offset, void* stream, qd_stats* out) {
  if (!h || !out) return QD_ERR_INVALID_ARG;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  if (dev != h->device) return QD_ERR_INVALID_ARG;   // the handle's device must be current
  double* scr = nullptr;
  const qd_status st = noalloc_scratch(dev, &scr);
  if (st != QD_OK) return st;
  static_assert(kScratchDoubles >= 4, "k_stats writes four results");
  return stats_into(h, qd_offset, (hipStream_t)stream, scr, out);
}

qd_status qd_archive_layout(const qd_archive* h, qd_layout* out) {
  if (!h || !out) return QD_ERR_INVALID_ARG;
  *out = h->lay;
  return QD_OK;
}

qd_status qd_set_kernel_timing(qd_archive* h, uint32_t kernel_mask) {
  if (!h || (kernel_mask >> QD_NUM_KERNELS) != 0u) return QD_ERR_INVALID_ARG;
  h->timing_mask = kernel_mask;
  return QD_OK;
}

qd_status qd_kernel_times(qd_archive* h, double* ms, int32_t* counts) {
  if (!h || !ms || !counts) return QD_ERR_INVALID_ARG;
  for (int k = 0; k < QD_NUM_KERNELS; ++k) {
    ms[k] = 0.0;
    counts[k] = 0;
  }
  qd_status st = QD_OK;
  for (auto& r : h->recs) {
    hipError_t e = hipEventSynchronize(r.b);
    float t = 0.0f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, r.a, r.b);
    if (e != hipSuccess) st = hip_fail(e);
    ms[r.kernel] += (double)t;
    counts[r.kernel] += 1;
    h->pool.push_back(r.a);
    h->pool.push_back(r.b);
  }
  h->recs.clear();
  return st;
}

qd_status qd_normal_table(float* out) {
  if (!out) return QD_ERR_INVALID_ARG;
  const NormalTable& tab = normal_table();
  std::memcpy(out, tab.data(), sizeof(float) * tab.size());
  return QD_OK;
}

qd_status qd_sample_normals(const qd_archive* h, const void* d_words, void* d_out, uint64_t count,
                            void* stream) {
  if (!h || count > ((uint64_t)1 << 32)) return QD_ERR_INVALID_ARG;
  if (count == 0) return QD_OK;
  if (!d_words || !d_out || ((uintptr_t)d_words % 4) != 0 || ((uintptr_t)d_out % 4) != 0)
    return QD_ERR_INVALID_ARG;
  const unsigned grid = std::min(blocks_for(count, 256), 4096u);
  hipLaunchKernelGGL(qd::k_sample_normals, dim3(grid), dim3(256), 0, (hipStream_t)stream, h->p.ntab,
                     (const uint32_t*)d_words, (float*)d_out, count);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? QD_OK : hip_fail(e);
}

qd_status qd_check_fast_arith(void* d_scratch, void* stream, uint64_t* mismatches) {
  if (!d_scratch || !mismatches) return QD_ERR_INVALID_ARG;
  if (((uintptr_t)d_scratch % 8) != 0) return QD_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  auto* count = (unsigned long long*)d_scratch;
  hipLaunchKernelGGL(qd::k_zero_u64, dim3(1), dim3(64), 0, s, count);
  hipLaunchKernelGGL(qd::k_check_fast, dim3(1u << 15), dim3(256), 0, s, count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e);
  unsigned long long host[2] = {0, 0};
  e = hipMemcpyAsync(host, count, sizeof(host), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e);
  for (int k = 0; k < 2; ++k) mismatches[k] = host[k];
  return QD_OK;
}

qd_status qd_archive_destroy(qd_archive* h) {
  if (!h) return QD_OK;
  for (auto& r : h->recs) {
    (void)hipEventSynchronize(r.b);
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : h->pool) (void)hipEventDestroy(e);
  delete h;
  return QD_OK;
}

const char* qd_status_str(qd_status s) {
  switch (s) {
    case QD_OK: return "ok";
    case QD_ERR_INVALID_ARG: return "invalid argument";
    case QD_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case QD_ERR_EMPTY_ARCHIVE: return "empty archive";
    case QD_ERR_UNSUPPORTED: return "unsupported configuration";
    case QD_ERR_HIP: return hipGetErrorString(g_last_hip);
  }
  return "unknown status";
}

}  // extern "C"
