// qd_rollout.hpp -- policy rollouts on the synthetic dynamics (gfx950).
//
// Evaluation of a batch of tanh MLP policies (two hidden tanh layers and a
// tanh output, as in Section 5.1 of the paper) for T steps of
// s' = tanh(A s + B a).  Every individual has its own weights, so this is a
// batch of independent GEMV chains, not one GEMM: no matrix core applies.
//
// One workgroup of H threads (H = hidden width, one or two waves) runs one
// individual with all its weights in VGPRs for the whole episode.  The
// summation order of every output is fixed (hidden layers and A s: four
// interleaved partial sums, then the bias; output layer: 8 slices folded
// pairwise, then the bias; dynamics: A s + B a), which keeps the result
// independent of the launch shape.
//
// The genotype is produced in the kernel's prologue straight from the parents
// (or the Glorot-uniform first batch) -- offspring weights never touch HBM.
#pragma once

#include "qd_kernels.hpp"

namespace qd {

constexpr int kObs = 27, kAct = 8;

inline bool rollout_supported(int obs, int hid, int act) {
  return obs == kObs && act == kAct && (hid == 64 || hid == 128);
}

// Glorot-uniform first-batch gene i (biases are zero).
__device__ __forceinline__ float mlp_init_gene(const Params& p, int i, float u) {
  const int o = p.obs, h = p.hid, a = p.act;
  const int e1 = h * o, e2 = e1 + h, e3 = e2 + h * h, e4 = e3 + h, e5 = e4 + a * h;
  float lim;
  if (i < e1) lim = __builtin_sqrtf(6.0f / (float)(o + h));
  else if (i < e2) lim = 0.0f;
  else if (i < e3) lim = __builtin_sqrtf(6.0f / (float)(h + h));
  else if (i < e4) lim = 0.0f;
  else if (i < e5) lim = __builtin_sqrtf(6.0f / (float)(h + a));
  else lim = 0.0f;
  return lim == 0.0f ? 0.0f : fma32(u, lim + lim, -lim);
}

// Genes 4 blk .. 4 blk + 3 of policy offspring j.
template <bool GEN0>
__device__ __forceinline__ float4 mlp_gene_block(const Params& p, const Pair& q, uint32_t g, int j,
                                                 int blk) {
  if (GEN0) {
    const uint4 x = philox((uint32_t)blk, (uint32_t)j, 0u, kTagInit, p.key);
    const int i = 4 * blk;
    return make_float4(mlp_init_gene(p, i, unit24(x.x)), mlp_init_gene(p, i + 1, unit24(x.y)),
                       mlp_init_gene(p, i + 2, unit24(x.z)), mlp_init_gene(p, i + 3, unit24(x.w)));
  }
  return make_genes<false>(p, q, g, j, 4 * blk);
}

// Makes the four genes opaque to the optimiser (an empty asm that claims to
// change them): the prologue's genes are then finished where they are made,
// instead of having the sampler's inputs carried into the episode loop where
// the genes are first read, which needs several times the registers.
__device__ __forceinline__ void settle(float4& v) {
  __asm__ volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
}

// The layers' dot products: four interleaved partial sums (input k goes to
// partial k mod 4, each an fma chain in input order from 0), folded as
// (p0 + p2) + (p1 + p3) -- four independent dependency chains per lane.  The
// inputs are broadcast from registers, not read from LDS one by one.
// With the DPP control row_newbcast:m, the first source of v_fmac_f32 is
// read from lane m of the executing lane's row of 16.  Component t of `v`
// holds, in lane 16 r + m, input 4 m + t of a run of 64 inputs (the same in
// every row r), so broadcast m of component t is input 4 m + t in every lane,
// and each partial sum below still takes its inputs in ascending order.  One
// float4 per lane per run replaces sixteen wave-wide LDS broadcasts.
// The compiler does not fold a DPP move into v_fmac, hence the asm.  No VGPR
// operand of a DPP instruction may be written by either of the two
// instructions before it: every block opens with s_nop 1, and inside a block
// each accumulator is written four instructions before it is read again.  The
// blocks must run with every lane of the wave active.
#define QD_BROW(B, W0, W1, W2, W3)                                                     \
  "v_fmac_f32_dpp %0, %4, %" #W0 " row_newbcast:" #B " row_mask:0xf bank_mask:0xf\n\t" \
  "v_fmac_f32_dpp %1, %5, %" #W1 " row_newbcast:" #B " row_mask:0xf bank_mask:0xf\n\t" \
  "v_fmac_f32_dpp %2, %6, %" #W2 " row_newbcast:" #B " row_mask:0xf bank_mask:0xf\n\t" \
  "v_fmac_f32_dpp %3, %7, %" #W3 " row_newbcast:" #B " row_mask:0xf bank_mask:0xf\n\t"
#define QD_BROW3(B, W0, W1, W2)                                                        \
  "v_fmac_f32_dpp %0, %4, %" #W0 " row_newbcast:" #B " row_mask:0xf bank_mask:0xf\n\t" \
  "v_fmac_f32_dpp %1, %5, %" #W1 " row_newbcast:" #B " row_mask:0xf bank_mask:0xf\n\t" \
  "v_fmac_f32_dpp %2, %6, %" #W2 " row_newbcast:" #B " row_mask:0xf bank_mask:0xf\n\t"
#define QD_BFMA_IO(w)                                                                   \
  : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3])                             \
  : "v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w), "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), \
    "v"(w[4]), "v"(w[5]), "v"(w[6]), "v"(w[7]), "v"(w[8]), "v"(w[9]), "v"(w[10])
#define QD_BFMA_IO16(w)                                                                 \
  QD_BFMA_IO(w), "v"(w[11]), "v"(w[12]), "v"(w[13]), "v"(w[14]), "v"(w[15])

// Inputs 16 B .. 16 B + 15 of a run (broadcasts 4 B .. 4 B + 3), weights w[0 .. 16).
template <int B>
__device__ __forceinline__ void bfma16(float (&acc)[4], const float4& v, const float* w) {
  if constexpr (B == 0) {
    __asm__("s_nop 1\n\t" QD_BROW(0, 8, 9, 10, 11) QD_BROW(1, 12, 13, 14, 15)
                QD_BROW(2, 16, 17, 18, 19) QD_BROW(3, 20, 21, 22, 23) QD_BFMA_IO16(w));
  } else if constexpr (B == 1) {
    __asm__("s_nop 1\n\t" QD_BROW(4, 8, 9, 10, 11) QD_BROW(5, 12, 13, 14, 15)
                QD_BROW(6, 16, 17, 18, 19) QD_BROW(7, 20, 21, 22, 23) QD_BFMA_IO16(w));
  } else if constexpr (B == 2) {
    __asm__("s_nop 1\n\t" QD_BROW(8, 8, 9, 10, 11) QD_BROW(9, 12, 13, 14, 15)
                QD_BROW(10, 16, 17, 18, 19) QD_BROW(11, 20, 21, 22, 23) QD_BFMA_IO16(w));
  } else {
    static_assert(B == 3, "four blocks per run");
    __asm__("s_nop 1\n\t" QD_BROW(12, 8, 9, 10, 11) QD_BROW(13, 12, 13, 14, 15)
                QD_BROW(14, 16, 17, 18, 19) QD_BROW(15, 20, 21, 22, 23) QD_BFMA_IO16(w));
  }
}

// Inputs 16 .. 26 of a run (broadcasts 4, 5 and 6 without input 27), weights w[0 .. 11).
__device__ __forceinline__ void bfma11(float (&acc)[4], const float4& v, const float* w) {
  __asm__("s_nop 1\n\t" QD_BROW(4, 8, 9, 10, 11) QD_BROW(5, 12, 13, 14, 15)
              QD_BROW3(6, 16, 17, 18) QD_BFMA_IO(w));
}

// That dot product for N a multiple of 64; run r of x is read as one float4 per lane
// from x + 64 r + 4 (lane mod 16), 16-byte aligned.
template <int N>
__device__ __forceinline__ float dot4_bcast(const float* w, const float* x) {
  static_assert(N % 64 == 0, "whole runs of 64 inputs");
  const int m = (int)(threadIdx.x & 15);
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int r = 0; r < N / 64; ++r) {
    const float4 v = *reinterpret_cast<const float4*>(x + 64 * r + 4 * m);
    bfma16<0>(acc, v, w + 64 * r);
    bfma16<1>(acc, v, w + 64 * r + 16);
    bfma16<2>(acc, v, w + 64 * r + 32);
    bfma16<3>(acc, v, w + 64 * r + 48);
  }
  return (acc[0] + acc[2]) + (acc[1] + acc[3]);
}

// That dot product for N = 27 on `v`, the float4 a lane reads from x + 4 (lane mod 8) of a
// 32-float, 16-byte aligned x (its input 27 and broadcast 7 are never used).
__device__ __forceinline__ float dot4_bcast27(const float* w, const float4& v) {
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  bfma16<0>(acc, v, w);
  bfma11(acc, v, w + 16);
  return (acc[0] + acc[2]) + (acc[1] + acc[3]);
}

__device__ __forceinline__ float pick4(const float4& v, int k) {
  return k == 0 ? v.x : (k == 1 ? v.y : (k == 2 ? v.z : v.w));
}

// Fills dst[0 .. LEN) with genes first .. first+LEN-1, first a multiple of 4.
template <bool GEN0, int LEN>
__device__ __forceinline__ void mlp_genes_aligned(const Params& p, const Pair& q, uint32_t g,
                                                  int j, int first, float* dst) {
  static_assert(LEN % 4 == 0, "aligned runs hold whole gene blocks");
#pragma unroll
  for (int t4 = 0; t4 < LEN / 4; ++t4) {
    float4 v = mlp_gene_block<GEN0>(p, q, g, j, (first >> 2) + t4);
    settle(v);
    dst[4 * t4] = v.x;
    dst[4 * t4 + 1] = v.y;
    dst[4 * t4 + 2] = v.z;
    dst[4 * t4 + 3] = v.w;
  }
}

// Fills dst[0 .. LEN) with genes first .. first+LEN-1 (any alignment).
template <bool GEN0, int LEN>
__device__ __forceinline__ void mlp_genes_run(const Params& p, const Pair& q, uint32_t g, int j,
                                              int first, float* dst) {
  const int b0 = first >> 2, b1 = (first + LEN - 1) >> 2;
  for (int blk = b0; blk <= b1; ++blk) {
    float4 v = mlp_gene_block<GEN0>(p, q, g, j, blk);
    settle(v);
#pragma unroll
    for (int t = 0; t < LEN; ++t) {
      const int gi = first + t;
      if ((gi >> 2) == blk) dst[t] = pick4(v, gi & 3);
    }
  }
}

// Steps a rollout records for its reward and descriptor sums (see k_rollout).
constexpr int kRing = 64;

// Orders the LDS accesses of one wave's lanes around this point.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Folds the first m ring slots into the running sums; called by all 64
// lanes of the output wave (o: lane index in it).  Lane i < m turns slot i
// into its step's reward s'_0 - 0.5 |a|^2 (|a|^2 as an fma chain over the
// actions in order) and the sigmoids of s'_1 .. s'_4; then lane 0 adds the m
// rewards and lanes 1 .. 4 their m sigmoids to `acc`, in slot (= step) order
// -- the same operations in the same order as adding each step's terms as
// the step ends.
template <int A>
__device__ __forceinline__ void flush_ring(float (*ra)[A], float (*rs)[kRing + 1], int m, int o,
                                           float& acc) {
  wave_sync();
  if (o < m) {
    float qa = 0.0f;
#pragma unroll
    for (int k = 0; k < A; ++k) qa = fma32(ra[o][k], ra[o][k], qa);
    rs[0][o] = fma32(-0.5f, qa, rs[0][o]);
#pragma unroll 1
    for (int c = 1; c <= 4; ++c) rs[c][o] = sigmoid32(rs[c][o]);
  }
  wave_sync();
  if (o <= 4) {
    const float* row = rs[o];
    int i = 0;
    for (; i + 8 <= m; i += 8) {   // eight loads in flight, then eight adds
      float v[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) v[t] = row[i + t];
#pragma unroll
      for (int t = 0; t < 8; ++t) acc = acc + v[t];
    }
    for (; i < m; ++i) acc = acc + row[i];
  }
  wave_sync();
}

// One individual per workgroup of H threads (H / 64 waves):
//   thread o      row o of W1 and W2, b1[o], b2[o] in VGPRs; hidden neuron o
//   output wave   the last wave.  Its 64 lanes (o3 = lane / 8, slice = lane %
//                 8) hold W3[o3][slice of H/8 inputs]; the 8 partial sums of an
//                 action are folded inside its group of 8 lanes.  Its lanes
//                 i < 27 also hold row i of A and B (shared environment) and
//                 compute state component i.
// Per step: layer 1 (and A s on the output wave), barrier, layer 2, barrier,
// then on the output wave alone the output layer, B a (the actions broadcast
// by readlane) and the new state, barrier.  The reward and the descriptor's
// sigmoids, which only lanes 0 .. 4 of the output wave need, are not
// evaluated in the step: the step's actions and new-state components 0 .. 4
// go to a ring in LDS, folded in every kRing steps by the output wave.
template <int H, bool GEN0, bool KEEP>
__global__ __launch_bounds__(H, H == 64 ? 3 : 2) void k_rollout(const Params p, uint32_t g) {
  constexpr int O = kObs, A = kAct, SL = H / 8;
  constexpr int E1 = H * O, E2 = E1 + H, E3 = E2 + H * H, E4 = E3 + H;   // W3 at E4, b3 after
  constexpr int OUT_WAVE_FIRST = H - 64;                                  // first lane of it
  __shared__ __attribute__((aligned(16))) float s_state[2][32];
  __shared__ __attribute__((aligned(16))) float s_h1[H];
  __shared__ float s_h2[H];
  // Ring of the last kRing valid steps: their actions, and their new states'
  // components 0 .. 4 (later the step's reward and four sigmoids).  Rows are
  // padded so that lanes 0 .. 4 reading one column hit different banks.
  __shared__ __attribute__((aligned(16))) float s_ra[kRing][A];
  __shared__ float s_rs[5][kRing + 1];
  __shared__ int s_fail;

  __shared__ float4 s_ntab[kNormalRows];

  const int o = threadIdx.x;
  const int j = blockIdx.x;

  Pair q{nullptr, nullptr, 0.0f, -1, -1, 0u};
  if (!GEN0) {
    const int nocc = p.counters[0];
    if (nocc <= 0) {
      if (o == 0) record_empty_archive(p, j);
      return;
    }
    stage_normal_table(s_ntab, p.ntab, o, H);
    __syncthreads();
    q = select_pair(p, g, j, nocc, Tables{s_ntab});
  }

  // ---- prologue: this individual's genotype, straight into registers
  const bool out_lane = o >= OUT_WAVE_FIRST;
  const int ol = o - OUT_WAVE_FIRST, o3 = (ol >> 3) & 7, slice = ol & 7;
  const bool dyn_lane = out_lane && ol < O;   // holds state component ol
  float w1[O], w2[H], w3[SL], arow[O], brow[A];
  float b1v, b2v, b3v = 0.0f;
  mlp_genes_run<GEN0, O>(p, q, g, j, o * O, w1);
  mlp_genes_aligned<GEN0, H>(p, q, g, j, E2 + o * H, w2);   // E2 = 28 H
  {
    float t[1];
    mlp_genes_run<GEN0, 1>(p, q, g, j, E1 + o, t);
    b1v = t[0];
    mlp_genes_run<GEN0, 1>(p, q, g, j, E3 + o, t);
    b2v = t[0];
    if (out_lane) {
      mlp_genes_run<GEN0, 1>(p, q, g, j, E4 + A * H + o3, t);
      b3v = t[0];
    }
  }
  if (out_lane) mlp_genes_aligned<GEN0, SL>(p, q, g, j, E4 + o3 * H + slice * SL, w3);
  if (KEEP) {
    float* row = p.off_geno + (size_t)j * (size_t)p.stride;
    for (int t = 0; t < O; ++t) row[o * O + t] = w1[t];
    for (int t = 0; t < H; ++t) row[E2 + o * H + t] = w2[t];
    row[E1 + o] = b1v;
    row[E3 + o] = b2v;
    if (out_lane) {
      for (int t = 0; t < SL; ++t) row[E4 + o3 * H + slice * SL + t] = w3[t];
      if (slice == 0) row[E4 + A * H + o3] = b3v;
    }
  }
  const float* envA = p.env;
  const float* envB = p.env + O * O;
  const float* envS = p.env + O * O + O * A;
#pragma unroll
  for (int k = 0; k < O; ++k) arow[k] = 0.0f;
  if (dyn_lane) {
#pragma unroll
    for (int k = 0; k < O; ++k) arow[k] = envA[ol * O + k];
#pragma unroll
    for (int k = 0; k < A; ++k) brow[k] = envB[ol * A + k];
    s_state[0][ol] = envS[ol];
  }
  if (o == 0) s_fail = 0;
  __syncthreads();

  // ---- episode; with death_mode != 0 it ends at the first new state whose
  // component 0 is below death_below, and that step counts for nothing.
  // Output-wave lane 0 sums the rewards, lanes 1 .. 4 the sigmoids of state
  // components 1 .. 4, each in step order; both are worked out from the ring,
  // kRing steps at a time (flush_ring), not inside the step.
  float acc = 0.0f;
  int cur = 0, valid = 0;
  for (int step = 0; step < p.T; ++step) {
    const int slot = valid & (kRing - 1);
    static_assert(O == 27, "the state is read as broadcasts 0 .. 6 of one float4");
    const float4 sv = *reinterpret_cast<const float4*>(&s_state[cur][4 * (o & 7)]);
    const float z1 = dot4_bcast27(w1, sv) + b1v;
    float as = 0.0f;
    if (out_lane) as = dot4_bcast27(arow, sv);   // the whole output wave (dyn_lane uses it)
    s_h1[o] = tanh32(z1);
    __syncthreads();
    const float z2 = dot4_bcast<H>(w2, s_h1) + b2v;
    s_h2[o] = tanh32(z2);
    __syncthreads();
    if (out_lane) {
      float pa = 0.0f;
#pragma unroll
      for (int t = 0; t < SL; ++t) pa = fma32(w3[t], s_h2[slice * SL + t], pa);
      pa = pa + row_shl<4>(pa);   // slices s and s + 4 (groups of 8 never straddle a row)
      pa = pa + row_shl<2>(pa);   // then s + 2
      pa = pa + row_shl<1>(pa);   // then s + 1
      const float act = tanh32(pa + b3v);   // action o3 in lane 8 o3 (slice 0)
      if (slice == 0) s_ra[slot][o3] = act;
      float ak[A];
#pragma unroll
      for (int k = 0; k < A; ++k)
        ak[k] = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(act), 8 * k));
      if (dyn_lane) {
        float ba = 0.0f;
#pragma unroll
        for (int k = 0; k < A; ++k) ba = fma32(brow[k], ak[k], ba);
        const float sn = tanh32(as + ba);
        s_state[cur ^ 1][ol] = sn;
        // lane 0 of this wave holds component 0 of the new state
        const bool fail = p.death_mode != 0 &&
                          __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(sn), 0)) <
                              p.death_below;
        if (fail) {
          if (ol == 0) s_fail = 1;
        } else if (ol <= 4) {
          s_rs[ol][slot] = sn;
        }
      }
    }
    cur ^= 1;
    __syncthreads();
    if (s_fail) break;   // the same value in every thread after the barrier
    ++valid;
    // a full ring: the output wave, its only writer, folds it in
    if ((valid & (kRing - 1)) == 0 && out_lane) flush_ring<A>(s_ra, s_rs, kRing, ol, acc);
  }
  if (out_lane) flush_ring<A>(s_ra, s_rs, valid & (kRing - 1), ol, acc);
  // death flag (Appendix A.4 i): a NaN objective is never inserted
  const bool dead = (p.death_mode == 2 && s_fail) || valid == 0;
  if (out_lane && ol == 0) {
    p.off_fit[j] = dead ? __builtin_nanf("") : acc;
    p.off_par[2 * j] = q.c1;
    p.off_par[2 * j + 1] = q.c2;
    p.off_bank[j] = (uint8_t)q.banks;
    p.off_won[j] = 0;
  } else if (out_lane && ol <= 4) {
    p.off_desc[(size_t)j * 4 + (ol - 1)] = valid > 0 ? acc / (float)valid : 0.0f;
  }
}

// Winners of a policy batch: a workgroup takes kRegenCellsMlp consecutive
// cells and, for each whose key names an offspring, all 256 threads write
// that offspring's genotype (same gene formula as the rollout's prologue) into
// the cell's other bank -- policy rows are long, so one row is spread over the
// whole workgroup.  After a barrier the cells record objective and descriptor,
// switch bank and take the incumbent key.
constexpr int kRegenCellsMlp = 8;

template <bool GEN0>
__global__ __launch_bounds__(256) void k_regen_mlp(const Params p, uint32_t g) {
  if (blockIdx.x == gridDim.x - 1) {
    compact_filled(p);
    return;
  }
  const int tid = threadIdx.x;
  const int first = blockIdx.x * kRegenCellsMlp;
  const int nblk = (p.n + 3) >> 2;
  __shared__ uint64_t s_key[kRegenCellsMlp];
  __shared__ float4 s_ntab[kNormalRows];
  if (!stage_keys<kRegenCellsMlp>(p, first, s_key)) return;
  if (!GEN0) {
    stage_normal_table(s_ntab, p.ntab, tid, 256);
    __syncthreads();
  }
  const Tables tb{s_ntab};
  for (int t = 0; t < kRegenCellsMlp; ++t) {
    const uint64_t key = s_key[t];
    if (!names_offspring(key)) continue;
    const int c = first + t;
    const int j = p.nb - 1 - (int)(uint32_t)key;
    Pair q{nullptr, nullptr, 0.0f, -1, -1, 0u};
    if (!GEN0) q = recorded_pair(p, g, j, tb);
    float* dst = geno_row(p, p.arch_slot[c] ^ 1u, c);
    for (int blk = tid; blk < nblk; blk += 256)
      *reinterpret_cast<float4*>(dst + 4 * blk) = mlp_gene_block<GEN0>(p, q, g, j, blk);
  }
  __syncthreads();
  if (tid < kRegenCellsMlp) {
    const uint64_t key = s_key[tid];
    if (names_offspring(key)) finish_winner(p, first + tid, p.nb - 1 - (int)(uint32_t)key, key);
  }
}

// Launchers: `go(kernel, grid, block, args...)` makes the launch.
template <class Go>
inline void launch_rollout(const Params& p, bool gen0, uint32_t g, bool keep, const Go& go) {
  const dim3 grid((unsigned)p.nb);
#define QD_RO(H)                                                        \
  do {                                                                  \
    if (gen0) {                                                         \
      if (keep) go(k_rollout<H, true, true>, grid, dim3(H), p, g);      \
      else go(k_rollout<H, true, false>, grid, dim3(H), p, g);          \
    } else {                                                            \
      if (keep) go(k_rollout<H, false, true>, grid, dim3(H), p, g);     \
      else go(k_rollout<H, false, false>, grid, dim3(H), p, g);         \
    }                                                                   \
  } while (0)
  if (p.hid == 64) QD_RO(64);
  else QD_RO(128);
#undef QD_RO
}

template <class Go>
inline void launch_mlp_regen(const Params& p, bool gen0, uint32_t g, const Go& go) {
  const dim3 grid(regen_blocks(p.C, kRegenCellsMlp)), block(256);
  if (gen0) go(k_regen_mlp<true>, grid, block, p, g);
  else go(k_regen_mlp<false>, grid, block, p, g);
}

}  // namespace qd
