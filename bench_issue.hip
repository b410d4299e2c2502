// VALU issue-rate probe for gfx950: what the roofline of an instruction-bound
// kernel rests on.  Every kernel runs independent dependency chains of one
// instruction form (or a fixed mix) in a loop and stores one value per thread;
// no kernel reads memory it did not write, and every store is inside the
// output buffer (one float per launched thread).
//
// Printed (one line per case): the kernel time and the cycles per wave
// instruction per SIMD at the published 2.4 GHz clock, for
//   * single instruction forms at 8 waves per SIMD (8 chains per wave);
//   * a 1:1 mix of an fma and a v_max_f32 (two instructions per issue slot);
//   * fma and DPP-broadcast fma on 8 and on 4 chains at 1, 2, 3, 4 and 8 waves
//     per SIMD;
//   * Philox4x32-10 with 64-bit multiply-adds against low/high multiplies.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

namespace {

constexpr int kThreads = 256;                 // four waves per workgroup
constexpr int kMaxBlocks = 2048;              // 8 waves per SIMD on 256 CUs

#define QD_CH8(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7)
#define QD_DECL_F(i) float a##i = (float)(gid + i) * 1e-3f;
#define QD_DECL_U(i) uint32_t a##i = gid * 7u + i;
#define QD_SUM_F (a0 + a1 + a2 + a3 + a4 + a5 + a6 + a7)
#define QD_SUM_U (float)(a0 ^ a1 ^ a2 ^ a3 ^ a4 ^ a5 ^ a6 ^ a7)

// one float kernel per instruction form: 16 instructions per iteration
#define QD_KF(NAME, STEP)                                                   \
  __global__ __launch_bounds__(kThreads) void NAME(float* out, int iters) { \
    const int gid = blockIdx.x * kThreads + threadIdx.x;                    \
    const float b = 1.0001f + gid * 1e-9f, c = 0.5f;                        \
    QD_CH8(QD_DECL_F)                                                       \
    for (int it = 0; it < iters; ++it) { QD_CH8(STEP) QD_CH8(STEP) }        \
    out[gid] = QD_SUM_F;                                                    \
  }
#define QD_KU(NAME, STEP)                                                   \
  __global__ __launch_bounds__(kThreads) void NAME(float* out, int iters) { \
    const int gid = blockIdx.x * kThreads + threadIdx.x;                    \
    const uint32_t m = 0xD2511F53u + gid, n = gid * 5u;                     \
    QD_CH8(QD_DECL_U)                                                       \
    for (int it = 0; it < iters; ++it) { QD_CH8(STEP) QD_CH8(STEP) }        \
    out[gid] = QD_SUM_U;                                                    \
  }

#define S_FMA(i) asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(a##i) : "v"(b), "v"(c));
#define S_ADD(i) asm volatile("v_add_f32 %0, %0, %1" : "+v"(a##i) : "v"(b));
#define S_MAX(i) asm volatile("v_max_f32 %0, %0, %1" : "+v"(a##i) : "v"(b));
#define S_MED3(i) asm volatile("v_med3_f32 %0, %0, %1, %2" : "+v"(a##i) : "v"(b), "v"(c));
#define S_EXP(i) asm volatile("v_exp_f32 %0, %0" : "+v"(a##i));
#define S_BOP3(i) asm volatile("v_bitop3_b32 %0, %0, %1, %2 bitop3:0x96" : "+v"(a##i) : "v"(m), "v"(n));
#define S_AND(i) asm volatile("v_and_b32 %0, %0, %1" : "+v"(a##i) : "v"(m));
#define S_CVT(i) asm volatile("v_cvt_f32_u32 %0, %0" : "+v"(a##i));
#define S_MUL24(i) asm volatile("v_mul_u32_u24 %0, %0, %1" : "+v"(a##i) : "v"(m));
#define S_MULHI(i) asm volatile("v_mul_hi_u32 %0, %0, %1" : "+v"(a##i) : "v"(m));
QD_KF(k_fma, S_FMA)
QD_KF(k_add, S_ADD)
QD_KF(k_max, S_MAX)
QD_KF(k_med3, S_MED3)
QD_KF(k_exp, S_EXP)
QD_KU(k_bop3, S_BOP3)
QD_KU(k_and, S_AND)
QD_KU(k_cvt, S_CVT)
QD_KU(k_mul24, S_MUL24)
QD_KU(k_mulhi, S_MULHI)

// v_mad_u64_u32 chains through the 64-bit addend (16 per iteration)
#define S_MAD64(i)                                                                         \
  {                                                                                        \
    uint64_t carry;                                                                        \
    asm volatile("v_mad_u64_u32 %0, %1, %2, %3, %0" : "+v"(w##i), "=s"(carry) : "v"(m), "v"(n)); \
  }
#define QD_DECL_W(i) uint64_t w##i = (uint64_t)(gid + i) * 7u;
__global__ __launch_bounds__(kThreads) void k_mad64(float* out, int iters) {
  const int gid = blockIdx.x * kThreads + threadIdx.x;
  const uint32_t m = 0xD2511F53u + gid, n = gid * 5u;
  QD_CH8(QD_DECL_W)
  for (int it = 0; it < iters; ++it) { QD_CH8(S_MAD64) QD_CH8(S_MAD64) }
  out[gid] = (float)(uint32_t)(w0 ^ w1 ^ w2 ^ w3 ^ w4 ^ w5 ^ w6 ^ w7);
}

// fma and v_max_f32 alternating, 16 instructions per iteration
__global__ __launch_bounds__(kThreads) void k_fma_max(float* out, int iters) {
  const int gid = blockIdx.x * kThreads + threadIdx.x;
  const float b = 1.0001f + gid * 1e-9f, c = 0.5f;
  QD_CH8(QD_DECL_F)
  for (int it = 0; it < iters; ++it) { QD_CH8(S_FMA) QD_CH8(S_MAX) }
  out[gid] = QD_SUM_F;
}

// fma with the first source broadcast from lane 3 of each row of 16 (DPP);
// the broadcast source is never written inside the loop, and the s_nop keeps
// two wait states after its last write before the loop
#define S_DPP(i)                                                                          \
  asm volatile("v_fmac_f32_dpp %0, %1, %2 row_newbcast:3 row_mask:0xf bank_mask:0xf"      \
               : "+v"(a##i) : "v"(src), "v"(b));
__global__ __launch_bounds__(kThreads) void k_dpp(float* out, int iters) {
  const int gid = blockIdx.x * kThreads + threadIdx.x;
  const float b = 1.0001f + gid * 1e-9f, src = 0.25f + gid * 1e-7f;
  QD_CH8(QD_DECL_F)
  for (int it = 0; it < iters; ++it) {
    asm volatile("s_nop 1");
    QD_CH8(S_DPP) QD_CH8(S_DPP)
  }
  out[gid] = QD_SUM_F;
}

// the same two forms on four accumulators (a dot product's four partial
// sums): each accumulator is written every fourth instruction
#define QD_CH4(X) X(0) X(1) X(2) X(3)
__global__ __launch_bounds__(kThreads) void k_fma4(float* out, int iters) {
  const int gid = blockIdx.x * kThreads + threadIdx.x;
  const float b = 1.0001f + gid * 1e-9f, c = 0.5f;
  QD_CH8(QD_DECL_F)
  for (int it = 0; it < iters; ++it) { QD_CH4(S_FMA) QD_CH4(S_FMA) QD_CH4(S_FMA) QD_CH4(S_FMA) }
  out[gid] = QD_SUM_F;
}
__global__ __launch_bounds__(kThreads) void k_dpp4(float* out, int iters) {
  const int gid = blockIdx.x * kThreads + threadIdx.x;
  const float b = 1.0001f + gid * 1e-9f, src = 0.25f + gid * 1e-7f;
  QD_CH8(QD_DECL_F)
  for (int it = 0; it < iters; ++it) {
    asm volatile("s_nop 1");
    QD_CH4(S_DPP) QD_CH4(S_DPP) QD_CH4(S_DPP) QD_CH4(S_DPP)
  }
  out[gid] = QD_SUM_F;
}

__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// Philox4x32-10 (Salmon et al., SC'11); WIDE: one 64-bit multiply-add per
// product, else a low and a high 32-bit multiply
template <bool WIDE>
__device__ __forceinline__ uint4 philox10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                          uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    uint32_t h0, l0, h1, l1;
    if (WIDE) {
      const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
      h0 = (uint32_t)(p0 >> 32);
      l0 = (uint32_t)p0;
      h1 = (uint32_t)(p1 >> 32);
      l1 = (uint32_t)p1;
    } else {
      asm("v_mul_hi_u32 %0, %1, %2" : "=v"(h0) : "s"(0xD2511F53u), "v"(c0));
      asm("v_mul_lo_u32 %0, %1, %2" : "=v"(l0) : "s"(0xD2511F53u), "v"(c0));
      asm("v_mul_hi_u32 %0, %1, %2" : "=v"(h1) : "s"(0xCD9E8D57u), "v"(c2));
      asm("v_mul_lo_u32 %0, %1, %2" : "=v"(l1) : "s"(0xCD9E8D57u), "v"(c2));
    }
    const uint32_t n0 = xor3(h1, c1, k0), n2 = xor3(h0, c3, k1);
    c0 = n0;
    c1 = l1;
    c2 = n2;
    c3 = l0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(c0, c1, c2, c3);
}

template <bool WIDE>
__global__ __launch_bounds__(kThreads) void k_philox(float* out, int iters) {
  const uint32_t gid = blockIdx.x * kThreads + threadIdx.x;
  uint32_t acc = 0;
  for (int it = 0; it < iters; ++it) {
    const uint4 x = philox10<WIDE>(gid, (uint32_t)it, 7u, 2u, 1u, 2u);
    acc ^= xor3(x.x, x.y, x.z) ^ x.w;
  }
  out[gid] = (float)acc;
}

typedef void (*kern_t)(float*, int);

bool ok(hipError_t e) {
  if (e == hipSuccess) return true;
  std::fprintf(stderr, "HIP error: %s\n", hipGetErrorString(e));
  return false;
}

// Best of three launches, in ms.
bool time_kernel(kern_t k, int blocks, int iters, float* out, hipEvent_t e0, hipEvent_t e1,
                 float* best, size_t lds = 0) {
  *best = 1e30f;
  for (int r = 0; r < 3; ++r) {
    if (!ok(hipEventRecord(e0, 0))) return false;
    hipLaunchKernelGGL(k, dim3(blocks), dim3(kThreads), lds, 0, out, iters);
    if (!ok(hipGetLastError()) || !ok(hipEventRecord(e1, 0)) || !ok(hipEventSynchronize(e1)))
      return false;
    float ms = 0.0f;
    if (!ok(hipEventElapsedTime(&ms, e0, e1))) return false;
    if (ms < *best) *best = ms;
  }
  return true;
}

}  // namespace

int main() {
  float* out = nullptr;
  if (!ok(hipMalloc(&out, sizeof(float) * kMaxBlocks * kThreads))) return 1;
  hipEvent_t e0, e1;
  if (!ok(hipEventCreate(&e0)) || !ok(hipEventCreate(&e1))) return 1;
  const int iters = 20000;
  // bring the clocks up before the first measurement
  for (int w = 0; w < 30; ++w) hipLaunchKernelGGL(k_fma, dim3(kMaxBlocks), dim3(kThreads), 0, 0, out, iters);
  if (!ok(hipDeviceSynchronize())) return 1;

  struct Case { const char* name; kern_t k; int per_iter; };
  const Case forms[] = {
      {"v_fma_f32", k_fma, 16},          {"v_add_f32", k_add, 16},
      {"v_bitop3_b32", k_bop3, 16},      {"v_and_b32", k_and, 16},
      {"v_max_f32", k_max, 16},          {"v_med3_f32", k_med3, 16},
      {"v_cvt_f32_u32", k_cvt, 16},      {"v_mul_u32_u24", k_mul24, 16},
      {"v_mul_hi_u32", k_mulhi, 16},     {"v_exp_f32", k_exp, 16},
      {"v_mad_u64_u32", k_mad64, 16},
      {"v_fma_f32 + v_max_f32 (1:1)", k_fma_max, 16},
      {"v_fmac_f32_dpp row_newbcast", k_dpp, 16},
  };
  std::printf("# cycles per wave instruction per SIMD at 2.4 GHz, 8 waves per SIMD\n");
  for (const Case& c : forms) {
    float ms;
    if (!time_kernel(c.k, kMaxBlocks, iters, out, e0, e1, &ms)) return 2;
    const double per_simd = (double)kMaxBlocks * kThreads / 64.0 / 1024.0 * iters * c.per_iter;
    std::printf("%-30s %8.3f ms  %5.2f cycles\n", c.name, ms, ms * 1e-3 * 2.4e9 / per_simd);
  }
  // Waves per SIMD pinned by LDS: a workgroup (4 waves) takes 160 KB / (w + 1)
  // < bytes <= 160 KB / w of dynamic LDS, so w workgroups fit a CU and w + 1 do
  // not; 2048 workgroups run in rounds at that occupancy.  One wave per SIMD:
  // 256 workgroups, one per CU, in a single round.
  int lds_per_cu = 0;
  if (!ok(hipDeviceGetAttribute(&lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, 0)))
    return 1;
  std::printf("# the same per SIMD at 1, 2, 3, 4, 8 waves per SIMD (LDS per CU %d bytes)\n", lds_per_cu);
  const Case chains[] = {{"v_fma_f32, 8 chains", k_fma, 16},
                         {"v_fmac_f32_dpp, 8 chains", k_dpp, 16},
                         {"v_fma_f32, 4 chains", k_fma4, 16},
                         {"v_fmac_f32_dpp, 4 chains", k_dpp4, 16}};
  const int chain_iters = 20000;
  for (const Case& c : chains) {
    for (int wps : {1, 2, 3, 4, 8}) {
      const int blocks = wps == 1 ? 256 : kMaxBlocks;
      const size_t lds = wps == 1 ? 0 : (size_t)(lds_per_cu / wps) & ~(size_t)1023;
      if (wps > 1 && (lds * (size_t)(wps + 1) <= (size_t)lds_per_cu ||
                      hipFuncSetAttribute((const void*)c.k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                          (int)lds) != hipSuccess)) {
        std::printf("%-30s %d waves/SIMD: LDS cannot pin it\n", c.name, wps);
        continue;
      }
      float ms;
      if (!time_kernel(c.k, blocks, chain_iters, out, e0, e1, &ms, lds)) return 2;
      const double per_simd = (double)blocks * 4.0 / 1024.0 * chain_iters * c.per_iter;
      std::printf("%-30s %d waves/SIMD %8.3f ms  %5.2f cycles\n", c.name, wps, ms,
                  ms * 1e-3 * 2.4e9 / per_simd);
    }
  }
  std::printf("# Philox4x32-10 draws per second, chip-wide\n");
  const Case px[] = {{"v_mad_u64_u32 products", k_philox<true>, 1},
                     {"v_mul_lo/hi_u32 products", k_philox<false>, 1}};
  for (const Case& c : px) {
    float ms;
    if (!time_kernel(c.k, kMaxBlocks, 2000, out, e0, e1, &ms)) return 2;
    std::printf("%-30s %8.3f ms  %.3e draws/s\n", c.name, ms,
                (double)kMaxBlocks * kThreads * 2000 / (ms * 1e-3));
  }
  const bool good = ok(hipDeviceSynchronize());
  (void)hipFree(out);
  return good ? 0 : 2;
}
