// Issue-cost microbenchmark for the VALU work of the FP8 attention kernel
// (not part of libtfm).  Per (query, key) score the kernel issues one
// v_fma_f32 (c*s + bias), one v_exp_f32, half a v_cvt_pk_fp8_f32 (two scores
// per instruction) and half a v_max3_f32 (two new scores per instruction),
// plus, at head_dim 64, 2 * 64 * 64 MACs of FP8 MFMA per 64 scores.  This
// probe times that mix with and without the MFMAs, and each instruction
// alone, on every compute unit (4 waves per SIMD, 16 independent chains per
// wave), and prints wall time and cost per wave64 instruction in cycles of a
// 2.4 GHz clock and of the shader clock the run actually got (each workgroup
// reads s_memtime, which counts shader cycles, and s_memrealtime, which counts
// at the fixed wall-clock rate, at its start and end).  The values it computes
// are meaningless; only time counts.
//
// Build and run (from the repository root):
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//     tests/valu_mix_probe.hip -o valu_mix_probe && ./valu_mix_probe
#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstdio>
#include <cstdlib>

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

#define CK(x)                                                                           \
  do {                                                                                  \
    hipError_t e_ = (x);                                                                \
    if (e_ != hipSuccess) {                                                             \
      printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);             \
      exit(1);                                                                          \
    }                                                                                   \
  } while (0)

#define R16(M) M(0) M(1) M(2) M(3) M(4) M(5) M(6) M(7) M(8) M(9) M(10) M(11) M(12) M(13) M(14) M(15)
#define FMA(i) asm volatile("v_fma_f32 %0, %0, %0, 1.0" : "+v"(a[i]));
#define EXP(i) asm volatile("v_exp_f32 %0, %0" : "+v"(a[i]));
#define CVT(i) asm volatile("v_cvt_pk_fp8_f32 %0, %1, %1" : "+v"(u[i]) : "v"(a[i]));
#define CVTH(i) asm volatile("v_cvt_pk_fp8_f32 %0, %1, %2" : "+v"(u[i]) : "v"(a[i]), "v"(a[i + 8]));
#define MAX3(i) asm volatile("v_max3_f32 %0, %0, %1, %1" : "+v"(a[i]) : "v"(a[(i + 1) & 15]));

// MODE 0..3: one instruction x16 per step; 4: four 32x32x64 FP8 MFMAs per step;
// 5: the per-score mix for 16 scores per lane; 6: the mix plus its 2 MFMAs at
// head_dim 64; 7: the mix plus its 4 MFMAs at head_dim 128.
template <int MODE>
__global__ __launch_bounds__(256) void probe(float* out, int iters, float seed, unsigned long long* clk) {
  const unsigned long long t0m = __builtin_amdgcn_s_memtime(), t0r = __builtin_amdgcn_s_memrealtime();
  float a[16];
  uint32_t u[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    a[i] = seed * (threadIdx.x + i);
    u[i] = threadIdx.x * 7 + i;
  }
  v16f acc0 = {}, acc1 = {};
  const v8i opa = {(int)threadIdx.x, 1, 2, 3, 4, 5, 6, 7};
  const v8i opb = {7, 6, 5, 4, 3, 2, 1, (int)threadIdx.x};
  for (int it = 0; it < iters; ++it) {
    if (MODE == 0) { R16(FMA) }
    if (MODE == 1) { R16(EXP) }
    if (MODE == 2) { R16(CVT) }
    if (MODE == 3) { R16(MAX3) }
    if (MODE == 4) {
      acc0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opa, opb, acc0, 0, 0, 0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opb, opa, acc1, 0, 0, 0, 0, 0, 0);
      acc0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opa, opb, acc0, 0, 0, 0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opb, opa, acc1, 0, 0, 0, 0, 0, 0);
    }
    if (MODE == 5 || MODE == 6 || MODE == 7) {
      R16(MAX3) R16(FMA) R16(EXP)
      CVTH(0) CVTH(1) CVTH(2) CVTH(3) CVTH(4) CVTH(5) CVTH(6) CVTH(7)
    }
    if (MODE == 6 || MODE == 7) {
      acc0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opa, opb, acc0, 0, 0, 0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opb, opa, acc1, 0, 0, 0, 0, 0, 0);
    }
    if (MODE == 7) {
      acc0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opa, opb, acc0, 0, 0, 0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opb, opa, acc1, 0, 0, 0, 0, 0, 0);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += a[i] + (float)u[i] + acc0[i] + acc1[i];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
  if (threadIdx.x == 0) {   // one lane per workgroup records its shader and wall-clock spans
    const unsigned long long t1m = __builtin_amdgcn_s_memtime(), t1r = __builtin_amdgcn_s_memrealtime();
    clk[2 * blockIdx.x] = t1m - t0m;
    clk[2 * blockIdx.x + 1] = t1r - t0r;
  }
}

struct Timing {
  float ms;      // wall time of the launch (HIP events)
  double ghz;    // mean shader clock over the workgroups' lifetimes
};

template <int M>
Timing run(float* d, unsigned long long* clk, int blocks, int iters, int wall_khz) {
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  probe<M><<<blocks, 256>>>(d, iters, 0.001f, clk);
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(e0));
  probe<M><<<blocks, 256>>>(d, iters, 0.001f, clk);
  CK(hipEventRecord(e1));
  CK(hipEventSynchronize(e1));
  Timing t;
  CK(hipEventElapsedTime(&t.ms, e0, e1));
  CK(hipEventDestroy(e0));
  CK(hipEventDestroy(e1));
  unsigned long long* h = (unsigned long long*)malloc(sizeof(unsigned long long) * 2 * blocks);
  CK(hipMemcpy(h, clk, sizeof(unsigned long long) * 2 * blocks, hipMemcpyDeviceToHost));
  double cycles = 0, ticks = 0;
  for (int b = 0; b < blocks; ++b) {
    cycles += (double)h[2 * b];
    ticks += (double)h[2 * b + 1];
  }
  free(h);
  t.ghz = cycles / ticks * wall_khz * 1e3 / 1e9;
  return t;
}

int main() {
  const int cus = 256, blocks = cus * 4, iters = 4000;  // 16 waves per CU, 4 per SIMD
  int wall_khz = 0;
  CK(hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, 0));
  float* d;
  unsigned long long* clk;
  CK(hipMalloc(&d, (size_t)blocks * 256 * sizeof(float)));
  CK(hipMalloc(&clk, (size_t)blocks * 2 * sizeof(unsigned long long)));
  const char* names[] = {"v_fma_f32", "v_exp_f32", "v_cvt_pk_fp8_f32", "v_max3_f32", "v_mfma_f32_32x32x64_f8f6f4",
                         "mix: 16 fma + 16 exp + 8 cvt + 16 max3", "mix + 2 MFMA 32x32x64 f8 (D = 64)",
                         "mix + 4 MFMA 32x32x64 f8 (D = 128)"};
  Timing t[8] = {run<0>(d, clk, blocks, iters, wall_khz), run<1>(d, clk, blocks, iters, wall_khz),
                 run<2>(d, clk, blocks, iters, wall_khz), run<3>(d, clk, blocks, iters, wall_khz),
                 run<4>(d, clk, blocks, iters, wall_khz), run<5>(d, clk, blocks, iters, wall_khz),
                 run<6>(d, clk, blocks, iters, wall_khz), run<7>(d, clk, blocks, iters, wall_khz)};
  const double scores = (double)blocks * 256 * iters * 16;  // scores per mix run (16 per lane per step)
  printf("wall-clock counter rate: %d kHz\n", wall_khz);
  for (int m = 0; m < 8; ++m) {
    const double per_step = t[m].ms * 1e-3 / iters;           // seconds per loop step (per SIMD: 4 waves)
    const double n = 4.0 * (m == 4 ? 4.0 : 16.0);            // wave64 instructions per step per SIMD
    printf("%-42s %8.3f ms  clock %.3f GHz", names[m], t[m].ms, t[m].ghz);
    if (m < 5)
      printf("  %6.2f cycles per wave64 instruction at 2.4 GHz, %6.2f at the measured clock", per_step * 2.4e9 / n,
             per_step * t[m].ghz * 1e9 / n);
    if (m >= 5) {
      const int hd = m == 7 ? 128 : 64;
      const double tf = scores / (t[m].ms * 1e-3) * 4 * hd / 1e12;
      printf("  -> %.4g scores/s = %.0f TFLOP/s at head_dim %d (%.0f TFLOP/s per GHz)", scores / (t[m].ms * 1e-3), tf,
             hd, tf / t[m].ghz);
    }
    printf("\n");
  }
  CK(hipFree(clk));
  CK(hipFree(d));
  return 0;
}
