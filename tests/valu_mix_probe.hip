// Issue-cost microbenchmark for the VALU work of the FP8 attention kernel
// (not part of libtfm).  Per (query, key) score the kernel issues one
// v_fma_f32 (c*s + bias), one v_exp_f32, half a v_cvt_pk_fp8_f32 (two scores
// per instruction) and half a v_max3_f32 (two new scores per instruction),
// plus, at head_dim 64, 2 * 64 * 64 MACs of FP8 MFMA per 64 scores.  This
// probe times that mix with and without the MFMAs, and each instruction
// alone, on every compute unit (4 waves per SIMD, 16 independent chains per
// wave), and prints wall time and cost per wave64 instruction in cycles of a
// 2.4 GHz clock.  The values it computes are meaningless; only time counts.
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
__global__ __launch_bounds__(256) void probe(float* out, int iters, float seed) {
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
}

template <int M>
float run(float* d, int blocks, int iters) {
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  probe<M><<<blocks, 256>>>(d, iters, 0.001f);
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(e0));
  probe<M><<<blocks, 256>>>(d, iters, 0.001f);
  CK(hipEventRecord(e1));
  CK(hipEventSynchronize(e1));
  float ms;
  CK(hipEventElapsedTime(&ms, e0, e1));
  CK(hipEventDestroy(e0));
  CK(hipEventDestroy(e1));
  return ms;
}

int main() {
  const int cus = 256, blocks = cus * 4, iters = 4000;  // 16 waves per CU, 4 per SIMD
  float* d;
  CK(hipMalloc(&d, (size_t)blocks * 256 * sizeof(float)));
  const char* names[] = {"v_fma_f32", "v_exp_f32", "v_cvt_pk_fp8_f32", "v_max3_f32", "v_mfma_f32_32x32x64_f8f6f4",
                         "mix: 16 fma + 16 exp + 8 cvt + 16 max3", "mix + 2 MFMA 32x32x64 f8 (D = 64)",
                         "mix + 4 MFMA 32x32x64 f8 (D = 128)"};
  float ms[8] = {run<0>(d, blocks, iters), run<1>(d, blocks, iters), run<2>(d, blocks, iters),
                 run<3>(d, blocks, iters), run<4>(d, blocks, iters), run<5>(d, blocks, iters),
                 run<6>(d, blocks, iters), run<7>(d, blocks, iters)};
  const double scores = (double)blocks * 256 * iters * 16;  // scores per mix run (16 per lane per step)
  for (int m = 0; m < 8; ++m) {
    const double cyc_step = ms[m] * 2.4e6 / iters;          // per SIMD, 2.4 GHz cycles
    const double per_instr = cyc_step / (4.0 * (m == 4 ? 4.0 : 16.0));
    printf("%-42s %8.3f ms", names[m], ms[m]);
    if (m < 5) printf("  %6.2f cycles per wave64 instruction", per_instr);
    if (m >= 5) {
      const int d = m == 7 ? 128 : 64;
      printf("  -> %.4g scores/s = %.0f TFLOP/s at head_dim %d (%d flop per score)", scores / (ms[m] * 1e-3),
             scores / (ms[m] * 1e-3) * 4 * d / 1e12, d, 4 * d);
    }
    printf("\n");
  }
  CK(hipFree(d));
  return 0;
}
