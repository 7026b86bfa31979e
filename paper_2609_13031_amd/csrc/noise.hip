// Per-head RMS-scaled Gaussian perturbation, Eq. (3) (appendix, noise
// experiment): X~ = X + eps * rho * Z per (table b, head h), where rho is the
// RMS of that head over its S rows and D channels and Z is a caller-drawn
// standard-normal field.  Three passes, all streams over HBM:
//   1. sumsq_kernel    -- per (row chunk, b, h) sum of x^2 in fp64 (squares of
//                         fp32 values are exact in fp64), reduced inside the
//                         block in a fixed order, so the result does not
//                         depend on scheduling (no atomics);
//   2. finalize_kernel -- rho = fl32(sqrt(sum over chunks / (S*D))), the chunks
//                         combined in a fixed order by one block per head;
//   3. apply_kernel    -- y = fmaf(fl32(eps * rho), z, x), one rounding, then
//                         to the output type (bf16: round to nearest even).
// Every 8-element group lies in one head (D % 8 == 0), which is the unit all
// three passes work on.
#include "common.h"

namespace tfm {
namespace {

constexpr int kThreads = 256;
constexpr int kGroup = 8;          // elements per group
constexpr int kChunkElems = 32768; // about this many elements per pass-1 block

__device__ inline void load8(const uint16_t* p, float* x) {
  const u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ inline void load8(const float* p, float* x) {
  const v4f a = *reinterpret_cast<const v4f*>(p);
  const v4f b = *reinterpret_cast<const v4f*>(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) { x[i] = a[i]; x[4 + i] = b[i]; }
}
__device__ inline void store8(uint16_t* p, const float* y) {
  typedef __bf16 v8b __attribute__((ext_vector_type(8)));
  v8b o;
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = (__bf16)y[i];
  *reinterpret_cast<v8b*>(p) = o;
}
__device__ inline void store8(float* p, const float* y) {
  *reinterpret_cast<v4f*>(p) = v4f{y[0], y[1], y[2], y[3]};
  *reinterpret_cast<v4f*>(p + 4) = v4f{y[4], y[5], y[6], y[7]};
}

// Pass 1.  Block (chunk, b) covers rows [chunk*rpc, +rpc) of table b.  A row
// is gpr = H*D/8 groups.  With gpr < 256 the block reads rpi = 256/gpr rows
// at a time and thread t owns group t % gpr of row offset t / gpr; otherwise
// thread t owns groups t, t+256, ...  Each (row offset, group) pair has one
// LDS slot, written by exactly one thread; head h then sums its slots in
// (row offset, group) order.
template <typename T>
__global__ __launch_bounds__(kThreads) void sumsq_kernel(int S, int H, int D, int rpc, const T* __restrict__ x,
                                                         double* __restrict__ partial) {
  extern __shared__ double slot[];
  const int chunk = blockIdx.x, b = blockIdx.y, B = gridDim.y;
  const int gpr = H * D / kGroup;
  const int lanes = gpr < kThreads ? gpr : kThreads;
  const int rpi = kThreads / lanes;
  const int t = threadIdx.x;
  const int r0 = chunk * rpc;
  const int r1 = min(S, r0 + rpc);
  if (t < rpi * lanes) {
    const int rr = t / lanes;
    for (int g = t % lanes; g < gpr; g += lanes) {
      double acc = 0.0;
      const T* base = x + ((size_t)b * S * H * D) + (size_t)g * kGroup;
      for (int row = r0 + rr; row < r1; row += rpi) {
        float v[kGroup];
        load8(base + (size_t)row * H * D, v);
#pragma unroll
        for (int i = 0; i < kGroup; ++i) acc = __builtin_fma((double)v[i], (double)v[i], acc);
      }
      slot[rr * gpr + g] = acc;
    }
  }
  __syncthreads();
  const int gph = D / kGroup;  // groups per head
  for (int h = t; h < H; h += kThreads) {
    double sum = 0.0;
    for (int rr = 0; rr < rpi; ++rr)
      for (int g = h * gph; g < (h + 1) * gph; ++g) sum += slot[rr * gpr + g];
    partial[((size_t)chunk * B + b) * H + h] = sum;
  }
}

// Pass 2: one block per (b, h).  Thread t sums chunks t, t+256, ... in order,
// then a fixed binary tree combines the 256 partial sums.
__global__ __launch_bounds__(kThreads) void finalize_kernel(int BH, int chunks, int S, int D,
                                                            const double* __restrict__ partial,
                                                            float* __restrict__ rho, float* rho_out) {
  __shared__ double red[kThreads];
  const int i = blockIdx.x, t = threadIdx.x;
  double sum = 0.0;
  for (int c = t; c < chunks; c += kThreads) sum += partial[(size_t)c * BH + i];
  red[t] = sum;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w /= 2) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) {
    const float r = (float)__builtin_sqrt(red[0] / ((double)S * (double)D));
    rho[i] = r;
    if (rho_out) rho_out[i] = r;
  }
}

// Pass 3: kPer consecutive groups per thread-iteration, blocks of 256*kPer groups.
constexpr int kPer = 4;
template <typename T, typename TZ>
__global__ __launch_bounds__(kThreads) void apply_kernel(long long groups, int S, int H, int D, float eps,
                                                         const T* x, const TZ* z, const float* __restrict__ rho,
                                                         T* out) {
  const long long base = (long long)blockIdx.x * kThreads * kPer + threadIdx.x;
  const long long per_table = (long long)S * H * D;
  float xv[kPer][kGroup], zv[kPer][kGroup];
  float e[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const long long gi = base + (long long)k * kThreads;
    if (gi < groups) {
      const long long el = gi * kGroup;
      load8(x + el, xv[k]);
      load8(z + el, zv[k]);
      const int b = (int)(el / per_table);
      const int h = (int)((el / D) % H);
      e[k] = eps * rho[b * H + h];
    }
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const long long gi = base + (long long)k * kThreads;
    if (gi < groups) {
      float y[kGroup];
#pragma unroll
      for (int i = 0; i < kGroup; ++i) y[i] = __builtin_fmaf(e[k], zv[k][i], xv[k][i]);
      store8(out + gi * kGroup, y);
    }
  }
}

}  // namespace

int noise_rows_per_chunk(int H, int D) {
  const int r = (kChunkElems + H * D - 1) / (H * D);
  return r < 1 ? 1 : r;
}

long long noise_grid_blocks(int B, int H, int S, int D) {
  const long long groups = (long long)B * S * H * D / kGroup;
  const long long apply = (groups + kThreads * kPer - 1) / (kThreads * kPer);
  const int rpc = noise_rows_per_chunk(H, D);
  const long long chunks = ((long long)S + rpc - 1) / rpc;
  return apply > chunks ? apply : chunks;
}

hipError_t launch_noise(int x_bf16, int z_bf16, int B, int H, int S, int D, const void* x, const void* z, float eps,
                        void* out, double* partial, float* rho, float* rho_out, hipStream_t s) {
  const int rpc = noise_rows_per_chunk(H, D);
  const int chunks = (S + rpc - 1) / rpc;
  const int gpr = H * D / kGroup;
  const int lanes = gpr < kThreads ? gpr : kThreads;
  const size_t lds = (size_t)(kThreads / lanes) * gpr * sizeof(double);
  dim3 g1(chunks, B);
  if (x_bf16)
    hipLaunchKernelGGL(sumsq_kernel<uint16_t>, g1, dim3(kThreads), lds, s, S, H, D, rpc, (const uint16_t*)x,
                       partial);
  else
    hipLaunchKernelGGL(sumsq_kernel<float>, g1, dim3(kThreads), lds, s, S, H, D, rpc, (const float*)x, partial);
  const int BH = B * H;
  hipLaunchKernelGGL(finalize_kernel, dim3(BH), dim3(kThreads), 0, s, BH, chunks, S, D, partial, rho, rho_out);
  const long long groups = (long long)B * S * H * D / kGroup;
  const long long blocks = (groups + kThreads * kPer - 1) / (kThreads * kPer);
  dim3 g3((unsigned)blocks);
  if (x_bf16) {
    if (z_bf16)
      hipLaunchKernelGGL((apply_kernel<uint16_t, uint16_t>), g3, dim3(kThreads), 0, s, groups, S, H, D, eps,
                         (const uint16_t*)x, (const uint16_t*)z, rho, (uint16_t*)out);
    else
      hipLaunchKernelGGL((apply_kernel<uint16_t, float>), g3, dim3(kThreads), 0, s, groups, S, H, D, eps,
                         (const uint16_t*)x, (const float*)z, rho, (uint16_t*)out);
  } else {
    if (z_bf16)
      hipLaunchKernelGGL((apply_kernel<float, uint16_t>), g3, dim3(kThreads), 0, s, groups, S, H, D, eps,
                         (const float*)x, (const uint16_t*)z, rho, (float*)out);
    else
      hipLaunchKernelGGL((apply_kernel<float, float>), g3, dim3(kThreads), 0, s, groups, S, H, D, eps,
                         (const float*)x, (const float*)z, rho, (float*)out);
  }
  return hipGetLastError();
}

}  // namespace tfm
