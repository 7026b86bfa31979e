// Per-head absmax quantization of Q, K, V to OCP e4m3fn on gfx950.
//
// Eq. (2) of the paper (Sec. 3): s = max|X^(h)| / 448 per head,
// X_8 = rn_fp8(clamp(X / s, -448, 448)), fp32 scale; test queries use the
// train-query scale.  Three passes, all HBM-bound streams of the inputs:
//   1. amax_kernel   -- per-(tensor, b, h) max|x| with 16-byte loads; the
//                       maximum of non-negative floats is taken on their bit
//                       patterns as uint32 (order-preserving, exact), first in
//                       LDS, then one global atomic max per head per block;
//   2. scales_kernel -- s = fl32(amax / 448) (IEEE division), 1 where 0;
//   3. quantize_*    -- fl32(x / s) (IEEE division), clamp, and the hardware
//                       fp32 -> e4m3fn conversion, which rounds to nearest
//                       even; codes go to (B,H,rows,D), or, for V on the fused
//                       path, to the tile-transposed layout of attn_fp8.hip.
#include "common.h"

namespace tfm {
namespace {

constexpr int kThreads = 256;

template <typename T> struct Vec;
template <> struct Vec<float> { static constexpr int n = 4; };
template <> struct Vec<uint16_t> { static constexpr int n = 8; };

// |x| of the VEC elements of a 16-byte vector, as order-preserving uint32 bits.
__device__ inline uint32_t absmax_bits(u32x4 w, float*) {
  uint32_t a = max(w.x & 0x7fffffffu, w.y & 0x7fffffffu);
  uint32_t b = max(w.z & 0x7fffffffu, w.w & 0x7fffffffu);
  return max(a, b);
}
__device__ inline uint32_t absmax_bits(u32x4 w, uint16_t*) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t hi = w[i] & 0x7fff0000u;
    uint32_t lo = (w[i] << 16) & 0x7fff0000u;
    m = max(m, max(hi, lo));
  }
  return m;
}

// The VEC elements of a 16-byte vector as floats.
__device__ inline void unpack(u32x4 w, float* x, float*) {
  x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
  x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
}
__device__ inline void unpack(u32x4 w, float* x, uint16_t*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// e4m3fn code of clamp(fl32(x / s), -448, 448), round to nearest even.
// The division is the IEEE-correct fp32 division (HIP's default for '/');
// v_cvt_pk_fp8_f32 rounds to nearest even and keeps the sign of zero.
__device__ inline uint32_t codes4(const float* x, float s) {
  float y[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) y[i] = __builtin_amdgcn_fmed3f(x[i] / s, -448.0f, 448.0f);
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], w, true);
  return (uint32_t)w;
}

// Thread -> (row offset, vector position) map shared by the row kernels: a
// row of H*D elements is `vpr` 16-byte vectors; with vpr <= 256 each thread
// keeps one fixed position (so one fixed head) and strides over rows.
struct RowMap {
  int vpr, lanes_per_row, rows_per_iter;
  __device__ RowMap(int H, int D, int vec) {
    vpr = H * D / vec;
    lanes_per_row = vpr < kThreads ? vpr : kThreads;
    rows_per_iter = kThreads / lanes_per_row;
  }
};

template <typename T>
__global__ __launch_bounds__(kThreads) void amax_kernel(int first_tensor, int B, int H, int D, int N, int M,
                                                        int rows_per_chunk,
                                                        const T* __restrict__ q, const T* __restrict__ k,
                                                        const T* __restrict__ v, const T* __restrict__ qt,
                                                        uint32_t* __restrict__ amax) {
  extern __shared__ uint32_t smax[];  // H entries
  constexpr int VEC = Vec<T>::n;
  const int tensor = first_tensor + blockIdx.y, b = blockIdx.z;
  const T* x = tensor == 0 ? q : (tensor == 1 ? k : (tensor == 2 ? v : qt));
  if (tensor == 3) N = M;   // the test queries have M rows
  if ((int)blockIdx.x * rows_per_chunk >= N) return;
  for (int i = threadIdx.x; i < H; i += kThreads) smax[i] = 0;
  __syncthreads();
  const RowMap rm(H, D, VEC);
  const int t = threadIdx.x;
  const int r0 = blockIdx.x * rows_per_chunk;
  const int r1 = min(N, r0 + rows_per_chunk);
  if (t < rm.rows_per_iter * rm.lanes_per_row) {
    const int rr = t / rm.lanes_per_row;
    for (int p = t % rm.lanes_per_row; p < rm.vpr; p += rm.lanes_per_row) {
      uint32_t m = 0;
      const T* base = x + ((size_t)b * N) * H * D + (size_t)p * VEC;
      const size_t step = (size_t)rm.rows_per_iter * H * D;
      int row = r0 + rr;
      // four independent 16-byte loads in flight per thread, then the remainder
      for (; row + 3 * rm.rows_per_iter < r1; row += 4 * rm.rows_per_iter) {
        const T* src = base + (size_t)row * H * D;
        const u32x4 w0 = *reinterpret_cast<const u32x4*>(src);
        const u32x4 w1 = *reinterpret_cast<const u32x4*>(src + step);
        const u32x4 w2 = *reinterpret_cast<const u32x4*>(src + 2 * step);
        const u32x4 w3 = *reinterpret_cast<const u32x4*>(src + 3 * step);
        m = max(max(m, absmax_bits(w0, (T*)nullptr)), absmax_bits(w1, (T*)nullptr));
        m = max(max(m, absmax_bits(w2, (T*)nullptr)), absmax_bits(w3, (T*)nullptr));
      }
      for (; row < r1; row += rm.rows_per_iter) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(base + (size_t)row * H * D);
        m = max(m, absmax_bits(w, (T*)nullptr));
      }
      atomicMax(&smax[p * VEC / D], m);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < H; i += kThreads)
    if (smax[i]) atomicMax(&amax[((size_t)tensor * B + b) * H + i], smax[i]);
}

__global__ void fill_zero_kernel(uint32_t* p, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// s = fl32(amax / 448), 1 where that is 0.  scales[4][BH] = s_q (train), s_k, s_v,
// s_q_test.  Query-scale modes: shared -> s_q_test = s_q; per call -> each from
// its own rows; joint -> both from the max over train and test rows.
__device__ inline float scale_of(uint32_t amax_bits) {
  float s = __uint_as_float(amax_bits) / 448.0f;
  return s == 0.0f ? 1.0f : s;
}
__global__ void scales_kernel(int BH, int q_scale_mode, const uint32_t* __restrict__ amax, float* __restrict__ scales,
                              float* s_q, float* s_k, float* s_v, float* s_q_test) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= BH) return;
  const uint32_t aq = amax[i], aqt = amax[3 * BH + i];
  const float sq = scale_of(q_scale_mode == TFM_QSCALE_JOINT ? max(aq, aqt) : aq);
  const float sqt = q_scale_mode == TFM_QSCALE_PER_CALL ? scale_of(aqt) : sq;
  const float sk = scale_of(amax[BH + i]), sv = scale_of(amax[2 * BH + i]);
  scales[i] = sq; scales[BH + i] = sk; scales[2 * BH + i] = sv; scales[3 * BH + i] = sqt;
  if (s_q) s_q[i] = sq;
  if (s_k) s_k[i] = sk;
  if (s_v) s_v[i] = sv;
  if (s_q_test) s_q_test[i] = sqt;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void quantize_rows_kernel(int H, int D, int rows, int rows_per_chunk,
                                                                 const T* __restrict__ x,
                                                                 const float* __restrict__ scale,
                                                                 uint8_t* __restrict__ codes) {
  constexpr int VEC = Vec<T>::n;
  const int b = blockIdx.y;
  const int r0 = blockIdx.x * rows_per_chunk;
  const RowMap rm(H, D, VEC);
  const int t = threadIdx.x;
  const int r1 = min(rows, r0 + rows_per_chunk);
  if (t >= rm.rows_per_iter * rm.lanes_per_row) return;
  const int rr = t / rm.lanes_per_row;
  for (int p = t % rm.lanes_per_row; p < rm.vpr; p += rm.lanes_per_row) {
    const int h = p * VEC / D, d0 = (p * VEC) % D;
    const float s = scale[b * H + h];
    const T* src = x + ((size_t)b * rows) * H * D + (size_t)p * VEC;
    uint8_t* dst = codes + (((size_t)b * H + h) * rows) * D + d0;
    // U rows per thread-iteration: their loads are all issued before any is converted
    constexpr int U = 4;
    int row = r0 + rr;
    for (; row < r1; row += U * rm.rows_per_iter) {
      u32x4 w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ru = row + u * rm.rows_per_iter;
        w[u] = ru < r1 ? *reinterpret_cast<const u32x4*>(src + (size_t)ru * H * D) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ru = row + u * rm.rows_per_iter;
        if (ru >= r1) break;
        float xv[VEC];
        unpack(w[u], xv, (T*)nullptr);
        if constexpr (VEC == 4) {
          *reinterpret_cast<uint32_t*>(dst + (size_t)ru * D) = codes4(xv, s);
        } else {
          uint2 o;
          o.x = codes4(xv, s);
          o.y = codes4(xv + 4, s);
          *reinterpret_cast<uint2*>(dst + (size_t)ru * D) = o;
        }
      }
    }
  }
}

// Position of key kk (0..63) of a 64-key tile inside the tile-transposed V
// layout: the PV product of attn_fp8.hip feeds lane half `hf` and byte j of
// its B operand with key ((j%16)/4)*8 + hf*4 + j%4 + 32*(j/16) (the row
// order of the QK^T accumulator), so V is stored in that order.
__device__ inline int v_tile_pos(int kk) {
  const int tile = kk >> 5, kp = kk & 31;
  const int g = kp >> 3, hf = (kp >> 2) & 1, i = kp & 3;
  return hf * 32 + tile * 16 + g * 4 + i;
}

// One block per (b*H + h, 64-key tile): codes of the tile's V rows (from
// inputs or from (B,H,N,D) codes) transposed through LDS into
// v8t[((b*H + h)*ntiles + tile)*D*64 + d*64 + pos].  Keys >= N get code 0.
template <typename T, bool FROM_CODES>
__global__ __launch_bounds__(kThreads) void v_tiles_kernel(int H, int D, int N, const T* __restrict__ src,
                                                           const float* __restrict__ scale,
                                                           uint8_t* __restrict__ v8t) {
  __shared__ uint8_t tile_codes[128 * 64];
  const int bh = blockIdx.y, kt = blockIdx.x;
  const int b = bh / H, h = bh % H;
  const int ntiles = (N + 63) / 64;
  if constexpr (FROM_CODES) {
    // src: (B,H,N,D) codes; 16 codes per thread-iteration
    const int per_row = D / 16;
    for (int i = threadIdx.x; i < 64 * per_row; i += kThreads) {
      const int kk = i / per_row, c = i % per_row;
      const int key = kt * 64 + kk;
      u32x4 w = {0u, 0u, 0u, 0u};
      if (key < N) w = *reinterpret_cast<const u32x4*>(src + ((size_t)bh * N + key) * D + c * 16);
      const int pos = v_tile_pos(kk);
#pragma unroll
      for (int j = 0; j < 16; ++j) tile_codes[(c * 16 + j) * 64 + pos] = (uint8_t)(w[j / 4] >> (8 * (j % 4)));
    }
  } else {
    constexpr int VEC = Vec<T>::n;
    const float s = scale[bh];
    const int per_row = D / VEC;
    const int items = 64 * per_row;       // a multiple of 2 * 256 for D = 64 and 128
    constexpr int U = 2;
    for (int i0 = threadIdx.x; i0 < items; i0 += U * kThreads) {
      u32x4 w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {       // loads first
        const int i = i0 + u * kThreads;
        const int key = kt * 64 + i / per_row;
        w[u] = (i < items && key < N)
                   ? *reinterpret_cast<const u32x4*>(src + (((size_t)b * N + key) * H + h) * D + (i % per_row) * VEC)
                   : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * kThreads;
        if (i >= items) break;
        const int kk = i / per_row, c = i % per_row;
        uint32_t cw[VEC / 4];
        float xv[VEC];
        unpack(w[u], xv, (T*)nullptr);
#pragma unroll
        for (int j = 0; j < VEC / 4; ++j) cw[j] = codes4(xv + 4 * j, s);   // zero inputs give code 0
        const int pos = v_tile_pos(kk);
#pragma unroll
        for (int j = 0; j < VEC; ++j) tile_codes[(c * VEC + j) * 64 + pos] = (uint8_t)(cw[j / 4] >> (8 * (j % 4)));
      }
    }
  }
  __syncthreads();
  uint8_t* dst = v8t + ((size_t)bh * ntiles + kt) * D * 64;
  for (int i = threadIdx.x; i < D * 4; i += kThreads)
    reinterpret_cast<u32x4*>(dst)[i] = reinterpret_cast<const u32x4*>(tile_codes)[i];
}

int chunk_rows(int rows, int H, int D, int esize) {
  // about 64 KiB of input per block (measured best among 64 KiB .. 512 KiB)
  long per_row = (long)H * D * esize;
  long r = (65536 + per_row - 1) / per_row;
  if (r < 1) r = 1;
  if (r > rows) r = rows > 0 ? rows : 1;
  return (int)r;
}

}  // namespace

hipError_t launch_fill_zero_u32(uint32_t* p, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_amax(int in_bf16, int first, int last, int B, int H, int D, int N, int M, const void* q_train,
                       const void* k, const void* v, const void* q_test, uint32_t* amax, hipStream_t s) {
  if (last == 3 && M == 0) last = 2;   // no test rows to scan
  if (last < first) return hipSuccess;
  const int esize = in_bf16 ? 2 : 4;
  const int rows = first == 3 ? M : ((last == 3 && M > N) ? M : N);   // the most rows of any launched tensor
  const int rpc = chunk_rows(first == 3 ? M : N, H, D, esize);
  dim3 grid((rows + rpc - 1) / rpc, last - first + 1, B);
  size_t lds = (size_t)H * sizeof(uint32_t);
  if (in_bf16)
    hipLaunchKernelGGL(amax_kernel<uint16_t>, grid, dim3(kThreads), lds, s, first, B, H, D, N, M, rpc,
                       (const uint16_t*)q_train, (const uint16_t*)k, (const uint16_t*)v, (const uint16_t*)q_test,
                       amax);
  else
    hipLaunchKernelGGL(amax_kernel<float>, grid, dim3(kThreads), lds, s, first, B, H, D, N, M, rpc,
                       (const float*)q_train, (const float*)k, (const float*)v, (const float*)q_test, amax);
  return hipGetLastError();
}

hipError_t launch_scales(int BH, int q_scale_mode, const uint32_t* amax, float* scales, float* s_q, float* s_k,
                         float* s_v, float* s_q_test, hipStream_t s) {
  hipLaunchKernelGGL(scales_kernel, dim3((BH + 255) / 256), dim3(256), 0, s, BH, q_scale_mode, amax, scales, s_q,
                     s_k, s_v, s_q_test);
  return hipGetLastError();
}

hipError_t launch_quantize_rows(int in_bf16, int B, int H, int D, int rows, const void* x, const float* scale,
                                uint8_t* codes, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int esize = in_bf16 ? 2 : 4;
  const int rpc = chunk_rows(rows, H, D, esize);
  dim3 grid((rows + rpc - 1) / rpc, B);
  if (in_bf16)
    hipLaunchKernelGGL(quantize_rows_kernel<uint16_t>, grid, dim3(kThreads), 0, s, H, D, rows, rpc,
                       (const uint16_t*)x, scale, codes);
  else
    hipLaunchKernelGGL(quantize_rows_kernel<float>, grid, dim3(kThreads), 0, s, H, D, rows, rpc,
                       (const float*)x, scale, codes);
  return hipGetLastError();
}

hipError_t launch_quantize_v_tiles(int in_bf16, int B, int H, int D, int N, const void* v, const float* scale,
                                   uint8_t* v8t, hipStream_t s) {
  dim3 grid((N + 63) / 64, B * H);
  if (in_bf16)
    hipLaunchKernelGGL((v_tiles_kernel<uint16_t, false>), grid, dim3(kThreads), 0, s, H, D, N,
                       (const uint16_t*)v, scale, v8t);
  else
    hipLaunchKernelGGL((v_tiles_kernel<float, false>), grid, dim3(kThreads), 0, s, H, D, N, (const float*)v,
                       scale, v8t);
  return hipGetLastError();
}

hipError_t launch_relayout_v_tiles(int B, int H, int D, int N, const uint8_t* v8, uint8_t* v8t, hipStream_t s) {
  dim3 grid((N + 63) / 64, B * H);
  hipLaunchKernelGGL((v_tiles_kernel<uint8_t, true>), grid, dim3(kThreads), 0, s, H, D, N, v8,
                     (const float*)nullptr, v8t);
  return hipGetLastError();
}

}  // namespace tfm
