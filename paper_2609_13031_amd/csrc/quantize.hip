// Per-head absmax quantization of Q, K, V to OCP e4m3fn on gfx950.
//
// Eq. (2) of the paper (Sec. 3): s = max|X^(h)| / 448 per head,
// X_8 = rn_fp8(clamp(X / s, -448, 448)), fp32 scale; test queries use the
// train-query scale.  Two launches, both HBM-bound streams of the inputs:
//   1. amax_kernel     -- one block per (row slice, tensor, table, head group)
//                         takes max|x| per head with 16-byte loads (the maximum
//                         of non-negative floats is taken on their bit patterns
//                         as uint32: order-preserving and exact), reduces the
//                         lanes of each head with cross-lane shuffles and the
//                         block's lanes in LDS, and writes the result to its own
//                         slot of partial[tensor][b][h][slice].  Every slot is
//                         written exactly once, so nothing has to be zeroed
//                         first and no global atomics are needed;
//   2. quantize_kernel -- one launch over all tensors (V, K, Q_train, Q_test,
//                         in that order).  Each block first reduces the slice
//                         maxima of the heads it covers to their scales,
//                         s = fl32(amax / 448) (IEEE division, 1 where 0), then
//                         writes fl32(x / s) (IEEE division), clamped, through
//                         the hardware fp32 -> e4m3fn conversion (round to
//                         nearest even) to (B,H,rows,D), or, for V on the fused
//                         path, to the tile-transposed layout of attn_fp8.hip.
//                         The first block of each (tensor, table, heads) also
//                         stores the scales.
// A third kernel re-lays V codes that are already quantized into the tile
// layout (the prequantized entry point).
#include "common.h"

namespace tfm {
namespace {

constexpr int kThreads = 256;
constexpr int kHeadGroup = 32;  // heads per block in the row kernels (their scales are kept in LDS)

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

// Thread -> (row offset, vector position) map of the row kernels for one block
// of `hn` heads: a row of hn*D elements is `vpr` 16-byte vectors; with vpr <=
// 256 each thread keeps one fixed position (so one fixed head) and strides over
// rows.
struct RowMap {
  int vpr, lanes_per_row, rows_per_iter;
  __device__ RowMap(int hn, int D, int vec) {
    vpr = hn * D / vec;
    lanes_per_row = vpr < kThreads ? vpr : kThreads;
    rows_per_iter = kThreads / lanes_per_row;
  }
};

__host__ __device__ inline int head_groups(int H) { return (H + kHeadGroup - 1) / kHeadGroup; }

struct AmaxArgs {
  int first_tensor;       // tensors first_tensor .. first_tensor + gridDim.y / groups - 1
  int B, H, D, N, M;
  const void* x[4];       // Q_train, K, V, Q_test
  uint32_t* partial;      // [4][B][H][kAmaxSlices]
};

template <typename T>
__global__ __launch_bounds__(kThreads) void amax_kernel(AmaxArgs a) {
  __shared__ uint32_t smax[kHeadGroup];
  constexpr int VEC = Vec<T>::n;
  const int groups = head_groups(a.H);
  const int tensor = a.first_tensor + blockIdx.y / groups;
  const int h0 = (blockIdx.y % groups) * kHeadGroup, hn = min(kHeadGroup, a.H - h0);
  const int b = blockIdx.z, g = blockIdx.x;
  const int rows = tensor == 3 ? a.M : a.N;
  if (g >= amax_slices(rows)) return;   // whole block: this tensor has fewer slices
  const int H = a.H, D = a.D;
  const int sr = amax_slice_rows(rows);
  const int r0 = g * sr, r1 = min(rows, r0 + sr);
  if (threadIdx.x < hn) smax[threadIdx.x] = 0;
  __syncthreads();
  const RowMap rm(hn, D, VEC);
  const int t = threadIdx.x;
  const int active = rm.rows_per_iter * rm.lanes_per_row;
  const int rr = t / rm.lanes_per_row;
  const T* x = (const T*)a.x[tensor] + ((size_t)b * rows) * H * D + (size_t)h0 * D;
  const size_t step = (size_t)rm.rows_per_iter * H * D;
  // The D / VEC lanes that hold one head's columns of one row slot are consecutive and
  // aligned (lanes_per_row and the position stride are multiples of D / VEC, which
  // divides 64), so they never straddle a wave.  Every thread runs the same number of
  // position rounds, so the shuffles below always see the whole wave.
  const int seg = D / VEC;
  for (int p0 = 0; p0 < rm.vpr; p0 += rm.lanes_per_row) {
    const int p = p0 + t % rm.lanes_per_row;
    const bool mine = t < active && p < rm.vpr;
    uint32_t m = 0;
    if (mine) {
      const T* base = x + (size_t)p * VEC;
      // eight independent 16-byte loads in flight per thread; rows past the slice read as 0
      for (int row = r0 + rr; row < r1; row += 8 * rm.rows_per_iter) {
        const T* src = base + (size_t)row * H * D;
        u32x4 w[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          w[u] = row + u * rm.rows_per_iter < r1 ? *reinterpret_cast<const u32x4*>(src + u * step)
                                                 : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int u = 0; u < 8; ++u) m = max(m, absmax_bits(w[u], (T*)nullptr));
      }
    }
    // the head's lanes combine their maxima with cross-lane shuffles; the first of them
    // folds the result into the block's per-head maximum
    for (int off = 1; off < seg; off <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
    if (mine && t % seg == 0) atomicMax(&smax[p / seg], m);
  }
  __syncthreads();
  if (threadIdx.x < hn)
    a.partial[(((size_t)tensor * a.B + b) * H + h0 + threadIdx.x) * kAmaxSlices + g] = smax[threadIdx.x];
}

// ---- quantize: one launch over the code tensors of a call ----

struct QSeg {
  const void* x;    // (B, rows, H, D) input
  uint8_t* codes;   // (B, H, rows, D) codes, or the V tile layout when v_tiles
  float* s_out;     // caller's copy of this tensor's (B, H) scales, or NULL
  int tensor;       // 0 Q_train, 1 K, 2 V, 3 Q_test (the amax and scale slot)
  int v_tiles;      // 1: 64-key tiles in the transposed layout of attn_fp8.hip
  int rows;         // N, or M for Q_test
  int rpc;          // rows per block (row layout)
  int per_table;    // blocks per table
  int first;        // first block of the segment in the grid
};

struct QArgs {
  QSeg seg[4];
  int nseg;
  int B, H, D, N, M, mode;
  int train_q_sets_test_slot;  // the Q_train segment also stores slot 3 (no Q_test segment)
  const uint32_t* partial;
  float* scales;               // [4][B*H]: s_q, s_k, s_v, s_q_test
  float* s_q_test_out;         // caller's copy of s_q_test, or NULL
};

// Max of the slice maxima of one (tensor, b, h), reduced by one wave; every lane returns it.
__device__ inline uint32_t wave_head_amax(const QArgs& a, int tensor, int b, int h, int lane) {
  const int n = amax_slices(tensor == 3 ? a.M : a.N);
  const uint32_t* p = a.partial + (((size_t)tensor * a.B + b) * a.H + h) * kAmaxSlices;
  uint32_t m = 0;
  for (int g = lane; g < n; g += 64) m = max(m, p[g]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  return m;
}

__device__ inline float scale_of(uint32_t amax_bits) {
  float s = __uint_as_float(amax_bits) / 448.0f;
  return s == 0.0f ? 1.0f : s;
}

// Scale of slot `tensor` for head (b, h) under the query-scale mode: shared ->
// test queries on the train-query scale; per call -> each query set on its own
// rows; joint -> both on the max over train and test rows.  The test-query
// maxima exist only when the mode needs them and there are test rows.
__device__ inline float wave_scale(const QArgs& a, int tensor, int b, int h, int lane) {
  if (tensor == 1 || tensor == 2) return scale_of(wave_head_amax(a, tensor, b, h, lane));
  const bool have_test = a.mode != TFM_QSCALE_SHARED && a.M > 0;
  if (a.mode == TFM_QSCALE_PER_CALL && tensor == 3) return scale_of(have_test ? wave_head_amax(a, 3, b, h, lane) : 0u);
  uint32_t m = wave_head_amax(a, 0, b, h, lane);
  if (a.mode == TFM_QSCALE_JOINT && have_test) m = max(m, wave_head_amax(a, 3, b, h, lane));
  return scale_of(m);
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

template <typename T>
__global__ __launch_bounds__(kThreads) void quantize_kernel(QArgs a) {
  __shared__ float sc[kHeadGroup];
  __shared__ uint8_t tile_codes[128 * 64];   // one 64-key V tile, transposed (D <= 128)
  constexpr int VEC = Vec<T>::n;
  int si = 0;
  while (si + 1 < a.nseg && (int)blockIdx.x >= a.seg[si + 1].first) ++si;
  const QSeg& sg = a.seg[si];
  const int local = blockIdx.x - sg.first;
  const int b = local / sg.per_table, rem = local % sg.per_table;
  const int H = a.H, D = a.D, rows = sg.rows;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;

  if (sg.v_tiles) {
    // one block per (b, h, 64-key tile) of V
    const int ntiles = (rows + 63) / 64;
    const int h = rem / ntiles, kt = rem % ntiles;
    if (wave == 0) {
      const float s = wave_scale(a, sg.tensor, b, h, lane);
      if (lane == 0) {
        sc[0] = s;
        if (kt == 0) {
          a.scales[(size_t)sg.tensor * a.B * H + b * H + h] = s;
          if (sg.s_out) sg.s_out[b * H + h] = s;
        }
      }
    }
    __syncthreads();
    const float s = sc[0];
    const int per_row = D / VEC;
    const int items = 64 * per_row;       // a multiple of 2 * 256 for D = 64 and 128
    constexpr int U = 2;
    for (int i0 = threadIdx.x; i0 < items; i0 += U * kThreads) {
      u32x4 w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {       // loads first
        const int i = i0 + u * kThreads;
        const int key = kt * 64 + i / per_row;
        w[u] = (i < items && key < rows)
                   ? *reinterpret_cast<const u32x4*>((const T*)sg.x + (((size_t)b * rows + key) * H + h) * D +
                                                     (i % per_row) * VEC)
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
    __syncthreads();
    uint8_t* dst = sg.codes + (((size_t)b * H + h) * ntiles + kt) * D * 64;
    for (int i = threadIdx.x; i < D * 4; i += kThreads)
      reinterpret_cast<u32x4*>(dst)[i] = reinterpret_cast<const u32x4*>(tile_codes)[i];
    return;
  }

  // row layout: one block per (b, row chunk, head group)
  const int groups = head_groups(H);
  const int chunk = rem / groups;
  const int h0 = (rem % groups) * kHeadGroup, hn = min(kHeadGroup, H - h0);
  const bool store = chunk == 0;
  const bool store_test = store && sg.tensor == 0 && a.train_q_sets_test_slot;
  for (int j = wave; j < hn; j += kThreads / 64) {
    const float s = wave_scale(a, sg.tensor, b, h0 + j, lane);
    const float st = store_test ? wave_scale(a, 3, b, h0 + j, lane) : 0.0f;
    if (lane == 0) {
      sc[j] = s;
      if (store) {
        const size_t bh = (size_t)b * H + h0 + j;
        a.scales[(size_t)sg.tensor * a.B * H + bh] = s;
        if (sg.s_out) sg.s_out[bh] = s;
        if (store_test) {
          a.scales[(size_t)3 * a.B * H + bh] = st;
          if (a.s_q_test_out) a.s_q_test_out[bh] = st;
        }
      }
    }
  }
  __syncthreads();
  const RowMap rm(hn, D, VEC);
  const int t = threadIdx.x;
  const int r0 = chunk * sg.rpc, r1 = min(rows, r0 + sg.rpc);
  if (t >= rm.rows_per_iter * rm.lanes_per_row) return;
  const int rr = t / rm.lanes_per_row;
  for (int p = t % rm.lanes_per_row; p < rm.vpr; p += rm.lanes_per_row) {
    const int hl = p * VEC / D, d0 = (p * VEC) % D;
    const float s = sc[hl];
    const T* src = (const T*)sg.x + ((size_t)b * rows) * H * D + (size_t)h0 * D + (size_t)p * VEC;
    uint8_t* dst = sg.codes + (((size_t)b * H + h0 + hl) * rows) * D + d0;
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

// One block per (b*H + h, 64-key tile): (B,H,N,D) codes transposed through LDS
// into v8t[((b*H + h)*ntiles + tile)*D*64 + d*64 + pos].  Keys >= N get code 0.
__global__ __launch_bounds__(kThreads) void relayout_v_tiles_kernel(int D, int N, const uint8_t* __restrict__ src,
                                                                    uint8_t* __restrict__ v8t) {
  __shared__ uint8_t tile_codes[128 * 64];
  const int bh = blockIdx.y, kt = blockIdx.x;
  const int ntiles = (N + 63) / 64;
  const int per_row = D / 16;   // 16 codes per thread-iteration
  for (int i = threadIdx.x; i < 64 * per_row; i += kThreads) {
    const int kk = i / per_row, c = i % per_row;
    const int key = kt * 64 + kk;
    u32x4 w = {0u, 0u, 0u, 0u};
    if (key < N) w = *reinterpret_cast<const u32x4*>(src + ((size_t)bh * N + key) * D + c * 16);
    const int pos = v_tile_pos(kk);
#pragma unroll
    for (int j = 0; j < 16; ++j) tile_codes[(c * 16 + j) * 64 + pos] = (uint8_t)(w[j / 4] >> (8 * (j % 4)));
  }
  __syncthreads();
  uint8_t* dst = v8t + ((size_t)bh * ntiles + kt) * D * 64;
  for (int i = threadIdx.x; i < D * 4; i += kThreads)
    reinterpret_cast<u32x4*>(dst)[i] = reinterpret_cast<const u32x4*>(tile_codes)[i];
}

// Input bytes per row-layout quantize block: 64 KiB (measured best among 64 KiB .. 512 KiB
// on large inputs), down to 8 KiB for a small launch, so that it still has about four
// blocks per CU and no block's chain of dependent loads sets the launch time.  The
// blocking changes no code.
long long chunk_target_bytes(long long launch_input_bytes) {
  const long long t = launch_input_bytes / (4 * 256);
  return t < 8192 ? 8192 : t > 65536 ? 65536 : t;
}

// Rows per row-layout quantize block at `target` input bytes per block.
int chunk_rows(int rows, int hn, int D, int esize, long long target) {
  long long per_row = (long long)hn * D * esize;
  long long r = (target + per_row - 1) / per_row;
  if (r < 1) r = 1;
  if (r > rows) r = rows > 0 ? rows : 1;
  return (int)r;
}

// Workgroups per table of one quantize segment: 64-key tiles of every head for V in
// the tile layout, else row chunks of every head group.
long long segment_blocks_per_table(int H, int D, int rows, int esize, bool v_tiles, long long target) {
  if (rows <= 0) return 0;
  if (v_tiles) return (long long)H * ((rows + 63) / 64);
  const int hn = H < kHeadGroup ? H : kHeadGroup;
  const int rpc = chunk_rows(rows, hn, D, esize, target);
  return (long long)((rows + rpc - 1) / rpc) * head_groups(H);
}

__global__ void fill_zero_kernel(uint32_t* p, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace

hipError_t launch_fill_zero_u32(uint32_t* p, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_amax(int in_bf16, int first, int last, int B, int H, int D, int N, int M, const void* q_train,
                       const void* k, const void* v, const void* q_test, uint32_t* partial, hipStream_t s) {
  if (last == 3 && M == 0) last = 2;   // no test rows to scan
  if (last < first) return hipSuccess;
  AmaxArgs a;
  a.first_tensor = first;
  a.B = B; a.H = H; a.D = D; a.N = N; a.M = M;
  a.x[0] = q_train; a.x[1] = k; a.x[2] = v; a.x[3] = q_test;
  a.partial = partial;
  int slices = 0;
  for (int t = first; t <= last; ++t) slices = max(slices, amax_slices(t == 3 ? M : N));
  dim3 grid(slices, (last - first + 1) * head_groups(H), B);
  if (in_bf16) hipLaunchKernelGGL(amax_kernel<uint16_t>, grid, dim3(kThreads), 0, s, a);
  else hipLaunchKernelGGL(amax_kernel<float>, grid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_quantize(int in_bf16, int q_scale_mode, int B, int H, int D, int N, int M, const void* q_train,
                           const void* k, const void* v, const void* q_test, uint8_t* q8_train, uint8_t* k8,
                           uint8_t* v8, uint8_t* v8t, uint8_t* q8_test, const uint32_t* partial, float* scales,
                           float* s_q, float* s_k, float* s_v, float* s_q_test, hipStream_t s) {
  QArgs a;
  a.B = B; a.H = H; a.D = D; a.N = N; a.M = M; a.mode = q_scale_mode;
  a.partial = partial; a.scales = scales; a.s_q_test_out = s_q_test;
  const int esize = in_bf16 ? 2 : 4;
  const int groups = head_groups(H);
  const int hn = H < kHeadGroup ? H : kHeadGroup;
  long long total = 0;
  const long long launch_rows = (long long)(v ? N : 0) + (k ? N : 0) + (q_train ? N : 0) + (q_test ? M : 0);
  const long long launch_bytes = (long long)B * H * D * esize * launch_rows;
  const long long target = chunk_target_bytes(launch_bytes);
  a.nseg = 0;
  auto add = [&](const void* x, uint8_t* codes, float* s_out, int tensor, int v_tiles, int rows) {
    if (!x || rows <= 0) return;
    QSeg& g = a.seg[a.nseg++];
    g.x = x; g.codes = codes; g.s_out = s_out; g.tensor = tensor; g.v_tiles = v_tiles; g.rows = rows;
    g.rpc = chunk_rows(rows, hn, D, esize, target);
    const long long per_table = segment_blocks_per_table(H, D, rows, esize, v_tiles, target);
    g.per_table = (int)per_table;   // launched only when the whole grid fits (below)
    g.first = (int)total;
    total += (long long)B * per_table;
  };
  // V, K, then the queries: the reverse of the order the amax pass reads them in, so the
  // second read of the most recently scanned tensors can still hit the memory-side cache
  add(v, v8t ? v8t : v8, s_v, 2, v8t != nullptr, N);
  add(k, k8, s_k, 1, 0, N);
  add(q_train, q8_train, s_q, 0, 0, N);
  add(q_test, q8_test, nullptr, 3, 0, M);
  a.train_q_sets_test_slot = !(q_test && M > 0);
  if (a.nseg > 0 && a.seg[a.nseg - 1].tensor == 3) a.seg[a.nseg - 1].s_out = s_q_test;
  if (total == 0) return hipSuccess;
  if (total > kMaxGridBlocks) return hipErrorInvalidValue;
  if (in_bf16) hipLaunchKernelGGL(quantize_kernel<uint16_t>, dim3((unsigned)total), dim3(kThreads), 0, s, a);
  else hipLaunchKernelGGL(quantize_kernel<float>, dim3((unsigned)total), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

long long quantize_grid_blocks(int esize, int B, int H, int D, int N, int M) {
  // the launch over all four tensors; a launch over fewer has less than 64 MiB of input
  // where its chunks shrink, and then far fewer blocks than the limit
  const long long target = chunk_target_bytes((long long)B * H * D * esize * (3LL * N + M));
  return (long long)B * (segment_blocks_per_table(H, D, N, esize, true, target) +
                         2 * segment_blocks_per_table(H, D, N, esize, false, target) +
                         segment_blocks_per_table(H, D, M, esize, false, target));
}

hipError_t launch_relayout_v_tiles(int B, int H, int D, int N, const uint8_t* v8, uint8_t* v8t, hipStream_t s) {
  dim3 grid((N + 63) / 64, B * H);
  hipLaunchKernelGGL(relayout_v_tiles_kernel, grid, dim3(kThreads), 0, s, D, N, v8, v8t);
  return hipGetLastError();
}

}  // namespace tfm
