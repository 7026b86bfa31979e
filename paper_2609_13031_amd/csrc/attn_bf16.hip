// bf16 ICL attention on gfx950: the 16-bit baseline built in the same library.
//
// The same two ICL calls as the FP8 kernel (N train + M test query rows of
// each (b, h) against the same N train keys/values, Eq. (1) of the paper),
// the same tiling (4 wave64s x 32 query rows, 64-key tiles through LDS) and
// the same one-pass fp32 online softmax in the exp2 domain, without any
// quantization: S^T = K Q^T and O^T += V^T P^T with
// v_mfma_f32_32x32x16_bf16, P rounded to bf16 (round to nearest even) for
// the PV product and l summed from the fp32 P.  The bf16 inputs are read in
// their (B, rows, H, D) layout; the V tile is transposed while it is written
// to LDS, with its keys in the row order of the QK^T accumulator.
#include "common.h"

namespace tfm {
namespace {

constexpr int kRowsPerBlock = 128;
constexpr int kPadB = 16;  // bytes

struct Bf16Args {
  int B, H, N, M, tiles;
  float alpha;
  const uint16_t* q_train;
  const uint16_t* q_test;
  const uint16_t* k;
  const uint16_t* v;
  void* o_train;
  void* o_test;
};

typedef uint16_t v8u16 __attribute__((ext_vector_type(8)));
typedef float v8f __attribute__((ext_vector_type(8)));

__device__ inline v8bf as_bf(u32x4 w) {
  v8bf r;
  __builtin_memcpy(&r, &w, 16);
  return r;
}

// Position of key kk (0..63) in a transposed V tile row: the B operand of the
// 32x32x16 PV product over keys [16q, 16q+16) holds, in lane half hf and
// element e, key 16q + (e/4)*8 + hf*4 + e%4.
__device__ inline int vt_pos(int kk) {
  const int q = kk >> 4, kp = kk & 15;
  const int hf = (kp >> 2) & 1, e = (kp >> 3) * 4 + (kp & 3);
  return q * 16 + hf * 8 + e;
}

template <int D, bool OUT_BF16>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(Bf16Args a) {
  constexpr int KS = 2 * D + kPadB;      // K tile row stride (bytes)
  constexpr int VS = 2 * 64 + kPadB;     // V^T tile row stride (bytes)
  __shared__ __attribute__((aligned(16))) uint8_t k_lds[64 * KS];
  __shared__ __attribute__((aligned(16))) uint8_t v_lds[D * VS];

  const int bh = blockIdx.x / a.tiles;
  const int tile = blockIdx.x % a.tiles;
  const int b = bh / a.H, h = bh % a.H, H = a.H;
  const int N = a.N, M = a.M;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int ql = lane % 32, half = lane / 32;
  const int row = tile * kRowsPerBlock + wave * 32 + ql;

  // Q fragment: for head_dim chunk j (16 wide) the lane holds d in [16j + 8*half, +8)
  v8bf qf[D / 16];
  {
    const uint16_t* qrow = nullptr;
    if (row < N) qrow = a.q_train + (((size_t)b * N + row) * H + h) * D;
    else if (row < N + M) qrow = a.q_test + (((size_t)b * M + (row - N)) * H + h) * D;
#pragma unroll
    for (int j = 0; j < D / 16; ++j)
      qf[j] = qrow ? as_bf(*reinterpret_cast<const u32x4*>(qrow + 16 * j + 8 * half)) : as_bf(u32x4{0u, 0u, 0u, 0u});
  }
  const float c = a.alpha * kLog2e;

  v16f acc_o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc_o[i] = v16f{};
  float l_run = 0.0f;
  float m_run = -__builtin_inff();

  const int ntiles = (N + 63) / 64;
  for (int kt = 0; kt < ntiles; ++kt) {
    __syncthreads();
    // K tile: 64 keys x D bf16, row-major
#pragma unroll
    for (int i = threadIdx.x; i < 64 * D / 8; i += 256) {
      const int r = i / (D / 8), cc = i % (D / 8);
      const int key = kt * 64 + r;
      u32x4 w = {0u, 0u, 0u, 0u};
      if (key < N) w = *reinterpret_cast<const u32x4*>(a.k + (((size_t)b * N + key) * H + h) * D + cc * 8);
      *reinterpret_cast<u32x4*>(k_lds + r * KS + cc * 16) = w;
    }
    // V tile transposed: v_lds[d][pos(key)]
#pragma unroll
    for (int i = threadIdx.x; i < 64 * D / 8; i += 256) {
      const int r = i % 64, cc = i / 64;
      const int key = kt * 64 + r;
      u32x4 w = {0u, 0u, 0u, 0u};
      if (key < N) w = *reinterpret_cast<const u32x4*>(a.v + (((size_t)b * N + key) * H + h) * D + cc * 8);
      const int pos = vt_pos(r);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint16_t x = (uint16_t)(w[e / 2] >> (16 * (e % 2)));
        *reinterpret_cast<uint16_t*>(v_lds + (cc * 8 + e) * VS + 2 * pos) = x;
      }
    }
    __syncthreads();

    v16f s0 = v16f{}, s1 = v16f{};
#pragma unroll
    for (int j = 0; j < D / 16; ++j) {
      v8bf k0 = as_bf(*reinterpret_cast<const u32x4*>(k_lds + ql * KS + 32 * j + 16 * half));
      v8bf k1 = as_bf(*reinterpret_cast<const u32x4*>(k_lds + (32 + ql) * KS + 32 * j + 16 * half));
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[j], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[j], s1, 0, 0, 0);
    }
    if (kt * 64 + 64 > N) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kt * 64 + (r / 4) * 8 + half * 4 + (r % 4);
        if (key >= N) s0[r] = -__builtin_inff();
        if (key + 32 >= N) s1[r] = -__builtin_inff();
      }
    }
    float mx = s0[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s0[r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s1[r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float rescale = __builtin_amdgcn_exp2f(c * (m_run - m_new));
    const float bias = -c * m_new;
    m_run = m_new;

    float lsum = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s0[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s0[r], c, bias));
      s1[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s1[r], c, bias));
      lsum += s0[r] + s1[r];
    }
    lsum += __shfl_xor(lsum, 32);
    l_run = l_run * rescale + lsum;
#pragma unroll
    for (int i = 0; i < D / 32; ++i) acc_o[i] *= rescale;

    // P fragments: chunk q covers keys [16q, 16q+16) = accumulator rows 8(q%2).. of s0 (q<2) / s1
    v8bf pfr[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const v16f& src = q < 2 ? s0 : s1;
      v8f pv;
#pragma unroll
      for (int e = 0; e < 8; ++e) pv[e] = src[8 * (q % 2) + e];
      pfr[q] = __builtin_convertvector(pv, v8bf);
    }
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v8bf va = as_bf(*reinterpret_cast<const u32x4*>(v_lds + (32 * i + ql) * VS + 2 * (16 * q + 8 * half)));
        acc_o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pfr[q], acc_o[i], 0, 0, 0);
      }
    }
  }

  if (row >= N + M) return;
  const float inv = 1.0f / l_run;
  const size_t orow = row < N ? (((size_t)b * N + row) * H + h) * D : (((size_t)b * M + (row - N)) * H + h) * D;
#pragma unroll
  for (int i = 0; i < D / 32; ++i) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d = 32 * i + 8 * g + 4 * half;
      const float o0 = acc_o[i][4 * g + 0] * inv, o1 = acc_o[i][4 * g + 1] * inv;
      const float o2 = acc_o[i][4 * g + 2] * inv, o3 = acc_o[i][4 * g + 3] * inv;
      if constexpr (OUT_BF16) {
        __bf16* op = (row < N ? (__bf16*)a.o_train : (__bf16*)a.o_test) + orow + d;
        typedef __bf16 v4bf __attribute__((ext_vector_type(4)));
        *reinterpret_cast<v4bf*>(op) = v4bf{(__bf16)o0, (__bf16)o1, (__bf16)o2, (__bf16)o3};
      } else {
        float* op = (row < N ? (float*)a.o_train : (float*)a.o_test) + orow + d;
        *reinterpret_cast<v4f*>(op) = v4f{o0, o1, o2, o3};
      }
    }
  }
}

}  // namespace

hipError_t launch_attn_bf16(int out_bf16, int B, int H, int D, int N, int M, float alpha, const void* q_train,
                            const void* q_test, const void* k, const void* v, void* o_train, void* o_test,
                            hipStream_t s) {
  Bf16Args a;
  a.B = B; a.H = H; a.N = N; a.M = M;
  a.tiles = (N + M + kRowsPerBlock - 1) / kRowsPerBlock;
  a.alpha = alpha;
  a.q_train = (const uint16_t*)q_train; a.q_test = (const uint16_t*)q_test;
  a.k = (const uint16_t*)k; a.v = (const uint16_t*)v;
  a.o_train = o_train; a.o_test = o_test;
  dim3 grid((unsigned)((long)a.tiles * B * H)), block(256);
  if (D == 64) {
    if (out_bf16) hipLaunchKernelGGL((attn_bf16_kernel<64, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<64, false>), grid, block, 0, s, a);
  } else {
    if (out_bf16) hipLaunchKernelGGL((attn_bf16_kernel<128, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<128, false>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace tfm
