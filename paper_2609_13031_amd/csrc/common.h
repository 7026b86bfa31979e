// Internal declarations shared by the libtfm translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/tfm.h"

namespace tfm {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v8f __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#ifndef TFM_FP8_BLOCK_KV
#define TFM_FP8_BLOCK_KV 128
#endif
constexpr int kBlockKv = TFM_FP8_BLOCK_KV;  // keys per block (running-max granularity) of the FP8 kernel
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kMinNormal = 1.17549435e-38f;   // smallest normal fp32
// Which of the two ICL calls an attention launch runs (a mask).
constexpr int kCallTrain = 1, kCallTest = 2;
// Most workgroups of 256 threads in one grid dimension: a dispatch holds fewer than
// 2^32 work-items per dimension.  The shape checks keep every launch within it.
constexpr long long kMaxGridBlocks = 0xFFFFFFFFLL / 256;

// The amax pass splits the rows of each (tensor, table) into at most kAmaxSlices
// slices of at least kMinSliceRows rows and keeps one maximum per (slice, head).
constexpr int kAmaxSlices = 128;
constexpr int kMinSliceRows = 16;
__host__ __device__ inline int amax_slice_rows(int rows) {
  const int r = (rows + kAmaxSlices - 1) / kAmaxSlices;
  return r < kMinSliceRows ? kMinSliceRows : r;
}
__host__ __device__ inline int amax_slices(int rows) {
  return rows <= 0 ? 0 : (rows + amax_slice_rows(rows) - 1) / amax_slice_rows(rows);
}
// uint32 words of the slice maxima of the four tensors: [4][B][H][kAmaxSlices]
inline size_t amax_partial_words(int B, int H) { return (size_t)4 * B * H * kAmaxSlices; }

// Byte offsets of the pieces of the FP8 workspace (all 256-byte aligned).  Everything
// before q8_test depends on the train rows only (the state a fit call leaves behind).
struct Fp8Workspace {
  size_t partial;   // [4][B][H][kAmaxSlices] uint32: slice maxima of |x| (float bits) of Q_train, K, V, Q_test
  size_t scales;    // 4*B*H float: s_q, s_k, s_v, s_q_test
  size_t q8_train;  // (B,H,N,D) codes
  size_t k8;        // (B,H,N,D) codes
  size_t v8t;       // (B,H,ceil(N/64),D,64) codes, tile-transposed (see attn_fp8.hip)
  size_t q8_test;   // (B,H,M,D) codes
  size_t total;
};
Fp8Workspace fp8_workspace_layout(int B, int H, int D, int N, int M);
size_t v8t_bytes(int B, int H, int D, int N);

// ---- launchers (return hipError_t of the launches) ----
// Zero `n` uint32 words.
hipError_t launch_fill_zero_u32(uint32_t* p, int n, hipStream_t s);
// Slice maxima of |x| per head of tensors first..last of (Q_train, K, V, Q_test) into
// partial[4][B][H][kAmaxSlices]; Q_test has M rows, the others N.
hipError_t launch_amax(int in_bf16, int first, int last, int B, int H, int D, int N, int M,
                       const void* q_train, const void* k, const void* v, const void* q_test,
                       uint32_t* partial, hipStream_t s);
// One launch quantizing every tensor whose input is non-NULL (Q_test only when M > 0)
// with the per-(b,h) scales of the query-scale mode, s = fl32(amax/448) (1 where that is
// 0), reduced from the slice maxima.  V goes to the tile layout v8t when it is non-NULL,
// else to (B,H,N,D) v8.  Stores scales[4][B][H] (s_q, s_k, s_v, s_q_test) for the tensors
// quantized (s_q_test with Q_train when there is no Q_test) and, when the pointers are
// non-NULL, copies of them.
hipError_t launch_quantize(int in_bf16, int q_scale_mode, int B, int H, int D, int N, int M,
                           const void* q_train, const void* k, const void* v, const void* q_test,
                           uint8_t* q8_train, uint8_t* k8, uint8_t* v8, uint8_t* v8t, uint8_t* q8_test,
                           const uint32_t* partial, float* scales, float* s_q, float* s_k, float* s_v,
                           float* s_q_test, hipStream_t s);
// Workgroups of the largest launch_quantize grid for these shapes: all four tensors, V as
// 64-key tiles, elements of esize bytes (fp32 inputs give the most).
long long quantize_grid_blocks(int esize, int B, int H, int D, int N, int M);
// Re-lay (B,H,N,D) V codes into the tile-transposed layout.
hipError_t launch_relayout_v_tiles(int B, int H, int D, int N, const uint8_t* v8,
                                   uint8_t* v8t, hipStream_t s);
// Fused FP8 attention over the N train (calls & kCallTrain) and M test (calls & kCallTest)
// query rows of every (b,h), all against the N train keys.
hipError_t launch_attn_fp8(int out_bf16, int calls, int B, int H, int D, int N, int M, int test_kv_heads,
                           float alpha, const uint8_t* q8_train, const uint8_t* q8_test,
                           const uint8_t* k8, const uint8_t* v8t, const float* s_q,
                           const float* s_k, const float* s_v, const float* s_q_test,
                           void* o_train, void* o_test, hipStream_t s);
// bf16 baseline attention over the N+M query rows of every (b,h); fp32 inputs are rounded to bf16.
hipError_t launch_attn_bf16(int in_f32, int out_bf16, int B, int H, int D, int N, int M, int test_kv_heads,
                            float alpha,
                            const void* q_train, const void* q_test, const void* k,
                            const void* v, void* o_train, void* o_test, hipStream_t s);

// Eq. (3) perturbation: sum of squares per (row chunk, b, h) into partial
// (chunks*B*H doubles), rho (B*H floats, also copied to rho_out when non-NULL),
// then out = x + fl32(eps*rho)*z.  Requires S >= 1, D % 8 == 0, H*D <= 16384.
int noise_rows_per_chunk(int H, int D);
// Workgroups of the largest noise launch (the elementwise pass) for these shapes.
long long noise_grid_blocks(int B, int H, int S, int D);
hipError_t launch_noise(int x_bf16, int z_bf16, int B, int H, int S, int D, const void* x, const void* z, float eps,
                        void* out, double* partial, float* rho, float* rho_out, hipStream_t s);

}  // namespace tfm
