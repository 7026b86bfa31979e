// bf16 ICL attention on gfx950: the 16-bit baseline built in the same library.
//
// The same two ICL calls as the FP8 kernel (N train + M test query rows of
// each (b, h) against the same N train keys/values, Eq. (1) of the paper)
// with the same structure, without quantization:
//  * a workgroup of W wave64s owns 32 W train rows or test rows of one
//    (b, h); 32 per wave; test rows may attend to a shared K/V head; W = 4,
//    or 8 at head dimension 128 where that grid still fills the chip (as in
//    the FP8 kernel; the width changes no output bit);
//  * fp32 inputs are rounded to bf16 (nearest even) as they are loaded;
//  * key blocks of kBlockKvBf16 keys; K and V are staged through LDS in their
//    row-major bf16 layout (double-buffered, one barrier per block);
//  * S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so each lane holds the scores
//    of one query row;
//  * one-pass online softmax in fp32 in the exp2 domain; the running state is
//    rescaled only on blocks where some row's max grew;
//  * P is rounded to bf16 (round to nearest even) and is directly the B
//    operand of O^T += V^T P^T (v_mfma_f32_32x32x16_bf16); the V^T operand is
//    read from the row-major V tile with ds_read_b64_tr_b16, the transposing
//    LDS read (in each 16-lane group, output lane i, element r is element i%4
//    of the 4 that input lane 4r + i/4 addressed);
//  * the row sum l = sum bf16(P) comes from v_mfma_f32_16x16x32_bf16 of a
//    constant 0/1 operand against the same P operand, so the weights used in
//    PV are normalised by their own sum.
#include <climits>

#include "common.h"

namespace tfm {
namespace {

constexpr int kRowsPerBlock = 128;      // query rows of a 4-wave workgroup
constexpr int kComputeUnitsBf16 = 256;  // MI355X; the width choice only affects speed
constexpr int kPadB = 16;        // bytes of LDS row padding
constexpr int kBlockKvBf16 = 64;

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

struct Bf16Args {
  int B, H, N, M;
  int tiles_train, tiles;  // query tiles per (b, h): train rows first, then test rows
  int test_group;          // test rows of query head h read K/V head h / test_group
  float alpha;
  const void* q_train;
  const void* q_test;
  const void* k;
  const void* v;
  void* o_train;
  void* o_test;
};

// Eight consecutive inputs as bf16 (fp32 inputs rounded to nearest even).
template <typename T>
__device__ inline u32x4 load8_as_bf16(const T* p) {
  if constexpr (sizeof(T) == 2) {
    return *reinterpret_cast<const u32x4*>(p);
  } else {
    const v4f lo = *reinterpret_cast<const v4f*>(p);
    const v4f hi = *reinterpret_cast<const v4f*>(p + 4);
    v8f x;
#pragma unroll
    for (int e = 0; e < 4; ++e) { x[e] = lo[e]; x[4 + e] = hi[e]; }
    const v8bf y = __builtin_convertvector(x, v8bf);
    u32x4 r;
    __builtin_memcpy(&r, &y, 16);
    return r;
  }
}

__device__ inline v8bf as_bf(u32x4 w) {
  v8bf r;
  __builtin_memcpy(&r, &w, 16);
  return r;
}

__device__ inline v8bf cat_bf(v4s lo, v4s hi) {
  v8bf r;
  __builtin_memcpy(&r, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char*>(&r) + 8, &hi, 8);
  return r;
}

__device__ inline v4s read_tr16(const uint8_t* lds_byte_ptr) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4s*)((__attribute__((address_space(3))) uint8_t*)(lds_byte_ptr)));
}

__device__ inline float max_across_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Stage one block of K and V (BKV keys x D bf16 each, rows >= N as zero) into registers.
template <int D, int BKV, typename T, int NT>
__device__ inline void stage_load(const T* kb_ptr, const T* vb_ptr, int row_stride, int key0, int N,
                                  u32x4* kr, u32x4* vr) {
  constexpr int PIECES = BKV * D / 8 / NT;
  static_assert(PIECES * NT == BKV * D / 8, "a key block splits evenly over the threads");
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    const int i = threadIdx.x + NT * j;
    const int r = i / (D / 8), cc = i % (D / 8);
    const int key = key0 + r;
    const size_t off = (size_t)key * row_stride + cc * 8;
    kr[j] = key < N ? load8_as_bf16(kb_ptr + off) : u32x4{0u, 0u, 0u, 0u};
    vr[j] = key < N ? load8_as_bf16(vb_ptr + off) : u32x4{0u, 0u, 0u, 0u};
  }
}

// A key block known to lie wholly below N: buffer loads from scalar resources based at
// the block's first key row (per-block scalar adds), with each lane's pieces at byte
// offsets `off` fixed for the whole launch, so the block costs no vector address
// arithmetic.  The caller uses it only where the block's BKV rows of row_stride
// elements span at most INT_MAX bytes, so every offset lies inside the resource.
template <int D, int BKV, typename T, int NT>
__device__ inline void stage_load_full(const T* kb_ptr, const T* vb_ptr, int row_stride, int key0, const int* off,
                                       u32x4* kr, u32x4* vr) {
  constexpr int PIECES = BKV * D / 8 / NT;
  constexpr int kRawBufferDword3 = 0x00020000;              // gfx9 untyped buffer: 32-bit data format
  const int bytes = BKV * row_stride * (int)sizeof(T);
  const size_t base = (size_t)key0 * row_stride;
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)(kb_ptr + base), 0, bytes, kRawBufferDword3);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)(vb_ptr + base), 0, bytes, kRawBufferDword3);
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    if constexpr (sizeof(T) == 2) {
      kr[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, off[j], 0, 0));
      vr[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, off[j], 0, 0));
    } else {
      v4f klo = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(rk, off[j], 0, 0));
      v4f khi = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(rk, off[j] + 16, 0, 0));
      v4f vlo = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(rv, off[j], 0, 0));
      v4f vhi = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(rv, off[j] + 16, 0, 0));
      v8f kx, vx;
#pragma unroll
      for (int e = 0; e < 4; ++e) { kx[e] = klo[e]; kx[4 + e] = khi[e]; vx[e] = vlo[e]; vx[4 + e] = vhi[e]; }
      const v8bf ky = __builtin_convertvector(kx, v8bf), vy = __builtin_convertvector(vx, v8bf);
      __builtin_memcpy(&kr[j], &ky, 16);
      __builtin_memcpy(&vr[j], &vy, 16);
    }
  }
}

template <int D, int BKV, int NT>
__device__ inline void stage_store(uint8_t* k_lds, uint8_t* v_lds, const u32x4* kr, const u32x4* vr) {
  constexpr int RS = 2 * D + kPadB;
  constexpr int PIECES = BKV * D / 8 / NT;
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    const int i = threadIdx.x + NT * j;
    const int off = (i / (D / 8)) * RS + (i % (D / 8)) * 16;
    *reinterpret_cast<u32x4*>(k_lds + off) = kr[j];
    *reinterpret_cast<u32x4*>(v_lds + off) = vr[j];
  }
}

template <int D, int BKV, typename T, bool OUT_BF16, int W>
__global__ __launch_bounds__(64 * W, 8 / W) void attn_bf16_kernel(Bf16Args a) {
  constexpr int NT = 64 * W;             // threads of the workgroup (W waves of 32 query rows)
  constexpr int RS = 2 * D + kPadB;      // LDS row stride (bytes) of both tiles
  constexpr int TBYTES = BKV * RS;
  constexpr int NS = BKV / 32;           // 32-key score tiles
  constexpr int NQ = BKV / 16;           // 16-key PV chunks
  constexpr int PIECES = BKV * D / 8 / NT;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * 2 * TBYTES];

  const int bh = blockIdx.x / a.tiles;
  const int tile = blockIdx.x % a.tiles;
  const int b = bh / a.H, h = bh % a.H, H = a.H;
  const int N = a.N, M = a.M;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int ql = lane % 32, half = lane / 32;
  const bool test = tile >= a.tiles_train;
  const int rows = test ? M : N;
  const int row = (test ? tile - a.tiles_train : tile) * (32 * W) + wave * 32 + ql;
  const int hkv = test ? h / a.test_group : h;   // the K/V head the rows attend to

  // Q fragment: for head_dim chunk j (16 wide) the lane holds d in [16j + 8*half, +8)
  v8bf qf[D / 16];
  {
    const T* qrow = row < rows ? (const T*)(test ? a.q_test : a.q_train) + (((size_t)b * rows + row) * H + h) * D
                               : nullptr;
#pragma unroll
    for (int j = 0; j < D / 16; ++j)
      qf[j] = qrow ? as_bf(load8_as_bf16(qrow + 16 * j + 8 * half)) : as_bf(u32x4{0u, 0u, 0u, 0u});
  }
  const float c = fmaxf(a.alpha * kLog2e, kMinNormal);   // as in the FP8 kernel: never 0

  // constant operand of the row-sum MFMA: 1.0 in rows {0,8} for k-groups {0,2}
  // and rows {4,12} for k-groups {1,3} (the lanes of one query in the P operand)
  v8bf ones;
  {
    const int r16 = lane % 16, g = lane / 16;
    const bool on = ((r16 == 0 || r16 == 8) && (g == 0 || g == 2)) || ((r16 == 4 || r16 == 12) && (g == 1 || g == 3));
    const uint32_t w = on ? 0x3f803f80u : 0u;
    ones = as_bf(u32x4{w, w, w, w});
  }

  v16f acc_o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc_o[i] = v16f{};
  v4f lacc = v4f{0.f, 0.f, 0.f, 0.f};
  float m_run = -__builtin_inff();

  const T* kb_ptr = (const T*)a.k + ((size_t)b * N * H + hkv) * D;
  const T* vb_ptr = (const T*)a.v + ((size_t)b * N * H + hkv) * D;
  const int row_stride = H * D;
  const int nblocks = (N + BKV - 1) / BKV;

  // per-lane byte offsets of the transposing V reads (see the header comment):
  // lane = 16g + 4r + j reads 4 consecutive d of key (g/2)*4 + r at d = 16(g%2) + 4j
  const int tg = lane / 16, tr = (lane / 4) % 4, tj = lane % 4;
  const int vtr_off = ((tg / 2) * 4 + tr) * RS + (16 * (tg % 2) + 4 * tj) * 2;

  u32x4 kr[PIECES], vr[PIECES];
  // buffer-load staging of full blocks where a block's byte span fits the 32-bit offsets
  const bool buf_ok = (long long)BKV * row_stride * (long long)sizeof(T) <= INT_MAX;
  int piece_off[PIECES];   // byte offset of each of this thread's pieces within a key block
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    const int i = threadIdx.x + NT * j;
    piece_off[j] = buf_ok ? ((i / (D / 8)) * row_stride + (i % (D / 8)) * 8) * (int)sizeof(T) : 0;
  }
  stage_load<D, BKV, T, NT>(kb_ptr, vb_ptr, row_stride, 0, N, kr, vr);
  stage_store<D, BKV, NT>(lds, lds + TBYTES, kr, vr);
  __syncthreads();

  for (int kb = 0; kb < nblocks; ++kb) {
    const uint8_t* k_lds = lds + (kb & 1) * 2 * TBYTES;
    const uint8_t* v_lds = k_lds + TBYTES;
    const bool more = kb + 1 < nblocks;
    if (more) {
      if (buf_ok && (kb + 2) * BKV <= N) stage_load_full<D, BKV, T, NT>(kb_ptr, vb_ptr, row_stride, (kb + 1) * BKV, piece_off, kr, vr);
      else stage_load<D, BKV, T, NT>(kb_ptr, vb_ptr, row_stride, (kb + 1) * BKV, N, kr, vr);
    }

    v16f st[NS];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      st[t] = v16f{};
#pragma unroll
      for (int j = 0; j < D / 16; ++j) {
        v8bf kf = as_bf(*reinterpret_cast<const u32x4*>(k_lds + (32 * t + ql) * RS + 32 * j + 16 * half));
        st[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[j], st[t], 0, 0, 0);
      }
    }
    if (kb * BKV + BKV > N) {
#pragma unroll
      for (int t = 0; t < NS; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kb * BKV + 32 * t + (r / 4) * 8 + half * 4 + (r % 4) >= N) st[t][r] = -__builtin_inff();
    }

    // softmax part at raised wave priority, as in the FP8 kernel
    __builtin_amdgcn_s_setprio(1);
    float mx = st[0][0];
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
      for (int r = (t == 0 ? 1 : 0); r < 16; ++r) mx = fmaxf(mx, st[t][r]);
    mx = max_across_halves(mx);
    const float m_old = m_run;
    const float m_new = fmaxf(m_run, mx);
    const float bias = -c * m_new;
    m_run = m_new;

    // P in bf16, 16-key chunk q = accumulator rows [8(q%2), +8) of score tile q/2
    v8bf pf[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const v16f& src = st[q / 2];
      v8f pv;
#pragma unroll
      for (int e = 0; e < 8; ++e) pv[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(src[8 * (q % 2) + e], c, bias));
      pf[q] = __builtin_convertvector(pv, v8bf);
    }

    // rescale by 2^(c (m_old - m_new)) only when some row's max grew (exactly 1 in the
    // rows where it did not, 0 in the first block)
    if (__builtin_amdgcn_ballot_w64(m_new != m_old)) {
      const float rescale = __builtin_amdgcn_exp2f(c * (m_old - m_new));
#pragma unroll
      for (int i = 0; i < D / 32; ++i)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc_o[i][j] = acc_o[i][j] * rescale;
#pragma unroll
      for (int j = 0; j < 4; ++j) lacc[j] = lacc[j] * rescale;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[q], lacc, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < D / 32; ++i) {
        const uint8_t* base = v_lds + (16 * q) * RS + 64 * i + vtr_off;
        const v8bf va = cat_bf(read_tr16(base), read_tr16(base + 8 * RS));
        acc_o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pf[q], acc_o[i], 0, 0, 0);
      }
    }

    __builtin_amdgcn_s_setprio(0);
    if (more) {
      uint8_t* nk = lds + ((kb + 1) & 1) * 2 * TBYTES;
      stage_store<D, BKV, NT>(nk, nk + TBYTES, kr, vr);
    }
    __syncthreads();
  }

  if (row >= rows) return;
  const float inv = 1.0f / lacc[0];
  const size_t orow = (((size_t)b * rows + row) * H + h) * D;
#pragma unroll
  for (int i = 0; i < D / 32; ++i) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d = 32 * i + 8 * g + 4 * half;
      const float o0 = acc_o[i][4 * g + 0] * inv, o1 = acc_o[i][4 * g + 1] * inv;
      const float o2 = acc_o[i][4 * g + 2] * inv, o3 = acc_o[i][4 * g + 3] * inv;
      if constexpr (OUT_BF16) {
        __bf16* op = (test ? (__bf16*)a.o_test : (__bf16*)a.o_train) + orow + d;
        typedef __bf16 v4bf __attribute__((ext_vector_type(4)));
        *reinterpret_cast<v4bf*>(op) = v4bf{(__bf16)o0, (__bf16)o1, (__bf16)o2, (__bf16)o3};
      } else {
        float* op = (test ? (float*)a.o_test : (float*)a.o_train) + orow + d;
        *reinterpret_cast<v4f*>(op) = v4f{o0, o1, o2, o3};
      }
    }
  }
}

}  // namespace

template <typename T>
static void launch_bf16_typed(int out_bf16, int D, bool wide, const Bf16Args& a, dim3 grid, hipStream_t s) {
  const dim3 block(wide ? 512 : 256);
  if (D == 64) {
    if (out_bf16) hipLaunchKernelGGL((attn_bf16_kernel<64, kBlockKvBf16, T, true, 4>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<64, kBlockKvBf16, T, false, 4>), grid, block, 0, s, a);
  } else if (wide) {
    if (out_bf16) hipLaunchKernelGGL((attn_bf16_kernel<128, kBlockKvBf16, T, true, 8>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<128, kBlockKvBf16, T, false, 8>), grid, block, 0, s, a);
  } else {
    if (out_bf16) hipLaunchKernelGGL((attn_bf16_kernel<128, kBlockKvBf16, T, true, 4>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<128, kBlockKvBf16, T, false, 4>), grid, block, 0, s, a);
  }
}

hipError_t launch_attn_bf16(int in_f32, int out_bf16, int B, int H, int D, int N, int M, int test_kv_heads,
                            float alpha, const void* q_train, const void* q_test, const void* k, const void* v,
                            void* o_train, void* o_test, hipStream_t s) {
  Bf16Args a;
  a.B = B; a.H = H; a.N = N; a.M = M;
  // At head dimension 128, workgroups of 8 waves (256 rows) share each staged key block when
  // that grid still gives every CU one and fits the launch limit, as in the FP8 kernel; the
  // width changes no output bit.
  const long long wide_blocks = (long long)((N + 255) / 256 + (M + 255) / 256) * B * H;
  const bool wide = D == 128 && wide_blocks >= kComputeUnitsBf16 && wide_blocks <= kMaxGridBlocks / 2;
  const int rpb = wide ? 256 : kRowsPerBlock;
  a.tiles_train = (N + rpb - 1) / rpb;
  a.tiles = a.tiles_train + (M + rpb - 1) / rpb;
  a.test_group = H / test_kv_heads;
  a.alpha = alpha;
  a.q_train = q_train; a.q_test = q_test; a.k = k; a.v = v;
  a.o_train = o_train; a.o_test = o_test;
  dim3 grid((unsigned)((long)a.tiles * B * H));
  if (in_f32) launch_bf16_typed<float>(out_bf16, D, wide, a, grid, s);
  else launch_bf16_typed<uint16_t>(out_bf16, D, wide, a, grid, s);
  return hipGetLastError();
}

}  // namespace tfm
