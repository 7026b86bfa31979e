// Fused FP8 ICL attention on gfx950 (train-train and test-train in one launch).
//
// The kernel of Sec. 3 / Fig. 2 of the paper, laid out for CDNA4:
//  * a workgroup of W wave64s owns 32 W consecutive train rows or test rows
//    of one (b, h) (both ICL calls share K_8 and V_8, so they are one
//    launch; the grid lists the train tiles of each (b, h), then its test
//    tiles, and a launch may run only one of the two calls); each wave owns
//    32 rows; test rows may attend to a shared K/V head (grouped-query
//    test-train call).  W = 4 at head dimension 64 (three workgroups per CU,
//    3 waves per SIMD).  At 128, W = 8 (one workgroup per CU, 2 waves per
//    SIMD, each staged key block shared by twice the rows) for long key
//    streams (N >= 65536) when that grid still gives every CU a workgroup,
//    else W = 4 (two per CU, whose waves on a SIMD come from different
//    workgroups and overlap each other's phases).  W changes no output bit:
//    every decision is per wave;
//  * keys are processed in blocks of kBlockKv (128), staged through LDS with
//    double buffering: the global loads of block k+1 are issued before the
//    math of block k and written to the other buffer after it, one barrier
//    per block;
//  * per 32-key tile each wave computes S^T = K_8 Q_8^T with
//    v_mfma_f32_32x32x64_f8f6f4 (fp32 accumulation; two per 64 of head_dim),
//    so every lane holds 32 scores of one query row, and the two lanes of a
//    row exchange their maxima with v_permlane32_swap;
//  * online softmax in the exp2 domain with one running max per block: P~ =
//    2^(c S + 8 - c m) with c = alpha * s_q * s_k * log2(e) (the Q and K
//    scales applied with the softmax scale), so the running row maximum maps
//    to 2^8; P~ is rounded to e4m3 by v_cvt_pk_fp8_f32 (round to nearest
//    even); the state is rescaled only in blocks where some row's max grew,
//    and a block whose lifted weights all round to zero is skipped exactly;
//  * the e4m3 P tile of the QK^T accumulator is directly the B operand of
//    O^T += V_8^T P_8^T (v_mfma_f32_32x32x64_f8f6f4): V is stored
//    tile-transposed with its keys in the accumulator's row order, so no
//    shuffle is needed;
//  * the row sum l = sum P_8 comes from one v_mfma_f32_16x16x128_f8f6f4 of a
//    constant 0/1 operand against the same P_8 operand;
//  * epilogue: O * s_v / l (the V scale applied last), fp32 or bf16 out.
// The VALU work per score (fma, exp, convert, max) bounds the kernel at head
// dimension 64; the MFMAs run beside it.
#include "common.h"

namespace tfm {
namespace {

constexpr int kRowsPerWave = 32;
constexpr int kComputeUnits = 256;   // MI355X; the wave-count choice below only affects speed
// Train rows from which 8-wave workgroups pay at head dimension 128 (measured: the
// 4-wave kernel is 2-11% faster below, level on generic inputs above, and the 8-wave
// one 14% faster on sharp heads whose blocks are mostly skipped at 262144 rows).
constexpr int kWideMinTrainRows = 65536;
constexpr int kPad = 16;  // padded-layout LDS row padding (bytes): conflict-free 16-byte lane reads
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;

struct Fp8Args {
  int B, H, N, M;
  int tiles_train, tiles;  // query tiles per (b, h): train rows first, then test rows
  int test_group;          // test rows of query head h read K/V head h / test_group
  float alpha;
  const uint8_t* q8_train;
  const uint8_t* q8_test;
  const uint8_t* k8;
  const uint8_t* v8t;
  const float* s_q;
  const float* s_k;
  const float* s_v;
  const float* s_q_test;
  void* o_train;
  void* o_test;
};

__device__ inline v8i load32(const uint8_t* p) {
  u32x4 a = *reinterpret_cast<const u32x4*>(p);
  u32x4 b = *reinterpret_cast<const u32x4*>(p + 16);
  return v8i{(int)a.x, (int)a.y, (int)a.z, (int)a.w, (int)b.x, (int)b.y, (int)b.z, (int)b.w};
}

__device__ inline v16f mfma_f8_32x32x64(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}
__device__ inline v4f mfma_f8_16x16x128(v8i a, v8i b, v4f c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// Max of x over the 64 lanes' two halves (lanes l and l+32 hold the same query).
__device__ inline float max_across_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Four P~ values rounded to e4m3 and packed little-endian into one dword.
__device__ inline int pack4_e4m3(float p0, float p1, float p2, float p3) {
  // the first conversion fills the low half; its high half is overwritten by the second
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(p0, p1, __float_as_int(p0), false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(p2, p3, lo, true);
}

// LDS rows of RB bytes hold 16-byte chunks XOR-swizzled instead of padded
// (the DMA below writes 1024 contiguous bytes per wave instruction): chunk c
// of row r sits at chunk position c ^ swz(r), which keeps the 16-byte MFMA
// operand reads free of bank conflicts (measured for both row sizes).
template <int RB>
__device__ inline int swz(int r) {
  static_assert(RB == 64 || RB == 128, "rows of 64 or 128 bytes");
  return RB == 64 ? (r >> 2) & 3 : (r >> 1) & 7;
}
template <int RB>
__device__ inline int lds_off(int r, int c) {
  return r * RB + ((c ^ swz<RB>(r)) << 4);
}
// Copy key block kb straight from global memory into LDS (global_load_lds_dwordx4:
// lane l of a wave instruction writes LDS bytes [base + 16 l, +16)): K as BKV rows
// of D bytes, V^T as BKV/64 stacked tiles of D rows of 64 bytes.  The 1024-byte
// pieces are shared out over the W waves.  Keys >= N read row N-1 and 64-key tiles
// past the end read the last tile: their scores are masked to -inf, so their
// weights are exactly 0.
template <int D, int BKV, int W>
__device__ inline void stage_dma(const uint8_t* kbase, const uint8_t* vbase, int kb, int N, int ntiles64,
                                 uint8_t* k_lds, uint8_t* v_lds, int wave, int lane) {
  constexpr int NP = BKV / 64;
  constexpr int KPIECES = BKV * D / 1024, VPIECES = NP * D * 64 / 1024;
  static_assert(KPIECES % W == 0 && VPIECES % W == 0, "pieces split evenly over the waves");
#pragma unroll
  for (int i = 0; i < KPIECES / W; ++i) {
    const int j = wave + W * i;
    const int at = j * 1024 + lane * 16;
    const int r = at / D, pos = (at % D) >> 4;
    const int key = min(kb * BKV + r, N - 1);
    const uint8_t* g = kbase + (size_t)key * D + ((pos ^ swz<D>(r)) << 4);
    __builtin_amdgcn_global_load_lds((global_void*)g, (lds_void*)(k_lds + j * 1024), 16, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < VPIECES / W; ++i) {
    const int j = wave + W * i;
    const int at = j * 1024 + lane * 16;
    const int r = at / 64, pos = (at % 64) >> 4;           // r = p * D + d
    const int t64 = min(kb * NP + r / D, ntiles64 - 1);
    const uint8_t* g = vbase + (size_t)t64 * D * 64 + (r % D) * 64 + ((pos ^ swz<64>(r)) << 4);
    __builtin_amdgcn_global_load_lds((global_void*)g, (lds_void*)(v_lds + j * 1024), 16, 0, 0);
  }
}

// A key block known to lie wholly below N, copied into LDS by buffer loads from scalar
// resources based at the block (per-block scalar adds): each lane's source offsets
// (voff: the K pieces, then the V pieces, fixed for the launch) and each piece's uniform
// LDS destination need no vector arithmetic per block.  The offsets are those of
// stage_dma without the clamp to the last key, which a full block never needs.
template <int D, int BKV, int W>
__device__ inline void stage_dma_full(const uint8_t* kbase, const uint8_t* vbase, int kb, const int* voff,
                                      uint8_t* k_lds, uint8_t* v_lds, int wave) {
  constexpr int NP = BKV / 64;
  constexpr int KPIECES = BKV * D / 1024, VPIECES = NP * D * 64 / 1024;
  constexpr int KB = BKV * D, VB = NP * D * 64;             // bytes of a K and a V^T block
  constexpr int kRawBufferDword3 = 0x00020000;              // gfx9 untyped buffer: 32-bit data format
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void*)(kbase + (size_t)kb * KB), 0, KB, kRawBufferDword3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void*)(vbase + (size_t)kb * VB), 0, VB, kRawBufferDword3);
#pragma unroll
  for (int i = 0; i < KPIECES / W; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(k_lds + (wave + W * i) * 1024), 16, voff[i], 0, 0, 0);
#pragma unroll
  for (int i = 0; i < VPIECES / W; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(v_lds + (wave + W * i) * 1024), 16,
                                             voff[KPIECES / W + i], 0, 0, 0);
}

// Wait for this wave's outstanding DMA into LDS (vmcnt(0)), before the barrier
// after which other waves read it.
__device__ inline void wait_dma() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// The other staging scheme (used at D = 64, where it measured faster): registers,
// then padded LDS rows (row stride RB + kPad).
// Stage one key block (BKV keys) of K (row-major, rows >= N read as zero) and
// V^T (BKV/64 tiles of D x 64 bytes, tiles past the end read as zero) into
// registers, 16 bytes per thread per piece.  In both tensors piece i of a block
// lies 16 i bytes after the block's start.
template <int D, int BKV>
__device__ inline void stage_load(const uint8_t* kbase, const uint8_t* vbase, int kb, int N, int ntiles64,
                                  u32x4* kr, u32x4* vr) {
  constexpr int PIECES = BKV * D / 16 / 256;
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    const int i = threadIdx.x + 256 * j;
    const int key = kb * BKV + i / (D / 16);
    kr[j] = key < N ? *reinterpret_cast<const u32x4*>(kbase + (size_t)kb * BKV * D + i * 16) : u32x4{0u, 0u, 0u, 0u};
    const int t64 = kb * (BKV / 64) + i / (D * 4);          // 64-key tile of this piece
    vr[j] = t64 < ntiles64 ? *reinterpret_cast<const u32x4*>(vbase + (size_t)kb * (BKV / 64) * D * 64 + i * 16)
                           : u32x4{0u, 0u, 0u, 0u};
  }
}

// A key block known to lie wholly below N: buffer loads through scalar resources
// based at the block (per-block scalar adds), with each lane's pieces at constant
// offsets, so the block costs no vector address arithmetic.  Every offset is
// inside the block, well within the resource's range.
template <int D, int BKV>
__device__ inline void stage_load_full(const uint8_t* kbase, const uint8_t* vbase, int kb, u32x4* kr, u32x4* vr) {
  constexpr int PIECES = BKV * D / 16 / 256;
  constexpr int KB = BKV * D, VB = (BKV / 64) * D * 64;     // bytes of a K and a V^T block
  constexpr int kRawBufferDword3 = 0x00020000;              // gfx9 untyped buffer: 32-bit data format
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void*)(kbase + (size_t)kb * KB), 0, KB, kRawBufferDword3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void*)(vbase + (size_t)kb * VB), 0, VB, kRawBufferDword3);
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    kr[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, threadIdx.x * 16, 4096 * j, 0));
    vr[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, threadIdx.x * 16, 4096 * j, 0));
  }
}

template <int D, int BKV>
__device__ inline void stage_store(uint8_t* k_lds, uint8_t* v_lds, const u32x4* kr, const u32x4* vr) {
  constexpr int KS = D + kPad, VS = 64 + kPad;
  constexpr int PIECES = BKV * D / 16 / 256;
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    const int i = threadIdx.x + 256 * j;
    *reinterpret_cast<u32x4*>(k_lds + (i / (D / 16)) * KS + (i % (D / 16)) * 16) = kr[j];
    // V^T tiles stacked: row (tile*D + d) of 64 bytes
    *reinterpret_cast<u32x4*>(v_lds + (i / 4) * VS + (i % 4) * 16) = vr[j];
  }
}

// Offset of 16-byte chunk c of LDS row r, in the swizzled (SWZ) or the padded layout.
template <int RB, bool SWZ>
__device__ inline int row_chunk(int r, int c) {
  if constexpr (SWZ) return lds_off<RB>(r, c);
  else return r * (RB + kPad) + (c << 4);
}
// 32 bytes of LDS row r starting at (even) chunk c0.
template <int RB, bool SWZ>
__device__ inline v8i load32_lds(const uint8_t* base, int r, int c0) {
  const u32x4 x = *reinterpret_cast<const u32x4*>(base + row_chunk<RB, SWZ>(r, c0));
  const u32x4 y = *reinterpret_cast<const u32x4*>(base + row_chunk<RB, SWZ>(r, c0 + 1));
  return v8i{(int)x.x, (int)x.y, (int)x.z, (int)x.w, (int)y.x, (int)y.y, (int)y.z, (int)y.w};
}

template <int D, int BKV, bool OUT_BF16, int W>
__global__ __launch_bounds__(64 * W, 8 / W) void attn_fp8_kernel(Fp8Args a) {
  constexpr int KD = D / 64;            // 64-wide head_dim chunks (k of one MFMA)
  constexpr int NS = BKV / 32;          // 32-key score tiles per key block
  constexpr int NP = BKV / 64;          // 64-key PV chunks per key block
  // D = 128: K/V copied into LDS by DMA, swizzled rows; D = 64: staged through
  // registers into padded rows (each measured the faster at its head dimension)
  constexpr bool kDma = D == 128;
  static_assert(kDma || W == 4, "register staging spreads a key block over exactly 256 threads");
  constexpr int KBYTES = BKV * (kDma ? D : D + kPad), VBYTES = NP * D * (kDma ? 64 : 64 + kPad);
  constexpr int PIECES = BKV * D / 16 / 256;
  // two K/V stages: the next key block is written while the current one is read
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * (KBYTES + VBYTES)];

  const int bh = blockIdx.x / a.tiles;
  const int tile = blockIdx.x % a.tiles;
  const int b = bh / a.H, h = bh % a.H;
  const int N = a.N, M = a.M;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int ql = lane % 32, half = lane / 32;
  // a workgroup serves either train rows (train-train call) or test rows (test-train call)
  const bool test = tile >= a.tiles_train;
  const int rows = test ? M : N;
  const int row = (test ? tile - a.tiles_train : tile) * (W * kRowsPerWave) + wave * kRowsPerWave + ql;
  const int bhkv = test ? b * a.H + h / a.test_group : bh;   // the (b, K/V head) the rows attend to

  // Q_8 fragment: lane holds head_dim bytes [64s + 32*half, +32) of its row
  v8i qf[KD];
  {
    const uint8_t* qrow = row < rows ? (test ? a.q8_test + ((size_t)bh * M + row) * D
                                             : a.q8_train + ((size_t)bh * N + row) * D)
                                     : nullptr;
#pragma unroll
    for (int s = 0; s < KD; ++s) qf[s] = qrow ? load32(qrow + 64 * s + 32 * half) : v8i{0, 0, 0, 0, 0, 0, 0, 0};
  }
  // A factor below the smallest normal fp32 (alpha s_q s_k underflowing) is taken as that
  // value: every lifted weight still rounds to exactly 2^8 (|c (S - m)| < 2^-100), as at
  // c = 0, while masked keys (S = -inf) and the empty first state keep weight 0 instead of
  // 0 * -inf = NaN.
  const float c = fmaxf(a.alpha * (test ? a.s_q_test[bh] : a.s_q[bh]) * a.s_k[bhkv] * kLog2e, kMinNormal);
  const float sv = a.s_v[bhkv];

  // constant operand of the row-sum MFMA (see the header comment)
  v8i ones;
  {
    const int r16 = lane % 16, g = lane / 16;
    const bool on = ((r16 == 0 || r16 == 8) && (g == 0 || g == 2)) || ((r16 == 4 || r16 == 12) && (g == 1 || g == 3));
    const int w = on ? 0x38383838 : 0;
    ones = v8i{w, w, w, w, w, w, w, w};
  }

  v16f acc_o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc_o[i] = v16f{};
  v4f lacc = v4f{0.f, 0.f, 0.f, 0.f};
  float m_run = -__builtin_inff();

  const int ntiles64 = (N + 63) / 64;
  const int nblocks = (N + BKV - 1) / BKV;
  const uint8_t* kbase = a.k8 + (size_t)bhkv * N * D;
  const uint8_t* vbase = a.v8t + (size_t)bhkv * ntiles64 * D * 64;

  u32x4 kr[kDma ? 1 : PIECES], vr[kDma ? 1 : PIECES];
  // DMA staging: this lane's byte offsets within a full key block for its pieces (K, then V),
  // and the wave index as a scalar so that the LDS destinations are scalar too
  constexpr int KPW = kDma ? BKV * D / 1024 / W : 1, VPW = kDma ? NP * D * 64 / 1024 / W : 1;
  int dma_off[KPW + VPW];
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  if constexpr (kDma) {
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const int at = (wave_s + W * i) * 1024 + lane * 16, r = at / D, pos = (at % D) >> 4;
      dma_off[i] = r * D + ((pos ^ swz<D>(r)) << 4);
    }
#pragma unroll
    for (int i = 0; i < VPW; ++i) {
      const int at = (wave_s + W * i) * 1024 + lane * 16, r = at / 64, pos = (at % 64) >> 4;
      dma_off[KPW + i] = r * 64 + ((pos ^ swz<64>(r)) << 4);
    }
  }
  if constexpr (kDma) {
    stage_dma<D, BKV, W>(kbase, vbase, 0, N, ntiles64, lds, lds + KBYTES, wave, lane);
    wait_dma();
  } else {
    stage_load<D, BKV>(kbase, vbase, 0, N, ntiles64, kr, vr);
    stage_store<D, BKV>(lds, lds + KBYTES, kr, vr);
  }
  __syncthreads();

  for (int kb = 0; kb < nblocks; ++kb) {
    uint8_t* k_lds = lds + (kb & 1) * (KBYTES + VBYTES);
    uint8_t* v_lds = k_lds + KBYTES;
    const bool more = kb + 1 < nblocks;
    if (more) {
      if constexpr (kDma) {
        uint8_t* nk = lds + ((kb + 1) & 1) * (KBYTES + VBYTES);
        if ((kb + 2) * BKV <= N) stage_dma_full<D, BKV, W>(kbase, vbase, kb + 1, dma_off, nk, nk + KBYTES, wave_s);
        else stage_dma<D, BKV, W>(kbase, vbase, kb + 1, N, ntiles64, nk, nk + KBYTES, wave, lane);
      } else if ((kb + 2) * BKV <= N) {
        stage_load_full<D, BKV>(kbase, vbase, kb + 1, kr, vr);
      } else {
        stage_load<D, BKV>(kbase, vbase, kb + 1, N, ntiles64, kr, vr);
      }
    }

    // ---- S^T = K_8 Q_8^T, 32 keys per accumulator tile ----
    v16f st[NS];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      st[t] = v16f{};
#pragma unroll
      for (int s = 0; s < KD; ++s) st[t] = mfma_f8_32x32x64(load32_lds<D, kDma>(k_lds, 32 * t + ql, 4 * s + 2 * half), qf[s], st[t]);
    }
    // keys beyond N (last block only) take no part
    if (kb * BKV + BKV > N) {
#pragma unroll
      for (int t = 0; t < NS; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kb * BKV + 32 * t + (r / 4) * 8 + half * 4 + (r % 4) >= N) st[t][r] = -__builtin_inff();
    }

    // ---- running max over the block; rescale the state by 2^(c (m_old - m_new)) ----
    // The softmax part runs at raised wave priority: where waves of a SIMD compete for
    // issue, the one with VALU work goes first while the others' MFMAs proceed.
    __builtin_amdgcn_s_setprio(1);
    float mx = st[0][0];
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
      for (int r = (t == 0 ? 1 : 0); r < 16; ++r) mx = fmaxf(mx, st[t][r]);
    mx = max_across_halves(mx);
    const float m_old = m_run;
    const float m_new = fmaxf(m_run, mx);
    const float bias = 8.0f - c * m_new;                                   // lifts the running max to 2^8
    m_run = m_new;

    // Exact skip: when every row's largest exponent in this block is <= -11, every
    // lifted weight 2^(c s + bias) < 2^-10 (with v_exp_f32's sub-ulp error) rounds
    // to e4m3 zero, and the running max did not move (the row max alone would
    // give exponent 8), so the block changes neither l nor O.
    if (__builtin_amdgcn_ballot_w64(__builtin_fmaf(mx, c, bias) > -11.0f)) {

      // ---- P~ = 2^(c S + bias) rounded to e4m3, directly the B operand of the PV product ----
      v8i pf[NP];
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          const v16f& src = st[2 * p + w / 4];
          const int r = 4 * (w % 4);
          pf[p][w] = pack4_e4m3(__builtin_amdgcn_exp2f(__builtin_fmaf(src[r + 0], c, bias)),
                                __builtin_amdgcn_exp2f(__builtin_fmaf(src[r + 1], c, bias)),
                                __builtin_amdgcn_exp2f(__builtin_fmaf(src[r + 2], c, bias)),
                                __builtin_amdgcn_exp2f(__builtin_fmaf(src[r + 3], c, bias)));
        }

      // ---- l += sum P_8 (row-sum MFMA) and O^T += V_8^T P_8^T ----
      // Rescale the running state by 2^(c (m_old - m_new)) only when some row's max
      // grew: the factor is exactly 1 in the rows where it did not, and 0 in the first
      // block (m_old = -inf, c > 0).  Written element-wise so the accumulators are
      // scaled in place inside the wave-uniform branch.
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
      for (int p = 0; p < NP; ++p) {
        lacc = mfma_f8_16x16x128(ones, pf[p], lacc);
#pragma unroll
        for (int i = 0; i < D / 32; ++i)
          acc_o[i] = mfma_f8_32x32x64(load32_lds<64, kDma>(v_lds, p * D + 32 * i + ql, 2 * half), pf[p], acc_o[i]);
      }
    }  // not skipped

    __builtin_amdgcn_s_setprio(0);
    if constexpr (kDma) {
      wait_dma();
    } else if (more) {
      uint8_t* nk = lds + ((kb + 1) & 1) * (KBYTES + VBYTES);
      stage_store<D, BKV>(nk, nk + KBYTES, kr, vr);
    }
    __syncthreads();
  }

  // ---- epilogue: O * s_v / l ----
  if (row >= rows) return;
  const float inv = sv / lacc[0];
  const size_t orow = (((size_t)b * rows + row) * a.H + h) * D;
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

hipError_t launch_attn_fp8(int out_bf16, int calls, int B, int H, int D, int N, int M, int test_kv_heads,
                           float alpha, const uint8_t* q8_train, const uint8_t* q8_test, const uint8_t* k8,
                           const uint8_t* v8t, const float* s_q, const float* s_k, const float* s_v,
                           const float* s_q_test, void* o_train, void* o_test, hipStream_t s) {
  Fp8Args a;
  a.B = B; a.H = H; a.N = N; a.M = M;
  auto tiles_of = [&](int rows_per_block) {
    return (long long)((calls & kCallTrain) ? (N + rows_per_block - 1) / rows_per_block : 0) +
           ((calls & kCallTest) ? (M + rows_per_block - 1) / rows_per_block : 0);
  };
  // (the shape check bounds the 4-wave grid; the 8-wave one, of 512-thread blocks, is used only where it fits too)
  const long long wide_blocks = tiles_of(8 * kRowsPerWave) * B * H;
  const bool wide = D == 128 && N >= kWideMinTrainRows && wide_blocks >= kComputeUnits &&
                    wide_blocks <= kMaxGridBlocks / 2;
  const int rpb = (wide ? 8 : 4) * kRowsPerWave;
  a.tiles_train = (calls & kCallTrain) ? (N + rpb - 1) / rpb : 0;
  a.tiles = a.tiles_train + ((calls & kCallTest) ? (M + rpb - 1) / rpb : 0);
  if (a.tiles == 0) return hipSuccess;
  a.test_group = H / test_kv_heads;
  a.alpha = alpha;
  a.q8_train = q8_train; a.q8_test = q8_test; a.k8 = k8; a.v8t = v8t;
  a.s_q = s_q; a.s_k = s_k; a.s_v = s_v; a.s_q_test = s_q_test; a.o_train = o_train; a.o_test = o_test;
  dim3 grid((unsigned)((long)a.tiles * B * H)), block(rpb * 2);   // 64 threads per 32-row wave
  if (D == 64) {
    if (out_bf16) hipLaunchKernelGGL((attn_fp8_kernel<64, kBlockKv, true, 4>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_fp8_kernel<64, kBlockKv, false, 4>), grid, block, 0, s, a);
  } else if (wide) {
    if (out_bf16) hipLaunchKernelGGL((attn_fp8_kernel<128, kBlockKv, true, 8>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_fp8_kernel<128, kBlockKv, false, 8>), grid, block, 0, s, a);
  } else {
    if (out_bf16) hipLaunchKernelGGL((attn_fp8_kernel<128, kBlockKv, true, 4>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_fp8_kernel<128, kBlockKv, false, 4>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace tfm
