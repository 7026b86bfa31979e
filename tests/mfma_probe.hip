// Test-only library: the matrix instructions the attention kernels use, one
// instruction per wave on operand tiles the caller chooses, so that their
// arithmetic (how a dot product of e4m3 or bf16 values is summed and rounded,
// and how it is added to the accumulator) can be compared with exact dot
// products on the host.  Not part of libtfm; built next to it.
//
// Tile layouts (row-major, one tile after another; every pointer 16-byte aligned):
//   f8 32x32x64   a (T,32,64) e4m3 bytes of A, bt (T,32,64) e4m3 bytes of B^T,
//                 c, d (T,32,32) float: D = A B + C
//   f8 16x16x128  a (T,16,128), bt (T,16,128), c, d (T,16,16)
//   bf16 32x32x16 a (T,32,16), bt (T,32,16) bf16 bits, c, d (T,32,32)
// Each instruction's k index of a lane's operand bytes is taken as
// k = (lane / rows) * per_lane + byte (rows = 32 or 16); A and B use the same
// mapping, so D is the dot product whatever the hardware's own k order is.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

namespace {

__device__ inline v8i load32(const uint8_t* p) {
  const u32x4 x = *reinterpret_cast<const u32x4*>(p);
  const u32x4 y = *reinterpret_cast<const u32x4*>(p + 16);
  return v8i{(int)x.x, (int)x.y, (int)x.z, (int)x.w, (int)y.x, (int)y.y, (int)y.z, (int)y.w};
}

__global__ __launch_bounds__(64) void f8_32x32x64(const uint8_t* a, const uint8_t* bt, const float* c, float* d,
                                                  int tiles) {
  const int t = blockIdx.x, l = threadIdx.x;
  if (t >= tiles) return;
  const size_t off = (size_t)t * 32 * 64 + (l % 32) * 64 + 32 * (l / 32);
  const v8i av = load32(a + off), bv = load32(bt + off);
  v16f acc;
  for (int r = 0; r < 16; ++r) acc[r] = c[(size_t)t * 1024 + (8 * (r / 4) + 4 * (l / 32) + r % 4) * 32 + l % 32];
  acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, acc, 0, 0, 0, 0, 0, 0);
  for (int r = 0; r < 16; ++r) d[(size_t)t * 1024 + (8 * (r / 4) + 4 * (l / 32) + r % 4) * 32 + l % 32] = acc[r];
}

__global__ __launch_bounds__(64) void f8_16x16x128(const uint8_t* a, const uint8_t* bt, const float* c, float* d,
                                                   int tiles) {
  const int t = blockIdx.x, l = threadIdx.x;
  if (t >= tiles) return;
  const size_t off = (size_t)t * 16 * 128 + (l % 16) * 128 + 32 * (l / 16);
  const v8i av = load32(a + off), bv = load32(bt + off);
  v4f acc;
  for (int r = 0; r < 4; ++r) acc[r] = c[(size_t)t * 256 + (4 * (l / 16) + r) * 16 + l % 16];
  acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, acc, 0, 0, 0, 0, 0, 0);
  for (int r = 0; r < 4; ++r) d[(size_t)t * 256 + (4 * (l / 16) + r) * 16 + l % 16] = acc[r];
}

__global__ __launch_bounds__(64) void bf16_32x32x16(const uint16_t* a, const uint16_t* bt, const float* c, float* d,
                                                    int tiles) {
  const int t = blockIdx.x, l = threadIdx.x;
  if (t >= tiles) return;
  const size_t off = (size_t)t * 32 * 16 + (l % 32) * 16 + 8 * (l / 32);
  const u32x4 x = *reinterpret_cast<const u32x4*>(a + off), y = *reinterpret_cast<const u32x4*>(bt + off);
  const v8bf av = __builtin_bit_cast(v8bf, x), bv = __builtin_bit_cast(v8bf, y);
  v16f acc;
  for (int r = 0; r < 16; ++r) acc[r] = c[(size_t)t * 1024 + (8 * (r / 4) + 4 * (l / 32) + r % 4) * 32 + l % 32];
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
  for (int r = 0; r < 16; ++r) d[(size_t)t * 1024 + (8 * (r / 4) + 4 * (l / 32) + r % 4) * 32 + l % 32] = acc[r];
}

bool bad(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15) != 0; }

}  // namespace

// kind: 0 = f8 32x32x64, 1 = f8 16x16x128, 2 = bf16 32x32x16.  Returns 0 on success,
// 1 for a bad argument (nothing launched), 2 when the launch failed.  Synchronous.
extern "C" int mfma_probe_run(int kind, const void* a, const void* bt, const float* c, float* d, int tiles) {
  if (kind < 0 || kind > 2 || tiles < 1 || tiles > (1 << 20) || bad(a) || bad(bt) || bad(c) || bad(d)) return 1;
  if (kind == 0)
    hipLaunchKernelGGL(f8_32x32x64, dim3(tiles), dim3(64), 0, 0, (const uint8_t*)a, (const uint8_t*)bt, c, d, tiles);
  else if (kind == 1)
    hipLaunchKernelGGL(f8_16x16x128, dim3(tiles), dim3(64), 0, 0, (const uint8_t*)a, (const uint8_t*)bt, c, d, tiles);
  else
    hipLaunchKernelGGL(bf16_32x32x16, dim3(tiles), dim3(64), 0, 0, (const uint16_t*)a, (const uint16_t*)bt, c, d,
                       tiles);
  if (hipGetLastError() != hipSuccess) return 2;
  return hipDeviceSynchronize() == hipSuccess ? 0 : 2;
}
