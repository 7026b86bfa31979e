// libtfm C ABI: argument validation, workspace layout and launch sequences.
// The operations and conventions are documented in include/tfm.h.
#include <atomic>
#include <climits>
#include <cmath>
#include <mutex>

#include "../../include/tfm.h"
#include "common.h"

namespace tfm {

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t v8t_bytes(int B, int H, int D, int N) {
  return (size_t)B * H * (size_t)((N + 63) / 64) * 64 * D;
}

Fp8Workspace fp8_workspace_layout(int B, int H, int D, int N, int M) {
  Fp8Workspace w;
  const size_t bh = (size_t)B * H;
  size_t off = 0;
  w.partial = off;   off += align256(amax_partial_words(B, H) * sizeof(uint32_t));
  w.scales = off;    off += align256(4 * bh * sizeof(float));
  w.q8_train = off;  off += align256(bh * N * D);
  w.k8 = off;        off += align256(bh * N * D);
  w.v8t = off;       off += align256(v8t_bytes(B, H, D, N));
  w.q8_test = off;   off += align256(bh * (size_t)M * D);
  w.total = off;
  return w;
}

}  // namespace tfm

namespace {

using namespace tfm;

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Shapes every entry point accepts.  Limits: B*H <= 65535 (a grid dimension),
// N + M below INT_MAX - 256 (row indices are 32-bit), and every grid within
// kMaxGridBlocks workgroups: the attention grid of at most B*H*(ceil(N/128) +
// ceil(M/128)) query tiles (128 or 256 rows each) and the quantize grid, whose V part alone has
// B*H*ceil(N/64) tiles (so the V relayout grid fits too).  The quantize grid is
// counted for fp32 inputs, its largest, whatever the dtype of the call.
int check_shape(int B, int H, int D, int N, int M) {
  if (B < 1 || H < 1 || N < 1 || M < 0) return TFM_ERR_BAD_SHAPE;
  if ((long long)B * H > 65535) return TFM_ERR_BAD_SHAPE;
  if ((long long)N + M > (long long)INT_MAX - 256) return TFM_ERR_BAD_SHAPE;
  if (D != 64 && D != 128) return TFM_ERR_UNSUPPORTED_HEAD_DIM;
  if ((((long long)N + 127) / 128 + ((long long)M + 127) / 128) * B * H > kMaxGridBlocks)
    return TFM_ERR_BAD_SHAPE;  // attention grid: query tiles of the train rows, then of the test rows
  if (quantize_grid_blocks(4, B, H, D, N, M) > kMaxGridBlocks) return TFM_ERR_BAD_SHAPE;
  return TFM_OK;
}

int check_io(bool need_test, const void* const* req, int nreq, const void* const* test_ptrs, int ntest) {
  for (int i = 0; i < nreq; ++i) if (!req[i]) return TFM_ERR_NULL_PTR;
  if (need_test) for (int i = 0; i < ntest; ++i) if (!test_ptrs[i]) return TFM_ERR_NULL_PTR;
  for (int i = 0; i < nreq; ++i) if (!aligned16(req[i])) return TFM_ERR_MISALIGNED;
  for (int i = 0; i < ntest; ++i) if (test_ptrs[i] && !aligned16(test_ptrs[i])) return TFM_ERR_MISALIGNED;
  return TFM_OK;
}

int check_alpha(float alpha) { return (std::isfinite(alpha) && alpha > 0.0f) ? TFM_OK : TFM_ERR_BAD_ARG; }

// Options with defaults filled in; TFM_ERR_BAD_ARG for an unknown query-scale
// mode or a test K/V head count that is not 0 or a divisor of H.
struct Opts {
  int q_scale_mode = TFM_QSCALE_SHARED;
  int test_kv_heads = 0;
};
int parse_opts(const tfm_icl_options* o, int H, Opts* out) {
  Opts r;
  if (o) {
    r.q_scale_mode = o->q_scale_mode;
    r.test_kv_heads = o->test_kv_heads;
  }
  if (r.q_scale_mode < TFM_QSCALE_SHARED || r.q_scale_mode > TFM_QSCALE_JOINT) return TFM_ERR_BAD_ARG;
  if (r.test_kv_heads == 0) r.test_kv_heads = H;
  if (r.test_kv_heads < 1 || r.test_kv_heads > H || H % r.test_kv_heads != 0) return TFM_ERR_BAD_ARG;
  *out = r;
  return TFM_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? TFM_OK : TFM_ERR_HIP; }

// Scratch of tfm_icl_attention_fp8_noalloc: one copy per GPU, at its own address on
// each.  In host code `scratch` only names the symbol; the device address comes
// from hipGetSymbolAddress, taken once per device (with that device current) and
// kept in scratch_ptr.
static __device__ __align__(256) uint8_t scratch[TFM_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::atomic<void*> scratch_ptr[kMaxDevices];
std::mutex scratch_mu;

// The device address of the current device's scratch (set up on the first call there).
int current_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TFM_ERR_HIP;
  void* p = scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(scratch_mu);
    p = scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TFM_ERR_HIP;
      scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return TFM_OK;
}

#define TFM_TRY(expr) do { int st_ = (expr); if (st_ != TFM_OK) return st_; } while (0)
#define TFM_HIP(expr) do { if ((expr) != hipSuccess) return TFM_ERR_HIP; } while (0)

// Slice maxima, then scales and the four code tensors in one launch.  v8 == nullptr
// writes V to v8t instead.  partial holds amax_partial_words(B, H) words and scales
// 4*B*H floats (s_q, s_k, s_v, s_q_test).
int quantize_all(int in_dtype, int q_scale_mode, int B, int H, int D, int N, int M, const void* q_train,
                 const void* k, const void* v, const void* q_test, uint8_t* q8_train, uint8_t* k8, uint8_t* v8,
                 uint8_t* v8t, uint8_t* q8_test, uint32_t* partial, float* scales, float* s_q, float* s_k,
                 float* s_v, float* s_q_test, hipStream_t s) {
  const int bf = in_dtype == TFM_BF16;
  const bool test_amax = q_scale_mode != TFM_QSCALE_SHARED && M > 0;
  TFM_HIP(launch_amax(bf, 0, test_amax ? 3 : 2, B, H, D, N, M, q_train, k, v, q_test, partial, s));
  TFM_HIP(launch_quantize(bf, q_scale_mode, B, H, D, N, M, q_train, k, v, M > 0 ? q_test : nullptr, q8_train, k8,
                          v8, v8 ? nullptr : v8t, q8_test, partial, scales, s_q, s_k, s_v, s_q_test, s));
  return TFM_OK;
}

}  // namespace

extern "C" {

const char* tfm_status_string(int status) {
  switch (status) {
    case TFM_OK: return "TFM_OK";
    case TFM_ERR_NULL_PTR: return "TFM_ERR_NULL_PTR: a required pointer is NULL";
    case TFM_ERR_BAD_SHAPE: return "TFM_ERR_BAD_SHAPE: B, H >= 1, N >= 1, M >= 0 (S >= 0) and sizes within limits required";
    case TFM_ERR_BAD_DTYPE: return "TFM_ERR_BAD_DTYPE: unsupported dtype code";
    case TFM_ERR_UNSUPPORTED_HEAD_DIM:
      return "TFM_ERR_UNSUPPORTED_HEAD_DIM: D must be 64 or 128 (a multiple of 8 for the noise operator)";
    case TFM_ERR_MISALIGNED: return "TFM_ERR_MISALIGNED: pointers must be 16-byte aligned";
    case TFM_ERR_WORKSPACE_TOO_SMALL: return "TFM_ERR_WORKSPACE_TOO_SMALL: workspace below the size query";
    case TFM_ERR_HIP: return "TFM_ERR_HIP: the HIP runtime reported an error";
    case TFM_ERR_BAD_ARG:
      return "TFM_ERR_BAD_ARG: alpha must be finite and positive, eps finite and >= 0, q_scale_mode one of "
             "TFM_QSCALE_*, test_kv_heads 0 or a divisor of H";
    default: return "TFM_ERR_UNKNOWN";
  }
}

int tfm_version(void) { return 200; }

size_t tfm_quantize_workspace_bytes(int B, int H) {
  if (B < 1 || H < 1 || (long long)B * H > 65535) return 0;
  return align256(amax_partial_words(B, H) * sizeof(uint32_t)) + align256(4 * (size_t)B * H * sizeof(float));
}

int tfm_quantize_qkv_per_head(int in_dtype, const tfm_icl_options* opts, int B, int H, int D, int N, int M,
                              const void* q_train, const void* k, const void* v, const void* q_test,
                              uint8_t* q8_train, uint8_t* k8, uint8_t* v8, uint8_t* q8_test, float* s_q, float* s_k,
                              float* s_v, float* s_q_test, void* workspace, size_t workspace_bytes,
                              tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (in_dtype != TFM_F32 && in_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  const void* req[] = {q_train, k, v, q8_train, k8, v8, s_q, s_k, s_v, workspace};
  const void* tst[] = {q_test, q8_test};
  TFM_TRY(check_io(M > 0, req, 10, tst, 2));
  if (s_q_test && !aligned16(s_q_test)) return TFM_ERR_MISALIGNED;
  if (workspace_bytes < tfm_quantize_workspace_bytes(B, H)) return TFM_ERR_WORKSPACE_TOO_SMALL;
  uint8_t* ws = (uint8_t*)workspace;
  uint32_t* partial = (uint32_t*)ws;
  float* scales = (float*)(ws + align256(amax_partial_words(B, H) * sizeof(uint32_t)));
  return quantize_all(in_dtype, o.q_scale_mode, B, H, D, N, M, q_train, k, v, q_test, q8_train, k8, v8, nullptr,
                      q8_test, partial, scales, s_q, s_k, s_v, s_q_test, (hipStream_t)stream);
}

size_t tfm_icl_attention_fp8_workspace_bytes(int B, int H, int D, int N, int M) {
  if (check_shape(B, H, D, N, M) != TFM_OK) return 0;
  return fp8_workspace_layout(B, H, D, N, M).total;
}

int tfm_icl_attention_fp8_quantize(int in_dtype, const tfm_icl_options* opts, int B, int H, int D, int N, int M,
                                   const void* q_train, const void* k, const void* v, const void* q_test,
                                   void* workspace, size_t workspace_bytes, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (in_dtype != TFM_F32 && in_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  const void* req[] = {q_train, k, v, workspace};
  const void* tst[] = {q_test};
  TFM_TRY(check_io(M > 0, req, 4, tst, 1));
  const Fp8Workspace L = fp8_workspace_layout(B, H, D, N, M);
  if (workspace_bytes < L.total) return TFM_ERR_WORKSPACE_TOO_SMALL;
  uint8_t* ws = (uint8_t*)workspace;
  return quantize_all(in_dtype, o.q_scale_mode, B, H, D, N, M, q_train, k, v, q_test, ws + L.q8_train, ws + L.k8,
                      nullptr, ws + L.v8t, ws + L.q8_test, (uint32_t*)(ws + L.partial), (float*)(ws + L.scales),
                      nullptr, nullptr, nullptr, nullptr, (hipStream_t)stream);
}

int tfm_icl_attention_fp8_attend(int out_dtype, const tfm_icl_options* opts, int B, int H, int D, int N, int M,
                                 float alpha, void* o_train, void* o_test, const void* workspace,
                                 size_t workspace_bytes, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (out_dtype != TFM_F32 && out_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  TFM_TRY(check_alpha(alpha));
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  const void* req[] = {o_train, workspace};
  const void* tst[] = {o_test};
  TFM_TRY(check_io(M > 0, req, 2, tst, 1));
  const Fp8Workspace L = fp8_workspace_layout(B, H, D, N, M);
  if (workspace_bytes < L.total) return TFM_ERR_WORKSPACE_TOO_SMALL;
  const uint8_t* ws = (const uint8_t*)workspace;
  const float* scales = (const float*)(ws + L.scales);
  const int BH = B * H;
  return hip_status(launch_attn_fp8(out_dtype == TFM_BF16, kCallTrain | kCallTest, B, H, D, N, M, o.test_kv_heads,
                                    alpha, ws + L.q8_train,
                                    ws + L.q8_test, ws + L.k8, ws + L.v8t, scales, scales + BH, scales + 2 * BH,
                                    scales + 3 * BH, o_train, o_test, (hipStream_t)stream));
}

int tfm_icl_attention_fp8(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H, int D, int N,
                          int M, float alpha, const void* q_train, const void* k, const void* v, const void* q_test,
                          void* o_train, void* o_test, void* workspace, size_t workspace_bytes, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (in_dtype != TFM_F32 && in_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  if (out_dtype != TFM_F32 && out_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  TFM_TRY(check_alpha(alpha));
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  const void* req[] = {q_train, k, v, o_train, workspace};
  const void* tst[] = {q_test, o_test};
  TFM_TRY(check_io(M > 0, req, 5, tst, 2));
  if (workspace_bytes < fp8_workspace_layout(B, H, D, N, M).total) return TFM_ERR_WORKSPACE_TOO_SMALL;
  TFM_TRY(tfm_icl_attention_fp8_quantize(in_dtype, opts, B, H, D, N, M, q_train, k, v, q_test, workspace,
                                         workspace_bytes, stream));
  return tfm_icl_attention_fp8_attend(out_dtype, opts, B, H, D, N, M, alpha, o_train, o_test, workspace,
                                      workspace_bytes, stream);
}

int tfm_icl_attention_fp8_noalloc(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H, int D,
                                  int N, int M, float alpha, const void* q_train, const void* k, const void* v,
                                  const void* q_test, void* o_train, void* o_test, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (fp8_workspace_layout(B, H, D, N, M).total > TFM_NOALLOC_SCRATCH_BYTES) return TFM_ERR_WORKSPACE_TOO_SMALL;
  if (in_dtype != TFM_F32 && in_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  if (out_dtype != TFM_F32 && out_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  TFM_TRY(check_alpha(alpha));
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  const void* req[] = {q_train, k, v, o_train};
  const void* tst[] = {q_test, o_test};
  TFM_TRY(check_io(M > 0, req, 4, tst, 2));
  void* ws = nullptr;
  TFM_TRY(current_scratch(&ws));
  return tfm_icl_attention_fp8(in_dtype, out_dtype, opts, B, H, D, N, M, alpha, q_train, k, v, q_test, o_train,
                               o_test, ws, TFM_NOALLOC_SCRATCH_BYTES, stream);
}

int tfm_icl_attention_fp8_fit(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H, int D, int N,
                              float alpha, const void* q_train, const void* k, const void* v, void* o_train,
                              void* workspace, size_t workspace_bytes, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, 0));
  if (in_dtype != TFM_F32 && in_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  if (out_dtype != TFM_F32 && out_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  TFM_TRY(check_alpha(alpha));
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  if (o.q_scale_mode == TFM_QSCALE_JOINT) return TFM_ERR_BAD_ARG;   // needs the test rows at fit time
  const void* req[] = {q_train, k, v, o_train, workspace};
  TFM_TRY(check_io(false, req, 5, nullptr, 0));
  const Fp8Workspace L = fp8_workspace_layout(B, H, D, N, 0);
  if (workspace_bytes < L.total) return TFM_ERR_WORKSPACE_TOO_SMALL;
  uint8_t* ws = (uint8_t*)workspace;
  hipStream_t s = (hipStream_t)stream;
  float* scales = (float*)(ws + L.scales);
  const int BH = B * H;
  TFM_TRY(quantize_all(in_dtype, TFM_QSCALE_SHARED, B, H, D, N, 0, q_train, k, v, nullptr, ws + L.q8_train,
                       ws + L.k8, nullptr, ws + L.v8t, nullptr, (uint32_t*)(ws + L.partial), scales, nullptr, nullptr,
                       nullptr, nullptr, s));
  return hip_status(launch_attn_fp8(out_dtype == TFM_BF16, kCallTrain, B, H, D, N, 0, o.test_kv_heads, alpha,
                                    ws + L.q8_train, nullptr, ws + L.k8, ws + L.v8t, scales, scales + BH,
                                    scales + 2 * BH, scales + 3 * BH, o_train, nullptr, s));
}

int tfm_icl_attention_fp8_predict(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H, int D,
                                  int N, int M, float alpha, const void* q_test, void* o_test, void* workspace,
                                  size_t workspace_bytes, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (in_dtype != TFM_F32 && in_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  if (out_dtype != TFM_F32 && out_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  TFM_TRY(check_alpha(alpha));
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  if (o.q_scale_mode == TFM_QSCALE_JOINT) return TFM_ERR_BAD_ARG;
  const void* req[] = {workspace};
  const void* tst[] = {q_test, o_test};
  TFM_TRY(check_io(M > 0, req, 1, tst, 2));
  const Fp8Workspace L = fp8_workspace_layout(B, H, D, N, M);
  if (workspace_bytes < L.total) return TFM_ERR_WORKSPACE_TOO_SMALL;
  if (M == 0) return TFM_OK;
  uint8_t* ws = (uint8_t*)workspace;
  hipStream_t s = (hipStream_t)stream;
  uint32_t* partial = (uint32_t*)(ws + L.partial);
  float* scales = (float*)(ws + L.scales);
  const int bf = in_dtype == TFM_BF16;
  const int BH = B * H;
  if (o.q_scale_mode == TFM_QSCALE_PER_CALL)
    TFM_HIP(launch_amax(bf, 3, 3, B, H, D, N, M, nullptr, nullptr, nullptr, q_test, partial, s));
  // Under the shared scale s_q_test comes from the fit's Q_train slice maxima, which the
  // workspace still holds; s_q, s_k and s_v stay as the fit stored them.
  TFM_HIP(launch_quantize(bf, o.q_scale_mode, B, H, D, N, M, nullptr, nullptr, nullptr, q_test, nullptr, nullptr,
                          nullptr, nullptr, ws + L.q8_test, partial, scales, nullptr, nullptr, nullptr, nullptr, s));
  return hip_status(launch_attn_fp8(out_dtype == TFM_BF16, kCallTest, B, H, D, N, M, o.test_kv_heads, alpha,
                                    ws + L.q8_train, ws + L.q8_test, ws + L.k8, ws + L.v8t, scales, scales + BH,
                                    scales + 2 * BH, scales + 3 * BH, nullptr, o_test, s));
}

size_t tfm_icl_attention_fp8_prequantized_workspace_bytes(int B, int H, int D, int N) {
  if (check_shape(B, H, D, N, 0) != TFM_OK) return 0;
  return align256(v8t_bytes(B, H, D, N));
}

int tfm_icl_attention_fp8_prequantized(int out_dtype, const tfm_icl_options* opts, int B, int H, int D, int N, int M,
                                       float alpha, const uint8_t* q8_train, const uint8_t* k8, const uint8_t* v8,
                                       const uint8_t* q8_test, const float* s_q, const float* s_k, const float* s_v,
                                       const float* s_q_test, void* o_train, void* o_test, void* workspace,
                                       size_t workspace_bytes, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (out_dtype != TFM_F32 && out_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  TFM_TRY(check_alpha(alpha));
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  const void* req[] = {q8_train, k8, v8, s_q, s_k, s_v, o_train, workspace};
  const void* tst[] = {q8_test, o_test};
  TFM_TRY(check_io(M > 0, req, 8, tst, 2));
  if (s_q_test && !aligned16(s_q_test)) return TFM_ERR_MISALIGNED;
  if (workspace_bytes < tfm_icl_attention_fp8_prequantized_workspace_bytes(B, H, D, N))
    return TFM_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* v8t = (uint8_t*)workspace;
  TFM_HIP(launch_relayout_v_tiles(B, H, D, N, v8, v8t, s));
  return hip_status(launch_attn_fp8(out_dtype == TFM_BF16, kCallTrain | kCallTest, B, H, D, N, M, o.test_kv_heads,
                                    alpha, q8_train, q8_test,
                                    k8, v8t, s_q, s_k, s_v, s_q_test ? s_q_test : s_q, o_train, o_test, s));
}

int tfm_icl_attention_fp8_block_kv(int D) { return (D == 64 || D == 128) ? kBlockKv : 0; }

int tfm_icl_attention_bf16(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H, int D, int N,
                           int M, float alpha, const void* q_train, const void* k, const void* v, const void* q_test,
                           void* o_train, void* o_test, tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  if (in_dtype != TFM_F32 && in_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  if (out_dtype != TFM_F32 && out_dtype != TFM_BF16) return TFM_ERR_BAD_DTYPE;
  TFM_TRY(check_alpha(alpha));
  Opts o;
  TFM_TRY(parse_opts(opts, H, &o));
  const void* req[] = {q_train, k, v, o_train};
  const void* tst[] = {q_test, o_test};
  TFM_TRY(check_io(M > 0, req, 4, tst, 2));
  return hip_status(launch_attn_bf16(in_dtype == TFM_F32, out_dtype == TFM_BF16, B, H, D, N, M, o.test_kv_heads, alpha,
                                     q_train, q_test, k, v, o_train, o_test, (hipStream_t)stream));
}

static int gate_rows(int fp8_min_train_rows) {
  return fp8_min_train_rows < 0 ? TFM_FP8_MIN_TRAIN_ROWS_DEFAULT : fp8_min_train_rows;
}

size_t tfm_icl_attention_workspace_bytes(int B, int H, int D, int N, int M, int fp8_min_train_rows) {
  if (check_shape(B, H, D, N, M) != TFM_OK) return 0;
  return N > gate_rows(fp8_min_train_rows) ? fp8_workspace_layout(B, H, D, N, M).total : 0;
}

int tfm_icl_attention(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H, int D, int N, int M,
                      float alpha, const void* q_train, const void* k, const void* v, const void* q_test, void* o_train,
                      void* o_test, int fp8_min_train_rows, int* used_fp8, void* workspace, size_t workspace_bytes,
                      tfm_stream stream) {
  TFM_TRY(check_shape(B, H, D, N, M));
  const bool fp8 = N > gate_rows(fp8_min_train_rows);
  int st;
  if (fp8)
    st = tfm_icl_attention_fp8(in_dtype, out_dtype, opts, B, H, D, N, M, alpha, q_train, k, v, q_test, o_train,
                               o_test, workspace, workspace_bytes, stream);
  else
    st = tfm_icl_attention_bf16(in_dtype, out_dtype, opts, B, H, D, N, M, alpha, q_train, k, v, q_test, o_train,
                                o_test, stream);
  if (st == TFM_OK && used_fp8) *used_fp8 = fp8 ? 1 : 0;
  return st;
}

// ---- Eq. (3) noise operator ----

static int check_noise_shape(int B, int H, int S, int D) {
  if (B < 1 || H < 1 || S < 0) return TFM_ERR_BAD_SHAPE;
  if (D < 8 || D % 8 != 0) return TFM_ERR_UNSUPPORTED_HEAD_DIM;
  if ((long long)B * H > 65535 || (long long)H * D > 16384) return TFM_ERR_BAD_SHAPE;
  if ((long double)B * S * H * D > 1099511627776.0L) return TFM_ERR_BAD_SHAPE;  // 2^40 elements
  if (noise_grid_blocks(B, H, S, D) > kMaxGridBlocks) return TFM_ERR_BAD_SHAPE;
  return TFM_OK;
}

static size_t noise_partial_bytes(int B, int H, int S, int D) {
  const int rpc = noise_rows_per_chunk(H, D);
  const size_t chunks = ((size_t)S + rpc - 1) / rpc;
  return align256(chunks * B * H * sizeof(double));
}

size_t tfm_noise_per_head_workspace_bytes(int B, int H, int S, int D) {
  if (check_noise_shape(B, H, S, D) != TFM_OK) return 0;
  return noise_partial_bytes(B, H, S, D) + align256((size_t)B * H * sizeof(float));
}

int tfm_noise_per_head(int x_dtype, int z_dtype, int B, int H, int S, int D, const void* x, const void* z, float eps,
                       void* out, float* rho, void* workspace, size_t workspace_bytes, tfm_stream stream) {
  TFM_TRY(check_noise_shape(B, H, S, D));
  if ((x_dtype != TFM_F32 && x_dtype != TFM_BF16) || (z_dtype != TFM_F32 && z_dtype != TFM_BF16))
    return TFM_ERR_BAD_DTYPE;
  if (!std::isfinite(eps) || eps < 0.0f) return TFM_ERR_BAD_ARG;
  if (rho && !aligned16(rho)) return TFM_ERR_MISALIGNED;
  hipStream_t s = (hipStream_t)stream;
  if (S == 0) {  // nothing to perturb; rho of an empty head is 0
    if (rho) TFM_HIP(launch_fill_zero_u32((uint32_t*)rho, B * H, s));
    return TFM_OK;
  }
  const void* req[] = {x, z, out, workspace};
  TFM_TRY(check_io(false, req, 4, nullptr, 0));
  if (workspace_bytes < tfm_noise_per_head_workspace_bytes(B, H, S, D)) return TFM_ERR_WORKSPACE_TOO_SMALL;
  uint8_t* ws = (uint8_t*)workspace;
  return hip_status(launch_noise(x_dtype == TFM_BF16, z_dtype == TFM_BF16, B, H, S, D, x, z, eps, out,
                                 (double*)ws, (float*)(ws + noise_partial_bytes(B, H, S, D)), rho, s));
}

}  // extern "C"
