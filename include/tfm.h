/*
 * tfm.h -- C ABI of libtfm: FP8 in-context-learning (ICL) attention for
 * tabular foundation models on AMD Instinct MI355X (gfx950).
 *
 * The operation is the one of "Attention Quantization for Tabular Foundation
 * Models" (Sec. 3, Method):
 *   - Eq. (1): Attn(Q,K,V) = P V with P = softmax(alpha Q K^T), row-wise;
 *   - the ICL layer evaluates it twice per head, train-train (N train queries
 *     against the N train keys) and test-train (M test queries against the
 *     same N train keys and values);
 *   - Eq. (2): every tensor is quantized per head to OCP e4m3fn with a
 *     dynamic absmax scale s = max|X| / 448 and X_8 = rn(clamp(X/s, +-448));
 *     by default test queries reuse the scale of the train queries, which
 *     makes each test row's output independent of its batch;
 *   - inside the fused kernel (Fig. 2): the Q and K scales are applied
 *     together with the softmax scale, P is lifted so that its row maximum is
 *     2^8 and rounded to e4m3, and the V scale is applied in the epilogue.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - B tables, H heads, D head_dim (64 or 128), N train rows (>= 1), M test
 *    rows (>= 0), with B*H <= 65535 and N + M < 2^31 - 256.  Every launch
 *    stays below 2^32 work-items per grid dimension, so that counted in
 *    workgroups of 256 threads, at most 2^24 - 1 of them: the attention grid
 *    has B*H*(ceil(N/128) + ceil(M/128)) query tiles of 128 rows (at head
 *    dimension 128, tiles of 256 rows are used only where they fit as well),
 *    and the quantize grid B*H*ceil(N/64) V tiles plus one workgroup per
 *    64 KiB of the other inputs, counted as fp32 whatever their dtype;
 *    TFM_ERR_BAD_SHAPE otherwise.  One GPU's memory does not reach these
 *    bounds.  Activations are row-major (B, rows, H, D), the layout the
 *    paper writes as X in R^{S x H x d}; quantized codes are row-major
 *    (B, H, rows, D) uint8; scales are (B, H) float32 dequantization scales.
 *  - All tensor pointers are device memory owned by the caller and borrowed
 *    for the call; they must be 16-byte aligned and must not alias each
 *    other.  A pointer whose element count is 0 (q_test / o_test / q8_test
 *    when M == 0) may be NULL.  The library never allocates device memory
 *    and keeps no state between calls (a fit leaves its train state in the
 *    caller's workspace), so calls are thread-safe; the one exception is
 *    tfm_icl_attention_fp8_noalloc, whose calls share a fixed per-GPU scratch
 *    (see there).
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *    null stream); no entry point synchronizes.
 *  - Every argument is validated before anything is enqueued; on a
 *    validation error nothing is enqueued and a tfm_status other than TFM_OK
 *    is returned.  TFM_ERR_HIP means the HIP runtime refused a launch; the
 *    launches of the same call before it may already be enqueued, so the
 *    outputs are then unspecified.  No C++ exception crosses this interface.
 *  - Inputs must be finite, and so must the logits they produce in fp32:
 *    alpha * q.k, and for the FP8 path the factor alpha * s_q * s_k * log2(e)
 *    (it overflows only for activations beyond about 1e19 in both Q and K).
 *    Otherwise the results are unspecified.
 */
#ifndef TFM_H_
#define TFM_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TFM_OK = 0,
  TFM_ERR_NULL_PTR = 1,             /* a required pointer is NULL */
  TFM_ERR_BAD_SHAPE = 2,            /* B, H < 1, N < 1, M < 0, or a size or grid overflows */
  TFM_ERR_BAD_DTYPE = 3,            /* dtype code not accepted by this entry point */
  TFM_ERR_UNSUPPORTED_HEAD_DIM = 4, /* D is not 64 or 128 */
  TFM_ERR_MISALIGNED = 5,           /* a pointer is not 16-byte aligned */
  TFM_ERR_WORKSPACE_TOO_SMALL = 6,  /* workspace_bytes below the size query */
  TFM_ERR_HIP = 7,                  /* the HIP runtime reported an error */
  TFM_ERR_BAD_ARG = 8               /* alpha not finite and positive, eps not finite and >= 0, or a bad option */
} tfm_status;

typedef enum { TFM_F32 = 0, TFM_BF16 = 1 } tfm_dtype;

/*
 * Options of the ICL calls (host memory; a NULL pointer means all defaults).
 *
 * q_scale_mode -- which dynamic scale the test queries are quantized with:
 *   TFM_QSCALE_SHARED   (0, default) the per-head scale of the train queries,
 *                       which makes test predictions independent of the test
 *                       batch (Sec. 3, the paragraph after Eq. (2); Table 1,
 *                       last row: the paper's final choice);
 *   TFM_QSCALE_PER_CALL (1) their own per-head absmax scale, computed over the
 *                       test rows of the call (Table 1, "per-call query scale");
 *   TFM_QSCALE_JOINT    (2) one per-head scale over the train and test queries
 *                       together, as for the single ICL call the paper uses for
 *                       TabICLv2 (Appendix, "Experiments on TabICLv2").
 * test_kv_heads -- the K/V heads the test rows attend to.  0 (default) or H:
 *   query head h attends to K/V head h, as the train rows do.  1 <= G < H with
 *   H % G == 0: grouped-query attention of the test rows over the first G K/V
 *   heads (query head h uses K/V head h / (H / G)), the way TabPFN-v3's test
 *   rows attend to the first K/V head (Appendix A).  The test call then reads
 *   exactly the quantized K/V (codes and scales) the train call reads.
 */
typedef enum { TFM_QSCALE_SHARED = 0, TFM_QSCALE_PER_CALL = 1, TFM_QSCALE_JOINT = 2 } tfm_qscale_mode;
typedef struct tfm_icl_options {
  int q_scale_mode;
  int test_kv_heads;
} tfm_icl_options;

/* A hipStream_t, passed as an opaque pointer. */
typedef void* tfm_stream;

/* Human-readable name of a status code (static storage, never NULL). */
const char* tfm_status_string(int status);

/* Library version as major*10000 + minor*100 + patch. */
int tfm_version(void);

/*
 * tfm_quantize_qkv_per_head -- Eq. (2) for the ICL layer (Sec. 3).
 *
 * For every (b, h): s_q = fl32(max|Q_train| / 448), s_k and s_v likewise
 * (fp32 division; a head whose scale would be 0 gets scale 1), and each
 * element becomes the e4m3fn code of clamp(fl32(x / s), -448, 448), rounded
 * to nearest, ties to even.  Q_test is quantized with s_q_test, which is s_q
 * of Q_train unless opts->q_scale_mode says otherwise (see tfm_icl_options).
 *
 *   in_dtype            TFM_F32 or TFM_BF16, the element type of the inputs
 *   opts                NULL or the options (only q_scale_mode is used)
 *   q_train, k, v       (B, N, H, D) inputs
 *   q_test              (B, M, H, D) input, NULL iff M == 0
 *   q8_train, k8, v8    (B, H, N, D) uint8 outputs
 *   q8_test             (B, H, M, D) uint8 output, NULL iff M == 0
 *   s_q, s_k, s_v       (B, H) float32 outputs
 *   s_q_test            (B, H) float32 output: the scale of Q_test (may be NULL)
 *   workspace           >= tfm_quantize_workspace_bytes(B, H) device bytes
 *                       of scratch (contents on entry are ignored)
 */
size_t tfm_quantize_workspace_bytes(int B, int H);
int tfm_quantize_qkv_per_head(int in_dtype, const tfm_icl_options* opts, int B, int H, int D, int N,
                              int M, const void* q_train, const void* k, const void* v,
                              const void* q_test, uint8_t* q8_train, uint8_t* k8,
                              uint8_t* v8, uint8_t* q8_test, float* s_q, float* s_k,
                              float* s_v, float* s_q_test, void* workspace,
                              size_t workspace_bytes, tfm_stream stream);

/*
 * tfm_icl_attention_fp8 -- the full hot path: Eq. (2) quantization of
 * Q_train, K, V and Q_test (test queries on the train-query scale unless
 * opts->q_scale_mode says otherwise), then
 * both ICL attention calls of Sec. 3 in one fused FP8 launch over the N + M
 * query rows, against the same quantized keys and values.
 *
 * Per (b, h) and query row i, over key tiles of tfm_icl_attention_fp8_block_kv(D)
 * keys in order: S = Q_8 K_8^T (FP8 products, fp32 accumulation); running
 * max m; P~ = 2^(c (S - m) + 8) with c = alpha * s_q * s_k * log2(e), so the
 * running row maximum maps to 2^8 (Sec. 3, the P paragraph); P_8 = e4m3(P~)
 * rounded to nearest even; l and O = sum P_8 V_8 are rescaled by
 * 2^(c (m_old - m)) when m grows; the epilogue writes O * s_v / l.  The row
 * sum l accumulates the rounded P_8.
 *
 *   in_dtype            TFM_F32 or TFM_BF16 (inputs)
 *   out_dtype           TFM_F32 or TFM_BF16 (outputs)
 *   opts                NULL (defaults) or the options: query-scale mode and
 *                       grouped test K/V heads (see tfm_icl_options); test rows
 *                       use c = alpha * s_q_test * s_k(h') * log2(e) and s_v(h')
 *                       of their K/V head h'
 *   alpha               softmax scale (finite, > 0), usually 1/sqrt(D)
 *   q_train, k, v       (B, N, H, D);  q_test (B, M, H, D), NULL iff M == 0
 *   o_train             (B, N, H, D) output;  o_test (B, M, H, D), NULL iff M == 0
 *   workspace           >= tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M)
 *                       device bytes of scratch (contents on entry ignored);
 *                       it holds the codes and scales of the call
 */
size_t tfm_icl_attention_fp8_workspace_bytes(int B, int H, int D, int N, int M);
int tfm_icl_attention_fp8(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H,
                          int D, int N, int M, float alpha, const void* q_train, const void* k, const void* v,
                          const void* q_test, void* o_train, void* o_test, void* workspace,
                          size_t workspace_bytes, tfm_stream stream);

/*
 * The two stages of tfm_icl_attention_fp8, which is exactly
 * tfm_icl_attention_fp8_quantize followed by tfm_icl_attention_fp8_attend on
 * the same workspace: for callers that time the stages or run the attention
 * again on codes that are already in the workspace.
 *
 * tfm_icl_attention_fp8_quantize -- Eq. (2) for Q_train, K, V and Q_test
 *   (Q_test on the scale opts->q_scale_mode selects) into `workspace`, in
 *   the private layout the attention stage reads (arguments as for
 *   tfm_icl_attention_fp8; only q_scale_mode of opts is used).
 * tfm_icl_attention_fp8_attend -- both ICL calls from a workspace filled by
 *   tfm_icl_attention_fp8_quantize with the same B, H, D, N, M; the scales
 *   it uses are the ones stored there, so only test_kv_heads of opts is
 *   used; the workspace is only read.  Outputs as for tfm_icl_attention_fp8.
 */
int tfm_icl_attention_fp8_quantize(int in_dtype, const tfm_icl_options* opts, int B, int H, int D,
                                   int N, int M,
                                   const void* q_train, const void* k, const void* v,
                                   const void* q_test, void* workspace, size_t workspace_bytes,
                                   tfm_stream stream);
int tfm_icl_attention_fp8_attend(int out_dtype, const tfm_icl_options* opts, int B, int H, int D,
                                 int N, int M, float alpha, void* o_train, void* o_test,
                                 const void* workspace,
                                 size_t workspace_bytes, tfm_stream stream);

/*
 * tfm_icl_attention_fp8_noalloc -- tfm_icl_attention_fp8 for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same arguments without a workspace,
 * the same kernels and the same results bit for bit.  The workspace is the
 * library's own fixed scratch of TFM_NOALLOC_SCRATCH_BYTES (64 MiB) per GPU,
 * a device array that each GPU the library runs on holds until the process
 * ends.  The scratch of the current device is used, so `stream` must belong
 * to the current device.  Nothing in it needs to start at zero: every call
 * writes what it later reads.
 *
 * Errors: TFM_ERR_WORKSPACE_TOO_SMALL when the call needs more scratch than
 * that (tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M) above
 * TFM_NOALLOC_SCRATCH_BYTES: up to about 64 M codes of Q_train, K, V and
 * Q_test together, e.g. B = 1, H = 8, D = 64, N = 32768, M = 4096); otherwise
 * as tfm_icl_attention_fp8.  The entry point calls no allocating routine; its
 * first call on a device looks up the scratch's device address there.
 * Calls that overlap on one GPU (different streams, or threads) share the
 * scratch and race: order them.
 */
#define TFM_NOALLOC_SCRATCH_BYTES (64u << 20)
int tfm_icl_attention_fp8_noalloc(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H,
                                  int D, int N, int M, float alpha, const void* q_train, const void* k,
                                  const void* v, const void* q_test, void* o_train, void* o_test,
                                  tfm_stream stream);

/*
 * tfm_icl_attention_fp8_fit / tfm_icl_attention_fp8_predict -- the two ICL
 * calls split the way a tabular foundation model is used: fit once on the
 * train rows, then predict any number of test batches against the same
 * quantized keys and values.  With the train-query scale shared by the test
 * queries (Sec. 3, the paragraph after Eq. (2)) a test row's output does not
 * depend on its batch, so the train-side state can be kept.
 *
 * fit: Eq. (2) for Q_train, K and V, then the train-train call into o_train.
 *   The workspace keeps the quantized train state (the per-head absmax
 *   partials, scales, Q_train, K, V codes) for later predict calls; size it with
 *   tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M_max) for the largest
 *   test batch M_max to come (M_max = 0 if none).
 * predict: Q_test (B, M, H, D) quantized with the train-query scale (or, with
 *   TFM_QSCALE_PER_CALL, its own per-head scale), then the test-train call into
 *   o_test (B, M, H, D), against the state of the last fit on this workspace.
 *   workspace_bytes must be >= tfm_icl_attention_fp8_workspace_bytes(B, H, D,
 *   N, M); B, H, D, N must be those of the fit.  M == 0 does nothing.
 *
 * Both produce, bit for bit, the rows tfm_icl_attention_fp8 returns for the
 * same inputs.  TFM_QSCALE_JOINT needs the test rows at fit time and is
 * rejected (TFM_ERR_BAD_ARG); opts->test_kv_heads applies to predict.  Calls
 * on one workspace must be ordered (one stream, or synchronized); a predict
 * overwrites the test part of the workspace only, so predicts on different
 * streams need different workspaces holding the same fit state.
 */
int tfm_icl_attention_fp8_fit(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H,
                              int D, int N, float alpha, const void* q_train, const void* k,
                              const void* v, void* o_train, void* workspace,
                              size_t workspace_bytes, tfm_stream stream);
int tfm_icl_attention_fp8_predict(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B,
                                  int H, int D, int N, int M, float alpha, const void* q_test,
                                  void* o_test, void* workspace, size_t workspace_bytes,
                                  tfm_stream stream);

/*
 * tfm_icl_attention_fp8_prequantized -- the attention part of
 * tfm_icl_attention_fp8 on codes and scales produced by
 * tfm_quantize_qkv_per_head (same layouts), e.g. to reuse K_8 / V_8 for
 * several test batches.  The workspace receives a re-laid-out copy of V_8.
 *
 *   q8_train, k8, v8    (B, H, N, D) uint8;  q8_test (B, H, M, D), NULL iff M == 0
 *   s_q, s_k, s_v       (B, H) float32;  s_q_test (B, H) float32 or NULL (then s_q)
 *   opts                NULL or the options (only test_kv_heads is used)
 *   workspace           >= tfm_icl_attention_fp8_prequantized_workspace_bytes(B, H, D, N)
 */
size_t tfm_icl_attention_fp8_prequantized_workspace_bytes(int B, int H, int D, int N);
int tfm_icl_attention_fp8_prequantized(int out_dtype, const tfm_icl_options* opts, int B, int H,
                                       int D, int N, int M, float alpha,
                                       const uint8_t* q8_train, const uint8_t* k8,
                                       const uint8_t* v8, const uint8_t* q8_test,
                                       const float* s_q, const float* s_k, const float* s_v,
                                       const float* s_q_test, void* o_train, void* o_test,
                                       void* workspace, size_t workspace_bytes,
                                       tfm_stream stream);

/* Number of keys per tile of the FP8 kernel for head_dim D (the granularity
 * of its running maximum); 0 for an unsupported D. */
int tfm_icl_attention_fp8_block_kv(int D);

/*
 * tfm_icl_attention_bf16 -- the 16-bit baseline of the same two ICL calls
 * (Eq. (1), no quantization): bf16 Q/K/V (fp32 inputs are rounded to bf16 on
 * load), fp32 online softmax in one pass, P rounded to bf16 for the PV
 * product and normalised by the sum of the rounded P, fp32 accumulation.
 *
 *   in_dtype            TFM_BF16 or TFM_F32
 *   opts                NULL or the options (only test_kv_heads is used)
 *   q_train, k, v       (B, N, H, D);  q_test (B, M, H, D), NULL iff M == 0
 *   out_dtype           TFM_F32 or TFM_BF16
 *   o_train, o_test     as for tfm_icl_attention_fp8
 */
int tfm_icl_attention_bf16(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H,
                           int D, int N, int M, float alpha, const void* q_train, const void* k, const void* v,
                           const void* q_test, void* o_train, void* o_test, tfm_stream stream);

/*
 * tfm_icl_attention -- the paper's final configuration (Sec. 3, last
 * paragraph; Sec. 4, "final configuration"): the FP8 path
 * (tfm_icl_attention_fp8) when the table has more than `fp8_min_train_rows`
 * train rows, where the quantization overhead is amortized, and the 16-bit
 * path (tfm_icl_attention_bf16) otherwise.  fp8_min_train_rows < 0 selects
 * the paper's gate of 8192 rows.  Arguments as for tfm_icl_attention_fp8;
 * `used_fp8` (host memory, may be NULL) receives 1 if the FP8 path ran.
 * The workspace is used only by the FP8 path.
 */
#define TFM_FP8_MIN_TRAIN_ROWS_DEFAULT 8192
size_t tfm_icl_attention_workspace_bytes(int B, int H, int D, int N, int M, int fp8_min_train_rows);
int tfm_icl_attention(int in_dtype, int out_dtype, const tfm_icl_options* opts, int B, int H, int D,
                      int N, int M, float alpha,
                      const void* q_train, const void* k, const void* v, const void* q_test,
                      void* o_train, void* o_test, int fp8_min_train_rows, int* used_fp8,
                      void* workspace, size_t workspace_bytes, tfm_stream stream);

/*
 * tfm_noise_per_head -- the per-head RMS-scaled Gaussian perturbation of
 * Eq. (3) (appendix, noise experiment), the explicit stand-in for quantization
 * error that the paper uses to study which calls may see perturbed inputs.
 *
 * For every table b and head h:
 *   rho[b,h] = fl32( sqrt( sum over rows i < S, channels j < D of x^2 / (S*D) ) )
 *   out      = fmaf( fl32(eps * rho[b,h]), z, x )         (one rounding in fp32)
 * then converted to the type of x (bf16: round to nearest even).  The sum is
 * taken in fp64 in a fixed order, so results are bitwise reproducible.  The
 * random field z is an input: the caller draws it (standard normal, from its
 * own seeded generator), which keeps a perturbation reproducible from the
 * field alone.  To perturb K and V once for both ICL calls (the paper's
 * "coordinated" setting), perturb them once and pass the results to the
 * attention entry points; the test call then reads the same perturbed K/V.
 *
 *   x_dtype, z_dtype  TFM_F32 or TFM_BF16 (out has the type of x)
 *   x, z              (B, S, H, D) device inputs
 *   eps               the perturbation strength, finite and >= 0
 *   out               (B, S, H, D) device output; may be x itself (in place)
 *                     or z itself, but must not partially overlap either
 *   rho               (B, H) float32 device output, or NULL
 *   workspace         >= tfm_noise_per_head_workspace_bytes(B, H, S, D) bytes
 *
 * D must be a multiple of 8 (TFM_ERR_UNSUPPORTED_HEAD_DIM otherwise);
 * H*D <= 16384, B*H <= 65535 and B*S*H*D below 2^37 (the elementwise pass
 * launches one 256-thread workgroup per 8192 elements, at most 2^24 - 1 of
 * them); TFM_ERR_BAD_SHAPE otherwise.
 * S == 0 is valid: nothing is read or written except rho, which is set to 0;
 * x, z, out and workspace may then be NULL.  Pointers 16-byte aligned.
 */
size_t tfm_noise_per_head_workspace_bytes(int B, int H, int S, int D);
int tfm_noise_per_head(int x_dtype, int z_dtype, int B, int H, int S, int D, const void* x,
                       const void* z, float eps, void* out, float* rho, void* workspace,
                       size_t workspace_bytes, tfm_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* TFM_H_ */
