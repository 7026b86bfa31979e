/* A plain C99 caller of the whole FP8 path on the GPU, with no Python or torch in the
 * process: it reads bf16 inputs from files, copies them to device memory with the HIP
 * runtime, runs tfm_quantize_qkv_per_head and tfm_icl_attention_fp8 on a stream of its
 * own, and writes the codes, scales and fp32 outputs back to files.  Built with the
 * host C compiler and run by tests/test_gpu_c_client.py, which checks the results.
 *
 * usage: c_abi_gpu_client DIR B H D N M ALPHA
 *   DIR/{q_train,k,v,q_test}.bin  bf16 (B, rows, H, D) row-major inputs
 *   writes DIR/{q8_train,k8,v8,q8_test}.bin (B, H, rows, D) codes, DIR/scales.bin
 *   (s_q, s_k, s_v, s_q_test as 4 x B*H float32) and DIR/{o_train,o_test}.bin float32. */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>

#include "tfm.h"

#define HIP_OK(x)                                                            \
  do {                                                                       \
    hipError_t e_ = (x);                                                     \
    if (e_ != hipSuccess) {                                                  \
      fprintf(stderr, "HIP error %d at line %d\n", (int)e_, __LINE__);       \
      exit(3);                                                               \
    }                                                                        \
  } while (0)
#define TFM_OK_(x)                                                           \
  do {                                                                       \
    int st_ = (x);                                                           \
    if (st_ != TFM_OK) {                                                     \
      fprintf(stderr, "tfm error %s at line %d\n", tfm_status_string(st_), __LINE__); \
      exit(4);                                                               \
    }                                                                        \
  } while (0)

static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[4096];
  FILE* f;
  void* p = malloc(bytes ? bytes : 1);
  snprintf(path, sizeof(path), "%s/%s", dir, name);
  f = fopen(path, "rb");
  if (!f || !p || fread(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "cannot read %zu bytes from %s\n", bytes, path);
    exit(2);
  }
  fclose(f);
  return p;
}

static void write_file(const char* dir, const char* name, const void* p, size_t bytes) {
  char path[4096];
  FILE* f;
  snprintf(path, sizeof(path), "%s/%s", dir, name);
  f = fopen(path, "wb");
  if (!f || fwrite(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "cannot write %s\n", path);
    exit(2);
  }
  fclose(f);
}

/* device copy of a host file (NULL when empty) */
static void* to_device(const char* dir, const char* name, size_t bytes) {
  void* h;
  void* d = NULL;
  if (bytes == 0) return NULL;
  h = read_file(dir, name, bytes);
  HIP_OK(hipMalloc(&d, bytes));
  HIP_OK(hipMemcpy(d, h, bytes, hipMemcpyHostToDevice));
  free(h);
  return d;
}

static void* device_buffer(size_t bytes) {
  void* d = NULL;
  if (bytes) HIP_OK(hipMalloc(&d, bytes));
  return d;
}

static void to_file(const char* dir, const char* name, const void* d, size_t bytes) {
  void* h = malloc(bytes ? bytes : 1);
  if (bytes) HIP_OK(hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost));
  write_file(dir, name, h, bytes);
  free(h);
}

int main(int argc, char** argv) {
  const char* dir;
  int B, H, D, N, M;
  float alpha;
  size_t tr, te, bh;
  void *q_train, *k, *v, *q_test, *q8_train, *k8, *v8, *q8_test, *o_train, *o_test, *ws, *qws;
  void* scale[4]; /* s_q, s_k, s_v, s_q_test: separate buffers, every pointer 16-byte aligned */
  int i;
  size_t ws_bytes, qws_bytes;
  hipStream_t s;
  if (argc != 8) {
    fprintf(stderr, "usage: %s DIR B H D N M ALPHA\n", argv[0]);
    return 1;
  }
  dir = argv[1];
  B = atoi(argv[2]);
  H = atoi(argv[3]);
  D = atoi(argv[4]);
  N = atoi(argv[5]);
  M = atoi(argv[6]);
  alpha = (float)atof(argv[7]);
  tr = (size_t)B * N * H * D;
  te = (size_t)B * M * H * D;
  bh = (size_t)B * H;

  q_train = to_device(dir, "q_train.bin", 2 * tr);
  k = to_device(dir, "k.bin", 2 * tr);
  v = to_device(dir, "v.bin", 2 * tr);
  q_test = to_device(dir, "q_test.bin", 2 * te);
  q8_train = device_buffer(tr);
  k8 = device_buffer(tr);
  v8 = device_buffer(tr);
  q8_test = device_buffer(te);
  for (i = 0; i < 4; ++i) scale[i] = device_buffer(bh * sizeof(float));
  o_train = device_buffer(4 * tr);
  o_test = device_buffer(4 * te);
  qws_bytes = tfm_quantize_workspace_bytes(B, H);
  ws_bytes = tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M);
  qws = device_buffer(qws_bytes);
  ws = device_buffer(ws_bytes);
  HIP_OK(hipStreamCreate(&s));

  TFM_OK_(tfm_quantize_qkv_per_head(TFM_BF16, NULL, B, H, D, N, M, q_train, k, v, q_test, (uint8_t*)q8_train,
                                    (uint8_t*)k8, (uint8_t*)v8, (uint8_t*)q8_test, (float*)scale[0],
                                    (float*)scale[1], (float*)scale[2], (float*)scale[3], qws, qws_bytes,
                                    (tfm_stream)s));
  TFM_OK_(tfm_icl_attention_fp8(TFM_BF16, TFM_F32, NULL, B, H, D, N, M, alpha, q_train, k, v, q_test, o_train,
                                o_test, ws, ws_bytes, (tfm_stream)s));
  HIP_OK(hipStreamSynchronize(s));

  to_file(dir, "q8_train.bin", q8_train, tr);
  to_file(dir, "k8.bin", k8, tr);
  to_file(dir, "v8.bin", v8, tr);
  to_file(dir, "q8_test.bin", q8_test, te);
  {
    float* all = (float*)malloc(4 * bh * sizeof(float));
    if (!all) return 2;
    for (i = 0; i < 4; ++i) HIP_OK(hipMemcpy(all + i * bh, scale[i], bh * sizeof(float), hipMemcpyDeviceToHost));
    write_file(dir, "scales.bin", all, 4 * bh * sizeof(float));
    free(all);
  }
  to_file(dir, "o_train.bin", o_train, 4 * tr);
  to_file(dir, "o_test.bin", o_test, 4 * te);

  HIP_OK(hipStreamDestroy(s));
  {
    void* bufs[] = {q_train, k, v, q_test, q8_train, k8, v8, q8_test, o_train, o_test, ws, qws};
    size_t j;
    for (j = 0; j < sizeof(bufs) / sizeof(bufs[0]); ++j)
      if (bufs[j]) HIP_OK(hipFree(bufs[j]));
    for (i = 0; i < 4; ++i) HIP_OK(hipFree(scale[i]));
  }
  printf("c gpu client: done\n");
  return 0;
}
