/* A plain-C consumer of the SelKV C ABI (include/selkv.h): device buffers
 * come from hipMalloc, and the five hot-path calls run in the paper's order
 * (Algorithm 1: score, select, merge, bias, then one biased decode step),
 * with the default parameters of selkv_params_init and fp32 storage.
 * It also checks, in C, that the fused selkv_merge_bias equals selkv_merge
 * + selkv_bias and that selkv_decode_attn_noalloc equals selkv_decode_attn,
 * bit for bit.
 *
 * Usage: selkv_c_demo IN OUT
 *   IN:  int32 B, H, G, d, n, W; then float32 K [B,H,n,d], V [B,H,n,d],
 *        Qwin [B,H*G,W,d], q [B,H*G,d]
 *   OUT: int32 m, m_r'; int32 kept [B,H,m], evicted [B,H,n-m],
 *        target [B,H,n-m]; float32 gate [B,H,n-m], K_out [B,H,m,d],
 *        V_out [B,H,m,d], bias [B,H,m], out [B,H*G,d], attn [B,H,n],
 *        score [B,H,n-m_r']
 * It then runs the fused selkv_merge_bias into fresh buffers and checks that
 * it reproduces the separate merge and bias bit for bit.
 * Exits 0 on success; on failure prints the failing call and its status. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "selkv.h"

#define HIP_OK(x)                                                              \
  do {                                                                         \
    hipError_t e_ = (x);                                                       \
    if (e_ != hipSuccess) {                                                    \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));          \
      exit(2);                                                                 \
    }                                                                          \
  } while (0)

#define SELKV_OK_(x)                                                           \
  do {                                                                         \
    selkv_status s_ = (x);                                                     \
    if (s_ != SELKV_OK) {                                                      \
      fprintf(stderr, "%s failed: %s\n", #x, selkv_status_string(s_));        \
      exit(3);                                                                 \
    }                                                                          \
  } while (0)

static void* dev_alloc(size_t bytes) {
  void* p = NULL;
  HIP_OK(hipMalloc(&p, bytes > 0 ? bytes : 1));
  return p;
}

static void* host_read(FILE* f, size_t bytes) {
  void* p = malloc(bytes > 0 ? bytes : 1);
  if (!p || fread(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "short input\n");
    exit(4);
  }
  return p;
}

static void to_file(FILE* f, const void* dev, size_t bytes) {
  void* h = malloc(bytes > 0 ? bytes : 1);
  if (!h) exit(5);
  HIP_OK(hipMemcpy(h, dev, bytes, hipMemcpyDeviceToHost));
  fwrite(h, 1, bytes, f);
  free(h);
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s IN OUT\n", argv[0]);
    return 1;
  }
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 1;
  int32_t dims[6];
  if (fread(dims, sizeof(int32_t), 6, in) != 6) return 4;
  const size_t B = dims[0], H = dims[1], G = dims[2], d = dims[3], n = dims[4], W = dims[5];

  selkv_params p;
  selkv_params_init(&p);
  p.batch = (int32_t)B;
  p.n_heads_kv = (int32_t)H;
  p.group = (int32_t)G;
  p.head_dim = (int32_t)d;
  p.seq_len = (int32_t)n;
  p.window = (int32_t)W;
  p.kv_dtype = SELKV_F32;
  int32_t mi = 0, mri = 0, msi = 0;
  SELKV_OK_(selkv_budget(&p, &mi, &mri, &msi));
  const size_t m = (size_t)mi, mr = (size_t)mri, ne = n - m;

  const size_t kv_bytes = B * H * n * d * sizeof(float);
  const size_t q_bytes = B * H * G * W * d * sizeof(float);
  const size_t qd_bytes = B * H * G * d * sizeof(float);
  void* hK = host_read(in, kv_bytes);
  void* hV = host_read(in, kv_bytes);
  void* hQ = host_read(in, q_bytes);
  void* hq = host_read(in, qd_bytes);
  fclose(in);

  void *K = dev_alloc(kv_bytes), *V = dev_alloc(kv_bytes), *Q = dev_alloc(q_bytes), *q = dev_alloc(qd_bytes);
  HIP_OK(hipMemcpy(K, hK, kv_bytes, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(V, hV, kv_bytes, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(Q, hQ, q_bytes, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(q, hq, qd_bytes, hipMemcpyHostToDevice));

  float* score = (float*)dev_alloc(B * H * (n - mr) * sizeof(float));
  float* attn = (float*)dev_alloc(B * H * n * sizeof(float));
  float* vnorm = (float*)dev_alloc(B * H * n * sizeof(float));
  int32_t* kept = (int32_t*)dev_alloc(B * H * m * sizeof(int32_t));
  int32_t* evicted = (int32_t*)dev_alloc(B * H * ne * sizeof(int32_t));
  int32_t* target = (int32_t*)dev_alloc(B * H * ne * sizeof(int32_t));
  float* gate = (float*)dev_alloc(B * H * ne * sizeof(float));
  void* K_out = dev_alloc(B * H * m * d * sizeof(float));
  void* V_out = dev_alloc(B * H * m * d * sizeof(float));
  float* bias = (float*)dev_alloc(B * H * m * sizeof(float));
  float* out = (float*)dev_alloc(qd_bytes);

  size_t ws_bytes = 0, sz = 0;
  const int32_t calls[4] = {SELKV_CALL_SCORE, SELKV_CALL_SELECT, SELKV_CALL_MERGE, SELKV_CALL_BIAS};
  for (int c = 0; c < 4; ++c) {
    SELKV_OK_(selkv_workspace_size(&p, calls[c], 0, &sz));
    if (sz > ws_bytes) ws_bytes = sz;
  }
  SELKV_OK_(selkv_workspace_size(&p, SELKV_CALL_DECODE, (int32_t)m, &sz));
  if (sz > ws_bytes) ws_bytes = sz;
  void* ws = dev_alloc(ws_bytes);   /* hipMalloc is 256-byte aligned; one workspace serves every call in turn */

  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));
  SELKV_OK_(selkv_score(&p, K, V, Q, score, attn, vnorm, ws, ws_bytes, st));
  SELKV_OK_(selkv_select(&p, score, kept, evicted, ws, ws_bytes, st));
  SELKV_OK_(selkv_merge(&p, K, V, attn, vnorm, kept, evicted, K_out, V_out, target, gate, ws, ws_bytes, st));
  SELKV_OK_(selkv_bias(&p, attn, kept, evicted, target, gate, bias, ws, ws_bytes, st));
  SELKV_OK_(selkv_decode_attn(&p, q, K_out, V_out, bias, (int32_t)m, out, ws, ws_bytes, st));

  /* the allocation-free decode (the library's own scratch) must match the workspace call bit for bit */
  float* out2 = (float*)dev_alloc(qd_bytes);
  SELKV_OK_(selkv_decode_attn_noalloc(&p, q, K_out, V_out, bias, (int32_t)m, out2, st));

  /* the fused call must reproduce selkv_merge + selkv_bias bit for bit */
  void* K_out2 = dev_alloc(B * H * m * d * sizeof(float));
  void* V_out2 = dev_alloc(B * H * m * d * sizeof(float));
  int32_t* target2 = (int32_t*)dev_alloc(B * H * ne * sizeof(int32_t));
  float* gate2 = (float*)dev_alloc(B * H * ne * sizeof(float));
  float* bias2 = (float*)dev_alloc(B * H * m * sizeof(float));
  SELKV_OK_(selkv_workspace_size(&p, SELKV_CALL_MERGE_BIAS, 0, &sz));
  if (sz > ws_bytes) return 6;
  SELKV_OK_(selkv_merge_bias(&p, K, V, attn, vnorm, kept, evicted, K_out2, V_out2, target2, gate2, bias2, ws,
                             ws_bytes, st));
  HIP_OK(hipStreamSynchronize(st));
  const struct { const void *a, *b; size_t bytes; const char* name; } same[] = {
      {K_out, K_out2, B * H * m * d * sizeof(float), "K_out"}, {V_out, V_out2, B * H * m * d * sizeof(float), "V_out"},
      {target, target2, B * H * ne * sizeof(int32_t), "target"}, {gate, gate2, B * H * ne * sizeof(float), "gate"},
      {bias, bias2, B * H * m * sizeof(float), "bias"}, {out, out2, qd_bytes, "decode out (noalloc)"}};
  for (size_t i = 0; i < sizeof(same) / sizeof(same[0]); ++i) {
    char* ha = (char*)malloc(same[i].bytes > 0 ? same[i].bytes : 1);
    char* hb = (char*)malloc(same[i].bytes > 0 ? same[i].bytes : 1);
    if (!ha || !hb) return 5;
    HIP_OK(hipMemcpy(ha, same[i].a, same[i].bytes, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hb, same[i].b, same[i].bytes, hipMemcpyDeviceToHost));
    if (memcmp(ha, hb, same[i].bytes) != 0) {
      fprintf(stderr, "two calls that must agree bit for bit differ in %s\n", same[i].name);
      return 7;
    }
    free(ha);
    free(hb);
  }

  FILE* o = fopen(argv[2], "wb");
  if (!o) return 1;
  fwrite(&mi, sizeof(int32_t), 1, o);
  fwrite(&mri, sizeof(int32_t), 1, o);
  to_file(o, kept, B * H * m * sizeof(int32_t));
  to_file(o, evicted, B * H * ne * sizeof(int32_t));
  to_file(o, target, B * H * ne * sizeof(int32_t));
  to_file(o, gate, B * H * ne * sizeof(float));
  to_file(o, K_out, B * H * m * d * sizeof(float));
  to_file(o, V_out, B * H * m * d * sizeof(float));
  to_file(o, bias, B * H * m * sizeof(float));
  to_file(o, out, qd_bytes);
  to_file(o, attn, B * H * n * sizeof(float));
  to_file(o, score, B * H * (n - mr) * sizeof(float));
  fclose(o);

  HIP_OK(hipStreamDestroy(st));
  void* bufs[] = {K, V, Q, q, score, attn, vnorm, kept, evicted, target, gate, K_out, V_out, bias, out, ws,
                  K_out2, V_out2, target2, gate2, bias2};
  for (size_t i = 0; i < sizeof(bufs) / sizeof(bufs[0]); ++i) HIP_OK(hipFree(bufs[i]));
  free(hK);
  free(hV);
  free(hQ);
  free(hq);
  printf("selkv_c_demo ok: m = %d\n", mi);
  return 0;
}
