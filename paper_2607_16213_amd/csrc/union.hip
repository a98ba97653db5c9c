// GQA union mode (Sec. 3.3 union selection, Sec. 3.6 GQA rule) for
// selkv_select / selkv_bias with SELKV_SELECT_UNION.
//
//   select  the per-KV-head top-m_s sets come from the ordinary selection
//           kernel; the heads of each cache then mark their picks in one flag
//           row, the flagged candidates get their mean score across the heads
//           (fp32, head order) and the rest -inf, and the same selection
//           kernel picks the m_s best means (lower position on ties) plus the
//           recent window; that set is copied to every head of the cache.
//   bias    the bias kernels write each head's R - 1 (absorbed / a); one pass
//           averages it over the heads of the cache in head order and writes
//           alpha * log1p(mean) for every head.
// Integer flags are written with plain stores of the same value, so the
// outcome does not depend on scheduling.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

__global__ __launch_bounds__(kThreads) void fill_int_kernel(int32_t* p, int64_t count, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < count) p[i] = v;
}

// flag[b][j] = 1 for every candidate j that KV head (b, h) picked.  The first
// m_s kept entries of a head are its picks (kept lists are ascending and the
// recent window sits above every candidate).
__global__ __launch_bounds__(kThreads) void union_flag_kernel(const int32_t* kept, int32_t* flag, int hkv, int m,
                                                              int ms, int n_cand) {
  const int64_t head = blockIdx.y;
  const int k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= ms) return;
  const int j = kept[head * m + k];
  if (j >= 0 && j < n_cand) flag[(head / hkv) * n_cand + j] = 1;
}

// key[b][j] = mean over the cache's heads of score[b, h, j] if flagged, else -inf.
__global__ __launch_bounds__(kThreads) void union_key_kernel(const float* score, const int32_t* flag, float* key,
                                                             int hkv, int n_cand) {
  const int64_t b = blockIdx.y;
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= n_cand) return;
  const size_t o = (size_t)b * n_cand + j;
  float v = kNegInf;
  if (flag[o]) {
    float acc = 0.f;
    for (int h = 0; h < hkv; ++h) acc += score[((size_t)b * hkv + h) * n_cand + j];
    v = acc / (float)hkv;
  }
  key[o] = v;
}

// Copies the cache's shared kept / evicted rows to each of its heads.
__global__ __launch_bounds__(kThreads) void union_broadcast_kernel(const int32_t* tkept, const int32_t* tev,
                                                                   int32_t* kept, int32_t* evicted, int hkv, int m,
                                                                   int ne) {
  const int64_t head = blockIdx.y;
  const int64_t b = head / hkv;
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < m) kept[head * m + i] = tkept[b * m + i];
  if (i < ne) evicted[head * ne + i] = tev[b * ne + i];
}

// bias[b, h, s] = alpha * log1p(mean over h' of r1[b, h', s]) for every h.
__global__ __launch_bounds__(kThreads) void union_bias_kernel(const float* r1, float* bias, int hkv, int m,
                                                              float alpha) {
  const int64_t b = blockIdx.y;
  const int s = blockIdx.x * kThreads + threadIdx.x;
  if (s >= m) return;
  float acc = 0.f;
  for (int h = 0; h < hkv; ++h) acc += r1[((size_t)b * hkv + h) * m + s];
  const float mean = acc / (float)hkv;
  const float v = mean > 0.f ? alpha * log1pf(mean) : 0.f;
  for (int h = 0; h < hkv; ++h) bias[((size_t)b * hkv + h) * m + s] = v;
}

}  // namespace

UnionPlan plan_union(const Shape& s) {
  UnionPlan p{};
  const size_t batch = (size_t)(s.heads / s.hkv);
  const size_t nc = s.n_cand > 0 ? (size_t)s.n_cand : 1;
  p.flag_off = 0;
  p.key_off = p.flag_off + align256(batch * nc * sizeof(int32_t));
  p.kept_off = p.key_off + align256(batch * nc * sizeof(float));
  p.ev_off = p.kept_off + align256(batch * (size_t)s.m * sizeof(int32_t));
  const size_t ne = (size_t)(s.n - s.m);
  p.select_bytes = p.ev_off + align256(batch * (ne > 0 ? ne : 1) * sizeof(int32_t));
  p.ratio_bytes = align256((size_t)s.heads * s.m * sizeof(float));
  return p;
}

hipError_t launch_union_select(const Shape& s, const UnionPlan& p, const float* score, int32_t* kept,
                               int32_t* evicted, void* ws, hipStream_t st) {
  hipError_t e = launch_select(s, score, kept, evicted, st);      // every head's own picks
  if (e != hipSuccess) return e;
  const int64_t batch = s.heads / s.hkv;
  if (s.ms == 0 || s.n_cand == 0) return hipSuccess;              // only the recent window: already shared
  char* w = static_cast<char*>(ws);
  int32_t* flag = reinterpret_cast<int32_t*>(w + p.flag_off);
  float* key = reinterpret_cast<float*>(w + p.key_off);
  int32_t* tkept = reinterpret_cast<int32_t*>(w + p.kept_off);
  int32_t* tev = reinterpret_cast<int32_t*>(w + p.ev_off);
  const int64_t nflag = batch * s.n_cand;
  hipLaunchKernelGGL(fill_int_kernel, dim3((unsigned)((nflag + kThreads - 1) / kThreads)), dim3(kThreads), 0, st,
                     flag, nflag, 0);
  hipLaunchKernelGGL(union_flag_kernel, dim3((s.ms + kThreads - 1) / kThreads, (unsigned)s.heads), dim3(kThreads),
                     0, st, kept, flag, s.hkv, s.m, s.ms, s.n_cand);
  hipLaunchKernelGGL(union_key_kernel, dim3((s.n_cand + kThreads - 1) / kThreads, (unsigned)batch), dim3(kThreads),
                     0, st, score, flag, key, s.hkv, s.n_cand);
  Shape su = s;
  su.heads = batch;
  su.hkv = 1;
  e = launch_select(su, key, tkept, tev, st);
  if (e != hipSuccess) return e;
  const int ne = s.n - s.m;
  const int rows = s.m > ne ? s.m : ne;
  hipLaunchKernelGGL(union_broadcast_kernel, dim3((rows + kThreads - 1) / kThreads, (unsigned)s.heads),
                     dim3(kThreads), 0, st, tkept, tev, kept, evicted, s.hkv, s.m, ne);
  return hipGetLastError();
}

hipError_t launch_union_bias(const Shape& s, const float* r1, float* bias, float alpha, hipStream_t st) {
  const int64_t batch = s.heads / s.hkv;
  hipLaunchKernelGGL(union_bias_kernel, dim3((s.m + kThreads - 1) / kThreads, (unsigned)batch), dim3(kThreads), 0,
                     st, r1, bias, s.hkv, s.m, alpha);
  return hipGetLastError();
}

}  // namespace selkv
