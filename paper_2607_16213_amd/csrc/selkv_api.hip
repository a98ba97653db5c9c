// C ABI of libselkv: argument validation, workspace sizing, dispatch.
// Every check happens on the host before anything is launched.
#include <math.h>
#include <string.h>

#include <mutex>

#include "internal.hpp"
#include "selkv.h"

using namespace selkv;

// Fixed scratch of selkv_decode_attn_noalloc: one copy per GPU, held until
// the process ends.  Host code never passes this name to a kernel (on the
// host it is only a stand-in for the symbol); it uses the device address
// that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[SELKV_NOALLOC_SCRATCH_BYTES];

namespace {

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Validates the fields every compression call uses and derives the sizes.
selkv_status make_shape(const selkv_params* p, Shape* s) {
  if (!p || p->struct_size != sizeof(selkv_params)) return SELKV_EINVAL;
  if (p->kv_dtype != SELKV_F32 && p->kv_dtype != SELKV_BF16) return SELKV_EDTYPE;
  if (p->batch < 1 || p->n_heads_kv < 1 || p->group < 1 || p->seq_len < 1) return SELKV_EINVAL;
  if (p->head_dim != 64 && p->head_dim != 128) return SELKV_EUNSUPPORTED;
  if (p->seq_len > (1 << 28)) return SELKV_EUNSUPPORTED;   // per-head arrays addressed by 32-bit byte offsets
  if (p->window < 1 || p->window > p->seq_len) return SELKV_EINVAL;
  if (p->pool_kernel < 1 || (p->pool_kernel % 2) == 0) return SELKV_EINVAL;
  if (p->pool_kernel > 1025) return SELKV_EUNSUPPORTED;
  if (p->recent < 0) return SELKV_EINVAL;
  if (p->bucket < 1) return SELKV_EINVAL;
  if (p->bucket > 64) return SELKV_EUNSUPPORTED;
  if (!(p->budget_ratio > 0.0 && p->budget_ratio <= 1.0)) return SELKV_EINVAL;
  if (!(p->scale >= 0.f) || !isfinite(p->scale)) return SELKV_EINVAL;
  if (!isfinite(p->alpha)) return SELKV_EINVAL;
  if (!(p->gate_temperature > 0.f) || !isfinite(p->gate_temperature) || !isfinite(p->gate_threshold))
    return SELKV_EINVAL;
  if (p->gate_mode < SELKV_GATE_COSINE || p->gate_mode > SELKV_GATE_MERGE_ALL) return SELKV_EINVAL;
  if (p->route_mode < SELKV_ROUTE_BUCKET || p->route_mode > SELKV_ROUTE_COATTN) return SELKV_EINVAL;
  if (p->merge_keys != 0 && p->merge_keys != 1) return SELKV_EINVAL;
  if (p->select_mode != SELKV_SELECT_PER_HEAD && p->select_mode != SELKV_SELECT_UNION) return SELKV_EINVAL;
  const int64_t heads = (int64_t)p->batch * p->n_heads_kv;
  if (heads > 65535) return SELKV_EUNSUPPORTED;              // grid y dimension
  const int64_t R = (int64_t)p->group * p->window;
  if (R > 4096) return SELKV_EUNSUPPORTED;
  const double md = floor(p->budget_ratio * (double)p->seq_len);
  const int m = (int)md;
  if (m < 1) return SELKV_EINVAL;
  s->heads = heads;
  s->hkv = p->n_heads_kv;
  s->n = p->seq_len;
  s->d = p->head_dim;
  s->G = p->group;
  s->W = p->window;
  s->R = (int)R;
  s->m = m;
  s->mr = p->recent < m ? p->recent : m;
  s->ms = m - s->mr;
  s->n_cand = s->n - s->mr;
  s->nb = (s->n + p->bucket - 1) / p->bucket;
  return SELKV_OK;
}

float eff_scale(const selkv_params* p) { return p->scale > 0.f ? p->scale : 1.f / sqrtf((float)p->head_dim); }

size_t elem_size(const selkv_params* p) { return p->kv_dtype == SELKV_BF16 ? 2 : 4; }

selkv_status hip_status(hipError_t e) { return e == hipSuccess ? SELKV_OK : SELKV_EHIP; }

bool is_union(const selkv_params* p) { return p->select_mode == SELKV_SELECT_UNION; }

size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }

// merge and bias workspace: the bucket offsets under the bucket routings,
// the grouping by target slot under full-cosine routing
size_t merge_bytes(const selkv_params* p, const Shape& s) {
  return p->route_mode == SELKV_ROUTE_FULL_COSINE ? plan_group(s, p->kv_dtype).bytes : bucket_offsets_bytes(s);
}

// co-attention routing workspace: the score pass's row statistics, then the bucket offsets
size_t route_bytes(const selkv_params* p, const Shape& s) {
  return round256(plan_score(s, p->kv_dtype).bytes) + bucket_offsets_bytes(s);
}

// bias workspace: the routing's own scratch, then (union mode) the per-head R - 1
size_t bias_base_bytes(const selkv_params* p, const Shape& s) { return merge_bytes(p, s); }

// bias workspace: the routing's own scratch, then (union mode) the per-head R - 1
size_t bias_bytes(const selkv_params* p, const Shape& s) {
  const size_t base = bias_base_bytes(p, s);
  return is_union(p) ? round256(base) + plan_union(s).ratio_bytes : base;
}

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

selkv_status scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SELKV_EHIP;
  if (dev >= kMaxDevices) return SELKV_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return SELKV_EHIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return SELKV_OK;
}

// Arguments of selkv_decode_attn and selkv_decode_attn_noalloc.
selkv_status check_decode_args(const selkv_params* p, const void* q, const void* K, const void* V, const float* bias,
                               int32_t cache_len, float* out) {
  if (!p || p->struct_size != sizeof(selkv_params)) return SELKV_EINVAL;
  if (p->kv_dtype != SELKV_F32 && p->kv_dtype != SELKV_BF16) return SELKV_EDTYPE;
  if (p->batch < 1 || p->n_heads_kv < 1 || p->group < 1 || cache_len < 1) return SELKV_EINVAL;
  if (p->group > 8) return SELKV_EUNSUPPORTED;
  if (p->head_dim != 64 && p->head_dim != 128) return SELKV_EUNSUPPORTED;
  if (!(p->scale >= 0.f) || !isfinite(p->scale)) return SELKV_EINVAL;
  const int64_t heads = (int64_t)p->batch * p->n_heads_kv;
  if (heads > 65535) return SELKV_EUNSUPPORTED;
  if (!q || !K || !V || !out) return SELKV_EINVAL;
  if (!aligned(q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(bias, 4) || !aligned(out, 16))
    return SELKV_EALIGN;
  return SELKV_OK;
}

selkv_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return SELKV_OK;
  if (!ws || ws_bytes < need) return SELKV_EWORKSPACE;
  if (!aligned(ws, 256)) return SELKV_EALIGN;
  return SELKV_OK;
}

selkv_status check_merge_args(const Shape& s, const void* K, const void* V, const float* attn, const float* vnorm,
                              const int32_t* kept_idx, const int32_t* evicted_idx, void* K_out, void* V_out,
                              int32_t* target, float* gate) {
  const bool has_ev = s.n > s.m;
  if (!K || !V || !attn || !vnorm || !kept_idx || !K_out || !V_out) return SELKV_EINVAL;
  if (has_ev && (!evicted_idx || !target || !gate)) return SELKV_EINVAL;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(K_out, 16) || !aligned(V_out, 16) || !aligned(attn, 4) ||
      !aligned(vnorm, 4) || !aligned(kept_idx, 4) || !aligned(evicted_idx, 4) || !aligned(target, 4) ||
      !aligned(gate, 4))
    return SELKV_EALIGN;
  return SELKV_OK;
}

// Steps 3 - 5 (and, when bias is set, the fused step 6) on validated arguments.
selkv_status run_merge(const selkv_params* p, const Shape& s, const void* K, const void* V, const float* attn,
                       const float* vnorm, const int32_t* kept_idx, const int32_t* evicted_idx, void* K_out,
                       void* V_out, int32_t* target, float* gate, float* bias, bool raw, void* ws,
                       hipStream_t stream) {
  const bool mk = p->merge_keys != 0;
  hipError_t e;
  if (p->route_mode == SELKV_ROUTE_COATTN) {
    // targets given by selkv_route_coattn: grouped by target inside each bucket
    int32_t* offs = static_cast<int32_t*>(ws);
    e = launch_bucket_offsets(s, p->bucket, kept_idx, offs, stream);
    if (e != hipSuccess) return SELKV_EHIP;
    return hip_status(launch_merge_targets(s, p->kv_dtype, p->bucket, p->gate_mode, p->gate_threshold,
                                           p->gate_temperature, K, V, attn, vnorm, kept_idx, evicted_idx, offs,
                                           target, K_out, V_out, gate, mk, bias, p->alpha, raw, stream));
  }
  if (p->route_mode != SELKV_ROUTE_FULL_COSINE) {
    // bucket routings: one wave per bucket (plus its runs of empty buckets under the nearest-kept fallback)
    int32_t* offs = static_cast<int32_t*>(ws);
    e = launch_bucket_offsets(s, p->bucket, kept_idx, offs, stream);
    if (e != hipSuccess) return SELKV_EHIP;
    return hip_status(launch_merge_bucket(s, p->kv_dtype, p->bucket, p->gate_mode, p->gate_threshold,
                                          p->gate_temperature, K, V, attn, vnorm, kept_idx, evicted_idx, offs, K_out,
                                          V_out, target, gate, mk, p->route_mode == SELKV_ROUTE_BUCKET_NEAREST, bias,
                                          p->alpha, raw, stream));
  }
  // all-pairs routing: match, group by target slot, merge per slot
  const GroupPlan gp = plan_group(s, p->kv_dtype);
  e = launch_cosine_match(s, gp, p->kv_dtype, p->gate_mode, p->gate_threshold, p->gate_temperature, V, vnorm,
                          kept_idx, evicted_idx, target, gate, ws, stream);
  if (e != hipSuccess) return SELKV_EHIP;
  e = launch_group(s, gp, target, ws, stream);
  if (e != hipSuccess) return SELKV_EHIP;
  return hip_status(launch_group_merge(s, gp, p->kv_dtype, K, V, attn, kept_idx, evicted_idx, gate, ws, K_out, V_out,
                                       bias, p->alpha, raw, mk, stream));
}

}  // namespace

extern "C" {

SELKV_API void selkv_params_init(selkv_params* p) {
  if (!p) return;
  memset(p, 0, sizeof(*p));
  p->struct_size = sizeof(selkv_params);
  p->batch = 1;
  p->n_heads_kv = 8;
  p->group = 4;
  p->head_dim = 128;
  p->seq_len = 0;
  p->window = 32;
  p->pool_kernel = 5;
  p->recent = 16;
  p->bucket = 32;
  p->kv_dtype = SELKV_BF16;
  p->gate_mode = SELKV_GATE_COSINE;
  p->route_mode = SELKV_ROUTE_BUCKET;
  p->scale = 0.f;
  p->alpha = 0.5f;
  p->gate_threshold = 0.f;
  p->gate_temperature = 1.f;
  p->budget_ratio = 0.25;
  p->select_mode = SELKV_SELECT_PER_HEAD;
}

SELKV_API selkv_status selkv_budget(const selkv_params* p, int32_t* m, int32_t* m_recent, int32_t* m_select) {
  Shape s;
  const selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  if (m) *m = s.m;
  if (m_recent) *m_recent = s.mr;
  if (m_select) *m_select = s.ms;
  return SELKV_OK;
}

SELKV_API selkv_status selkv_workspace_size(const selkv_params* p, int32_t call, int32_t cache_len, size_t* bytes) {
  if (!bytes) return SELKV_EINVAL;
  if (call == SELKV_CALL_DECODE) {
    if (!p || p->struct_size != sizeof(selkv_params)) return SELKV_EINVAL;
    if (p->batch < 1 || p->n_heads_kv < 1 || p->group < 1 || p->group > 8 || cache_len < 1) return SELKV_EINVAL;
    if (p->head_dim != 64 && p->head_dim != 128) return SELKV_EUNSUPPORTED;
    *bytes = decode_workspace_bound((int64_t)p->batch * p->n_heads_kv, cache_len, p->head_dim, p->group);
    return SELKV_OK;
  }
  Shape s;
  const selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  switch (call) {
    case SELKV_CALL_SCORE: *bytes = plan_score(s, p->kv_dtype).bytes; return SELKV_OK;
    case SELKV_CALL_SELECT: *bytes = is_union(p) ? plan_union(s).select_bytes : 0; return SELKV_OK;
    case SELKV_CALL_MERGE: *bytes = merge_bytes(p, s); return SELKV_OK;
    case SELKV_CALL_ROUTE: *bytes = route_bytes(p, s); return SELKV_OK;
    case SELKV_CALL_BIAS:
    case SELKV_CALL_MERGE_BIAS: *bytes = bias_bytes(p, s); return SELKV_OK;
    default: return SELKV_EINVAL;
  }
}

SELKV_API selkv_status selkv_score(const selkv_params* p, const void* K, const void* V, const void* Qwin,
                                   float* score, float* attn, float* vnorm, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  Shape s;
  selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  if (!K || !V || !Qwin || !score || !attn || !vnorm) return SELKV_EINVAL;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(Qwin, 16) || !aligned(score, 4) || !aligned(attn, 4) ||
      !aligned(vnorm, 4))
    return SELKV_EALIGN;
  const ScorePlan plan = plan_score(s, p->kv_dtype);
  if ((st = check_ws(ws, ws_bytes, plan.bytes)) != SELKV_OK) return st;
  return hip_status(launch_score(s, plan, p->kv_dtype, eff_scale(p), K, V, Qwin, score, attn, vnorm,
                                 p->pool_kernel, ws, stream));
}

SELKV_API selkv_status selkv_select(const selkv_params* p, const float* score, int32_t* kept_idx,
                                    int32_t* evicted_idx, void* ws, size_t ws_bytes, hipStream_t stream) {
  Shape s;
  selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  if (!score || !kept_idx || (!evicted_idx && s.n > s.m)) return SELKV_EINVAL;
  if (!aligned(score, 4) || !aligned(kept_idx, 4) || !aligned(evicted_idx, 4)) return SELKV_EALIGN;
  if (is_union(p)) {
    const UnionPlan up = plan_union(s);
    if ((st = check_ws(ws, ws_bytes, up.select_bytes)) != SELKV_OK) return st;
    return hip_status(launch_union_select(s, up, score, kept_idx, evicted_idx, ws, stream));
  }
  return hip_status(launch_select(s, score, kept_idx, evicted_idx, stream));
}

SELKV_API selkv_status selkv_route_coattn(const selkv_params* p, const void* K, const void* Qwin,
                                          const int32_t* kept_idx, const int32_t* evicted_idx, int32_t* target,
                                          void* ws, size_t ws_bytes, hipStream_t stream) {
  Shape s;
  selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  const bool has_ev = s.n > s.m;
  if (!K || !Qwin || !kept_idx) return SELKV_EINVAL;
  if (has_ev && (!evicted_idx || !target)) return SELKV_EINVAL;
  if (!aligned(K, 16) || !aligned(Qwin, 16) || !aligned(kept_idx, 4) || !aligned(evicted_idx, 4) ||
      !aligned(target, 4))
    return SELKV_EALIGN;
  if ((st = check_ws(ws, ws_bytes, route_bytes(p, s))) != SELKV_OK) return st;
  if (!has_ev) return SELKV_OK;
  const ScorePlan sp = plan_score(s, p->kv_dtype);
  int32_t* offs = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + round256(sp.bytes));
  const float scale = eff_scale(p);
  hipError_t e = launch_row_stats(s, sp, p->kv_dtype, scale, K, Qwin, ws, stream);
  if (e != hipSuccess) return SELKV_EHIP;
  e = launch_bucket_offsets(s, p->bucket, kept_idx, offs, stream);
  if (e != hipSuccess) return SELKV_EHIP;
  return hip_status(launch_coattn_route(s, sp, p->kv_dtype, p->bucket, p->window, K, Qwin, ws, kept_idx, offs, target,
                                        scale * 1.4426950408889634f, stream));   // log2(e): logits in the log2 domain
}

SELKV_API selkv_status selkv_merge(const selkv_params* p, const void* K, const void* V, const float* attn,
                                   const float* vnorm, const int32_t* kept_idx, const int32_t* evicted_idx,
                                   void* K_out, void* V_out, int32_t* target, float* gate, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
  Shape s;
  selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  if ((st = check_merge_args(s, K, V, attn, vnorm, kept_idx, evicted_idx, K_out, V_out, target, gate)) != SELKV_OK)
    return st;
  if ((st = check_ws(ws, ws_bytes, merge_bytes(p, s))) != SELKV_OK) return st;
  return run_merge(p, s, K, V, attn, vnorm, kept_idx, evicted_idx, K_out, V_out, target, gate, nullptr, false, ws,
                   stream);
}

SELKV_API selkv_status selkv_merge_bias(const selkv_params* p, const void* K, const void* V, const float* attn,
                                        const float* vnorm, const int32_t* kept_idx, const int32_t* evicted_idx,
                                        void* K_out, void* V_out, int32_t* target, float* gate, float* bias,
                                        void* ws, size_t ws_bytes, hipStream_t stream) {
  Shape s;
  selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  if ((st = check_merge_args(s, K, V, attn, vnorm, kept_idx, evicted_idx, K_out, V_out, target, gate)) != SELKV_OK)
    return st;
  if (!bias) return SELKV_EINVAL;
  if (!aligned(bias, 4)) return SELKV_EALIGN;
  const bool uni = is_union(p);
  if ((st = check_ws(ws, ws_bytes, bias_bytes(p, s))) != SELKV_OK) return st;
  // union mode: the merge writes each head's R - 1 into the workspace
  float* dst = uni ? reinterpret_cast<float*>(static_cast<char*>(ws) + round256(merge_bytes(p, s))) : bias;
  if ((st = run_merge(p, s, K, V, attn, vnorm, kept_idx, evicted_idx, K_out, V_out, target, gate, dst, uni, ws,
                      stream)) != SELKV_OK || !uni)
    return st;
  return hip_status(launch_union_bias(s, dst, bias, p->alpha, stream));
}

SELKV_API selkv_status selkv_bias(const selkv_params* p, const float* attn, const int32_t* kept_idx,
                                  const int32_t* evicted_idx, const int32_t* target, const float* gate,
                                  float* bias, void* ws, size_t ws_bytes, hipStream_t stream) {
  Shape s;
  selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  const bool has_ev = s.n > s.m;
  if (!attn || !kept_idx || !bias) return SELKV_EINVAL;
  if (has_ev && (!evicted_idx || !target || !gate)) return SELKV_EINVAL;
  if (!aligned(attn, 4) || !aligned(kept_idx, 4) || !aligned(evicted_idx, 4) || !aligned(target, 4) ||
      !aligned(gate, 4) || !aligned(bias, 4))
    return SELKV_EALIGN;
  // union mode: the routing kernels write each head's R - 1 into the
  // workspace and one more pass averages it over the heads of each cache
  const bool uni = is_union(p);
  const size_t base = bias_base_bytes(p, s);
  if ((st = check_ws(ws, ws_bytes, bias_bytes(p, s))) != SELKV_OK) return st;
  float* dst = uni ? reinterpret_cast<float*>(static_cast<char*>(ws) + round256(base)) : bias;
  hipError_t e;
  if (p->route_mode == SELKV_ROUTE_FULL_COSINE) {
    const GroupPlan gp = plan_group(s, p->kv_dtype);
    e = launch_group(s, gp, target, ws, stream);
    if (e != hipSuccess) return SELKV_EHIP;
    e = launch_group_merge(s, gp, p->kv_dtype, nullptr, nullptr, attn, kept_idx, evicted_idx, gate, ws, nullptr,
                           nullptr, dst, p->alpha, uni, false, stream);
  } else {
    int32_t* offs = static_cast<int32_t*>(ws);
    e = launch_bucket_offsets(s, p->bucket, kept_idx, offs, stream);
    if (e != hipSuccess) return SELKV_EHIP;
    e = launch_bias_bucket(s, p->bucket, p->alpha, attn, kept_idx, evicted_idx, offs, target, gate, dst, uni,
                           p->route_mode == SELKV_ROUTE_BUCKET_NEAREST, stream);
  }
  if (e != hipSuccess || !uni) return hip_status(e);
  return hip_status(launch_union_bias(s, dst, bias, p->alpha, stream));
}

SELKV_API selkv_status selkv_rope_reposition(const selkv_params* p, const int32_t* kept_idx, void* K_out,
                                             double rope_theta, hipStream_t stream) {
  Shape s;
  selkv_status st = make_shape(p, &s);
  if (st != SELKV_OK) return st;
  if (!kept_idx || !K_out) return SELKV_EINVAL;
  if (!(rope_theta > 1.0) || !isfinite(rope_theta)) return SELKV_EINVAL;
  if (!aligned(kept_idx, 4) || !aligned(K_out, 16)) return SELKV_EALIGN;
  return hip_status(launch_rope_reposition(s, p->kv_dtype, kept_idx, K_out, rope_theta, stream));
}

SELKV_API selkv_status selkv_decode_attn(const selkv_params* p, const void* q, const void* K, const void* V,
                                         const float* bias, int32_t cache_len, float* out, void* ws,
                                         size_t ws_bytes, hipStream_t stream) {
  selkv_status st = check_decode_args(p, q, K, V, bias, cache_len, out);
  if (st != SELKV_OK) return st;
  const int64_t heads = (int64_t)p->batch * p->n_heads_kv;
  const DecodePlan plan = plan_decode(heads, cache_len, p->head_dim, p->group);
  st = check_ws(ws, ws_bytes, plan.bytes);
  if (st != SELKV_OK) return st;
  return hip_status(launch_decode(heads, p->n_heads_kv, cache_len, cache_len, p->head_dim, p->group, p->kv_dtype,
                                  eff_scale(p), plan, q, K, V, bias, out, ws, stream));
}

SELKV_API selkv_status selkv_decode_attn_noalloc(const selkv_params* p, const void* q, const void* K, const void* V,
                                                 const float* bias, int32_t cache_len, float* out,
                                                 hipStream_t stream) {
  selkv_status st = check_decode_args(p, q, K, V, bias, cache_len, out);
  if (st != SELKV_OK) return st;
  const int64_t heads = (int64_t)p->batch * p->n_heads_kv;
  const DecodePlan plan = plan_decode(heads, cache_len, p->head_dim, p->group);
  if (plan.bytes > (size_t)SELKV_NOALLOC_SCRATCH_BYTES) return SELKV_EWORKSPACE;
  void* ws = nullptr;
  st = scratch_of_current_device(&ws);
  if (st != SELKV_OK) return st;
  return hip_status(launch_decode(heads, p->n_heads_kv, cache_len, cache_len, p->head_dim, p->group, p->kv_dtype,
                                  eff_scale(p), plan, q, K, V, bias, out, ws, stream));
}

SELKV_API selkv_status selkv_decode_append(const selkv_params* p, const void* q, const void* k_new,
                                           const void* v_new, void* K, void* V, float* bias, int32_t cache_len,
                                           int32_t capacity, float* out, void* ws, size_t ws_bytes,
                                           hipStream_t stream) {
  if (!p || p->struct_size != sizeof(selkv_params)) return SELKV_EINVAL;
  if (p->kv_dtype != SELKV_F32 && p->kv_dtype != SELKV_BF16) return SELKV_EDTYPE;
  if (p->batch < 1 || p->n_heads_kv < 1 || p->group < 1 || cache_len < 0 || capacity < 1) return SELKV_EINVAL;
  if (cache_len >= capacity) return SELKV_EINVAL;                 // no room for the new entry
  if (p->group > 8) return SELKV_EUNSUPPORTED;
  if (p->head_dim != 64 && p->head_dim != 128) return SELKV_EUNSUPPORTED;
  if (!(p->scale >= 0.f) || !isfinite(p->scale)) return SELKV_EINVAL;
  const int64_t heads = (int64_t)p->batch * p->n_heads_kv;
  if (heads > 65535) return SELKV_EUNSUPPORTED;
  if (!q || !k_new || !v_new || !K || !V || !out) return SELKV_EINVAL;
  if (!aligned(q, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(K, 16) || !aligned(V, 16) ||
      !aligned(bias, 4) || !aligned(out, 16))
    return SELKV_EALIGN;
  const DecodePlan plan = plan_decode(heads, cache_len + 1, p->head_dim, p->group);
  selkv_status st = check_ws(ws, ws_bytes, plan.bytes);
  if (st != SELKV_OK) return st;
  // one launch: the new entry is read from k_new / v_new and stored into the cache on the way
  return hip_status(launch_decode(heads, p->n_heads_kv, cache_len + 1, capacity, p->head_dim, p->group,
                                  p->kv_dtype, eff_scale(p), plan, q, K, V, bias, out, ws, stream, k_new, v_new));
}

SELKV_API const char* selkv_status_string(selkv_status s) {
  switch (s) {
    case SELKV_OK: return "success";
    case SELKV_EINVAL: return "invalid argument";
    case SELKV_EDTYPE: return "unknown kv dtype";
    case SELKV_EUNSUPPORTED: return "unsupported configuration";
    case SELKV_EALIGN: return "misaligned pointer";
    case SELKV_EWORKSPACE: return "workspace missing or too small";
    case SELKV_EHIP: return "HIP launch error";
    default: return "unknown status";
  }
}

SELKV_API int32_t selkv_abi_version(void) { return SELKV_ABI_VERSION; }

}  // extern "C"
