/*
 * selkv.h - C ABI of the SelKV one-shot KV-cache compression and biased
 * decode library for AMD Instinct MI355X (gfx950).
 *
 * Paper: "SelKV: Selective KV Cache Merging with Per-Token Merge-or-Drop
 * and Attention Compensation" (arXiv 2607.16213), Sec. 3 and Algorithm 1.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every tensor pointer is a DEVICE pointer owned by the caller.  The
 *    library never allocates, frees or retains memory, and keeps no state
 *    between calls.  Scratch memory is passed in as `ws` / `ws_bytes`,
 *    sized by selkv_workspace_size(); a call whose workspace size is 0 may
 *    pass NULL.  A workspace needs no initialisation: every call writes the
 *    scratch it reads, so its contents on entry never change a result.
 *  - Tensors are dense, row-major, contiguous.  "B" is any leading batch of
 *    independent caches: sequences, or sequences x layers when a whole
 *    model's caches are stored back to back, since every step is
 *    independent per (sequence, layer, KV head).
 *  - Storage dtype of K, V and queries is params.kv_dtype (fp32 or bf16);
 *    all arithmetic accumulates in fp32.  Scores, attention masses, norms,
 *    gates and biases are fp32; indices are int32.
 *  - K, V, query and decode-output pointers must be 16-byte aligned; other
 *    fp32 / int32 arrays 4-byte aligned.
 *  - Calls are asynchronous on `stream` (0 = the null stream) and never
 *    synchronise the host.  Arguments are validated on the host before
 *    anything is launched; an invalid call returns an error status and
 *    launches nothing.  A failed launch returns SELKV_EHIP.  Faults inside a
 *    kernel surface at the caller's next synchronisation.
 *  - Every call is deterministic: the same inputs give bitwise-identical
 *    outputs (no floating-point atomics).
 *  - Index inputs (kept_idx, evicted_idx, target) are meant to come from the
 *    library's own calls.  Positions are clamped into [0, n) and target slots
 *    checked against [0, m) before any memory access, so a malformed list
 *    gives wrong outputs but never an access outside the caller's buffers.
 *  - No C++ exception crosses this interface.
 */
#ifndef SELKV_H_
#define SELKV_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__)
#define SELKV_API __attribute__((visibility("default")))
#else
#define SELKV_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

#define SELKV_ABI_VERSION 6

/* Bytes of the fixed per-GPU scratch of selkv_decode_attn_noalloc (16 MiB). */
#define SELKV_NOALLOC_SCRATCH_BYTES (16u << 20)

typedef enum selkv_status {
  SELKV_OK = 0,
  SELKV_EINVAL = 1,        /* a NULL pointer, a size or parameter out of range */
  SELKV_EDTYPE = 2,        /* kv_dtype is not one of selkv_dtype */
  SELKV_EUNSUPPORTED = 3,  /* valid request the library does not implement (e.g. head_dim not 64/128) */
  SELKV_EALIGN = 4,        /* a pointer violates the alignment rule above */
  SELKV_EWORKSPACE = 5,    /* ws is NULL or ws_bytes is below selkv_workspace_size() */
  SELKV_EHIP = 6           /* a HIP launch returned an error */
} selkv_status;

typedef enum selkv_dtype { SELKV_F32 = 0, SELKV_BF16 = 1 } selkv_dtype;

/* Gate of Sec. 3.5.  COSINE is the paper's soft cosine gate (generalised by
 * gate_threshold / gate_temperature, see selkv_params); DROP (g = 0) and
 * MERGE_ALL (g = 1) are the "eviction only" and "merge all" ablations of
 * Sec. 4.3. */
typedef enum selkv_gate_mode {
  SELKV_GATE_COSINE = 0,
  SELKV_GATE_DROP = 1,
  SELKV_GATE_MERGE_ALL = 2
} selkv_gate_mode;

/* Merge-target routing of Sec. 3.4.  BUCKET is Eq. 3 (bucket-attention
 * routing; the evicted tokens of a bucket that keeps nothing are dropped);
 * FULL_COSINE is the all-pairs cosine routing that Eq. 3 replaces;
 * BUCKET_NEAREST is Eq. 3 with the other reading of the empty-bucket case
 * the paper leaves open: those tokens go to the kept token nearest by
 * position (the lower position when two are equally near).
 * COATTN reads Eq. 3's A_{h,j,i} as co-attention: targets come from
 * selkv_route_coattn, and selkv_merge takes them as input. */
typedef enum selkv_route_mode {
  SELKV_ROUTE_BUCKET = 0,
  SELKV_ROUTE_FULL_COSINE = 1,
  SELKV_ROUTE_BUCKET_NEAREST = 2,
  SELKV_ROUTE_COATTN = 3
} selkv_route_mode;

/* Token selection of Sec. 3.3.  PER_HEAD: every KV head keeps its own
 * top-m_s set (Eq. 2; the MHA rule, and per-KV-head selection for GQA).
 * UNION: the GQA rule - each KV head picks its top-m_s, the union over the
 * n_heads_kv heads of one cache is trimmed to m_s by the mean score across
 * those heads, and that one kept set is shared by all of them; selkv_bias
 * then averages R across the heads (Sec. 3.6). */
typedef enum selkv_select_mode {
  SELKV_SELECT_PER_HEAD = 0,
  SELKV_SELECT_UNION = 1
} selkv_select_mode;

/* Which call a workspace size is asked for. */
typedef enum selkv_call {
  SELKV_CALL_SCORE = 0,
  SELKV_CALL_SELECT = 1,
  SELKV_CALL_MERGE = 2,
  SELKV_CALL_BIAS = 3,
  SELKV_CALL_DECODE = 4,
  SELKV_CALL_ROUTE = 5,     /* selkv_route_coattn */
  SELKV_CALL_MERGE_BIAS = 6 /* selkv_merge_bias */
} selkv_call;

/* Problem description, named as in the paper.  Fill it with
 * selkv_params_init() and override fields. */
typedef struct selkv_params {
  uint32_t struct_size;      /* = sizeof(selkv_params); guards ABI drift */
  int32_t batch;             /* B: independent caches (sequences, or sequences x layers) */
  int32_t n_heads_kv;        /* H_kv */
  int32_t group;             /* G: query heads per KV head; H_q = G * H_kv; query head h reads KV head h / G */
  int32_t head_dim;          /* d: 64 or 128 */
  int32_t seq_len;           /* n: prompt length (tokens in the uncompressed cache), at most 2^28 */
  int32_t window;            /* W: observation window, 1 <= W <= n (Sec. 3.2, default 32) */
  int32_t pool_kernel;       /* K: odd smoothing kernel (Sec. 3.2, default 5; at most 1025) */
  int32_t recent;            /* m_r: recent tokens always kept (Sec. 3.1, default 16) */
  int32_t bucket;            /* B: routing bucket size, 1..64 (Sec. 3.4, default 32) */
  int32_t kv_dtype;          /* selkv_dtype of K, V and queries */
  int32_t gate_mode;         /* selkv_gate_mode */
  int32_t route_mode;        /* selkv_route_mode */
  float scale;               /* softmax scale of the window pass and of decode; 0 means 1/sqrt(d) */
  float alpha;               /* compensation strength alpha (Sec. 3.6, default 0.5) */
  float gate_threshold;      /* tau: g = clamp((sim - tau) / T, 0, 1); tau = 0, T = 1 is max(sim, 0) */
  float gate_temperature;    /* T > 0 */
  double budget_ratio;       /* rho in (0, 1]; m = floor(rho * n) computed in IEEE double (Sec. 3.1) */
  int32_t select_mode;       /* selkv_select_mode (default PER_HEAD) */
  int32_t merge_keys;        /* 0: keys gathered (Eq. 5 defines only values; default); 1: keys merged with
                                the value weights of Eq. 5 (the alternative reading) */
} selkv_params;

/* Fill `p` with the paper's defaults (App. F: W = 32, K = 5, B = 32,
 * m_r = 16, alpha = 0.5, rho = 0.25; cosine gate, bucket routing, bf16),
 * batch = 1, H_kv = 8, G = 4, d = 128, n = 0 (to be set). */
SELKV_API void selkv_params_init(selkv_params* p);

/* Budget of Sec. 3.1: m = floor(rho * n) entries per KV head, of which
 * m_r' = min(m_r, m) are the most recent tokens and m_s = m - m_r' are
 * chosen by score.  Returns SELKV_EINVAL if m < 1 or a field is invalid.
 * Host-only; touches no device. */
SELKV_API selkv_status selkv_budget(const selkv_params* p, int32_t* m, int32_t* m_recent,
                                    int32_t* m_select);

/* Bytes of scratch the call `call` (selkv_call) needs for `p`.
 * `cache_len` is used only for SELKV_CALL_DECODE (entries per KV head);
 * the size returned then serves every cache length up to `cache_len`.
 * Host-only. */
SELKV_API selkv_status selkv_workspace_size(const selkv_params* p, int32_t call, int32_t cache_len,
                                            size_t* bytes);

/* Step 1 of Algorithm 1: contribution scores (Sec. 3.2, Eq. 1).
 *
 * Recomputes the observation-window attention of Sec. 3.1 (the eager
 * re-pass of the last W query positions over the cached keys) without
 * materialising it: window row i of a query head is position n-W+i and
 * attends causally to keys j <= n-W+i with logits scale * q.k.  For each KV
 * head it produces
 *   attn[j]  = a_j = (1/G) * sum over the G query heads and W rows of A[row, j]
 *              (the cumulative window attention of Eq. 5, averaged over the
 *              query heads that share the KV head, Sec. 3.3),
 *   vnorm[j] = ||v_j||_2,
 *   score[j] = the K-wide centred moving average of c = a * ||v|| (Eq. 1)
 *              over the candidate range [0, n - m_r'), zero outside it,
 *              divisor K (Sec. 3.2 smoothing).
 * In:  K, V  [B, H_kv, n, d]   Qwin [B, H_kv*G, W, d]   (kv_dtype)
 * Out: score [B, H_kv, n - m_r'] fp32; attn, vnorm [B, H_kv, n] fp32.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_SCORE, 0). */
SELKV_API selkv_status selkv_score(const selkv_params* p, const void* K, const void* V, const void* Qwin,
                                   float* score, float* attn, float* vnorm, void* ws, size_t ws_bytes,
                                   hipStream_t stream);

/* Step 2 of Algorithm 1: token selection (Sec. 3.3, Eq. 2).
 *
 * PER_HEAD: per KV head, keeps the m_s candidates with the largest score
 * (equal scores: the lower position wins) plus the m_r' most recent
 * positions.  UNION (GQA): per cache b, each of the H_kv heads picks its
 * top-m_s as above; a candidate picked by any head is in the union; the
 * union is cut to its m_s candidates of largest mean score across the heads
 * (the mean is the fp32 sum in head order divided by H_kv; equal means: the
 * lower position wins); that set plus the recent positions is written for
 * every head of the cache.  Every head contributes m_s candidates, so the
 * union is never short and each head keeps exactly m entries.
 * In:  score [B, H_kv, n - m_r'] fp32 (NaN is outside the contract)
 * Out: kept_idx [B, H_kv, m] and evicted_idx [B, H_kv, n - m], int32
 *      positions, each ascending; together a partition of 0..n-1.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_SELECT, 0) (0 for
 *      PER_HEAD; the union flags, means and shared set for UNION). */
SELKV_API selkv_status selkv_select(const selkv_params* p, const float* score, int32_t* kept_idx,
                                    int32_t* evicted_idx, void* ws, size_t ws_bytes, hipStream_t stream);

/* Step 3 of Algorithm 1 under the co-attention reading of Eq. 3 (Sec. 3.4;
 * the route_mode COATTN alternative).
 *
 * Eq. 3 ranks candidate targets by A_{h,j,i}, which the window pass does not
 * produce as such; this call reads it as how much the observation window
 * attends to evicted j and kept i together:
 *   co(j, i) = sum over the G*W window rows r of the KV head of P[r, j] P[r, i]
 * with P the softmax window attention of selkv_score (scale, causal mask).
 * Evicted token j goes to the kept token of its bucket floor(j/B) with the
 * largest co(j, i), lowest position on ties, or nowhere (-1) if the bucket
 * keeps no token.  The row statistics over all n keys are recomputed here,
 * then the logits of each bucket's keys and their Gram matrix P^T P are
 * formed on MFMA; the attention matrix is never stored.
 * In:  K [B, H_kv, n, d], Qwin [B, H_kv*G, W, d] (kv_dtype, as for
 *      selkv_score); kept_idx, evicted_idx (from selkv_select).
 * Out: target [B, H_kv, n - m] int32 kept slot or -1; pass it to selkv_merge
 *      and selkv_bias with route_mode COATTN.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_ROUTE, 0). */
SELKV_API selkv_status selkv_route_coattn(const selkv_params* p, const void* K, const void* Qwin,
                                          const int32_t* kept_idx, const int32_t* evicted_idx, int32_t* target,
                                          void* ws, size_t ws_bytes, hipStream_t stream);

/* Steps 3-5 of Algorithm 1: routing (Sec. 3.4, Eq. 3), soft cosine gate
 * (Sec. 3.5, Eq. 4) and gated merge (Eq. 5).
 *
 * BUCKET routing: evicted token j goes to the kept token of its bucket
 * floor(j/B) with the largest attn (lowest position on ties), or nowhere
 * (-1, dropped) if the bucket keeps no token.  FULL_COSINE routing: to the
 * kept token with the most cosine-similar value (lowest slot on ties),
 * found by an all-pairs MFMA contraction per KV head; the tokens routed to
 * each slot are then merged in ascending order.
 * Gate: sim = v_j . v_t / (||v_j|| ||v_t||) against the pre-merge target
 * value (0 if a norm is 0), g = clamp((sim - tau)/T, 0, 1) in COSINE mode,
 * 0 in DROP, 1 in MERGE_ALL; unrouted tokens get g = 0.
 * Merge: V~_i = (a_i v_i + sum_{j->i} g_j a_j v_j) / (a_i + sum g_j a_j);
 * a kept token that absorbs nothing is copied bit for bit.  Keys are not
 * merged (K~_i = k_i) unless merge_keys = 1, which gives them the same
 * weights as the values.  BUCKET_NEAREST routes like BUCKET where a bucket
 * keeps a token and sends the tokens of a bucket that keeps none to the
 * kept token nearest by position (the lower one when equally near); a run
 * of such buckets is absorbed by the non-empty buckets on either side, so
 * the merge stays bucket-local (it takes the run's positions from kept_idx,
 * whose complement evicted_idx must be).  COATTN takes `target` as INPUT
 * (from selkv_route_coattn) instead of routing: a target outside the
 * token's own bucket counts as -1; the merge per kept slot runs over its
 * tokens in ascending order.
 * In:  K, V [B, H_kv, n, d]; attn, vnorm [B, H_kv, n] (from selkv_score);
 *      kept_idx, evicted_idx (from selkv_select).  Every kept token must
 *      have attn > 0.
 * Out: K_out, V_out [B, H_kv, m, d] (kv_dtype; row s is kept_idx[s]);
 *      target [B, H_kv, n - m] int32 kept slot or -1 (read, not written,
 *      under COATTN); gate [B, H_kv, n - m] fp32.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_MERGE, 0). */
SELKV_API selkv_status selkv_merge(const selkv_params* p, const void* K, const void* V, const float* attn,
                                   const float* vnorm, const int32_t* kept_idx, const int32_t* evicted_idx,
                                   void* K_out, void* V_out, int32_t* target, float* gate, void* ws,
                                   size_t ws_bytes, hipStream_t stream);

/* Step 6 of Algorithm 1: attention-ratio compensation (Sec. 3.6, Eq. 6).
 *
 * R_s = (a_i + sum_{j->s} g_j a_j) / a_i for kept slot s (position i), and
 * bias[s] = alpha * ln R_s, the per-KV-head logit bias that decode adds
 * (the per-head rule of Sec. 3.6).  R_s = 1 (bias exactly 0) where nothing
 * was absorbed.  With select_mode UNION (one kept set shared by the H_kv
 * heads of a cache, the GQA rule) R is averaged across those heads first:
 * bias[b, h, s] = alpha * ln(mean_h' R_{h', s}) for every h, the mean being
 * the fp32 sum of (R - 1) in head order divided by H_kv.
 * In:  attn [B, H_kv, n]; kept_idx, evicted_idx; target, gate (from
 *      selkv_merge with the same params: under BUCKET routing every routed
 *      token lies in its target's bucket, and under BUCKET_NEAREST in it
 *      or in the run of empty buckets beside it on the nearer side, which
 *      this call relies on; under COATTN a target outside the token's
 *      bucket counts as -1; under FULL_COSINE any target slot is allowed).
 * Out: bias [B, H_kv, m] fp32.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_BIAS, 0) (UNION adds the
 *      per-head ratios). */
SELKV_API selkv_status selkv_bias(const selkv_params* p, const float* attn, const int32_t* kept_idx,
                                  const int32_t* evicted_idx, const int32_t* target, const float* gate,
                                  float* bias, void* ws, size_t ws_bytes, hipStream_t stream);

/* Steps 3 to 6 of Algorithm 1 in one call: selkv_merge and selkv_bias
 * (Sec. 3.4 - 3.6, Eq. 3 - 6) with the same params, fused.
 *
 * The merge pass already forms, for every kept slot, the absorbed mass
 * sum_{j->s} g_j a_j that Eq. 5 divides by; it writes bias[s] = alpha * ln R_s
 * from that same sum, so attn, target and gate are not read back and the
 * bias pass over the evicted tokens disappears.  Outputs are bit for bit
 * those of selkv_merge followed by selkv_bias (both sum a slot's weights in
 * one fixed order).  Under UNION selection the per-head R - 1 go to the
 * workspace and one more small pass averages them over the heads of each
 * cache, as selkv_bias does.
 * In:  as selkv_merge (under COATTN routing, target from selkv_route_coattn).
 * Out: K_out, V_out, target, gate as selkv_merge; bias [B, H_kv, m] fp32 as
 *      selkv_bias.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_MERGE_BIAS, 0). */
SELKV_API selkv_status selkv_merge_bias(const selkv_params* p, const void* K, const void* V, const float* attn,
                                        const float* vnorm, const int32_t* kept_idx, const int32_t* evicted_idx,
                                        void* K_out, void* V_out, int32_t* target, float* gate, float* bias,
                                        void* ws, size_t ws_bytes, hipStream_t stream);

/* Step 7 of Algorithm 1: RoPE repositioning (Sec. 3.7,
 * Eq. 7; the paper leaves it off for long contexts).
 *
 * K~_s = RoPE(RoPE^-1(K_out[s], kept_idx[s]), s): the key in kept slot s
 * moves from its original position to the contiguous position s.  RoPE is
 * the rotate-half form: dimension j < d/2 pairs with j + d/2 and turns by
 * position * rope_theta^(-2j/d).  The two rotations are applied as one turn
 * by (s - kept_idx[s]) * rope_theta^(-2j/d), formed in fp64 and reduced
 * modulo one turn there; sine and cosine of the remainder are fp32;
 * rows already at their slot are left bit for bit.
 * In:  kept_idx [B, H_kv, m] (from selkv_select); rope_theta > 1 (10000 for
 *      Llama 2, 500000 for Llama 3).
 * In/out: K_out [B, H_kv, m, d] (kv_dtype, from selkv_merge), rewritten in place.
 * Workspace: none. */
SELKV_API selkv_status selkv_rope_reposition(const selkv_params* p, const int32_t* kept_idx, void* K_out,
                                             double rope_theta, hipStream_t stream);

/* Decode with the compressed cache (Sec. 3.1 last paragraph, Algorithm 1
 * "Decode with compressed cache + alpha log R bias").
 *
 * out[b, h] = sum_s softmax_s(scale * q[b, h] . K[b, h/G, s] + bias[b, h/G, s]) V[b, h/G, s]
 * over the cache_len entries of KV head h/G.  bias may be NULL (plain
 * attention, e.g. the uncompressed cache); a zero bias gives bitwise the
 * same result as NULL.  Split-K over the cache; a second kernel on the same
 * stream combines the splits in split order.
 * In:  q [B, H_kv*G, d] (kv_dtype); K, V [B, H_kv, cache_len, d] (kv_dtype);
 *      bias [B, H_kv, cache_len] fp32 or NULL.  Uses params batch,
 *      n_heads_kv, group (1..8), head_dim, kv_dtype and scale only.
 * Out: out [B, H_kv*G, d] fp32.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_DECODE, cache_len) bytes
 *      for the per-split partials; no initialisation is needed.  Calls that
 *      may overlap in time need separate workspaces. */
SELKV_API selkv_status selkv_decode_attn(const selkv_params* p, const void* q, const void* K, const void* V,
                                         const float* bias, int32_t cache_len, float* out, void* ws,
                                         size_t ws_bytes, hipStream_t stream);

/* selkv_decode_attn without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, kernels and
 * result as selkv_decode_attn; the split partials live in a fixed scratch
 * array of SELKV_NOALLOC_SCRATCH_BYTES that the library holds on each GPU
 * it runs on until the process ends.  The call allocates nothing: the
 * scratch address is looked up (hipGetSymbolAddress) on the first call on a
 * device, with that device current; the stream must belong to the current
 * device.  Every call on a GPU shares that GPU's scratch, so calls that may
 * overlap in time on one GPU (different streams, other threads) race and
 * must be serialised by the caller; the scratch needs no clearing between
 * calls.  Returns SELKV_EWORKSPACE when the shape's split partials exceed
 * the scratch (never while selkv_workspace_size(p, SELKV_CALL_DECODE,
 * cache_len) is within SELKV_NOALLOC_SCRATCH_BYTES: at most 256 KV heads of
 * any cache length, or about 4000 with G = 8 and d = 128), SELKV_EHIP if
 * the scratch address cannot be obtained. */
SELKV_API selkv_status selkv_decode_attn_noalloc(const selkv_params* p, const void* q, const void* K,
                                                 const void* V, const float* bias, int32_t cache_len, float* out,
                                                 hipStream_t stream);

/* One generation step over a cache that grows (the decode loop after
 * compression, Sec. 4.4): the step attends over the cache_len + 1 entries
 * exactly as selkv_decode_attn, the last one being the new token, whose
 * key and value it reads from k_new / v_new with bias 0 (a new token
 * absorbed nothing, so R = 1).  The same launch stores them at entry
 * cache_len of every KV head (and bias 0 there when bias is given) for the
 * later steps.
 * In:  q [B, H_kv*G, d]; k_new, v_new [B, H_kv, d] (kv_dtype; must not
 *      overlap the cache); 0 <= cache_len < capacity.
 * In/out: K, V [B, H_kv, capacity, d] (entries past cache_len + 1 are not
 *      read); bias [B, H_kv, capacity] fp32 or NULL.
 * Out: out [B, H_kv*G, d] fp32.
 * Workspace: selkv_workspace_size(p, SELKV_CALL_DECODE, capacity) covers every
 *      cache_len below capacity. */
SELKV_API selkv_status selkv_decode_append(const selkv_params* p, const void* q, const void* k_new,
                                           const void* v_new, void* K, void* V, float* bias, int32_t cache_len,
                                           int32_t capacity, float* out, void* ws, size_t ws_bytes,
                                           hipStream_t stream);

/* Static, NUL-terminated description of a status code. */
SELKV_API const char* selkv_status_string(selkv_status s);

/* SELKV_ABI_VERSION of the built library. */
SELKV_API int32_t selkv_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SELKV_H_ */
