// Host-side launch plans and kernel launchers (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "selkv.h"

namespace selkv {

// Validated, derived sizes of one problem.
struct Shape {
  int64_t heads;     // batch * n_heads_kv
  int hkv;           // n_heads_kv (heads of one cache)
  int n, d, G, W, R; // R = G * W window rows per KV head
  int m, mr, ms;     // budget of Sec. 3.1
  int n_cand;        // n - mr
  int nb;            // number of routing buckets
};

// Score pass layout: key chunks per KV head and row groups.
struct ScorePlan {
  int chunk_keys;    // keys per workgroup (multiple of 64)
  int nchunks;       // chunks per KV head
  int rows_per_group;  // rows held in registers by one pass (16 * row blocks)
  int nrg;           // row groups
  int rpad;          // nrg * rows_per_group
  int tiled;         // 1: shared-tile passes (bf16, at most 128 window rows)
  int chunk_keys2;   // shared-tile pass 2: keys per workgroup (outputs staged in LDS)
  int nchunks2;      // shared-tile pass 2: chunks per KV head
  size_t part_off, stats_off, bytes;
};

struct DecodePlan {
  int chunk;            // keys per workgroup (multiple of 32)
  int nsplit;           // workgroups per KV head
  size_t ml_bytes;      // per-chunk (max, sum) partials, at the start of the workspace
  size_t bytes;
};

// Workspace of the grouping by target slot (full-cosine routing).
struct GroupPlan {
  size_t off_off, table_off, keys_off[2], vals_off[2], list_off, bytes;   // list: the last sort pass's values
  int passes;               // 8-bit radix passes over the keys 0 .. m
  int match_parts;          // runs the bf16 match splits the kept range into
  size_t match_slot_off;    // their per-run results: values at 0, slots at match_slot_off
  int match_mpad;           // bf16: rows per head of the gathered kept value block
  size_t match_vk_off, match_ik_off;   // the gathered block and its inverse norms
};

// Workspace of the GQA union mode: flags, mean keys and the shared set per
// cache for selection; the per-head R - 1 for the bias.
struct UnionPlan {
  size_t flag_off, key_off, kept_off, ev_off, select_bytes;
  size_t ratio_bytes;
};

ScorePlan plan_score(const Shape& s, int dtype);
UnionPlan plan_union(const Shape& s);
GroupPlan plan_group(const Shape& s, int dtype);
DecodePlan plan_decode(int64_t heads, int cache_len, int d, int G);
// bytes that cover plan_decode(heads, L, d, G).bytes for every L <= capacity
size_t decode_workspace_bound(int64_t heads, int capacity, int d, int G);
size_t bucket_offsets_bytes(const Shape& s);

// Launchers return hipSuccess or the launch error.
hipError_t launch_score(const Shape& s, const ScorePlan& plan, int dtype, float scale, const void* K,
                        const void* V, const void* Qwin, float* score, float* attn, float* vnorm,
                        int pool_kernel, void* ws, hipStream_t st);
hipError_t launch_select(const Shape& s, const float* score, int32_t* kept, int32_t* evicted, hipStream_t st);
hipError_t launch_bucket_offsets(const Shape& s, int bucket, const int32_t* kept, int32_t* offs, hipStream_t st);
hipError_t launch_merge_bucket(const Shape& s, int dtype, int bucket, int gate_mode, float tau, float temp,
                               const void* K, const void* V, const float* attn, const float* vnorm,
                               const int32_t* kept, const int32_t* evicted, const int32_t* offs, void* K_out,
                               void* V_out, int32_t* target, float* gate, bool merge_keys, bool nearest,
                               float* bias, float alpha, bool raw, hipStream_t st);
// bias (nullable): the fused Eq. 6 output per kept slot, alpha * ln R or (raw) R - 1
// targets given (co-attention routing): per bucket, grouped by target slot
hipError_t launch_merge_targets(const Shape& s, int dtype, int bucket, int gate_mode, float tau, float temp,
                                const void* K, const void* V, const float* attn, const float* vnorm,
                                const int32_t* kept, const int32_t* evicted, const int32_t* offs,
                                const int32_t* target, void* K_out, void* V_out, float* gate, bool merge_keys,
                                float* bias, float alpha, bool raw, hipStream_t st);
// score pass 1 and its combine only: the row statistics at plan.stats_off of ws
hipError_t launch_row_stats(const Shape& s, const ScorePlan& p, int dtype, float scale, const void* K,
                            const void* Qwin, void* ws, hipStream_t st);
hipError_t launch_coattn_route(const Shape& s, const ScorePlan& sp, int dtype, int bucket, int W, const void* K,
                               const void* Qwin, const void* score_ws, const int32_t* kept, const int32_t* offs,
                               int32_t* target, float c2, hipStream_t st);
// raw: write R - 1 = absorbed / a instead of alpha * ln R (the union mode averages it)
hipError_t launch_bias_bucket(const Shape& s, int bucket, float alpha, const float* attn, const int32_t* kept,
                              const int32_t* evicted, const int32_t* offs, const int32_t* target,
                              const float* gate, float* bias, bool raw, bool nearest, hipStream_t st);
// ws: the grouping workspace (plan gp); the per-run match results use it before the grouping does
hipError_t launch_cosine_match(const Shape& s, const GroupPlan& gp, int dtype, int gate_mode, float tau, float temp,
                               const void* V, const float* vnorm, const int32_t* kept, const int32_t* evicted,
                               int32_t* target, float* gate, void* ws, hipStream_t st);
hipError_t launch_group(const Shape& s, const GroupPlan& p, const int32_t* target, void* ws, hipStream_t st);
// values pass when V_out is set (bias, when also set, from the same sums); bias pass alone otherwise
hipError_t launch_group_merge(const Shape& s, const GroupPlan& p, int dtype, const void* K, const void* V,
                              const float* attn, const int32_t* kept, const int32_t* evicted, const float* gate,
                              void* ws, void* K_out, void* V_out, float* bias, float alpha, bool raw,
                              bool merge_keys, hipStream_t st);
hipError_t launch_union_select(const Shape& s, const UnionPlan& p, const float* score, int32_t* kept,
                               int32_t* evicted, void* ws, hipStream_t st);
hipError_t launch_union_bias(const Shape& s, const float* r1, float* bias, float alpha, hipStream_t st);
hipError_t launch_rope_reposition(const Shape& s, int dtype, const int32_t* kept, void* K_out, double theta,
                                  hipStream_t st);
// cache_len valid entries per head, `stride` entries apart in memory (stride >= cache_len).
// With k_new / v_new the last entry (cache_len - 1) is read from them (bias 0)
// and stored into K, V (and bias, if any) by the same launch.
hipError_t launch_decode(int64_t heads, int n_heads_kv, int cache_len, int stride, int d, int G, int dtype,
                         float scale, const DecodePlan& plan, const void* q, const void* K, const void* V,
                         const float* bias, float* out, void* ws, hipStream_t st, const void* k_new = nullptr,
                         const void* v_new = nullptr);

}  // namespace selkv
