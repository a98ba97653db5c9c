// selkv_merge (BUCKET routing) and selkv_bias: Sec. 3.4 - 3.6, Eq. 3 - 6.
//
// Under bucket routing every evicted token and its target share one
// positional bucket of B <= 64 tokens, so one wave owns one bucket and the
// whole merge is local: no sort, no atomics, fixed summation order.
//   offsets  start[b] = number of kept positions < b*B (one pass over kept)
//   merge    per bucket: route (argmax attn over the bucket's kept tokens,
//            lowest position on ties), gate each evicted token by its value
//            cosine with the target, accumulate g*a*v in a fixed order,
//            write the merged target value, copy the other kept values and
//            gather every kept key
//   bias     per bucket: R = 1 + (sum over routed tokens of g*a) / a_i,
//            bias = alpha * ln R (exactly 0 when nothing was absorbed)
// Row layout of one wave: lane group g = lane / 16 takes one token (row) and
// each of its 16 lanes one contiguous slice of d/16 elements, so a wave
// instruction moves four consecutive rows.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / 64;

template <typename T, int D>
__device__ __forceinline__ void load_slice(const char* row, int col, float (&x)[Slice<T, D>::kElems]) {
  constexpr int E = Slice<T, D>::kElems;
  constexpr int B = Slice<T, D>::kBytes;
  const char* p = row + col * B;
  if constexpr (B >= 16) {
#pragma unroll
    for (int c = 0; c < B / 16; ++c) {
      const Chunk16 ch = load16(p + c * 16);
#pragma unroll
      for (int e = 0; e < Elem<T>::kPerChunk; ++e) x[c * Elem<T>::kPerChunk + e] = Elem<T>::get(ch, e);
    }
  } else {  // 8 bytes: four bf16
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    x[0] = __uint_as_float(v.x << 16);
    x[1] = __uint_as_float(v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.y << 16);
    x[3] = __uint_as_float(v.y & 0xffff0000u);
    static_assert(E == 4, "8-byte slices hold four bf16");
  }
}

// start[head][b] = lower_bound(kept, b * B) for b = 0 .. nb (start[nb] = m).
__global__ __launch_bounds__(kThreads) void bucket_offsets_kernel(const int32_t* kept, int32_t* offs, int m,
                                                                 int nb, int B) {
  const int64_t head = blockIdx.y;
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s > m) return;
  const int32_t* kh = kept + (size_t)head * m;
  int32_t* oh = offs + (size_t)head * (nb + 1);
  // positions outside [0, n) (a caller error) are clamped so writes stay in [0, nb]
  const int prev_b = s == 0 ? -1 : min(max(kh[s - 1], 0) / B, nb);
  const int cur_b = s == m ? nb : min(max(kh[s], 0) / B, nb);
  for (int b = prev_b + 1; b <= cur_b; ++b) oh[b] = s;
}

struct MergeArgs {
  const char* K;
  const char* V;
  const float* attn;
  const float* vnorm;
  const int32_t* kept;
  const int32_t* evicted;
  const int32_t* offs;
  char* K_out;
  char* V_out;
  int32_t* target;
  float* gate;
  int n, m, nb, B, gate_mode;
  float tau, inv_temp;
};

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void merge_bucket_kernel(MergeArgs a) {
  constexpr int E = Slice<T, D>::kElems;
  constexpr int RB = D * (int)sizeof(T);
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int bucket = blockIdx.x * kWavesPerBlock + wave;
  if (bucket >= a.nb) return;   // whole wave; no block barrier below

  const int n = a.n, m = a.m;
  const int32_t* kh = a.kept + (size_t)head * m;
  const int32_t* eh = a.evicted + (size_t)head * (n - m);
  const int32_t* oh = a.offs + (size_t)head * (a.nb + 1);
  const float* ah = a.attn + (size_t)head * n;
  const float* vnh = a.vnorm + (size_t)head * n;
  const char* Kh = a.K + (size_t)head * n * RB;
  const char* Vh = a.V + (size_t)head * n * RB;
  char* Ko = a.K_out + (size_t)head * m * RB;
  char* Vo = a.V_out + (size_t)head * m * RB;
  int32_t* th = a.target + (size_t)head * (n - m);
  float* gh = a.gate + (size_t)head * (n - m);

  const int start = bucket * a.B;
  const int end = min(n, start + a.B);
  const int k0 = oh[bucket], k1 = oh[bucket + 1];
  const int e0 = start - k0, e1 = end - k1;
  if (k0 > k1 || k1 > m || e0 < 0 || e0 > e1 || e1 > n - m) return;   // inconsistent kept list
  const int nk = k1 - k0, ne = e1 - e0;   // both <= B <= 64

  // lane-parallel metadata of the bucket: lane i holds kept entry i and evicted entry i
  int pos_k = 0, pos_e = 0;
  float a_k = kNegInf, a_e = 0.f, vn_e = 0.f;
  if (lane < nk) {
    pos_k = kh[k0 + lane];
    a_k = ah[pos_k];
  }
  if (lane < ne) {
    pos_e = eh[e0 + lane];
    a_e = ah[pos_e];
    vn_e = vnh[pos_e];
  }

  // route: kept token of the bucket with the largest attention, lowest slot on ties
  float best_a = a_k;
  int best = lane < nk ? lane : 0x7fffffff;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float oa = xor_shfl(best_a, off);
    const int ob = xor_shfl(best, off);
    if (oa > best_a || (oa == best_a && ob < best)) {
      best_a = oa;
      best = ob;
    }
  }
  const int tslot = nk > 0 ? k0 + best : -1;
  const int tpos = __shfl(pos_k, nk > 0 ? best : 0, 64);
  const float a_t = nk > 0 ? best_a : 0.f;

  float vt[E];
  float vn_t = 0.f;
  if (tslot >= 0) {
    load_slice<T, D>(Vh + (size_t)tpos * RB, col, vt);
    vn_t = vnh[tpos];
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) vt[e] = 0.f;
  }

  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  float wsum = 0.f;
  // evicted rows, kBatch per lane group with their loads issued together;
  // lane group q takes entries 4u + q (uniform trip count, masked)
  constexpr int kBatch = 4;
  for (int ib0 = 0; ib0 < ne; ib0 += 4 * kBatch) {
    int jj[kBatch];
    float ajv[kBatch], vnjv[kBatch];
    RawSlice<T, D> vr[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = ib0 + 4 * u + grp;
      const int src = i < ne ? i : 0;
      jj[u] = __shfl(pos_e, src, 64);
      ajv[u] = __shfl(a_e, src, 64);
      vnjv[u] = __shfl(vn_e, src, 64);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) vr[u].load(Vh + (size_t)jj[u] * RB, col);
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = ib0 + 4 * u + grp;
      const bool valid = i < ne;
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) dot = fmaf(vr[u].get(e), vt[e], dot);
      dot = sum16(dot);
      float g = 0.f;
      if (tslot >= 0) {
        if (a.gate_mode == SELKV_GATE_MERGE_ALL) {
          g = 1.f;
        } else if (a.gate_mode == SELKV_GATE_COSINE) {
          const float sim = (vnjv[u] > 0.f && vn_t > 0.f) ? dot / (vnjv[u] * vn_t) : 0.f;
          g = fminf(1.f, fmaxf(0.f, (sim - a.tau) * a.inv_temp));
        }
      }
      if (valid) {
        const float w = g * ajv[u];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(w, vr[u].get(e), acc[e]);
        wsum += w;
        if (col == 0) {
          th[e0 + i] = tslot;
          gh[e0 + i] = g;
        }
      }
    }
  }
  // combine the four lane groups (fixed order)
#pragma unroll
  for (int e = 0; e < E; ++e) {
    acc[e] += xor_shfl(acc[e], 16);
    acc[e] += xor_shfl(acc[e], 32);
  }
  wsum += xor_shfl(wsum, 16);
  wsum += xor_shfl(wsum, 32);

  // write the bucket's kept rows: keys gathered, values copied or merged;
  // kBatch rows per lane group loaded before any is stored
  for (int kb0 = 0; kb0 < nk; kb0 += 4 * kBatch) {
    RawSlice<T, D> kr[kBatch], vr[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = kb0 + 4 * u + grp;
      const int pos = __shfl(pos_k, i < nk ? i : 0, 64);
      kr[u].load(Kh + (size_t)pos * RB, col);
      vr[u].load(Vh + (size_t)pos * RB, col);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = kb0 + 4 * u + grp;
      if (i < nk) {
        const int k = k0 + i;
        kr[u].store(Ko + (size_t)k * RB, col);
        if (k == tslot && wsum > 0.f) {
          const float den = a_t + wsum;
          RawSlice<T, D> mv;
#pragma unroll
          for (int e = 0; e < E; ++e) mv.put(e, fmaf(a_t, vt[e], acc[e]) / den);
          mv.store(Vo + (size_t)k * RB, col);
        } else {
          vr[u].store(Vo + (size_t)k * RB, col);
        }
      }
    }
  }
}

struct BiasArgs {
  const float* attn;
  const int32_t* kept;
  const int32_t* evicted;
  const int32_t* offs;
  const int32_t* target;
  const float* gate;
  float* bias;
  int n, m, nb, B;
  float alpha;
  int raw;   // write absorbed / a (R - 1) instead of alpha * ln R
};

// One wave per kBiasBuckets consecutive buckets.  For each bucket lane e
// loads the e-th evicted entry and its contribution g * a, lane i the i-th
// kept slot; the loads of all the wave's buckets are issued level by level
// (offsets, then indices / targets / gates, then attention masses).  Lane i
// then adds the contributions routed to its slot (one wave sum when, as
// bucket routing guarantees, all routed tokens of the bucket share a target;
// otherwise in ascending evicted order): R = 1 + absorbed / a_i,
// bias = alpha * ln R (exactly 0 if nothing was absorbed).
constexpr int kBiasBuckets = 4;

__global__ __launch_bounds__(kThreads) void bias_bucket_kernel(BiasArgs a) {
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b0 = (blockIdx.x * kWavesPerBlock + wave) * kBiasBuckets;
  if (b0 >= a.nb) return;
  const int n = a.n, m = a.m;
  const int32_t* kh = a.kept + (size_t)head * m;
  const int32_t* eh = a.evicted + (size_t)head * (n - m);
  const int32_t* th = a.target + (size_t)head * (n - m);
  const float* gh = a.gate + (size_t)head * (n - m);
  const int32_t* oh = a.offs + (size_t)head * (a.nb + 1);
  const float* ah = a.attn + (size_t)head * n;

  const int offv = oh[min(b0 + lane, a.nb)];
  int k0[kBiasBuckets], k1[kBiasBuckets], e0[kBiasBuckets], ne[kBiasBuckets];
  bool ok[kBiasBuckets];
#pragma unroll
  for (int bi = 0; bi < kBiasBuckets; ++bi) {
    const int bucket = b0 + bi;
    k0[bi] = __shfl(offv, bi, 64);
    k1[bi] = __shfl(offv, bi + 1, 64);
    const int start = bucket * a.B;
    const int end = min(n, start + a.B);
    e0[bi] = start - k0[bi];
    const int e1 = end - k1[bi];
    ne[bi] = e1 - e0[bi];
    ok[bi] = bucket < a.nb && k0[bi] <= k1[bi] && k1[bi] <= m && e0[bi] >= 0 && e0[bi] <= e1 && e1 <= n - m;
  }
  int t_e[kBiasBuckets], j_e[kBiasBuckets], pos_k[kBiasBuckets];
  float g_e[kBiasBuckets];
#pragma unroll
  for (int bi = 0; bi < kBiasBuckets; ++bi) {
    const bool has_e = ok[bi] && lane < ne[bi];
    const bool has_k = ok[bi] && lane < k1[bi] - k0[bi];
    t_e[bi] = has_e ? th[e0[bi] + lane] : -1;
    g_e[bi] = has_e ? gh[e0[bi] + lane] : 0.f;
    j_e[bi] = has_e ? eh[e0[bi] + lane] : 0;
    pos_k[bi] = has_k ? kh[k0[bi] + lane] : 0;
  }
  float c_e[kBiasBuckets], a_k[kBiasBuckets];
#pragma unroll
  for (int bi = 0; bi < kBiasBuckets; ++bi) {
    c_e[bi] = g_e[bi] * ah[j_e[bi]];
    a_k[bi] = ah[pos_k[bi]];
  }
#pragma unroll
  for (int bi = 0; bi < kBiasBuckets; ++bi) {
    if (!ok[bi]) continue;                       // wave-uniform
    const int k = k0[bi] + lane;
    float absorbed = 0.f;
    // bucket routing sends every routed token of a bucket to one slot: then
    // one wave sum does; otherwise add per slot in ascending evicted order
    const int t0 = __shfl(t_e[bi], 0, 64);
    const bool same = __ballot(lane >= ne[bi] || t_e[bi] == t0) == ~0ull;
    if (same) {
      float tot = c_e[bi];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) tot += xor_shfl(tot, off);
      absorbed = (k == t0) ? tot : 0.f;
    } else {
      for (int i = 0; i < ne[bi]; ++i) {
        const int t = __shfl(t_e[bi], i, 64);
        const float c = __shfl(c_e[bi], i, 64);
        if (t == k) absorbed += c;
      }
    }
    if (k < k1[bi])
      a.bias[(size_t)head * m + k] =
          absorbed > 0.f ? (a.raw ? absorbed / a_k[bi] : a.alpha * log1pf(absorbed / a_k[bi])) : 0.f;
  }
}

}  // namespace

size_t bucket_offsets_bytes(const Shape& s) {
  return ((size_t)s.heads * (s.nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255;
}

hipError_t launch_bucket_offsets(const Shape& s, int bucket, const int32_t* kept, int32_t* offs, hipStream_t st) {
  const dim3 grid((s.m + 1 + kThreads - 1) / kThreads, (unsigned)s.heads);
  hipLaunchKernelGGL(bucket_offsets_kernel, grid, dim3(kThreads), 0, st, kept, offs, s.m, s.nb, bucket);
  return hipGetLastError();
}

hipError_t launch_merge_bucket(const Shape& s, int dtype, int bucket, int gate_mode, float tau, float temp,
                               const void* K, const void* V, const float* attn, const float* vnorm,
                               const int32_t* kept, const int32_t* evicted, const int32_t* offs, void* K_out,
                               void* V_out, int32_t* target, float* gate, hipStream_t st) {
  MergeArgs a{};
  a.K = static_cast<const char*>(K);
  a.V = static_cast<const char*>(V);
  a.attn = attn;
  a.vnorm = vnorm;
  a.kept = kept;
  a.evicted = evicted;
  a.offs = offs;
  a.K_out = static_cast<char*>(K_out);
  a.V_out = static_cast<char*>(V_out);
  a.target = target;
  a.gate = gate;
  a.n = s.n;
  a.m = s.m;
  a.nb = s.nb;
  a.B = bucket;
  a.gate_mode = gate_mode;
  a.tau = tau;
  a.inv_temp = 1.f / temp;
  const dim3 grid((s.nb + kWavesPerBlock - 1) / kWavesPerBlock, (unsigned)s.heads);
  if (dtype == SELKV_BF16) {
    if (s.d == 128)
      hipLaunchKernelGGL((merge_bucket_kernel<bf16_t, 128>), grid, dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL((merge_bucket_kernel<bf16_t, 64>), grid, dim3(kThreads), 0, st, a);
  } else {
    if (s.d == 128)
      hipLaunchKernelGGL((merge_bucket_kernel<float, 128>), grid, dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL((merge_bucket_kernel<float, 64>), grid, dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_bias_bucket(const Shape& s, int bucket, float alpha, const float* attn, const int32_t* kept,
                              const int32_t* evicted, const int32_t* offs, const int32_t* target,
                              const float* gate, float* bias, bool raw, hipStream_t st) {
  BiasArgs a{};
  a.raw = raw ? 1 : 0;
  a.attn = attn;
  a.kept = kept;
  a.evicted = evicted;
  a.offs = offs;
  a.target = target;
  a.gate = gate;
  a.bias = bias;
  a.n = s.n;
  a.m = s.m;
  a.nb = s.nb;
  a.B = bucket;
  a.alpha = alpha;
  const int per_block = kWavesPerBlock * kBiasBuckets;
  const dim3 grid((s.nb + per_block - 1) / per_block, (unsigned)s.heads);
  hipLaunchKernelGGL(bias_bucket_kernel, grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace selkv
