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

// Lane slice of one row: d/16 elements of type T.
template <typename T, int D>
struct Slice {
  static constexpr int kElems = D / 16;
  static constexpr int kBytes = kElems * (int)sizeof(T);   // 8, 16 or 32
  static constexpr int kChunks = kBytes >= 16 ? kBytes / 16 : 1;
};

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

template <typename T, int D>
__device__ __forceinline__ void copy_slice(char* dst, const char* src, int col) {
  constexpr int B = Slice<T, D>::kBytes;
  if constexpr (B >= 16) {
#pragma unroll
    for (int c = 0; c < B / 16; ++c) store16(dst + col * B + c * 16, load16(src + col * B + c * 16));
  } else {
    *reinterpret_cast<uint2*>(dst + col * B) = *reinterpret_cast<const uint2*>(src + col * B);
  }
}

template <typename T, int D>
__device__ __forceinline__ void store_slice(char* row, int col, const float (&x)[Slice<T, D>::kElems]) {
  constexpr int B = Slice<T, D>::kBytes;
  char* p = row + col * B;
  if constexpr (B >= 16) {
#pragma unroll
    for (int c = 0; c < B / 16; ++c) {
      Chunk16 ch = zero16();
#pragma unroll
      for (int e = 0; e < Elem<T>::kPerChunk; ++e) Elem<T>::put(ch, e, x[c * Elem<T>::kPerChunk + e]);
      store16(p + c * 16, ch);
    }
  } else {
    uint2 v;
    v.x = (uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
    v.y = (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
    *reinterpret_cast<uint2*>(p) = v;
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
#pragma unroll 2
  for (int ib = 0; ib < ne; ib += 4) {     // uniform trip count; lane group q takes entry ib + q
    const int i = ib + grp;
    const bool valid = i < ne;
    const int src = valid ? i : 0;
    const int j = __shfl(pos_e, src, 64);
    const float aj = __shfl(a_e, src, 64);
    const float vnj = __shfl(vn_e, src, 64);
    float vj[E];
    if (valid) {
      load_slice<T, D>(Vh + (size_t)j * RB, col, vj);
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) vj[e] = 0.f;
    }
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) dot = fmaf(vj[e], vt[e], dot);
    dot = sum16(dot);
    float g = 0.f;
    if (tslot >= 0) {
      if (a.gate_mode == SELKV_GATE_MERGE_ALL) {
        g = 1.f;
      } else if (a.gate_mode == SELKV_GATE_COSINE) {
        const float sim = (vnj > 0.f && vn_t > 0.f) ? dot / (vnj * vn_t) : 0.f;
        g = fminf(1.f, fmaxf(0.f, (sim - a.tau) * a.inv_temp));
      }
    }
    if (valid) {
      const float w = g * aj;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(w, vj[e], acc[e]);
      wsum += w;
      if (col == 0) {
        th[e0 + i] = tslot;
        gh[e0 + i] = g;
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

  // write the bucket's kept rows: keys gathered, values copied or merged
  for (int kb = 0; kb < nk; kb += 4) {
    const int i = kb + grp;
    const int pos = __shfl(pos_k, i < nk ? i : 0, 64);
    if (i < nk) {
      const int k = k0 + i;
      copy_slice<T, D>(Ko + (size_t)k * RB, Kh + (size_t)pos * RB, col);
      if (k == tslot && wsum > 0.f) {
        const float den = a_t + wsum;
        float out[E];
#pragma unroll
        for (int e = 0; e < E; ++e) out[e] = fmaf(a_t, vt[e], acc[e]) / den;
        store_slice<T, D>(Vo + (size_t)k * RB, col, out);
      } else {
        copy_slice<T, D>(Vo + (size_t)k * RB, Vh + (size_t)pos * RB, col);
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
};

// One wave per bucket.  Lane e loads the bucket's e-th evicted entry and its
// contribution g * a (all loads in parallel); lane i then owns kept slot
// k0 + i and adds, in ascending evicted order, the contributions routed to it.
__global__ __launch_bounds__(kThreads) void bias_bucket_kernel(BiasArgs a) {
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int bucket = blockIdx.x * kWavesPerBlock + wave;
  if (bucket >= a.nb) return;
  const int n = a.n, m = a.m;
  const int32_t* kh = a.kept + (size_t)head * m;
  const int32_t* eh = a.evicted + (size_t)head * (n - m);
  const int32_t* th = a.target + (size_t)head * (n - m);
  const float* gh = a.gate + (size_t)head * (n - m);
  const int32_t* oh = a.offs + (size_t)head * (a.nb + 1);
  const float* ah = a.attn + (size_t)head * n;
  const int start = bucket * a.B;
  const int end = min(n, start + a.B);
  const int k0 = oh[bucket], k1 = oh[bucket + 1];
  const int e0 = start - k0, e1 = end - k1;
  if (k0 > k1 || k1 > m || e0 < 0 || e0 > e1 || e1 > n - m) return;   // inconsistent kept list
  const int ne = e1 - e0;
  int t_e = -1;
  float c_e = 0.f;
  if (lane < ne) {
    t_e = th[e0 + lane];
    c_e = gh[e0 + lane] * ah[eh[e0 + lane]];
  }
  const int k = k0 + lane;
  const float ai = lane < k1 - k0 ? ah[kh[k]] : 1.f;
  float absorbed = 0.f;
  for (int i = 0; i < ne; ++i) {
    const int t = __shfl(t_e, i, 64);
    const float c = __shfl(c_e, i, 64);
    if (t == k) absorbed += c;
  }
  if (k < k1) a.bias[(size_t)head * m + k] = absorbed > 0.f ? a.alpha * log1pf(absorbed / ai) : 0.f;
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
                              const float* gate, float* bias, hipStream_t st) {
  BiasArgs a{};
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
  const dim3 grid((s.nb + kWavesPerBlock - 1) / kWavesPerBlock, (unsigned)s.heads);
  hipLaunchKernelGGL(bias_bucket_kernel, grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace selkv
