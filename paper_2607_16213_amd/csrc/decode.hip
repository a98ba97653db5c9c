// selkv_decode_attn: one decode step over a (compressed) cache with the
// additive per-entry logit bias of Sec. 3.6 (alpha * ln R).
//
// Split-K flash-decode.  Work item = (sequence x KV head, chunk of entries);
// the G query heads of the KV head share every K/V load.  Inside a wave,
// lane group g = lane / 16 takes one cache entry and each of its 16 lanes a
// d/16-element slice, so one load instruction moves four consecutive rows
// (fully coalesced).  A wave handles 8 entries per lane group per step:
// logits (slice dot products reduced across the 16 lanes), + bias, in the
// log2 domain; then one running-max rescale per head per step.  The four
// lane groups and four waves are merged in a fixed order and every
// workgroup writes (max, sum, o[d]) per head to the workspace; a second
// kernel combines the chunks of each KV head in chunk order.  Deterministic.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kUnroll = 8;                       // entries per lane group per step
constexpr int kKeysPerStep = 4 * kUnroll;        // per wave
constexpr int kChunkQuant = kWaves * kKeysPerStep;   // 128
constexpr int kTargetBlocks = 2048;

template <typename T, int D>
struct Slice {
  static constexpr int kElems = D / 16;
  static constexpr int kBytes = kElems * (int)sizeof(T);
};

template <typename T, int D>
__device__ __forceinline__ void load_slice(const char* row, int col, float (&x)[Slice<T, D>::kElems]) {
  constexpr int B = Slice<T, D>::kBytes;
  const char* p = row + col * B;
  if constexpr (B >= 16) {
#pragma unroll
    for (int c = 0; c < B / 16; ++c) {
      const Chunk16 ch = load16(p + c * 16);
#pragma unroll
      for (int e = 0; e < Elem<T>::kPerChunk; ++e) x[c * Elem<T>::kPerChunk + e] = Elem<T>::get(ch, e);
    }
  } else {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    x[0] = __uint_as_float(v.x << 16);
    x[1] = __uint_as_float(v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.y << 16);
    x[3] = __uint_as_float(v.y & 0xffff0000u);
  }
}

struct DecodeArgs {
  const char* q;
  const char* K;
  const char* V;
  const float* bias;
  float* out;
  float* part;      // [heads, nsplit, G, D + 2]
  int L, chunk, nsplit;
  float c2;         // scale * log2(e)
};

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(DecodeArgs a) {
  constexpr int E = Slice<T, D>::kElems;
  constexpr int RB = D * (int)sizeof(T);
  const int split = blockIdx.x;
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int L = a.L;
  const char* Kh = a.K + (size_t)head * L * RB;
  const char* Vh = a.V + (size_t)head * L * RB;
  const float* bh = a.bias ? a.bias + (size_t)head * L : nullptr;

  float q[G][E];
#pragma unroll
  for (int g = 0; g < G; ++g) load_slice<T, D>(a.q + ((size_t)head * G + g) * RB, col, q[g]);

  float mrun[G], lrun[G], o[G][E];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    mrun[g] = kNegInf;
    lrun[g] = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) o[g][e] = 0.f;
  }

  const int kb = split * a.chunk;
  const int ke = min(L, kb + a.chunk);
  for (int base = kb + wave * kKeysPerStep; base < ke; base += kWaves * kKeysPerStep) {
    float x[kUnroll][G];
    float vv[kUnroll][E];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int key = base + u * 4 + grp;
      const bool valid = key < ke;
      float kk[E];
      if (valid) {
        load_slice<T, D>(Kh + (size_t)key * RB, col, kk);
        load_slice<T, D>(Vh + (size_t)key * RB, col, vv[u]);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) kk[e] = vv[u][e] = 0.f;
      }
      const float b2 = (valid && bh) ? bh[key] * kLog2e : 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) dot = fmaf(q[g][e], kk[e], dot);
        dot = sum16(dot);
        x[u][g] = valid ? fmaf(dot, a.c2, b2) : kNegInf;
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = x[0][g];
#pragma unroll
      for (int u = 1; u < kUnroll; ++u) mx = fmaxf(mx, x[u][g]);
      const float mnew = fmaxf(mrun[g], mx);
      if (mnew == kNegInf) continue;              // nothing valid yet for this group
      const float corr = fast_exp2(mrun[g] - mnew);   // 0 when mrun was -inf
      lrun[g] *= corr;
#pragma unroll
      for (int e = 0; e < E; ++e) o[g][e] *= corr;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const float p = fast_exp2(x[u][g] - mnew);   // 0 for invalid entries
        lrun[g] += p;
#pragma unroll
        for (int e = 0; e < E; ++e) o[g][e] = fmaf(p, vv[u][e], o[g][e]);
      }
      mrun[g] = mnew;
    }
  }

  // merge the four lane groups of the wave (xor 16, then xor 32)
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float m2 = xor_shfl(mrun[g], off);
      const float l2 = xor_shfl(lrun[g], off);
      const float M = fmaxf(mrun[g], m2);
      const float c1 = M == kNegInf ? 0.f : fast_exp2(mrun[g] - M);
      const float cb = M == kNegInf ? 0.f : fast_exp2(m2 - M);
      lrun[g] = lrun[g] * c1 + l2 * cb;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float o2 = xor_shfl(o[g][e], off);
        o[g][e] = o[g][e] * c1 + o2 * cb;
      }
      mrun[g] = M;
    }
  }

  // merge the four waves through LDS, in wave order
  __shared__ float s_m[kWaves][G], s_l[kWaves][G];
  __shared__ float s_o[kWaves][G][D];
  if (grp == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (col == 0) {
        s_m[wave][g] = mrun[g];
        s_l[wave][g] = lrun[g];
      }
#pragma unroll
      for (int e = 0; e < E; ++e) s_o[wave][g][col * E + e] = o[g][e];
    }
  }
  __syncthreads();
  float* part = a.part + ((size_t)head * a.nsplit + split) * G * (D + 2);
  for (int idx = threadIdx.x; idx < G * D; idx += kThreads) {
    const int g = idx / D, dd = idx % D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][g]);
    float l = 0.f, ov = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float c = fast_exp2(s_m[w][g] - M);
        l = fmaf(s_l[w][g], c, l);
        ov = fmaf(s_o[w][g][dd], c, ov);
      }
    }
    float* pg = part + (size_t)g * (D + 2);
    pg[2 + dd] = ov;
    if (dd == 0) {
      pg[0] = M;
      pg[1] = l;
    }
  }
}

// out[head*G + g][dd] = sum over chunks of o * 2^(m - M) / sum of l * 2^(m - M)
template <int D>
__global__ __launch_bounds__(kThreads) void decode_combine_kernel(const float* part, float* out, int nsplit, int G) {
  const int64_t head = blockIdx.x;
  for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
    const int g = idx / D, dd = idx % D;
    const float* p = part + (size_t)head * nsplit * G * (D + 2) + (size_t)g * (D + 2);
    const size_t stride = (size_t)G * (D + 2);
    float M = kNegInf;
    for (int s = 0; s < nsplit; ++s) M = fmaxf(M, p[s * stride]);
    float l = 0.f, ov = 0.f;
    for (int s = 0; s < nsplit; ++s) {
      const float ms = p[s * stride];
      if (ms == kNegInf) continue;
      const float c = fast_exp2(ms - M);
      l = fmaf(p[s * stride + 1], c, l);
      ov = fmaf(p[s * stride + 2 + dd], c, ov);
    }
    out[((size_t)head * G + g) * D + dd] = ov / l;
  }
}

template <typename T, int D, int G>
hipError_t launch_g(int64_t heads, const DecodePlan& p, DecodeArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((decode_split_kernel<T, D, G>), dim3(p.nsplit, (unsigned)heads), dim3(kThreads), 0, st, a);
  hipLaunchKernelGGL((decode_combine_kernel<D>), dim3((unsigned)heads), dim3(kThreads), 0, st, a.part, a.out,
                     p.nsplit, G);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_td(int64_t heads, int G, const DecodePlan& p, DecodeArgs& a, hipStream_t st) {
  switch (G) {
    case 1: return launch_g<T, D, 1>(heads, p, a, st);
    case 2: return launch_g<T, D, 2>(heads, p, a, st);
    case 3: return launch_g<T, D, 3>(heads, p, a, st);
    case 4: return launch_g<T, D, 4>(heads, p, a, st);
    case 5: return launch_g<T, D, 5>(heads, p, a, st);
    case 6: return launch_g<T, D, 6>(heads, p, a, st);
    case 7: return launch_g<T, D, 7>(heads, p, a, st);
    case 8: return launch_g<T, D, 8>(heads, p, a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

DecodePlan plan_decode(int64_t heads, int cache_len, int d, int G) {
  DecodePlan p{};
  int64_t ck = ((int64_t)cache_len * heads + kTargetBlocks - 1) / kTargetBlocks;
  ck = (ck + kChunkQuant - 1) / kChunkQuant * kChunkQuant;
  if (ck < kChunkQuant) ck = kChunkQuant;
  if (ck > 16384) ck = 16384;
  p.chunk = (int)ck;
  p.nsplit = (int)((cache_len + ck - 1) / ck);
  if (p.nsplit < 1) p.nsplit = 1;
  p.bytes = ((size_t)heads * p.nsplit * G * (d + 2) * sizeof(float) + 255) & ~(size_t)255;
  return p;
}

hipError_t launch_decode(int64_t heads, int n_heads_kv, int cache_len, int d, int G, int dtype, float scale,
                         const DecodePlan& p, const void* q, const void* K, const void* V, const float* bias,
                         float* out, void* ws, hipStream_t st) {
  (void)n_heads_kv;
  DecodeArgs a{};
  a.q = static_cast<const char*>(q);
  a.K = static_cast<const char*>(K);
  a.V = static_cast<const char*>(V);
  a.bias = bias;
  a.out = out;
  a.part = static_cast<float*>(ws);
  a.L = cache_len;
  a.chunk = p.chunk;
  a.nsplit = p.nsplit;
  a.c2 = scale * kLog2e;
  if (dtype == SELKV_BF16) {
    if (d == 128) return launch_td<bf16_t, 128>(heads, G, p, a, st);
    return launch_td<bf16_t, 64>(heads, G, p, a, st);
  }
  if (d == 128) return launch_td<float, 128>(heads, G, p, a, st);
  return launch_td<float, 64>(heads, G, p, a, st);
}

}  // namespace selkv
