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
// workgroup writes (max, sum, o[d]) per head to the workspace.  A second,
// small kernel (one workgroup per query head) combines the chunks of each
// head in chunk order.  The kernel boundary makes the partials visible: a
// cross-workgroup hand-off inside one kernel would need device-scope cache
// write-back / invalidate on every workgroup, and on a multi-XCD device that
// costs more than the second launch.  Deterministic.
// Appending (selkv_decode_append): the last entry is read from the caller's
// new key / value rows while the step runs, and the workgroup that owns it
// also stores those rows into the cache, so a generation step is one launch
// pair like any other decode step.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
#ifndef SELKV_DECODE_UNROLL
#define SELKV_DECODE_UNROLL 8
#endif
constexpr int kUnroll = SELKV_DECODE_UNROLL;     // entries per lane group per step
constexpr int kKeysPerStep = 4 * kUnroll;        // per wave
#ifndef SELKV_DECODE_TARGET_BLOCKS
#define SELKV_DECODE_TARGET_BLOCKS 256
#endif
constexpr int kTargetBlocks = SELKV_DECODE_TARGET_BLOCKS;   // workgroups per launch (one per CU)
constexpr int kMaxSplit = 1024;
constexpr int kReduceThreads = 256;   // 256 measured 0.4 - 0.6 us faster per call than 512 or 128

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

// Loads of one step: kUnroll entries per lane group, K and V slices and the bias.
template <typename T, int D, bool BIAS>
__device__ __forceinline__ void load_step(const char* Kh, const char* Vh, const float* bh, int base, int ke, int grp,
                                          int col, RawSlice<T, D> (&kr)[kUnroll], RawSlice<T, D> (&vr)[kUnroll],
                                          float (&br)[kUnroll]) {
  constexpr int RB = D * (int)sizeof(T);
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int key = base + u * 4 + grp;
    const int kc = key < ke ? key : ke - 1;
    kr[u].load(Kh + (size_t)kc * RB, col);
    vr[u].load(Vh + (size_t)kc * RB, col);
    if constexpr (BIAS) br[u] = bh[kc];
    else br[u] = 0.f;
  }
}

// Online-softmax update of the G heads with one loaded step.
template <typename T, int D, int G>
__device__ __forceinline__ void attend_step(const float (&q)[G][Slice<T, D>::kElems], float c2, int base, int ke,
                                            int grp, const RawSlice<T, D> (&kr)[kUnroll],
                                            const RawSlice<T, D> (&vr)[kUnroll], const float (&br)[kUnroll],
                                            float (&mrun)[G], float (&lrun)[G], float (&o)[G][Slice<T, D>::kElems]) {
  constexpr int E = Slice<T, D>::kElems;
  float x[kUnroll][G];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const bool valid = base + u * 4 + grp < ke;
    const float b2 = br[u] * kLog2e;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) dot = fmaf(q[g][e], kr[u].get(e), dot);
      dot = sum16(dot);
      x[u][g] = valid ? fmaf(dot, c2, b2) : kNegInf;
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
      const float p = fast_exp2(x[u][g] - mnew);   // 0 for masked entries
      lrun[g] += p;
#pragma unroll
      for (int e = 0; e < E; ++e) o[g][e] = fmaf(p, vr[u].get(e), o[g][e]);
    }
    mrun[g] = mnew;
  }
}

struct DecodeArgs {
  const char* q;
  const char* K;
  const char* V;
  const float* bias;
  float* out;
  float* part_o;    // [heads, nsplit, G, D]
  float2* part_ml;  // [heads, nsplit, G]: running max (log2 domain) and sum
  int L, chunk, nsplit;
  int stride;       // entries between consecutive heads in K, V and bias (>= L)
  float c2;         // scale * log2(e)
  // appended token (new_key = L - 1) or none (new_key = -1): its rows per
  // head in k_new / v_new; the workgroup holding it also stores them (and a
  // zero bias) into the cache through K_w / V_w / bias_w
  const char* k_new;
  const char* v_new;
  char* K_w;
  char* V_w;
  float* bias_w;
  int new_key;
};

// Store the appended token's rows (and bias 0) into the cache: wave 0 of the
// workgroup whose chunk holds it, at the end of the kernel.  Nothing else
// reads those cache rows in this launch (they are read from k_new / v_new).
template <int RB>
__device__ __forceinline__ void store_new_row(const DecodeArgs& a, int64_t head, int split, int wave, int lane) {
  if (a.new_key < 0 || split != a.new_key / a.chunk || wave != 0) return;
  const size_t row = (size_t)head * a.stride + a.new_key;
  for (int c = lane; c * 16 < RB; c += 64) {
    store16(a.K_w + row * RB + c * 16, load16(a.k_new + (size_t)head * RB + c * 16));
    store16(a.V_w + row * RB + c * 16, load16(a.v_new + (size_t)head * RB + c * 16));
  }
  if (a.bias_w && lane == 0) a.bias_w[row] = 0.f;
}

template <typename T, int D, int G, bool BIAS, bool APP>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(DecodeArgs a) {
  constexpr int E = Slice<T, D>::kElems;
  constexpr int RB = D * (int)sizeof(T);
  const int split = blockIdx.x;
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int L = a.L;
  const char* Kh = a.K + (size_t)head * a.stride * RB;
  const char* Vh = a.V + (size_t)head * a.stride * RB;
  const float* bh = BIAS ? a.bias + (size_t)head * a.stride : nullptr;

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
  // APP: the loop stops before the appended entry, which is taken below
  const int ke = min(APP ? a.new_key : L, kb + a.chunk);
  // two register buffers: the loads of the next step are in flight while
  // the current one is computed (rows past the chunk end re-read the last
  // row of the chunk and are masked, so no load sits behind a branch)
  RawSlice<T, D> kA[kUnroll], vA[kUnroll], kB[kUnroll], vB[kUnroll];
  float bA[kUnroll], bB[kUnroll];
  const int stride = kWaves * kKeysPerStep;
  int base = kb + wave * kKeysPerStep;
  if (base < ke) load_step<T, D, BIAS>(Kh, Vh, bh, base, ke, grp, col, kA, vA, bA);
  while (base < ke) {
    load_step<T, D, BIAS>(Kh, Vh, bh, base + stride, ke, grp, col, kB, vB, bB);
    attend_step<T, D, G>(q, a.c2, base, ke, grp, kA, vA, bA, mrun, lrun, o);
    base += stride;
    if (base >= ke) break;
    load_step<T, D, BIAS>(Kh, Vh, bh, base + stride, ke, grp, col, kA, vA, bA);
    attend_step<T, D, G>(q, a.c2, base, ke, grp, kB, vB, bB, mrun, lrun, o);
    base += stride;
  }
  // the appended entry: one masked step of wave 0 of the workgroup that owns
  // it, reading the caller's rows (bias 0)
  if (APP && wave == 0 && a.new_key >= kb && a.new_key < kb + a.chunk) {
    load_step<T, D, false>(a.k_new + (size_t)head * RB, a.v_new + (size_t)head * RB, nullptr, 0, 1, grp, col, kA, vA,
                           bA);
    attend_step<T, D, G>(q, a.c2, 0, 1, grp, kA, vA, bA, mrun, lrun, o);
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
  float* po = a.part_o + ((size_t)head * a.nsplit + split) * G * D;
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
    po[idx] = ov;
    if (dd == 0) a.part_ml[((size_t)head * a.nsplit + split) * G + g] = make_float2(M, l);
  }
  // after the streaming loop, so these stores never sit among its loads
  if constexpr (APP) store_new_row<RB>(a, head, split, wave, lane);

}

// bf16 variant with Q K^T on MFMA.  A wave step covers one 16-entry MFMA
// tile: Q (the G query rows, zero-padded to 16) is the A operand, the K tile
// the B operand, so lane (c, r) receives the logits of heads 4r .. 4r+3 for
// entry c.  The running max is kept wave-uniform per head (row-wise DPP max,
// then read into scalars), so every entry's probability shares one
// reference and the four lane groups sum without rescaling.  P V stays in
// fp32 on the VALU in the row-per-lane-group layout; lanes fetch the
// probabilities of their entries with ds_bpermute.  Two register buffers
// keep the next step's loads in flight during the current step's math.
template <int D>
struct Bf16Step {
  static constexpr int NCH = D * 2 / 64;
  Chunk16 kf[NCH];             // K tile, MFMA B layout
  RawSlice<bf16_t, D> vr[4];   // V rows base + 4u + r, lane-group layout
  float bias;                  // bias of entry base + c
};

template <int D, bool BIAS>
__device__ __forceinline__ void load_bf16_step(const char* Kh, const char* Vh, const float* bh, int base, int ke,
                                               int col, int grp, Bf16Step<D>& s) {
  constexpr int RB = D * 2;
  const int key = min(base + col, ke - 1);
#pragma unroll
  for (int c = 0; c < Bf16Step<D>::NCH; ++c) s.kf[c] = load16(Kh + (size_t)key * RB + (c * 4 + grp) * 16);
#pragma unroll
  for (int u = 0; u < 4; ++u) s.vr[u].load(Vh + (size_t)min(base + 4 * u + grp, ke - 1) * RB, col);
  if constexpr (BIAS) s.bias = bh[key];
  else s.bias = 0.f;
}

template <int D, int G>
__device__ __forceinline__ void attend_bf16_step(const Chunk16 (&qf)[Bf16Step<D>::NCH], float c2, int base, int ke,
                                                 int col, int grp, const Bf16Step<D>& s, float (&mrun)[G],
                                                 float (&lpart)[4], float (&o)[G][D / 16]) {
  constexpr int E = D / 16;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < Bf16Step<D>::NCH; ++c) acc = Mma<bf16_t>::step(qf[c], s.kf[c], acc);
  const bool valid = base + col < ke;
  float x[4], mrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[i] = valid ? fmaf(acc[i], c2, s.bias * kLog2e) : kNegInf;
    float v = x[i];
    v = fmaxf(v, row_ror<8>(v));
    v = fmaxf(v, row_ror<4>(v));
    v = fmaxf(v, row_ror<2>(v));
    v = fmaxf(v, row_ror<1>(v));
    mrow[i] = v;
  }
  float corr[G];
  bool moved = false;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float mstep = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mrow[g % 4]), 16 * (g / 4)));
    const float mnew = fmaxf(mrun[g], mstep);
    corr[g] = mnew == mrun[g] ? 1.f : fast_exp2(mrun[g] - mnew);   // 0 when mrun was -inf
    moved |= mnew != mrun[g];
    mrun[g] = mnew;
  }
  // probabilities in the MFMA layout: lane row r holds heads 4r + i
  float pb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float m_i = kNegInf, c_i = 1.f;
#pragma unroll
    for (int g = 0; g < G; ++g)
      if (g % 4 == i && grp == g / 4) {
        m_i = mrun[g];
        c_i = corr[g];
      }
    pb[i] = m_i == kNegInf ? 0.f : fast_exp2(x[i] - m_i);
    lpart[i] = fmaf(lpart[i], c_i, pb[i]);
  }
  if (moved) {   // wave-uniform: the running maxima are scalars
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < E; ++e) o[g][e] *= corr[g];
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int src = 4 * u + grp;          // MFMA column of this lane's entry
    float pg[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
      pg[g] = __int_as_float(__builtin_amdgcn_ds_bpermute((src + 16 * (g / 4)) * 4, __float_as_int(pb[g % 4])));
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const float vv = s.vr[u].get(e);
#pragma unroll
      for (int g = 0; g < G; ++g) o[g][e] = fmaf(pg[g], vv, o[g][e]);
    }
  }
}

template <int D, int G, bool BIAS, bool APP>
__global__ __launch_bounds__(kThreads) void decode_mfma_kernel(DecodeArgs a) {
  static_assert(G <= 8, "heads of a group live in lane rows 0 and 1");
  constexpr int NCH = Bf16Step<D>::NCH;
  constexpr int E = D / 16;
  constexpr int RB = D * 2;
  constexpr int KPS = 16;                  // entries per wave step
  const int split = blockIdx.x;
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int L = a.L;
  const char* Kh = a.K + (size_t)head * a.stride * RB;
  const char* Vh = a.V + (size_t)head * a.stride * RB;
  const float* bh = BIAS ? a.bias + (size_t)head * a.stride : nullptr;

  // Q as the MFMA A operand: lane (c, r) holds chunks 4j + r of query row c
  Chunk16 qf[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
    qf[c] = col < G ? load16(a.q + ((size_t)head * G + col) * RB + (c * 4 + grp) * 16) : zero16();

  float mrun[G], o[G][E], lpart[4];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    mrun[g] = kNegInf;
#pragma unroll
    for (int e = 0; e < E; ++e) o[g][e] = 0.f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) lpart[i] = 0.f;

  const int kb = split * a.chunk;
  // APP: the loop stops before the appended entry, which is taken below
  const int ke = min(APP ? a.new_key : L, kb + a.chunk);
  const int stride = kWaves * KPS;
  int base = kb + wave * KPS;
  Bf16Step<D> sA, sB;
  if (base < ke) load_bf16_step<D, BIAS>(Kh, Vh, bh, base, ke, col, grp, sA);
  while (base < ke) {
    load_bf16_step<D, BIAS>(Kh, Vh, bh, base + stride, ke, col, grp, sB);
    attend_bf16_step<D, G>(qf, a.c2, base, ke, col, grp, sA, mrun, lpart, o);
    base += stride;
    if (base >= ke) break;
    load_bf16_step<D, BIAS>(Kh, Vh, bh, base + stride, ke, col, grp, sA);
    attend_bf16_step<D, G>(qf, a.c2, base, ke, col, grp, sB, mrun, lpart, o);
    base += stride;
  }
  // the appended entry: one masked step of wave 0 of the workgroup that owns
  // it, reading the caller's rows (bias 0)
  if (APP && wave == 0 && a.new_key >= kb && a.new_key < kb + a.chunk) {
    load_bf16_step<D, false>(a.k_new + (size_t)head * RB, a.v_new + (size_t)head * RB, nullptr, 0, 1, col, grp, sA);
    attend_bf16_step<D, G>(qf, a.c2, 0, 1, col, grp, sA, mrun, lpart, o);
  }

  // l per head: sum the 16 columns of its lane row
  float lrun[G];
#pragma unroll
  for (int i = 0; i < 4; ++i) lpart[i] = sum16(lpart[i]);
#pragma unroll
  for (int g = 0; g < G; ++g)
    lrun[g] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lpart[g % 4]), 16 * (g / 4)));
  // the four lane groups share the reference max: plain sums
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      o[g][e] += xor_shfl(o[g][e], 16);
      o[g][e] += xor_shfl(o[g][e], 32);
    }

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
  float* po = a.part_o + ((size_t)head * a.nsplit + split) * G * D;
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
    po[idx] = ov;
    if (dd == 0) a.part_ml[((size_t)head * a.nsplit + split) * G + g] = make_float2(M, l);
  }
  // after the streaming loop, so these stores never sit among its loads
  if constexpr (APP) store_new_row<RB>(a, head, split, wave, lane);
}

// out[head * G + g] = sum over chunks of o * 2^(m - M) / sum of l * 2^(m - M),
// one workgroup per (KV head, query head of the group).  Thread (d, s) takes
// the chunks s, s + S, ... of output element d and loads their outputs and
// (max, sum) pairs together (one memory round trip for up to 16 chunks),
// merging them against its own running max; the S subsets are then merged
// in order through LDS.  The result is independent of scheduling.
template <int D>
__global__ __launch_bounds__(kReduceThreads) void decode_reduce_kernel(const float* part_o, const float2* part_ml,
                                                                       float* out, int nsplit, int G) {
  constexpr int S = kReduceThreads / D;   // chunk subsets per output element
  constexpr int kBatch = 16;
  const int64_t head = blockIdx.x;
  const int g = blockIdx.y;
  const int tid = threadIdx.x;
  const int dd = tid % D, sub = tid / D;
  __shared__ float s_m[S], s_l[S];
  __shared__ float s_o[S][D];
  const float2* ml = part_ml + (size_t)head * nsplit * G + g;
  const float* po = part_o + (size_t)head * nsplit * G * D + (size_t)g * D + dd;
  const size_t stride = (size_t)G * D;
  float m = kNegInf, acc = 0.f, lsum = 0.f;
  for (int sp0 = sub; sp0 < nsplit; sp0 += S * kBatch) {
    float ov[kBatch];
    float2 mlv[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int sp = min(sp0 + u * S, nsplit - 1);
      ov[u] = po[(size_t)sp * stride];
      mlv[u] = ml[(size_t)sp * G];
    }
    float mb = m;
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (sp0 + u * S < nsplit) mb = fmaxf(mb, mlv[u].x);
    if (mb == kNegInf) continue;
    const float c = fast_exp2(m - mb);     // 0 while m is -inf
    acc *= c;
    lsum *= c;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (sp0 + u * S < nsplit) {
        const float w = fast_exp2(mlv[u].x - mb);
        acc = fmaf(ov[u], w, acc);
        lsum = fmaf(mlv[u].y, w, lsum);
      }
    }
    m = mb;
  }
  s_o[sub][dd] = acc;
  if (dd == 0) {
    s_m[sub] = m;
    s_l[sub] = lsum;
  }
  __syncthreads();
  if (sub == 0) {
    float M = s_m[0];
#pragma unroll
    for (int k = 1; k < S; ++k) M = fmaxf(M, s_m[k]);
    float t = 0.f, L = 0.f;
#pragma unroll
    for (int k = 0; k < S; ++k) {
      const float w = s_m[k] == kNegInf ? 0.f : fast_exp2(s_m[k] - M);
      t = fmaf(s_o[k][dd], w, t);
      L = fmaf(s_l[k], w, L);
    }
    out[((size_t)head * G + g) * D + dd] = t / L;
  }
}

template <typename T, int D, int G>
hipError_t launch_g(int64_t heads, const DecodePlan& p, DecodeArgs& a, hipStream_t st) {
  const dim3 grid(p.nsplit, (unsigned)heads), blk(kThreads);
  const bool app = a.new_key >= 0;
  if constexpr (sizeof(T) == 2) {
    if (a.bias && app) hipLaunchKernelGGL((decode_mfma_kernel<D, G, true, true>), grid, blk, 0, st, a);
    else if (a.bias) hipLaunchKernelGGL((decode_mfma_kernel<D, G, true, false>), grid, blk, 0, st, a);
    else if (app) hipLaunchKernelGGL((decode_mfma_kernel<D, G, false, true>), grid, blk, 0, st, a);
    else hipLaunchKernelGGL((decode_mfma_kernel<D, G, false, false>), grid, blk, 0, st, a);
  } else {
    if (a.bias && app) hipLaunchKernelGGL((decode_split_kernel<T, D, G, true, true>), grid, blk, 0, st, a);
    else if (a.bias) hipLaunchKernelGGL((decode_split_kernel<T, D, G, true, false>), grid, blk, 0, st, a);
    else if (app) hipLaunchKernelGGL((decode_split_kernel<T, D, G, false, true>), grid, blk, 0, st, a);
    else hipLaunchKernelGGL((decode_split_kernel<T, D, G, false, false>), grid, blk, 0, st, a);
  }
  hipLaunchKernelGGL((decode_reduce_kernel<D>), dim3((unsigned)heads, G), dim3(kReduceThreads), 0, st, a.part_o,
                     a.part_ml, a.out, p.nsplit, G);
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
  int64_t nsplit = (kTargetBlocks + heads - 1) / heads;
  const int64_t max_split = (cache_len + kKeysPerStep - 1) / kKeysPerStep;
  if (nsplit > max_split) nsplit = max_split;
  if (nsplit > kMaxSplit) nsplit = kMaxSplit;
  if (nsplit < 1) nsplit = 1;
  int64_t ck = (cache_len + nsplit - 1) / nsplit;
  ck = (ck + kKeysPerStep - 1) / kKeysPerStep * kKeysPerStep;
  p.chunk = (int)ck;
  p.nsplit = (int)((cache_len + ck - 1) / ck);
  p.ml_bytes = ((size_t)heads * p.nsplit * G * sizeof(float2) + 255) & ~(size_t)255;
  p.bytes = p.ml_bytes + (((size_t)heads * p.nsplit * G * d * sizeof(float) + 255) & ~(size_t)255);
  return p;
}

// Workspace that covers plan_decode(heads, L, d, G) for every L <= capacity.
// Rounding the chunk up to whole steps can only lower the split count below
// min(ceil(kTargetBlocks / heads), ceil(L / kKeysPerStep), kMaxSplit), and
// that bound grows with L, so its value at L = capacity is the largest.
size_t decode_workspace_bound(int64_t heads, int capacity, int d, int G) {
  int64_t nsplit = (kTargetBlocks + heads - 1) / heads;
  const int64_t max_split = (capacity + kKeysPerStep - 1) / kKeysPerStep;
  if (nsplit > max_split) nsplit = max_split;
  if (nsplit > kMaxSplit) nsplit = kMaxSplit;
  if (nsplit < 1) nsplit = 1;
  const size_t ml = ((size_t)heads * nsplit * G * sizeof(float2) + 255) & ~(size_t)255;
  return ml + (((size_t)heads * nsplit * G * d * sizeof(float) + 255) & ~(size_t)255);
}

hipError_t launch_decode(int64_t heads, int n_heads_kv, int cache_len, int stride, int d, int G, int dtype,
                         float scale, const DecodePlan& p, const void* q, const void* K, const void* V,
                         const float* bias, float* out, void* ws, hipStream_t st, const void* k_new,
                         const void* v_new) {
  (void)n_heads_kv;
  DecodeArgs a{};
  if (k_new) {   // the last entry is appended by this step
    a.k_new = static_cast<const char*>(k_new);
    a.v_new = static_cast<const char*>(v_new);
    a.K_w = const_cast<char*>(static_cast<const char*>(K));
    a.V_w = const_cast<char*>(static_cast<const char*>(V));
    a.bias_w = const_cast<float*>(bias);
    a.new_key = cache_len - 1;
  } else {
    a.k_new = a.v_new = static_cast<const char*>(K);   // never selected: no entry has key -1
    a.new_key = -1;
  }
  a.stride = stride;
  a.q = static_cast<const char*>(q);
  a.K = static_cast<const char*>(K);
  a.V = static_cast<const char*>(V);
  a.bias = bias;
  a.out = out;
  a.part_ml = reinterpret_cast<float2*>(ws);
  a.part_o = reinterpret_cast<float*>(static_cast<char*>(ws) + p.ml_bytes);
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
