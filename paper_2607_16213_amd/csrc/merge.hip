// selkv_merge, selkv_bias and selkv_merge_bias under the bucket routings: Sec. 3.4 - 3.6, Eq. 3 - 6.
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
//            bias = alpha * ln R (exactly 0 when nothing was absorbed); the
//            sums are taken in the merge's order, and the fused call
//            (selkv_merge_bias) has the merge wave write them directly
// Options: keys merged with the value weights (merge_keys), and the
// nearest-kept fallback, under which the waves of the non-empty buckets also
// absorb the runs of empty buckets beside them (still local, still ordered).
// The given-targets merge (co-attention routing) groups each bucket's
// entries by target slot instead of routing them itself.
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
// Each thread takes kOffSlots consecutive slots s (their kept positions and
// the one before them loaded together) and writes the starts of the buckets
// that begin after kept[s - 1] and at or before kept[s].
constexpr int kOffSlots = 4;

__global__ __launch_bounds__(kThreads) void bucket_offsets_kernel(const int32_t* kept, int32_t* offs, int m,
                                                                 int nb, int B) {
  const int64_t head = blockIdx.y;
  const int s0 = (blockIdx.x * blockDim.x + threadIdx.x) * kOffSlots;
  if (s0 > m) return;
  const int32_t* kh = kept + (size_t)head * m;
  int32_t* oh = offs + (size_t)head * (nb + 1);
  // positions outside [0, n) (a caller error) are clamped so writes stay in [0, nb];
  // loads are clamped to [0, m) and none is made when m = 0
  int bk[kOffSlots + 1];   // bucket of kept[s0 - 1 + u]; -1 before slot 0, nb at slot m
#pragma unroll
  for (int u = 0; u <= kOffSlots; ++u) {
    const int s = s0 - 1 + u;
    const int pos = m > 0 ? kh[min(max(s, 0), m - 1)] : 0;
    bk[u] = s < 0 ? -1 : s >= m ? nb : min(max(pos, 0) / B, nb);
  }
#pragma unroll
  for (int u = 0; u < kOffSlots; ++u) {
    const int s = s0 + u;
    if (s > m) break;
    for (int b = bk[u] + 1; b <= bk[u + 1]; ++b) oh[b] = s;
  }
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
  float* bias;      // fused Eq. 6 output per kept slot, or null
  int n, m, nb, B, gate_mode;
  float tau, inv_temp;
  float alpha;
  int raw;          // bias holds R - 1 (union mode) instead of alpha * ln R
};

// base[i] = v through a 32-bit byte offset from a wave-uniform base, which
// lets the store take its base from scalar registers (one offset VGPR
// instead of a 64-bit address pair).  Valid while i * 4 < 2^32: per-head
// arrays here hold at most seq_len < 2^28 entries.
template <typename T>
__device__ __forceinline__ void store_u32off(T* base, uint32_t i, T v) {
  *reinterpret_cast<T*>(reinterpret_cast<char*>(base) + i * (uint32_t)sizeof(T)) = v;
}

// Eq. 4 gate of a token whose value has dot product `dot` with its target's
// value: clamp((cos - tau) / T, 0, 1), the cosine 0 when a norm is 0; 0
// under DROP, 1 under MERGE_ALL.  The norm product is divided through the
// hardware reciprocal (within 2 ulp of the quotient), which keeps the IEEE
// division's temporaries out of the merge loops.
__device__ __forceinline__ float gate_of(const MergeArgs& a, float dot, float vn_j, float vn_t) {
  if (a.gate_mode == SELKV_GATE_MERGE_ALL) return 1.f;
  if (a.gate_mode != SELKV_GATE_COSINE) return 0.f;
  const float sim = (vn_j > 0.f && vn_t > 0.f) ? dot * __builtin_amdgcn_rcpf(vn_j * vn_t) : 0.f;
  return fminf(1.f, fmaxf(0.f, (sim - a.tau) * a.inv_temp));
}

// Nearest-kept fallback: the evicted tokens of the empty buckets between two
// non-empty ones all lie between the last kept token P before them and the
// first kept token Q after them, so they go to P up to floor((P + Q) / 2)
// (the lower one when equally near) and to Q beyond.  A run before the first
// or after the last non-empty bucket goes wholly to that bucket's outer kept
// token.  For the non-empty bucket [bstart, bend) with kept slots [k0, k1)
// this gives the evicted-index ranges it absorbs on either side:
// [eL0, eL1) into slot k0 (positions e + k0) and [eR0, eR1) into slot k1 - 1
// (positions e + k1); the ranges of neighbouring buckets meet exactly.
struct GapRuns {
  int eL0, eL1, eR0, eR1;
};

__device__ __forceinline__ GapRuns gap_runs(const int32_t* kh, int n, int m, int B, int bstart, int bend, int k0,
                                            int k1) {
  GapRuns r;
  int jL0 = 0;
  if (k0 > 0) {
    const int P = kh[k0 - 1], Q = kh[k0];
    jL0 = max((P / B + 1) * B, (int)(((int64_t)P + Q) / 2) + 1);
  }
  jL0 = min(max(jL0, 0), bstart);
  int jR1 = n;
  if (k1 < m) {
    const int P = kh[k1 - 1], Q = kh[k1];
    jR1 = min((Q / B) * B, (int)(((int64_t)P + Q) / 2) + 1);
  }
  jR1 = min(max(jR1, bend), n);
  // clamped so that an inconsistent kept list cannot leave [0, n - m)
  r.eL1 = bstart - k0;
  r.eL0 = min(max(jL0 - k0, 0), r.eL1);
  r.eR0 = bend - k1;
  r.eR1 = max(min(jR1 - k1, n - m), r.eR0);
  return r;
}

// Absorb the evicted entries [ea, eb) (positions e + shift, consecutive) into
// kept slot `slot` with value vt and norm vn_t: gate each by its value cosine
// with vt, accumulate g*a*v (and g*a*k under MK) in a fixed order, and write
// target and gate.  Wave-uniform trip counts; lane group q takes entries 4u + q.
template <typename T, int D, bool MK>
__device__ __forceinline__ void absorb_run(const MergeArgs& a, const char* Kh, const char* Vh, const float* ah,
                                           const float* vnh, int32_t* th, float* gh, int ea, int eb, int shift,
                                           int slot, const float (&vt)[Slice<T, D>::kElems], float vn_t,
                                           float (&acc)[Slice<T, D>::kElems],
                                           float (&kacc)[MK ? Slice<T, D>::kElems : 1], float& wsum, int lane,
                                           int grp, int col) {
  constexpr int E = Slice<T, D>::kElems;
  constexpr int RB = D * (int)sizeof(T);
  constexpr int kBatch = 4;
  for (int c0 = ea; c0 < eb; c0 += 64) {
    const int cnt = min(64, eb - c0);
    const int pos_l = c0 + shift + min(lane, cnt - 1);
    const float a_l = ah[pos_l], vn_l = vnh[pos_l];
    for (int ib0 = 0; ib0 < cnt; ib0 += 4 * kBatch) {
      int jj[kBatch];
      float ajv[kBatch], vnjv[kBatch];
      RawSlice<T, D> vr[kBatch], kre[MK ? kBatch : 1];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = ib0 + 4 * u + grp;
        const int src = i < cnt ? i : 0;
        jj[u] = c0 + shift + src;
        ajv[u] = __shfl(a_l, src, 64);
        vnjv[u] = __shfl(vn_l, src, 64);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) vr[u].load(Vh + (size_t)jj[u] * RB, col);
      if constexpr (MK) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) kre[u].load(Kh + (size_t)jj[u] * RB, col);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = ib0 + 4 * u + grp;
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) dot = fmaf(vr[u].get(e), vt[e], dot);
        dot = sum16(dot);
        const float g = gate_of(a, dot, vnjv[u], vn_t);
        if (i < cnt) {
          const float w = weight_rn(g, ajv[u]);
#pragma unroll
          for (int e = 0; e < E; ++e) acc[e] = fmaf(w, vr[u].get(e), acc[e]);
          if constexpr (MK) {
#pragma unroll
            for (int e = 0; e < E; ++e) kacc[e] = fmaf(w, kre[u].get(e), kacc[e]);
          }
          wsum += w;
          if (col == 0) {
            store_u32off(th, (uint32_t)(c0 + i), slot);
            store_u32off(gh, (uint32_t)(c0 + i), g);
          }
        }
      }
    }
  }
}

template <int N>
__device__ __forceinline__ void reduce_groups(float (&x)[N]) {
#pragma unroll
  for (int e = 0; e < N; ++e) {
    x[e] += xor_shfl(x[e], 16);
    x[e] += xor_shfl(x[e], 32);
  }
}

// MK: keys merged with the value weights (the merge_keys reading) instead of gathered.
// NR: nearest-kept fallback; a bucket that keeps no token is absorbed by its neighbours.
template <typename T, int D, bool MK, bool NR>
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
  if (NR && nk == 0) return;               // the neighbouring buckets absorb this one

  // lane-parallel metadata of the bucket: lane i holds kept entry i and evicted entry i
  int pos_k = 0, pos_e = 0;
  float a_k = kNegInf, a_e = 0.f, vn_e = 0.f;
  if (lane < nk) {
    pos_k = clamp_pos(kh[k0 + lane], n);
    a_k = ah[pos_k];
  }
  if (lane < ne) {
    pos_e = clamp_pos(eh[e0 + lane], n);
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

  float acc[E], kacc[MK ? E : 1];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
#pragma unroll
  for (int e = 0; e < (MK ? E : 1); ++e) kacc[e] = 0.f;
  float wsum = 0.f;
  // a bucket that keeps nothing (the wave agrees on tslot): its evicted tokens
  // go nowhere with gate 0 and their rows are not read
  if (tslot < 0 && lane < ne) {
    store_u32off(th, (uint32_t)(e0 + lane), -1);
    store_u32off(gh, (uint32_t)(e0 + lane), 0.f);
  }
  // evicted rows, kBatch per lane group with their loads issued together;
  // lane group q takes entries 4u + q (uniform trip count, masked)
  constexpr int kBatch = 4;
  for (int ib0 = 0; ib0 < (tslot >= 0 ? ne : 0); ib0 += 4 * kBatch) {
    int jj[kBatch];
    float ajv[kBatch], vnjv[kBatch];
    RawSlice<T, D> vr[kBatch], kre[MK ? kBatch : 1];
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
    if constexpr (MK) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) kre[u].load(Kh + (size_t)jj[u] * RB, col);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = ib0 + 4 * u + grp;
      const bool valid = i < ne;
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) dot = fmaf(vr[u].get(e), vt[e], dot);
      dot = sum16(dot);
      const float g = tslot >= 0 ? gate_of(a, dot, vnjv[u], vn_t) : 0.f;
      if (valid) {
        const float w = weight_rn(g, ajv[u]);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(w, vr[u].get(e), acc[e]);
        if constexpr (MK) {
#pragma unroll
          for (int e = 0; e < E; ++e) kacc[e] = fmaf(w, kre[u].get(e), kacc[e]);
        }
        wsum += w;
        if (col == 0) {
          store_u32off(th, (uint32_t)(e0 + i), tslot);
          store_u32off(gh, (uint32_t)(e0 + i), g);
        }
      }
    }
  }
  // nearest-kept fallback: the runs of empty buckets on either side
  constexpr int EN = NR ? E : 1, EK = NR && MK ? E : 1;
  float accf[EN], kaccf[EK], accl[EN], kaccl[EK];
  float wf = 0.f, wl = 0.f;
  if constexpr (NR) {
#pragma unroll
    for (int e = 0; e < E; ++e) accf[e] = accl[e] = 0.f;
#pragma unroll
    for (int e = 0; e < EK; ++e) kaccf[e] = kaccl[e] = 0.f;
    const GapRuns r = gap_runs(kh, n, m, a.B, start, end, k0, k1);
    const int pf = __shfl(pos_k, 0, 64), pl = __shfl(pos_k, nk - 1, 64);
    if (r.eL1 > r.eL0) {
      float vf[E];
      load_slice<T, D>(Vh + (size_t)pf * RB, col, vf);
      absorb_run<T, D, MK>(a, Kh, Vh, ah, vnh, th, gh, r.eL0, r.eL1, k0, k0, vf, vnh[pf], accf, kaccf, wf, lane, grp,
                           col);
    }
    if (r.eR1 > r.eR0) {
      float vl[E];
      load_slice<T, D>(Vh + (size_t)pl * RB, col, vl);
      absorb_run<T, D, MK>(a, Kh, Vh, ah, vnh, th, gh, r.eR0, r.eR1, k1, k1 - 1, vl, vnh[pl], accl, kaccl, wl, lane,
                           grp, col);
    }
  }

  // combine the four lane groups (fixed order)
  reduce_groups(acc);
  if constexpr (MK) reduce_groups(kacc);
  wsum += xor_shfl(wsum, 16);
  wsum += xor_shfl(wsum, 32);
  if constexpr (NR) {
    reduce_groups(accf);
    reduce_groups(accl);
    if constexpr (MK) {
      reduce_groups(kaccf);
      reduce_groups(kaccl);
    }
    wf += xor_shfl(wf, 16);
    wf += xor_shfl(wf, 32);
    wl += xor_shfl(wl, 16);
    wl += xor_shfl(wl, 32);
  }

  // the fused Eq. 6 bias: only the target slot (and, with the fallback, the
  // bucket's outer slots) absorbed anything, so the ratios are formed once
  // per wave, from the same sums the merged rows divide by; one coalesced
  // store of the bucket's nk <= 64 biases, ahead of the row loop
  if (a.bias != nullptr) {
    auto slot_w = [&](int k) {
      if constexpr (NR) return (k == tslot ? wsum : 0.f) + (k == k0 ? wf : 0.f) + (k == k1 - 1 ? wl : 0.f);
      else return k == tslot ? wsum : 0.f;
    };
    const bool raw = a.raw != 0;
    const float b_t = ratio_bias(slot_w(tslot), a_t, a.alpha, raw);
    float b_0 = 0.f, b_1 = 0.f;
    if constexpr (NR) {
      b_0 = ratio_bias(slot_w(k0), __shfl(a_k, 0, 64), a.alpha, raw);
      b_1 = ratio_bias(slot_w(k1 - 1), __shfl(a_k, nk - 1, 64), a.alpha, raw);
    }
    const int k = k0 + lane;
    if (lane < nk)
      a.bias[(size_t)head * m + k] = k == tslot ? b_t : (NR && k == k0) ? b_0 : (NR && k == k1 - 1) ? b_1 : 0.f;
  }

  // write the bucket's kept rows: keys gathered (or merged), values copied or merged;
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
    float akv[NR ? kBatch : 1];
    if constexpr (NR) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = kb0 + 4 * u + grp;
        akv[u] = __shfl(a_k, i < nk ? i : 0, 64);
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = kb0 + 4 * u + grp;
      if (i < nk) {
        const int k = k0 + i;
        if constexpr (NR) {
          // up to three sources: the bucket's own tokens, the left run, the right run
          const bool own = k == tslot, left = k == k0, right = k == k1 - 1;
          const float w = (own ? wsum : 0.f) + (left ? wf : 0.f) + (right ? wl : 0.f);
          if (w > 0.f) {
            const float ak = akv[u], den = ak + w;
            RawSlice<T, D> mv;
#pragma unroll
            for (int e = 0; e < E; ++e) {
              const float num = (own ? acc[e] : 0.f) + (left ? accf[e] : 0.f) + (right ? accl[e] : 0.f);
              mv.put(e, fmaf(ak, vr[u].get(e), num) / den);
            }
            mv.store(Vo + (size_t)k * RB, col);
            if constexpr (MK) {
              RawSlice<T, D> mk;
#pragma unroll
              for (int e = 0; e < E; ++e) {
                const float num = (own ? kacc[e] : 0.f) + (left ? kaccf[e] : 0.f) + (right ? kaccl[e] : 0.f);
                mk.put(e, fmaf(ak, kr[u].get(e), num) / den);
              }
              mk.store(Ko + (size_t)k * RB, col);
            } else {
              kr[u].store(Ko + (size_t)k * RB, col);
            }
          } else {
            kr[u].store(Ko + (size_t)k * RB, col);
            vr[u].store(Vo + (size_t)k * RB, col);
          }
        } else if (k == tslot && wsum > 0.f) {
          const float den = a_t + wsum;
          RawSlice<T, D> mv;
#pragma unroll
          for (int e = 0; e < E; ++e) mv.put(e, fmaf(a_t, vt[e], acc[e]) / den);
          mv.store(Vo + (size_t)k * RB, col);
          if constexpr (MK) {
            RawSlice<T, D> mk;
#pragma unroll
            for (int e = 0; e < E; ++e) mk.put(e, fmaf(a_t, kr[u].get(e), kacc[e]) / den);
            mk.store(Ko + (size_t)k * RB, col);
          } else {
            kr[u].store(Ko + (size_t)k * RB, col);
          }
        } else {
          kr[u].store(Ko + (size_t)k * RB, col);
          vr[u].store(Vo + (size_t)k * RB, col);
        }
      }
    }
  }
}

// Targets given (the co-attention routing): any kept slot of a bucket may
// absorb any of its evicted tokens.  One wave per bucket ranks the bucket's
// routed entries by (target, position), then merges one target slot at a
// time over its entries in ascending position, and copies the kept rows
// that absorbed nothing.  A target outside the token's bucket counts as -1.
template <typename T, int D, bool MK>
__global__ __launch_bounds__(kThreads) void merge_targets_kernel(MergeArgs a) {
  constexpr int E = Slice<T, D>::kElems;
  constexpr int RB = D * (int)sizeof(T);
  constexpr int kBatch = 4;
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
  const int32_t* th = a.target + (size_t)head * (n - m);
  float* gh = a.gate + (size_t)head * (n - m);

  const int start = bucket * a.B;
  const int end = min(n, start + a.B);
  const int k0 = oh[bucket], k1 = oh[bucket + 1];
  const int e0 = start - k0, e1 = end - k1;
  if (k0 > k1 || k1 > m || e0 < 0 || e0 > e1 || e1 > n - m) return;   // inconsistent kept list
  const int nk = k1 - k0, ne = e1 - e0;   // both <= B <= 64

  int pos_k = 0, pos_e = 0, t_e = -1;
  float a_k = 1.f, a_e = 0.f, vn_e = 0.f;
  if (lane < nk) {
    pos_k = clamp_pos(kh[k0 + lane], n);
    a_k = ah[pos_k];
  }
  if (lane < ne) {
    pos_e = clamp_pos(eh[e0 + lane], n);
    a_e = ah[pos_e];
    vn_e = vnh[pos_e];
    const int t = th[e0 + lane];
    t_e = (t >= k0 && t < k1) ? t : -1;
    if (t_e < 0) gh[e0 + lane] = 0.f;
  }
  const bool routed = t_e >= 0;
  // rank by (target, lane); unrouted lanes after every routed one
  // (routed lanes all lie below ne, so both loops stop there: a routed
  // lane's rank and the source of every rank below nrouted are exact)
  const int key = routed ? t_e : 0x7fffffff;
  int rank = 0;
  for (int q = 0; q < ne; ++q) {
    const int kq = __builtin_amdgcn_readlane(key, q);
    rank += (kq < key || (kq == key && q < lane)) ? 1 : 0;
  }
  int src = 0;   // the lane whose rank is this lane
  for (int q = 0; q < ne; ++q)
    if (__builtin_amdgcn_readlane(rank, q) == lane) src = q;
  const int nrouted = __popcll(__ballot(routed));
  const int s_t = __shfl(t_e, src, 64), s_pos = __shfl(pos_e, src, 64);
  const float s_a = __shfl(a_e, src, 64), s_vn = __shfl(vn_e, src, 64);
  const int prev_t = __shfl(s_t, lane > 0 ? lane - 1 : 0, 64);
  uint64_t heads = __ballot(lane < nrouted && (lane == 0 || prev_t != s_t));
  const int s_e = e0 + src;

  uint64_t written = 0;   // kept slots (bucket-relative) already stored
  while (heads) {         // one target slot per iteration, in ascending slot order
    const int s0 = __builtin_ctzll(heads);
    heads &= heads - 1;
    const int s1 = heads ? __builtin_ctzll(heads) : nrouted;
    const int k = __builtin_amdgcn_readlane(s_t, s0);
    const int ki = k - k0;
    const int tpos = __builtin_amdgcn_readlane(pos_k, ki);
    const float a_t = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(a_k), ki));
    float vt[E];
    load_slice<T, D>(Vh + (size_t)tpos * RB, col, vt);
    const float vn_t = vnh[tpos];
    float acc[E], kacc[MK ? E : 1];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
#pragma unroll
    for (int e = 0; e < (MK ? E : 1); ++e) kacc[e] = 0.f;
    float wsum = 0.f;
    for (int ib0 = s0; ib0 < s1; ib0 += 4 * kBatch) {
      int jj[kBatch], ev[kBatch];
      float ajv[kBatch], vnjv[kBatch];
      RawSlice<T, D> vr[kBatch], kre[MK ? kBatch : 1];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = ib0 + 4 * u + grp;
        const int sl = i < s1 ? i : s0;
        jj[u] = __shfl(s_pos, sl, 64);
        ajv[u] = __shfl(s_a, sl, 64);
        vnjv[u] = __shfl(s_vn, sl, 64);
        ev[u] = __shfl(s_e, sl, 64);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) vr[u].load(Vh + (size_t)jj[u] * RB, col);
      if constexpr (MK) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) kre[u].load(Kh + (size_t)jj[u] * RB, col);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = ib0 + 4 * u + grp;
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) dot = fmaf(vr[u].get(e), vt[e], dot);
        dot = sum16(dot);
        const float g = gate_of(a, dot, vnjv[u], vn_t);
        if (i < s1) {
          const float w = weight_rn(g, ajv[u]);
#pragma unroll
          for (int e = 0; e < E; ++e) acc[e] = fmaf(w, vr[u].get(e), acc[e]);
          if constexpr (MK) {
#pragma unroll
            for (int e = 0; e < E; ++e) kacc[e] = fmaf(w, kre[u].get(e), kacc[e]);
          }
          wsum += w;
          if (col == 0) store_u32off(gh, (uint32_t)ev[u], g);
        }
      }
    }
    reduce_groups(acc);
    if constexpr (MK) reduce_groups(kacc);
    wsum += xor_shfl(wsum, 16);
    wsum += xor_shfl(wsum, 32);
    if (grp == 0) {
      RawSlice<T, D> kr, vr;
      kr.load(Kh + (size_t)tpos * RB, col);
      vr.load(Vh + (size_t)tpos * RB, col);
      if (wsum > 0.f) {
        const float den = a_t + wsum;
        RawSlice<T, D> mv;
#pragma unroll
        for (int e = 0; e < E; ++e) mv.put(e, fmaf(a_t, vt[e], acc[e]) / den);
        mv.store(Vo + (size_t)k * RB, col);
        if constexpr (MK) {
          RawSlice<T, D> mk;
#pragma unroll
          for (int e = 0; e < E; ++e) mk.put(e, fmaf(a_t, kr.get(e), kacc[e]) / den);
          mk.store(Ko + (size_t)k * RB, col);
        } else {
          kr.store(Ko + (size_t)k * RB, col);
        }
      } else {
        kr.store(Ko + (size_t)k * RB, col);
        vr.store(Vo + (size_t)k * RB, col);
      }
      if (a.bias != nullptr && col == 0) a.bias[(size_t)head * m + k] = ratio_bias(wsum, a_t, a.alpha, a.raw != 0);
    }
    written |= 1ull << ki;
  }
  // the kept rows that absorbed nothing: copied bit for bit
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
      if (i < nk && !((written >> i) & 1ull)) {
        kr[u].store(Ko + (size_t)(k0 + i) * RB, col);
        vr[u].store(Vo + (size_t)(k0 + i) * RB, col);
        if (a.bias != nullptr && col == 0) a.bias[(size_t)head * m + k0 + i] = 0.f;
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

// Sum of g * a over a bucket's evicted entries routed to slot k (lane e holds
// entry e: its target t_e and contribution c_e, 0 past ne), in the order in
// which the merge kernels accumulate a slot's weights: one segment when, as
// bucket routing guarantees, every routed token of the bucket shares a
// target; otherwise the entries routed to k in ascending evicted order (the
// segment order of the given-targets merge).
__device__ __forceinline__ float bucket_mass(int t_e, float c_e, int k, int ne, int lane) {
  const int t0 = __shfl(t_e, 0, 64);
  if (__ballot(lane >= ne || t_e == t0) == ~0ull) {
    const float tot = seg_sum_total(seg_sum_add(0.f, c_e, lane));
    return k == t0 ? tot : 0.f;
  }
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  int r = 0;   // entries of k's segment so far
  for (int i = 0; i < ne; ++i) {
    const int t = __shfl(t_e, i, 64);
    const float c = __shfl(c_e, i, 64);
    if (t == k) {
      const int q = r & 3;
      if (q == 0) s0 += c;
      else if (q == 1) s1 += c;
      else if (q == 2) s2 += c;
      else s3 += c;
      ++r;
    }
  }
  return (s0 + s1) + (s2 + s3);
}

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
    j_e[bi] = has_e ? clamp_pos(eh[e0[bi] + lane], n) : 0;
    pos_k[bi] = has_k ? clamp_pos(kh[k0[bi] + lane], n) : 0;
  }
  float c_e[kBiasBuckets], a_k[kBiasBuckets];
#pragma unroll
  for (int bi = 0; bi < kBiasBuckets; ++bi) {
    c_e[bi] = weight_rn(g_e[bi], ah[j_e[bi]]);
    a_k[bi] = ah[pos_k[bi]];
  }
#pragma unroll
  for (int bi = 0; bi < kBiasBuckets; ++bi) {
    if (!ok[bi]) continue;                       // wave-uniform
    const int k = k0[bi] + lane;
    const float absorbed = bucket_mass(t_e[bi], c_e[bi], k, ne[bi], lane);
    if (k < k1[bi]) a.bias[(size_t)head * m + k] = ratio_bias(absorbed, a_k[bi], a.alpha, a.raw != 0);
  }
}

// Sum of g * a over the evicted entries [ea, eb) (positions e + shift) whose
// target is `slot`; the wave total, in a fixed order.
__device__ __forceinline__ float run_mass(const BiasArgs& a, const int32_t* th, const float* gh, const float* ah,
                                          int ea, int eb, int shift, int slot, int lane) {
  float s = 0.f;
  for (int c0 = ea; c0 < eb; c0 += 64) {
    const int e = c0 + lane;
    const float c = (e < eb && th[e] == slot) ? weight_rn(gh[e], ah[e + shift]) : 0.f;
    s = seg_sum_add(s, c, lane);
  }
  return seg_sum_total(s);
}

// Nearest-kept fallback: one wave per non-empty bucket adds to its kept
// slots the bucket's own routed tokens and, for its outer slots, the runs of
// empty buckets on either side (the split of the merge).
__global__ __launch_bounds__(kThreads) void bias_nearest_kernel(BiasArgs a) {
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
  const int start = bucket * a.B, end = min(n, start + a.B);
  const int k0 = oh[bucket], k1 = oh[bucket + 1];
  const int e0 = start - k0, e1 = end - k1;
  if (k0 >= k1 || k1 > m || e0 < 0 || e0 > e1 || e1 > n - m) return;   // empty bucket or inconsistent list
  const int nk = k1 - k0, ne = e1 - e0;
  const int t_e = lane < ne ? th[e0 + lane] : -1;
  const float c_e = lane < ne ? weight_rn(gh[e0 + lane], ah[clamp_pos(eh[e0 + lane], n)]) : 0.f;
  const float a_k = lane < nk ? ah[clamp_pos(kh[k0 + lane], n)] : 1.f;
  const int k = k0 + lane;
  // the merge's order: the bucket's own tokens, then the left run, then the right run
  float absorbed = bucket_mass(t_e, c_e, k, ne, lane);
  const GapRuns r = gap_runs(kh, n, m, a.B, start, end, k0, k1);
  const float left = run_mass(a, th, gh, ah, r.eL0, r.eL1, k0, k0, lane);
  const float right = run_mass(a, th, gh, ah, r.eR0, r.eR1, k1, k1 - 1, lane);
  if (k == k0) absorbed += left;
  if (k == k1 - 1) absorbed += right;
  if (lane < nk) a.bias[(size_t)head * m + k] = ratio_bias(absorbed, a_k, a.alpha, a.raw != 0);
}

}  // namespace

size_t bucket_offsets_bytes(const Shape& s) {
  return ((size_t)s.heads * (s.nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255;
}

hipError_t launch_bucket_offsets(const Shape& s, int bucket, const int32_t* kept, int32_t* offs, hipStream_t st) {
  const int per_block = kThreads * kOffSlots;
  const dim3 grid((s.m + 1 + per_block - 1) / per_block, (unsigned)s.heads);
  hipLaunchKernelGGL(bucket_offsets_kernel, grid, dim3(kThreads), 0, st, kept, offs, s.m, s.nb, bucket);
  return hipGetLastError();
}

hipError_t launch_merge_bucket(const Shape& s, int dtype, int bucket, int gate_mode, float tau, float temp,
                               const void* K, const void* V, const float* attn, const float* vnorm,
                               const int32_t* kept, const int32_t* evicted, const int32_t* offs, void* K_out,
                               void* V_out, int32_t* target, float* gate, bool merge_keys, bool nearest,
                               float* bias, float alpha, bool raw, hipStream_t st) {
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
  a.bias = bias;
  a.alpha = alpha;
  a.raw = raw ? 1 : 0;
  a.n = s.n;
  a.m = s.m;
  a.nb = s.nb;
  a.B = bucket;
  a.gate_mode = gate_mode;
  a.tau = tau;
  a.inv_temp = 1.f / temp;
  const dim3 grid((s.nb + kWavesPerBlock - 1) / kWavesPerBlock, (unsigned)s.heads);
#define SELKV_MB(T, D)                                                                                    \
  do {                                                                                                    \
    if (nearest) {                                                                                        \
      if (merge_keys) hipLaunchKernelGGL((merge_bucket_kernel<T, D, true, true>), grid, dim3(kThreads), 0, st, a); \
      else hipLaunchKernelGGL((merge_bucket_kernel<T, D, false, true>), grid, dim3(kThreads), 0, st, a);          \
    } else {                                                                                              \
      if (merge_keys) hipLaunchKernelGGL((merge_bucket_kernel<T, D, true, false>), grid, dim3(kThreads), 0, st, a); \
      else hipLaunchKernelGGL((merge_bucket_kernel<T, D, false, false>), grid, dim3(kThreads), 0, st, a);          \
    }                                                                                                     \
  } while (0)
  if (dtype == SELKV_BF16) {
    if (s.d == 128) SELKV_MB(bf16_t, 128);
    else SELKV_MB(bf16_t, 64);
  } else {
    if (s.d == 128) SELKV_MB(float, 128);
    else SELKV_MB(float, 64);
  }
#undef SELKV_MB
  return hipGetLastError();
}

hipError_t launch_merge_targets(const Shape& s, int dtype, int bucket, int gate_mode, float tau, float temp,
                                const void* K, const void* V, const float* attn, const float* vnorm,
                                const int32_t* kept, const int32_t* evicted, const int32_t* offs,
                                const int32_t* target, void* K_out, void* V_out, float* gate, bool merge_keys,
                                float* bias, float alpha, bool raw, hipStream_t st) {
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
  a.target = const_cast<int32_t*>(target);   // read only by this kernel
  a.gate = gate;
  a.bias = bias;
  a.alpha = alpha;
  a.raw = raw ? 1 : 0;
  a.n = s.n;
  a.m = s.m;
  a.nb = s.nb;
  a.B = bucket;
  a.gate_mode = gate_mode;
  a.tau = tau;
  a.inv_temp = 1.f / temp;
  const dim3 grid((s.nb + kWavesPerBlock - 1) / kWavesPerBlock, (unsigned)s.heads);
#define SELKV_MT(T, D)                                                                                  \
  do {                                                                                                  \
    if (merge_keys) hipLaunchKernelGGL((merge_targets_kernel<T, D, true>), grid, dim3(kThreads), 0, st, a); \
    else hipLaunchKernelGGL((merge_targets_kernel<T, D, false>), grid, dim3(kThreads), 0, st, a);           \
  } while (0)
  if (dtype == SELKV_BF16) {
    if (s.d == 128) SELKV_MT(bf16_t, 128);
    else SELKV_MT(bf16_t, 64);
  } else {
    if (s.d == 128) SELKV_MT(float, 128);
    else SELKV_MT(float, 64);
  }
#undef SELKV_MT
  return hipGetLastError();
}

hipError_t launch_bias_bucket(const Shape& s, int bucket, float alpha, const float* attn, const int32_t* kept,
                              const int32_t* evicted, const int32_t* offs, const int32_t* target,
                              const float* gate, float* bias, bool raw, bool nearest, hipStream_t st) {
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
  if (nearest) {
    const dim3 grid((s.nb + kWavesPerBlock - 1) / kWavesPerBlock, (unsigned)s.heads);
    hipLaunchKernelGGL(bias_nearest_kernel, grid, dim3(kThreads), 0, st, a);
    return hipGetLastError();
  }
  const int per_block = kWavesPerBlock * kBiasBuckets;
  const dim3 grid((s.nb + per_block - 1) / per_block, (unsigned)s.heads);
  hipLaunchKernelGGL(bias_bucket_kernel, grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace selkv
