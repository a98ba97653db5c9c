// selkv_select: per-head top-m_s selection of Sec. 3.3 (Eq. 2).
//
// One workgroup (16 waves) per KV head.  Scores are mapped to order-
// preserving 32-bit keys; an MSB-first radix select finds the m_s-th largest
// key T and how many keys equal to T must be taken:
//   pass 1   histogram of the top 12 bits (4096 LDS bins, integer atomics)
//   pass 2   the keys of the bin holding T (a few percent of the head) are
//            copied into LDS, and the low 20 bits are resolved there in two
//            10-bit passes; a bin too large for LDS is resolved with two
//            more global passes instead
// A single ordered pass then keeps every key > T and the first `need` keys
// == T (lowest positions win ties), compacting kept and evicted positions in
// ascending order with one block prefix sum per 4096-key chunk.  The m_r'
// recent positions are appended to the kept list.  Outputs do not depend on
// scheduling: bitwise deterministic.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kPerThread = 4;                   // consecutive keys per thread in the compaction
constexpr int kChunk = kThreads * kPerThread;
static_assert(kChunk < 65536, "packed scan fields are 16 bits");
constexpr int kHistBatch = 16;    // score loads in flight per thread
constexpr int kTopBits = 12;
constexpr int kTopBins = 1 << kTopBits;
constexpr int kLowBits = 10;      // the two passes over the low 20 bits
constexpr int kCandCap = 12288;   // keys of T's top bin held in LDS (48 KB)
static_assert(kTopBits + 2 * kLowBits == 32, "the passes cover the 32-bit key");

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;  // -0 ranks with +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the block; `total` receives the block sum.
__device__ __forceinline__ int block_exclusive_scan(int v, int* lds_waves, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int incl = wave_inclusive_scan(v, lane);
  if (lane == 63) lds_waves[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int w = lane < kWaves ? lds_waves[lane] : 0;
    const int wi = wave_inclusive_scan(w, lane);
    if (lane < kWaves) lds_waves[kWaves + lane] = wi - w;   // exclusive wave offsets
    if (lane == kWaves - 1) lds_waves[2 * kWaves] = wi;
  }
  __syncthreads();
  const int r = lds_waves[kWaves + wave] + incl - v;
  total = lds_waves[2 * kWaves];
  __syncthreads();
  return r;
}

struct Pick {
  uint32_t bin;   // the digit of the need-th largest key
  int need;       // its rank among the keys of that bin
  int count;      // keys in that bin
};

// Walks the nbins bins from the top (thread t covers nbins / kThreads
// consecutive bins, or one) and finds the bin holding the need-th largest key.
__device__ Pick find_bin(const int* hist, int nbins, int need, int* scan_lds, Pick* sh) {
  const int tid = threadIdx.x;
  const int bpt = nbins > kThreads ? nbins / kThreads : 1;
  const int top = nbins - 1 - tid * bpt;   // this thread's highest bin
  int c = 0;
  for (int k = 0; k < bpt; ++k)
    if (top - k >= 0) c += hist[top - k];
  int total;
  const int excl = block_exclusive_scan(c, scan_lds, total);
  if (excl < need && excl + c >= need) {
    int cum = excl;
    for (int k = 0; k < bpt; ++k) {
      const int h = hist[top - k];
      if (cum + h >= need) {
        sh->bin = (uint32_t)(top - k);
        sh->need = need - cum;
        sh->count = h;
        break;
      }
      cum += h;
    }
  }
  __syncthreads();
  const Pick r = *sh;
  __syncthreads();
  return r;
}

// Histogram of digit (key >> shift) & (nbins - 1) over the keys matching
// prefix under mask: from the global scores (LDS_SRC false) or the staged keys.
template <bool LDS_SRC>
__device__ void histogram(const float* s, const uint32_t* cand, int count, int shift, int nbins, uint32_t mask,
                          uint32_t prefix, int* hist) {
  const int tid = threadIdx.x;
  for (int b = tid; b < nbins; b += kThreads) hist[b] = 0;
  __syncthreads();
  const uint32_t dmask = (uint32_t)nbins - 1u;
  if constexpr (LDS_SRC) {
    for (int j = tid; j < count; j += kThreads) {
      const uint32_t key = cand[j];
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1);
    }
  } else {
    for (int j0 = tid; j0 < count; j0 += kThreads * kHistBatch) {
      float v[kHistBatch];
#pragma unroll
      for (int u = 0; u < kHistBatch; ++u) v[u] = s[min(j0 + u * kThreads, count - 1)];
#pragma unroll
      for (int u = 0; u < kHistBatch; ++u) {
        const uint32_t key = order_key(v[u]);
        if (j0 + u * kThreads < count && (key & mask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1);
      }
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kThreads) void select_kernel(const float* score, int32_t* kept, int32_t* evicted,
                                                         int n, int n_cand, int m, int mr, int ms) {
  const int64_t head = blockIdx.x;
  const float* s = score + (size_t)head * n_cand;
  int32_t* kh = kept + (size_t)head * m;
  int32_t* eh = evicted + (size_t)head * (n - m);
  const int tid = threadIdx.x, lane = tid & 63;

  __shared__ int hist[kTopBins];
  __shared__ uint32_t cand[kCandCap];
  __shared__ int scan_lds[2 * kWaves + 1];
  __shared__ Pick sh_pick;
  __shared__ int sh_pos;

  // ---- radix select of the ms-th largest key
  uint32_t prefix = 0u, mask = 0u;
  int need = ms;
  if (ms > 0) {
    histogram<false>(s, nullptr, n_cand, 32 - kTopBits, kTopBins, 0u, 0u, hist);
    Pick pk = find_bin(hist, kTopBins, need, scan_lds, &sh_pick);
    prefix = pk.bin << (32 - kTopBits);
    mask = ~0u << (32 - kTopBits);
    need = pk.need;
    const bool staged = pk.count <= kCandCap;
    if (staged) {
      // copy the bin's keys into LDS (order is irrelevant to the threshold)
      if (tid == 0) sh_pos = 0;
      __syncthreads();
      for (int j0 = tid; j0 < n_cand; j0 += kThreads * kHistBatch) {
        float v[kHistBatch];
#pragma unroll
        for (int u = 0; u < kHistBatch; ++u) v[u] = s[min(j0 + u * kThreads, n_cand - 1)];
#pragma unroll
        for (int u = 0; u < kHistBatch; ++u) {
          const uint32_t key = order_key(v[u]);
          const bool hit = j0 + u * kThreads < n_cand && (key & mask) == prefix;
          const uint64_t bal = __ballot(hit);
          if (bal) {                              // wave-uniform
            int base = 0;
            if (lane == 0) base = atomicAdd(&sh_pos, __popcll(bal));
            base = __shfl(base, 0, 64);
            const int at = base + __popcll(bal & ((1ull << lane) - 1ull));
            if (hit && at < kCandCap) cand[at] = key;
          }
        }
      }
      __syncthreads();
    }
    for (int shift = 32 - kTopBits - kLowBits; shift >= 0; shift -= kLowBits) {
      if (staged) histogram<true>(nullptr, cand, pk.count, shift, 1 << kLowBits, mask, prefix, hist);
      else histogram<false>(s, nullptr, n_cand, shift, 1 << kLowBits, mask, prefix, hist);
      const Pick q = find_bin(hist, 1 << kLowBits, need, scan_lds, &sh_pick);
      prefix |= q.bin << shift;
      mask |= ((1u << kLowBits) - 1u) << shift;
      need = q.need;
    }
  } else {
    prefix = 0xffffffffu;  // nothing is strictly greater; take no ties
    need = 0;
  }
  const uint32_t T = prefix;

  // ---- ordered compaction: keep u > T, and the first `need` keys equal to T.
  // The kept list index of key j is (keys > T before j) + min(keys == T
  // before j, need), so one block scan of the packed (> T, == T) counts per
  // chunk places every key; its evicted index is j minus that.
  // The scores of chunk c + 1 are loaded before chunk c is scanned, so each
  // chunk's memory latency hides behind the previous chunk's scan.
  int run_gt = 0, run_eq = 0;
  float nxt[kPerThread];
  auto load_chunk = [&](int base) {
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) nxt[e] = s[min(base + tid * kPerThread + e, n_cand - 1)];   // clamped
  };
  if (n_cand > 0) load_chunk(0);
  for (int base = 0; base < n_cand; base += kChunk) {
    uint32_t u[kPerThread];
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) u[e] = order_key(nxt[e]);
    load_chunk(base + kChunk);   // past the end: re-reads the last score, unused
    int ngt = 0, neq = 0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int j = base + tid * kPerThread + e;
      ngt += (j < n_cand && u[e] > T) ? 1 : 0;
      neq += (j < n_cand && u[e] == T) ? 1 : 0;
    }
    int total;
    const int pre = block_exclusive_scan(ngt | (neq << 16), scan_lds, total);
    int gt_b = run_gt + (pre & 0xffff), eq_b = run_eq + (pre >> 16);
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int j = base + tid * kPerThread + e;
      if (j < n_cand) {
        const int kb = gt_b + min(eq_b, need);
        const bool keep = u[e] > T || (u[e] == T && eq_b < need);
        if (keep) {
          if (kb < ms) kh[kb] = j;
        } else if (j - kb < n - m) {
          eh[j - kb] = j;
        }
        gt_b += u[e] > T ? 1 : 0;
        eq_b += u[e] == T ? 1 : 0;
      }
    }
    run_gt += total & 0xffff;
    run_eq += total >> 16;
  }
  for (int r = tid; r < mr; r += kThreads) kh[ms + r] = n_cand + r;
}

}  // namespace

hipError_t launch_select(const Shape& s, const float* score, int32_t* kept, int32_t* evicted, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3((unsigned)s.heads), dim3(kThreads), 0, st, score, kept, evicted, s.n,
                     s.n_cand, s.m, s.mr, s.ms);
  return hipGetLastError();
}

}  // namespace selkv
