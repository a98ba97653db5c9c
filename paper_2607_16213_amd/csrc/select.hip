// selkv_select: per-head top-m_s selection of Sec. 3.3 (Eq. 2).
//
// One workgroup (16 waves) per KV head.  Scores are mapped to order-
// preserving 32-bit keys; a radix select finds the m_s-th largest key T and
// how many keys equal to T must be taken, on the offsets d = key - min key:
//   pass 0   the head's smallest and largest key above that of -inf, and
//            how many keys lie above it (-inf marks candidates that must not
//            be chosen; when fewer than m_s keys lie above, every key and
//            the whole key range are used instead)
//   pass 1   histogram of d >> s over 4096 LDS bins (integer atomics), s the
//            smallest shift that fits the head's key range into them, so
//            the bins span the scores actually present
//   pass 2   the keys of the bin holding T (a few hundred for the scores
//            the workloads produce) are copied into LDS, and the s low bits
//            are resolved there in passes of at most 10 bits; a bin too
//            large for LDS is resolved with global passes instead
// Scores that concentrate in a narrow range (the usual case) would otherwise
// put nearly every key of a head into one top-bits bin, one LDS counter.
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
constexpr int kLowBits = 10;      // bits per pass below the top bins
constexpr int kCandCap = 12288;   // keys of T's top bin held in LDS (48 KB)
// a key range of up to 2^32 - 1 fits the top bins at a shift of at most 20,
// which two low passes resolve
static_assert(kTopBits + 2 * kLowBits == 32, "two low passes cover the bits below the top bins");

constexpr uint32_t kNegInfKey = 0x007fffffu;   // order_key(-inf)

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

// Histogram of digit (d >> shift) & (nbins - 1), d = key - base, over the
// keys >= kfloor whose d matches prefix under mask: from the global scores
// (LDS_SRC false) or the staged offsets (which are d already, all admitted).
template <bool LDS_SRC>
__device__ void histogram(const float* s, const uint32_t* cand, int count, uint32_t kfloor, uint32_t base, int shift,
                          int nbins, uint32_t mask, uint32_t prefix, int* hist) {
  const int tid = threadIdx.x;
  for (int b = tid; b < nbins; b += kThreads) hist[b] = 0;
  __syncthreads();
  const uint32_t dmask = (uint32_t)nbins - 1u;
  if constexpr (LDS_SRC) {
    for (int j = tid; j < count; j += kThreads) {
      const uint32_t d = cand[j];
      if ((d & mask) == prefix) atomicAdd(&hist[(d >> shift) & dmask], 1);
    }
  } else {
    for (int j0 = tid; j0 < count; j0 += kThreads * kHistBatch) {
      float v[kHistBatch];
#pragma unroll
      for (int u = 0; u < kHistBatch; ++u) v[u] = s[min(j0 + u * kThreads, count - 1)];
#pragma unroll
      for (int u = 0; u < kHistBatch; ++u) {
        const uint32_t key = order_key(v[u]), d = key - base;
        if (j0 + u * kThreads < count && key >= kfloor && (d & mask) == prefix)
          atomicAdd(&hist[(d >> shift) & dmask], 1);
      }
    }
  }
  __syncthreads();
}

// Smallest and largest key above the key of -inf, and how many keys are
// above it, visible to every thread (lo > hi when there are none).
__device__ void key_range(const float* s, int count, uint32_t* red, uint32_t& kmin, uint32_t& kmax, int& above) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t lo = 0xffffffffu, hi = 0u;
  int c = 0;
  for (int j0 = tid; j0 < count; j0 += kThreads * kHistBatch) {
    float v[kHistBatch];
#pragma unroll
    for (int u = 0; u < kHistBatch; ++u) v[u] = s[min(j0 + u * kThreads, count - 1)];
#pragma unroll
    for (int u = 0; u < kHistBatch; ++u) {
      const uint32_t key = order_key(v[u]);
      if (j0 + u * kThreads < count && key > kNegInfKey) {
        lo = min(lo, key);
        hi = max(hi, key);
        ++c;
      }
    }
  }
  for (int o = 32; o >= 1; o >>= 1) {
    lo = min(lo, (uint32_t)__shfl_xor((int)lo, o, 64));
    hi = max(hi, (uint32_t)__shfl_xor((int)hi, o, 64));
    c += __shfl_xor(c, o, 64);
  }
  if (lane == 0) {
    red[wave] = lo;
    red[kWaves + wave] = hi;
    red[2 * kWaves + wave] = (uint32_t)c;
  }
  __syncthreads();
  lo = red[0];
  hi = red[kWaves];
  c = (int)red[2 * kWaves];
  for (int w = 1; w < kWaves; ++w) {
    lo = min(lo, red[w]);
    hi = max(hi, red[kWaves + w]);
    c += (int)red[2 * kWaves + w];
  }
  kmin = lo;
  kmax = hi;
  above = c;
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

  // ---- radix select of the ms-th largest key, on d = key - kmin
  __shared__ uint32_t red[3 * kWaves];
  uint32_t kmin = 0u, prefix = 0u, mask = 0u;
  int need = ms;
  if (ms > 0) {
    uint32_t kmax;
    int above;
    key_range(s, n_cand, red, kmin, kmax, above);
    // With at least ms keys above -inf the threshold is one of them: those
    // keys alone are binned (-inf marks what must not be chosen, e.g. the
    // non-members of the GQA union, and would stretch the range over the
    // whole key space).  Otherwise every key and the whole range are used.
    uint32_t kfloor = kNegInfKey + 1u;
    if (above < ms) {
      kfloor = 0u;
      kmin = 0u;
      kmax = 0xffffffffu;
    }
    int hi_bit = 0;   // the smallest shift that fits d into the top bins
    while (hi_bit < 32 && ((kmax - kmin) >> hi_bit) >= (uint32_t)kTopBins) ++hi_bit;
    histogram<false>(s, nullptr, n_cand, kfloor, kmin, hi_bit, kTopBins, 0u, 0u, hist);
    Pick pk = find_bin(hist, kTopBins, need, scan_lds, &sh_pick);
    prefix = pk.bin << hi_bit;
    mask = ~0u << hi_bit;
    need = pk.need;
    const bool staged = pk.count <= kCandCap;
    if (staged && hi_bit > 0) {
      // copy the bin's offsets into LDS (order is irrelevant to the threshold)
      if (tid == 0) sh_pos = 0;
      __syncthreads();
      for (int j0 = tid; j0 < n_cand; j0 += kThreads * kHistBatch) {
        float v[kHistBatch];
#pragma unroll
        for (int u = 0; u < kHistBatch; ++u) v[u] = s[min(j0 + u * kThreads, n_cand - 1)];
#pragma unroll
        for (int u = 0; u < kHistBatch; ++u) {
          const uint32_t key = order_key(v[u]), d = key - kmin;
          const bool hit = j0 + u * kThreads < n_cand && key >= kfloor && (d & mask) == prefix;
          const uint64_t bal = __ballot(hit);
          if (bal) {                              // wave-uniform
            int base = 0;
            if (lane == 0) base = atomicAdd(&sh_pos, __popcll(bal));
            base = __shfl(base, 0, 64);
            const int at = base + __popcll(bal & ((1ull << lane) - 1ull));
            if (hit && at < kCandCap) cand[at] = d;
          }
        }
      }
      __syncthreads();
    }
    // the hi_bit low bits of d, at most kLowBits per pass
    while (hi_bit > 0) {
      const int shift = hi_bit > kLowBits ? hi_bit - kLowBits : 0;
      const int nbins = 1 << (hi_bit - shift);
      if (staged) histogram<true>(nullptr, cand, pk.count, 0u, 0u, shift, nbins, mask, prefix, hist);
      else histogram<false>(s, nullptr, n_cand, kfloor, kmin, shift, nbins, mask, prefix, hist);
      const Pick q = find_bin(hist, nbins, need, scan_lds, &sh_pick);
      prefix |= q.bin << shift;
      mask |= ((uint32_t)nbins - 1u) << shift;
      need = q.need;
      hi_bit = shift;
    }
    prefix += kmin;   // the threshold key
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
