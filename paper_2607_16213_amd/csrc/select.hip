// selkv_select: per-head top-m_s selection of Sec. 3.3 (Eq. 2).
//
// One workgroup (16 waves) per KV head.  Scores are mapped to order-
// preserving 32-bit keys; the kernel finds the m_s-th largest key T and how
// many keys equal to T must be taken (`need`), then compacts.
//
// Threshold, usual path (two reads of the scores in all):
//   sample   4096 keys at evenly spaced positions; a histogram of the
//            sampled keys above -inf over their own key range gives a band of
//            keys around the sample rank where T is expected (128 sample
//            ranks on either side)
//   band     one pass over the scores: keys above the band are counted per
//            wave, keys inside it are staged in LDS with their positions
//   resolve  when T lies inside the band and the band fits in LDS (nearly
//            always), T and `need` are resolved among the staged keys by LDS
//            radix passes, and the staged keys complete the per-wave counts
// Heads of at most 12288 candidates stage every key and skip the sample.
// Otherwise (a band that misses T or overflows, e.g. very many equal keys):
//   pass 0   the head's smallest and largest key above that of -inf, and
//            how many keys lie above it (-inf marks candidates that must not
//            be chosen; when fewer than m_s keys lie above, every key and
//            the whole key range are used instead)
//   pass 1   histogram of d >> s over 4096 LDS bins (integer atomics), d the
//            offset from the smallest key and s the smallest shift that fits
//            the key range into them, so the bins span the scores present
//   pass 2   the keys of the bin holding T are copied into LDS and the s low
//            bits are resolved there in passes of at most 10 bits; a bin too
//            large for LDS is resolved with global passes instead
//   count    each wave counts its segment's keys > T and == T
// Either way the result is the exact m_s-th largest key: the paths differ
// only in cost.  Compaction: wave w owns one contiguous segment of the
// candidates; the per-wave counts are prefixed once, and each wave walks its
// segment keeping every key > T and the first `need` keys == T (lowest
// positions win ties), ranking its keys with ballots, so kept and evicted
// positions come out ascending with no barrier inside the walk.  The m_r'
// recent positions are appended to the kept list.  Outputs do not depend on
// scheduling: bitwise deterministic.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kIter = 256;        // keys of one wave step (four per lane: positions e * 64 + lane)
constexpr int kRing = 8;          // wave steps whose loads are in flight together
constexpr int kSample = 4096;     // sampled keys (four per thread)
constexpr int kBandRanks = 128;   // sample ranks on either side of T's expected rank
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

// Block-wide min / max / sum of the per-thread partial ranges, visible to
// every thread.
__device__ void reduce_range(uint32_t lo, uint32_t hi, int c, uint32_t* red, uint32_t& kmin, uint32_t& kmax,
                             int& count) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
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
  count = c;
  __syncthreads();
}

// Smallest and largest key above the key of -inf, and how many keys are
// above it, visible to every thread (lo > hi when there are none).
__device__ void key_range(const float* s, int count, uint32_t* red, uint32_t& kmin, uint32_t& kmax, int& above) {
  const int tid = threadIdx.x;
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
  reduce_range(lo, hi, c, red, kmin, kmax, above);
}

// The smallest shift that fits the key range [kmin, kmax] into the top bins.
__device__ __forceinline__ int top_shift(uint32_t kmin, uint32_t kmax) {
  int hb = 0;
  while (hb < 32 && ((kmax - kmin) >> hb) >= (uint32_t)kTopBins) ++hb;
  return hb;
}

// Walks the wave's segment [begin, end) of the scores: step t holds
// positions begin + t * kIter + e * 64 + lane (e = 0 .. 3), so every load
// instruction reads 256 contiguous bytes and the keys of a step ascend in
// (e, lane) order.  The loads of kRing steps are issued together, the next
// group's before the current group is handled.  f(t, v) gets the lane's four
// scores of step t; reads past the end are clamped (the caller masks them by
// position).
template <class F>
__device__ __forceinline__ void walk_segment(const float* s, int begin, int end, F&& f) {
  const int lane = threadIdx.x & 63;
  const int steps = (end - begin + kIter - 1) / kIter;
  if (steps <= 0) return;
  float cur[kRing][4], nxt[kRing][4];
  auto load = [&](float (&v)[kRing][4], int g) {
#pragma unroll
    for (int r = 0; r < kRing; ++r)
#pragma unroll
      for (int e = 0; e < 4; ++e) v[r][e] = s[min(begin + (g + r) * kIter + e * 64 + lane, end - 1)];
  };
  load(cur, 0);
  for (int g = 0; g < steps; g += kRing) {
    if (g + kRing < steps) load(nxt, g + kRing);
#pragma unroll
    for (int r = 0; r < kRing; ++r)
      if (g + r < steps) f(g + r, cur[r]);
#pragma unroll
    for (int r = 0; r < kRing; ++r)
#pragma unroll
      for (int e = 0; e < 4; ++e) cur[r][e] = nxt[r][e];
  }
}

// Resolves the need-th largest of the staged offsets cand[0 .. count) whose
// values lie in [0, 2^32): the offset itself, and `need` becomes its rank
// among the offsets equal to it.
__device__ uint32_t resolve_staged(const uint32_t* cand, int count, uint32_t dmax, int& need, int* hist, int* scan_lds,
                                   Pick* sh) {
  int hb = top_shift(0u, dmax);
  histogram<true>(nullptr, cand, count, 0u, 0u, hb, kTopBins, 0u, 0u, hist);
  const Pick pk = find_bin(hist, kTopBins, need, scan_lds, sh);
  uint32_t prefix = pk.bin << hb;
  uint32_t mask = hb >= 32 ? 0u : ~0u << hb;
  need = pk.need;
  while (hb > 0) {
    const int shift = hb > kLowBits ? hb - kLowBits : 0;
    const int nbins = 1 << (hb - shift);
    histogram<true>(nullptr, cand, count, 0u, 0u, shift, nbins, mask, prefix, hist);
    const Pick q = find_bin(hist, nbins, need, scan_lds, sh);
    prefix |= q.bin << shift;
    mask |= ((uint32_t)nbins - 1u) << shift;
    need = q.need;
    hb = shift;
  }
  return prefix;
}

__global__ __launch_bounds__(kThreads) void select_kernel(const float* score, int32_t* kept, int32_t* evicted,
                                                         int n, int n_cand, int m, int mr, int ms) {
  const int64_t head = blockIdx.x;
  const float* s = score + (size_t)head * n_cand;
  int32_t* kh = kept + (size_t)head * m;
  int32_t* eh = evicted + (size_t)head * (n - m);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t below = (1ull << lane) - 1ull;

  __shared__ int hist[kTopBins];
  __shared__ uint32_t cand[kCandCap];   // staged key offsets (the sample first)
  __shared__ int cpos[kCandCap];        // their positions (band path)
  __shared__ int scan_lds[2 * kWaves + 1];
  __shared__ uint32_t red[3 * kWaves];
  __shared__ int wgt[kWaves], weq[kWaves];   // per wave: keys > T, keys == T in its segment
  __shared__ Pick sh_pick;
  __shared__ int sh_pos;

  // wave w owns candidates [w * seg, (w + 1) * seg)
  const int seg = (n_cand + kWaves * kIter - 1) / (kWaves * kIter) * kIter;
  const int wb = min(wave * seg, n_cand), we = min(wb + seg, n_cand);
  if (tid < kWaves) {
    wgt[tid] = 0;
    weq[tid] = 0;
  }

  uint32_t T = 0xffffffffu;   // ms == 0: nothing is strictly greater, and no ties are taken
  int need = 0;
  if (ms > 0) {
    // ---- the band [lo, hi) of keys around T's expected place (hi = 2^32: no key above)
    uint32_t lo = 0u;
    uint64_t hi = 1ull << 32;
    if (n_cand > kCandCap) {
      // the sample's keys above -inf span the bins (-inf ranks below them
      // all and would stretch the range over the whole key space)
      uint32_t smin = 0xffffffffu, smax = 0u;
      int fin = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = tid * 4 + e;
        const uint32_t key = order_key(s[(int)(((int64_t)i * n_cand) / kSample)]);
        cand[i] = key;
        if (key > kNegInfKey) {
          smin = min(smin, key);
          smax = max(smax, key);
          ++fin;
        }
      }
      reduce_range(smin, smax, fin, red, smin, smax, fin);   // its barriers also publish the sample
      if (fin > 0) {
        const int sh = top_shift(smin, smax);
        for (int b = tid; b < kTopBins; b += kThreads) hist[b] = 0;
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t key = cand[tid * 4 + e];
          if (key > kNegInfKey) atomicAdd(&hist[(key - smin) >> sh], 1);
        }
        __syncthreads();
        // T's expected rank in the sample, 1-based from the top
        const int rr = (int)(((int64_t)ms * kSample + n_cand - 1) / n_cand);
        const Pick ph = find_bin(hist, kTopBins, max(1, min(fin, rr - kBandRanks)), scan_lds, &sh_pick);
        const Pick pl = find_bin(hist, kTopBins, min(fin, rr + kBandRanks), scan_lds, &sh_pick);
        lo = smin + (pl.bin << sh);
        hi = (uint64_t)smin + ((uint64_t)(ph.bin + 1u) << sh);
      }
    }
    // ---- one pass: count the keys above the band per wave, stage the band
    if (tid == 0) sh_pos = 0;
    __syncthreads();
    int up_count = 0;
    walk_segment(s, wb, we, [&](int t, const float (&v)[4]) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int pos = wb + t * kIter + e * 64 + lane;
        const uint32_t key = order_key(v[e]);
        const bool ok = pos < we;
        const bool up = ok && (uint64_t)key >= hi;
        const bool in = ok && !up && key >= lo;
        up_count += up ? 1 : 0;
        const uint64_t bal = __ballot(in);
        if (bal) {                              // wave-uniform
          int base = 0;
          if (lane == 0) base = atomicAdd(&sh_pos, __popcll(bal));
          base = __shfl(base, 0, 64);
          const int at = base + __popcll(bal & below);
          if (in && at < kCandCap) {
            cand[at] = key - lo;
            cpos[at] = pos;
          }
        }
      }
    });
    for (int o = 32; o >= 1; o >>= 1) up_count += __shfl_xor(up_count, o, 64);
    if (lane == 0) wgt[wave] = up_count;
    __syncthreads();
    int above = 0;
    for (int w = 0; w < kWaves; ++w) above += wgt[w];
    const int banded = sh_pos;
    if (above < ms && above + banded >= ms && banded <= kCandCap) {
      // T is the (ms - above)-th largest staged key; the staged keys then
      // complete the per-wave counts
      need = ms - above;
      const uint32_t td = resolve_staged(cand, banded, (uint32_t)min<uint64_t>(hi - lo - 1u, 0xffffffffull), need,
                                         hist, scan_lds, &sh_pick);
      T = lo + td;
      for (int j = tid; j < banded; j += kThreads) {
        const uint32_t d = cand[j];
        if (d > td) atomicAdd(&wgt[cpos[j] / seg], 1);
        else if (d == td) atomicAdd(&weq[cpos[j] / seg], 1);
      }
      __syncthreads();
    } else {
      // ---- the band missed T or overflowed LDS: radix select on
      // d = key - (smallest key), then count per wave
      uint32_t kmin, kmax, prefix, mask;
      int kabove;
      need = ms;
      key_range(s, n_cand, red, kmin, kmax, kabove);
      // With at least ms keys above -inf the threshold is one of them: those
      // keys alone are binned (-inf marks what must not be chosen, e.g. the
      // non-members of the GQA union, and would stretch the range over the
      // whole key space).  Otherwise every key and the whole range are used.
      uint32_t kfloor = kNegInfKey + 1u;
      if (kabove < ms) {
        kfloor = 0u;
        kmin = 0u;
        kmax = 0xffffffffu;
      }
      int hi_bit = top_shift(kmin, kmax);
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
              const int at = base + __popcll(bal & below);
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
      T = prefix + kmin;
      int cg = 0, ce = 0;
      walk_segment(s, wb, we, [&](int t, const float (&v)[4]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int pos = wb + t * kIter + e * 64 + lane;
          const uint32_t key = order_key(v[e]);
          cg += (pos < we && key > T) ? 1 : 0;
          ce += (pos < we && key == T) ? 1 : 0;
        }
      });
      for (int o = 32; o >= 1; o >>= 1) {
        cg += __shfl_xor(cg, o, 64);
        ce += __shfl_xor(ce, o, 64);
      }
      if (lane == 0) {
        wgt[wave] = cg;
        weq[wave] = ce;
      }
      __syncthreads();
    }
  } else {
    __syncthreads();   // the zeroed counts
  }

  // ---- compaction.  The kept list index of key j is (keys > T before j) +
  // min(keys == T before j, need); its evicted index is j minus that.
  int gt0 = 0, eq0 = 0;
  for (int w = 0; w < wave; ++w) {
    gt0 += wgt[w];
    eq0 += weq[w];
  }
  walk_segment(s, wb, we, [&](int t, const float (&v)[4]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int pos = wb + t * kIter + e * 64 + lane;
      const bool ok = pos < we;
      const uint32_t key = order_key(v[e]);
      const bool gt = ok && key > T, eq = ok && key == T;
      const uint64_t bg = __ballot(gt), be = __ballot(eq);
      const int gb = gt0 + __popcll(bg & below), eb = eq0 + __popcll(be & below);
      if (ok) {
        const int kb = gb + min(eb, need);
        if (gt || (eq && eb < need)) {
          if (kb < ms) kh[kb] = pos;
        } else if (pos - kb < n - m) {
          eh[pos - kb] = pos;
        }
      }
      gt0 += __popcll(bg);
      eq0 += __popcll(be);
    }
  });
  for (int r = tid; r < mr; r += kThreads) kh[ms + r] = n_cand + r;
}

}  // namespace

hipError_t launch_select(const Shape& s, const float* score, int32_t* kept, int32_t* evicted, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3((unsigned)s.heads), dim3(kThreads), 0, st, score, kept, evicted, s.n,
                     s.n_cand, s.m, s.mr, s.ms);
  return hipGetLastError();
}

}  // namespace selkv
