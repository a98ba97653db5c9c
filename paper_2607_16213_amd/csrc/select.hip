// selkv_select: per-head top-m_s selection of Sec. 3.3 (Eq. 2).
//
// One workgroup (16 waves) per KV head.  Scores are mapped to order-
// preserving 32-bit keys; an MSB-first radix select with 8-bit digits and
// LDS histograms (integer atomics only) finds the m_s-th largest key T and
// how many keys equal to T must be taken.  A single ordered pass then keeps
// every key > T and the first `need` keys == T (lowest positions win ties),
// compacting kept and evicted positions in ascending order with two block
// prefix sums per chunk.  The m_r' recent positions are appended to the
// kept list.  Outputs do not depend on scheduling: bitwise deterministic.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kPerThread = 4;
constexpr int kChunk = kThreads * kPerThread;
constexpr int kHistBatch = 8;   // score loads in flight per thread

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

__global__ __launch_bounds__(kThreads) void select_kernel(const float* score, int32_t* kept, int32_t* evicted,
                                                         int n, int n_cand, int m, int mr, int ms) {
  const int64_t head = blockIdx.x;
  const float* s = score + (size_t)head * n_cand;
  int32_t* kh = kept + (size_t)head * m;
  int32_t* eh = evicted + (size_t)head * (n - m);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  __shared__ int hist[256];
  __shared__ int scan_lds[2 * kWaves + 1];
  __shared__ uint32_t sh_sel;
  __shared__ int sh_need;

  // ---- radix select of the ms-th largest key
  uint32_t prefix = 0u, mask = 0u;
  int need = ms;
  if (ms > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int b = tid; b < 256; b += kThreads) hist[b] = 0;
      __syncthreads();
      for (int j0 = tid; j0 < n_cand; j0 += kThreads * kHistBatch) {
        float v[kHistBatch];
#pragma unroll
        for (int u = 0; u < kHistBatch; ++u) v[u] = s[min(j0 + u * kThreads, n_cand - 1)];
#pragma unroll
        for (int u = 0; u < kHistBatch; ++u) {
          const uint32_t key = order_key(v[u]);
          if (j0 + u * kThreads < n_cand && (key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
      }
      __syncthreads();
      if (wave == 0) {
        // lane L covers bins 255-4L .. 252-4L, walked from the top
        int c[4], lsum = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          c[k] = hist[255 - (lane * 4 + k)];
          lsum += c[k];
        }
        const int incl = wave_inclusive_scan(lsum, lane);
        const int excl = incl - lsum;
        if (excl < need && incl >= need) {
          int cum = excl;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if (cum + c[k] >= need) {
              sh_sel = 255u - (uint32_t)(lane * 4 + k);
              sh_need = need - cum;
              break;
            }
            cum += c[k];
          }
        }
      }
      __syncthreads();
      prefix |= sh_sel << shift;
      mask |= 255u << shift;
      need = sh_need;
      __syncthreads();
    }
  } else {
    prefix = 0xffffffffu;  // nothing is strictly greater; take no ties
    need = 0;
  }
  const uint32_t T = prefix;

  // ---- ordered compaction: keep u > T, and the first `need` keys equal to T
  int run_kept = 0, run_eq = 0;
  for (int base = 0; base < n_cand; base += kChunk) {
    uint32_t u[kPerThread];
    int neq = 0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int j = base + tid * kPerThread + e;
      u[e] = order_key(s[min(j, n_cand - 1)]);   // clamped: no load behind a branch
      neq += (j < n_cand && u[e] == T) ? 1 : 0;
    }
    int eq_total;
    const int eq_before = run_eq + block_exclusive_scan(neq, scan_lds, eq_total);
    bool keep[kPerThread];
    int nk = 0, eqr = eq_before;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int j = base + tid * kPerThread + e;
      bool k = false;
      if (j < n_cand) {
        if (u[e] > T) {
          k = true;
        } else if (u[e] == T) {
          k = eqr < need;
          ++eqr;
        }
      }
      keep[e] = k;
      nk += k ? 1 : 0;
    }
    int kept_total;
    int kb = run_kept + block_exclusive_scan(nk, scan_lds, kept_total);
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int j = base + tid * kPerThread + e;
      if (j < n_cand) {
        if (keep[e]) {
          if (kb < ms) kh[kb] = j;
          ++kb;
        } else if (j - kb < n - m) {
          eh[j - kb] = j;
        }
      }
    }
    run_kept += kept_total;
    run_eq += eq_total;
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
