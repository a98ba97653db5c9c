// selkv_route_coattn: the co-attention reading of Eq. 3 (Sec. 3.4).
//
// Eq. 3 ranks the kept tokens of an evicted token's bucket by A_{h,j,i}.
// Here that is how much the observation window attends to j and i together:
//   co(j, i) = sum over the G*W window rows r of P[r, j] * P[r, i],
// P the softmax window attention (scale, causal mask) of the score pass.
//
//   row statistics  the score pass 1 kernels and their combine give every
//                   window row's exponent offset -M - log2 L over all n keys
//   routing         one wave per bucket of B <= 64 keys.  The K fragments of
//                   the bucket's keys stay in registers; per 16-row block of
//                   window rows the logits Q K^T come from MFMA, become
//                   P = 2^(c2 x - M - log2 L) (0 where masked), and the
//                   bucket's Gram matrix C = P^T P accumulates on fp32 MFMA.
//                   Then every evicted row of C takes the argmax over the
//                   bucket's kept columns (lowest position on ties).
//
// Gram operands: the 16x16 logits tile leaves lane (g, c) holding rows
// 4g .. 4g+3 of key column c.  In the 16x16x4 fp32 MFMA, lane (g, c) gives
// A[c][g] and B[g][c], so step s that feeds element s of the P tiles of key
// tiles tj (as A) and ti (as B) adds sum_g P[4g+s][tj:c] P[4g+s][ti:c']; the
// four steps cover the 16 rows and no data moves between lanes.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

struct CoArgs {
  const char* K;
  const char* Q;
  const float2* stats;   // per row (-M - log2 L, unused), rpad rows per head
  const int32_t* kept;
  const int32_t* offs;   // bucket offsets into kept
  int32_t* target;
  int n, m, nb, B, W, R, rpad;
  float c2;
};

// NT = 16-key tiles per bucket (B <= 16 * NT).
template <typename T, int D, int NT>
__global__ __launch_bounds__(kThreads) void coattn_route_kernel(CoArgs a) {
  constexpr int RB = D * (int)sizeof(T);
  constexpr int NCH = RB / 64;   // 16-byte chunk steps of one row (4 lane groups x 16 bytes each)
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int bucket = blockIdx.x * kWaves + wave;
  if (bucket >= a.nb) return;   // whole wave; no block barrier below
  const int n = a.n, m = a.m, ne_all = n - m;
  const int32_t* kh = a.kept + (size_t)head * m;
  const int32_t* oh = a.offs + (size_t)head * (a.nb + 1);
  int32_t* th = a.target + (size_t)head * ne_all;
  const int start = bucket * a.B, end = min(n, start + a.B);
  const int k0 = oh[bucket], k1 = oh[bucket + 1];
  const int e0 = start - k0, e1 = end - k1;
  if (k0 > k1 || k1 > m || e0 < 0 || e0 > e1 || e1 > ne_all) return;   // inconsistent kept list
  const int nk = k1 - k0, ne = e1 - e0;
  if (ne == 0) return;
  if (nk == 0) {
    for (int i = lane; i < ne; i += 64) th[e0 + i] = -1;
    return;
  }
  // bucket-relative positions of the kept tokens as a bit mask
  const int kp = lane < nk ? kh[k0 + lane] - start : 0;
  uint64_t kmask = 0;
  for (int i = 0; i < nk; ++i) kmask |= 1ull << (__builtin_amdgcn_readlane(kp, i) & 63);

  // K fragments of the bucket's keys (past the end: the last key, masked below)
  Chunk16 kf[NT][NCH];
  const char* Kh = a.K + (size_t)head * n * RB;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int key = min(start + 16 * t + col, end - 1);
#pragma unroll
    for (int c = 0; c < NCH; ++c) kf[t][c] = load16(Kh + (size_t)key * RB + (c * 4 + grp) * 16);
  }

  f32x4 C[NT][NT];
#pragma unroll
  for (int tj = 0; tj < NT; ++tj)
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) C[tj][ti] = f32x4{0.f, 0.f, 0.f, 0.f};

  const float2* st = a.stats + (size_t)head * a.rpad;
  const char* Qh = a.Q + (size_t)head * a.R * RB;
  const int R = a.R, nrb = (R + 15) / 16;
  const int win0 = n - a.W;
  // query rows and row statistics of the next 16-row block load while the
  // current block is used (indices clamped; rows past R are masked by off)
  Chunk16 qf[NCH];
  float offn[4];
#pragma unroll
  for (int c = 0; c < NCH; ++c) qf[c] = load16(Qh + (size_t)min(col, R - 1) * RB + (c * 4 + grp) * 16);
#pragma unroll
  for (int i = 0; i < 4; ++i) offn[i] = st[min(grp * 4 + i, R - 1)].x;
  for (int rb = 0; rb < nrb; ++rb) {
    float off[4];
    int rpos[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = rb * 16 + grp * 4 + i;
      off[i] = r < R ? offn[i] : kNegInf;
      rpos[i] = win0 + (r < R ? r % a.W : 0);
      offn[i] = st[min(r + 16, R - 1)].x;
    }
    // logits of the block's 16 rows against the bucket's keys
    f32x4 x[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      x[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NCH; ++c) x[t] = Mma<T>::step(qf[c], kf[t][c], x[t]);
    }
    // the next block's query rows load while this one is used
    if (rb + 1 < nrb) {
      const int qr = min((rb + 1) * 16 + col, R - 1);
#pragma unroll
      for (int c = 0; c < NCH; ++c) qf[c] = load16(Qh + (size_t)qr * RB + (c * 4 + grp) * 16);
    }
    f32x4 P[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int key = start + 16 * t + col;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        P[t][i] = (key < end && key <= rpos[i] && off[i] != kNegInf) ? fast_exp2(fmaf(x[t][i], a.c2, off[i])) : 0.f;
    }
#pragma unroll
    for (int tj = 0; tj < NT; ++tj)
#pragma unroll
      for (int ti = 0; ti < NT; ++ti)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          C[tj][ti] = __builtin_amdgcn_mfma_f32_16x16x4f32(P[tj][s], P[ti][s], C[tj][ti], 0, 0, 0);
  }

  // argmax over the kept columns for every row (lane (g, c) holds rows
  // 16 tj + 4g + i, column 16 ti + c); ties to the lower column
#pragma unroll
  for (int tj = 0; tj < NT; ++tj) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float best = kNegInf;
      int bcol = 64;
#pragma unroll
      for (int ti = 0; ti < NT; ++ti) {
        const int cc = 16 * ti + col;
        const float v = ((kmask >> cc) & 1ull) ? C[tj][ti][i] : kNegInf;
        if (v > best) {             // ti ascends, so the first (lowest) column keeps equal values
          best = v;
          bcol = cc;
        }
      }
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) {
        const float ob = xor_shfl(best, o);
        const int oc = xor_shfl(bcol, o);
        if (ob > best || (ob == best && oc < bcol)) {
          best = ob;
          bcol = oc;
        }
      }
      const int jj = 16 * tj + 4 * grp + i;     // bucket-relative row
      if (col == 0 && start + jj < end && !((kmask >> jj) & 1ull) && bcol < 64) {
        const int e = e0 + jj - __popcll(kmask & ((1ull << jj) - 1));
        th[e] = k0 + __popcll(kmask & ((1ull << bcol) - 1));
      }
    }
  }
}

}  // namespace

hipError_t launch_coattn_route(const Shape& s, const ScorePlan& sp, int dtype, int bucket, int W, const void* K,
                               const void* Qwin, const void* score_ws, const int32_t* kept, const int32_t* offs,
                               int32_t* target, float c2, hipStream_t st) {
  if (s.n - s.m <= 0) return hipSuccess;
  CoArgs a{};
  a.K = static_cast<const char*>(K);
  a.Q = static_cast<const char*>(Qwin);
  a.stats = reinterpret_cast<const float2*>(static_cast<const char*>(score_ws) + sp.stats_off);
  a.kept = kept;
  a.offs = offs;
  a.target = target;
  a.n = s.n;
  a.m = s.m;
  a.nb = s.nb;
  a.B = bucket;
  a.W = W;
  a.R = s.R;
  a.rpad = sp.rpad;
  a.c2 = c2;
  const dim3 grid((s.nb + kWaves - 1) / kWaves, (unsigned)s.heads), blk(kThreads);
  const int nt = (bucket + 15) / 16;
#define SELKV_CO(T, D)                                                                            \
  do {                                                                                            \
    switch (nt) {                                                                                 \
      case 1: hipLaunchKernelGGL((coattn_route_kernel<T, D, 1>), grid, blk, 0, st, a); break;     \
      case 2: hipLaunchKernelGGL((coattn_route_kernel<T, D, 2>), grid, blk, 0, st, a); break;     \
      case 3: hipLaunchKernelGGL((coattn_route_kernel<T, D, 3>), grid, blk, 0, st, a); break;     \
      default: hipLaunchKernelGGL((coattn_route_kernel<T, D, 4>), grid, blk, 0, st, a); break;    \
    }                                                                                             \
  } while (0)
  if (dtype == SELKV_BF16) {
    if (s.d == 128) SELKV_CO(bf16_t, 128);
    else SELKV_CO(bf16_t, 64);
  } else {
    if (s.d == 128) SELKV_CO(float, 128);
    else SELKV_CO(float, 64);
  }
#undef SELKV_CO
  return hipGetLastError();
}

}  // namespace selkv
