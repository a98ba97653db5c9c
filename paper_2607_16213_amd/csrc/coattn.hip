// selkv_route_coattn: the co-attention reading of Eq. 3 (Sec. 3.4).
//
// Eq. 3 ranks the kept tokens of an evicted token's bucket by A_{h,j,i}.
// Here that is how much the observation window attends to j and i together:
//   co(j, i) = sum over the G*W window rows r of P[r, j] * P[r, i],
// P the softmax window attention (scale, causal mask) of the score pass.
//
//   row statistics  the score pass 1 kernels and their combine give every
//                   window row's max M and 1/L over all n keys
//   routing         a workgroup stages one head's window queries and row
//                   offsets in LDS (when they fit in 32 KB) for its four
//                   waves; each wave routes eight consecutive buckets of
//                   B <= 64 keys in turn, a bucket's columns ordered kept
//                   tokens first, then evicted ones.  The K fragments
//                   of the bucket's keys stay in registers; per 16-row block
//                   of window rows the logits Q K^T come from MFMA, become
//                   P = 2^(c2 x - M) / L (0 where masked), and the
//                   Gram blocks C = P^T P that pair an evicted row tile with
//                   a kept column tile accumulate on fp32 MFMA (at 25%
//                   retention one kept tile: half of the B x B blocks).  Then
//                   every evicted row takes the argmax over the kept columns
//                   (lowest position on ties: kept columns are ascending).
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
  const float2* stats;   // per row (-M, 1/L), rpad rows per head
  const int32_t* kept;
  const int32_t* offs;   // bucket offsets into kept
  int32_t* target;
  int n, m, nb, B, W, R, rpad;
  float c2;
};

// Window queries staged in LDS per workgroup (the four waves route buckets
// of one head and share them) when they fit; otherwise each wave reads them
// from global memory.
constexpr int kQldsBytes = 32 * 1024;

// Buckets one wave routes in turn (the workgroup's staged queries serve 32).
constexpr int kBucketsPerWave = 8;

// One bucket: the body of the routing described at the top of the file.
template <typename T, int D, int NT, bool QL>
__device__ __forceinline__ void route_bucket(const CoArgs& a, int bucket, int64_t head, int lane,
                                             const char* q_lds, const float2* off_lds) {
  constexpr int RB = D * (int)sizeof(T);
  constexpr int NCH = RB / 64;
  constexpr int NCHUNK = RB / 16;
  const int col = lane & 15, grp = lane >> 4;
  const char* Qh = a.Q + (size_t)head * a.R * RB;
  const float2* st = a.stats + (size_t)head * a.rpad;
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
  const int bsize = end - start;   // <= 64
  const int kp = lane < nk ? kh[k0 + lane] - start : 0;
  uint64_t kmask = 0;
  for (int i = 0; i < nk; ++i) kmask |= 1ull << (__builtin_amdgcn_readlane(kp, i) & 63);
  // Column order of the tiles: the bucket's kept tokens (ascending), then its
  // evicted ones (ascending), so the Gram blocks that pair an evicted row
  // with a kept column are the only ones formed.  Lane L (a bucket position)
  // sends L to the lane of its column; lanes past the bucket map to themselves.
  const int below = __popcll(kmask & ((1ull << lane) - 1ull));
  const int column = lane >= bsize ? lane : (((kmask >> lane) & 1ull) ? below : nk + lane - below);
  const int colpos = __builtin_amdgcn_ds_permute(column * 4, lane);   // lane j: position of column j

  // K fragments of the columns' keys (past the bucket: the last key, masked below)
  Chunk16 kf[NT][NCH];
  int ckey[NT];   // this lane's column key in tile t, or -1 past the bucket
  const char* Kh = a.K + (size_t)head * n * RB;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int j = 16 * t + col;
    const int pos = __shfl(colpos, j, 64);
    ckey[t] = j < bsize ? start + pos : -1;
    const int key = j < bsize ? start + pos : end - 1;
#pragma unroll
    for (int c = 0; c < NCH; ++c) kf[t][c] = load16(Kh + (size_t)key * RB + (c * 4 + grp) * 16);
  }

  f32x4 C[NT][NT];
#pragma unroll
  for (int tj = 0; tj < NT; ++tj)
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) C[tj][ti] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int R = a.R, nrb = (R + 15) / 16;
  const int win0 = n - a.W;
  // fragment c of query row r for this lane, and row r's exponent offset
  auto q_frag = [&](int r, int c) {
    if constexpr (QL) return *reinterpret_cast<const Chunk16*>(q_lds + r * RB + (((c * 4 + grp) ^ (r % NCHUNK)) * 16));
    else return load16(Qh + (size_t)r * RB + (c * 4 + grp) * 16);
  };
  auto row_off = [&](int r) {
    if constexpr (QL) return off_lds[r];
    else return st[r];
  };
  // query rows and row statistics of the next 16-row block load while the
  // current block is used (indices clamped; rows past R are masked by off)
  Chunk16 qf[NCH];
  float2 offn[4];
#pragma unroll
  for (int c = 0; c < NCH; ++c) qf[c] = q_frag(min(col, R - 1), c);
#pragma unroll
  for (int i = 0; i < 4; ++i) offn[i] = row_off(min(grp * 4 + i, R - 1));
  for (int rb = 0; rb < nrb; ++rb) {
    float off[4], inv[4];
    int rpos[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = rb * 16 + grp * 4 + i;
      off[i] = r < R ? offn[i].x : kNegInf;
      inv[i] = offn[i].y;
      rpos[i] = win0 + (r < R ? r % a.W : 0);
      offn[i] = row_off(min(r + 16, R - 1));
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
      for (int c = 0; c < NCH; ++c) qf[c] = q_frag(qr, c);
    }
    f32x4 P[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        P[t][i] = (ckey[t] >= 0 && ckey[t] <= rpos[i] && off[i] != kNegInf)
                      ? fast_exp2(fmaf(x[t][i], a.c2, off[i])) * inv[i]
                      : 0.f;
    }
    // Gram blocks of evicted row tiles against kept column tiles only
#pragma unroll
    for (int tj = 0; tj < NT; ++tj) {
      if (16 * (tj + 1) <= nk || 16 * tj >= bsize) continue;   // no evicted column in tile tj
#pragma unroll
      for (int ti = 0; ti < NT; ++ti) {
        if (16 * ti >= nk) continue;                           // no kept column in tile ti
#pragma unroll
        for (int s = 0; s < 4; ++s)
          C[tj][ti] = __builtin_amdgcn_mfma_f32_16x16x4f32(P[tj][s], P[ti][s], C[tj][ti], 0, 0, 0);
      }
    }
  }

  // argmax over the kept columns (ordinals 0 .. nk-1) for every evicted row
  // (ordinal nk .. bsize-1); lane (g, c) holds rows 16 tj + 4g + i, column
  // 16 ti + c; ties to the lower column, i.e. the lower kept position
#pragma unroll
  for (int tj = 0; tj < NT; ++tj) {
    if (16 * (tj + 1) <= nk || 16 * tj >= bsize) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float best = kNegInf;
      int bcol = 64;
#pragma unroll
      for (int ti = 0; ti < NT; ++ti) {
        const int cc = 16 * ti + col;
        const float v = (16 * ti < nk && cc < nk) ? C[tj][ti][i] : kNegInf;
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
      const int row = 16 * tj + 4 * grp + i;   // column ordinal of the evicted token
      if (col == 0 && row >= nk && row < bsize && bcol < nk) th[e0 + row - nk] = k0 + bcol;
    }
  }
}

// NT = 16-key tiles per bucket (B <= 16 * NT); QL: queries and row
// statistics in LDS (R * row bytes <= kQldsBytes).
template <typename T, int D, int NT, bool QL>
__global__ __launch_bounds__(kThreads) void coattn_route_kernel(CoArgs a) {
  constexpr int RB = D * (int)sizeof(T);
  constexpr int NCH = RB / 64;      // 16-byte chunk steps of one row (4 lane groups x 16 bytes each)
  constexpr int NCHUNK = RB / 16;   // 16-byte chunks of one row
  constexpr int QB = QL ? kQldsBytes : 16;
  constexpr int QR = QL ? kQldsBytes / RB : 1;
  __shared__ __align__(16) char q_lds[QB];   // row r, chunk ch at r * RB + (ch ^ (r mod NCHUNK)) * 16
  __shared__ float2 off_lds[QR];
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const char* Qh = a.Q + (size_t)head * a.R * RB;
  const float2* st = a.stats + (size_t)head * a.rpad;
  if constexpr (QL) {
    // every thread helps stage the head's queries and row offsets (before
    // any wave leaves: this is the kernel's only block barrier)
    for (int idx = threadIdx.x; idx < a.R * NCHUNK; idx += kThreads) {
      const int r = idx / NCHUNK, ch = idx % NCHUNK;
      store16(q_lds + r * RB + ((ch ^ (r % NCHUNK)) * 16), load16(Qh + (size_t)r * RB + ch * 16));
    }
    for (int r = threadIdx.x; r < a.R; r += kThreads) off_lds[r] = st[r];
    __syncthreads();
  }
  const int first = (blockIdx.x * kWaves + wave) * kBucketsPerWave;
  for (int bucket = first; bucket < min(a.nb, first + kBucketsPerWave); ++bucket) route_bucket<T, D, NT, QL>(
      a, bucket, head, lane, q_lds, off_lds);   // whole waves; no block barrier below
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
  const int per_block = kWaves * kBucketsPerWave;
  const dim3 grid((s.nb + per_block - 1) / per_block, (unsigned)s.heads), blk(kThreads);
  const int nt = (bucket + 15) / 16;
  const bool ql = (size_t)s.R * s.d * (dtype == SELKV_BF16 ? 2 : 4) <= (size_t)kQldsBytes;
#define SELKV_CO_NT(T, D, QL)                                                                      \
  do {                                                                                             \
    switch (nt) {                                                                                  \
      case 1: hipLaunchKernelGGL((coattn_route_kernel<T, D, 1, QL>), grid, blk, 0, st, a); break;  \
      case 2: hipLaunchKernelGGL((coattn_route_kernel<T, D, 2, QL>), grid, blk, 0, st, a); break;  \
      case 3: hipLaunchKernelGGL((coattn_route_kernel<T, D, 3, QL>), grid, blk, 0, st, a); break;  \
      default: hipLaunchKernelGGL((coattn_route_kernel<T, D, 4, QL>), grid, blk, 0, st, a); break; \
    }                                                                                              \
  } while (0)
#define SELKV_CO(T, D)                         \
  do {                                         \
    if (ql) SELKV_CO_NT(T, D, true);           \
    else SELKV_CO_NT(T, D, false);             \
  } while (0)
  if (dtype == SELKV_BF16) {
    if (s.d == 128) SELKV_CO(bf16_t, 128);
    else SELKV_CO(bf16_t, 64);
  } else {
    if (s.d == 128) SELKV_CO(float, 128);
    else SELKV_CO(float, 64);
  }
#undef SELKV_CO
#undef SELKV_CO_NT
  return hipGetLastError();
}

}  // namespace selkv
