// selkv_score: contribution scores of Sec. 3.2 (Eq. 1) from the
// observation-window attention of Sec. 3.1, recomputed on the fly.
//
// For one KV head the window rows are the G*W query rows of its G query
// heads (row r = h*W + i is position n-W+i, causal).  The logits
// scale * Q K^T are produced on MFMA (16x16x32 bf16, or 16x16x4 fp32) with
// Q fragments in registers and K streamed from HBM:
//   pass 1  per (key chunk, row group): online row max / sum of exp  -> ws
//   combine per KV head: merge the chunk partials in chunk order     -> ws
//   pass 2  per key chunk: recompute the logits, normalise, sum the G*W
//           rows of every key column (a_j, divided by G), value norms from
//           V, write attn, vnorm and c = a * ||v||
//   pool    centred K-wide moving average of c over [0, n - m_r')
// The attention matrix itself is never stored.
//
// Work split inside a 4-wave workgroup: RW waves share each K tile, each
// holding NRB 16-row blocks of Q (RW * NRB * 16 rows per row group); the
// 4 / RW pairs walk interleaved 16-key tiles of the chunk.  Every K load is
// issued unconditionally (rows past the chunk end re-read its last row and
// are masked) and the next tile is loaded before the current one is used.
// Tiles that every row sees in full skip all masking.
//
// Fragment layout (both MFMA operands, all dtypes): lane l handles matrix
// index l % 16 (a window row for Q, a key for K) and lane group g = l / 16
// owns the 16-byte chunks c*4 + g of that row, so one load instruction reads
// 64 contiguous bytes from each of 16 rows.  MFMA output lane l holds rows
// 4g .. 4g+3 of the 16-row block for key l % 16.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;          // 4 waves
constexpr int kMaxChunkKeys = 4096;    // LDS column accumulator bound
constexpr int kMinChunkKeys = 128;
constexpr int kTargetBlocks = 2048;

template <typename T, int D>
struct Row {
  static constexpr int kBytes = D * (int)sizeof(T);
  static constexpr int kNch = kBytes / 64;   // 16-byte chunks per lane per row
};

struct ScoreArgs {
  const char* K;
  const char* V;
  const char* Q;
  float* attn;
  float* vnorm;
  float2* part;
  float2* stats;
  float* cbuf;
  int n, W, R, G;
  int chunk_keys, nchunks, rpad, nrg;
  float c2;  // scale * log2(e): logits are kept in the log2 domain
};

__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == kNegInf) {
    s = 0.f;
  } else {
    s = s * fast_exp2(m - M) + s2 * fast_exp2(m2 - M);
  }
  m = M;
}

template <typename T, int D, int NRB>
__device__ __forceinline__ void load_q(const char* Qh, int R, int row0, int col, int grp,
                                       Chunk16 (&q)[NRB][Row<T, D>::kNch]) {
  constexpr int NCH = Row<T, D>::kNch;
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    const int row = row0 + rb * 16 + col;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      q[rb][c] = row < R ? load16(Qh + (size_t)row * Row<T, D>::kBytes + (c * 4 + grp) * 16) : zero16();
  }
}

// K (or V) fragments of the 16-key tile starting at t; keys past `last` re-read row `last`.
template <typename T, int D>
__device__ __forceinline__ void load_tile(const char* Xh, int t, int last, int col, int grp,
                                          Chunk16 (&f)[Row<T, D>::kNch]) {
  constexpr int NCH = Row<T, D>::kNch;
  const int key = min(t + col, last);
#pragma unroll
  for (int c = 0; c < NCH; ++c) f[c] = load16(Xh + (size_t)key * Row<T, D>::kBytes + (c * 4 + grp) * 16);
}

// Pass 1: per-row (max, sum of exp2) over this block's key chunk.
template <typename T, int D, int NRB, int RW>
__global__ __launch_bounds__(kThreads) void score_rowstats_kernel(ScoreArgs a) {
  constexpr int NCH = Row<T, D>::kNch;
  constexpr int TS = 4 / RW;
  constexpr int ROWS = RW * NRB * 16;
  const int chunk = blockIdx.x;
  const int64_t head = blockIdx.y;
  const int rg = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int half = wave % RW, stream = wave / RW;
  const int n = a.n, W = a.W;
  const char* Kh = a.K + (size_t)head * n * Row<T, D>::kBytes;
  const char* Qh = a.Q + (size_t)head * a.R * Row<T, D>::kBytes;
  const int row0 = rg * ROWS + half * NRB * 16;

  Chunk16 q[NRB][NCH];
  load_q<T, D, NRB>(Qh, a.R, row0, col, grp, q);

  float m[NRB][4], s[NRB][4];
  int wi[NRB][4];  // window index of the row, -1 for padding rows
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row0 + rb * 16 + grp * 4 + i;
      wi[rb][i] = row < a.R ? row % W : -1;
      m[rb][i] = kNegInf;
      s[rb][i] = 0.f;
    }

  const int kb = chunk * a.chunk_keys;
  const int ke = min(n, kb + a.chunk_keys);
  const int full_end = min(ke, n - W + 1);     // keys below this are seen by every row
  int t = kb + stream * 16;
  Chunk16 kcur[NCH], knxt[NCH];
  if (t < ke) load_tile<T, D>(Kh, t, ke - 1, col, grp, kcur);
  for (; t < ke; t += TS * 16) {
    load_tile<T, D>(Kh, t + TS * 16, ke - 1, col, grp, knxt);
    const bool fast = t + 16 <= full_end;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NCH; ++c) acc = Mma<T>::step(q[rb][c], kcur[c], acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = t + col;
        const bool valid = fast || (key < ke && wi[rb][i] >= 0 && key <= n - W + wi[rb][i]);
        if (valid) {
          const float x = acc[i] * a.c2;
          const float dlt = x - m[rb][i];
          const float e = fast_exp2(-fabsf(dlt));
          if (dlt > 0.f) {
            s[rb][i] = fmaf(s[rb][i], e, 1.f);
            m[rb][i] = x;
          } else {
            s[rb][i] += e;
          }
        }
      }
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) kcur[c] = knxt[c];
  }

  // merge the 16 lanes (keys) that share each row
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float m2 = xor_shfl(m[rb][i], off);
        const float s2 = xor_shfl(s[rb][i], off);
        lse_merge(m[rb][i], s[rb][i], m2, s2);
      }

  __shared__ float2 red[TS][ROWS];
  if (col == 0) {
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        red[stream][half * NRB * 16 + rb * 16 + grp * 4 + i] = make_float2(m[rb][i], s[rb][i]);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < ROWS; r += kThreads) {
    float mm = red[0][r].x, ss = red[0][r].y;
#pragma unroll
    for (int w = 1; w < TS; ++w) lse_merge(mm, ss, red[w][r].x, red[w][r].y);
    a.part[((size_t)head * a.nchunks + chunk) * a.rpad + rg * ROWS + r] = make_float2(mm, ss);
  }
}

// Combine the chunk partials of every row, in chunk order: (max, 1/sum).
__global__ __launch_bounds__(kThreads) void score_combine_kernel(ScoreArgs a) {
  constexpr int kBatch = 8;   // partial loads in flight per thread
  const int64_t head = blockIdx.x;
  for (int row = threadIdx.x; row < a.rpad; row += blockDim.x) {
    const float2* p = a.part + (size_t)head * a.nchunks * a.rpad + row;
    float M = kNegInf, L = 0.f;
    for (int c0 = 0; c0 < a.nchunks; c0 += kBatch) {
      float2 v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) v[u] = p[(size_t)min(c0 + u, a.nchunks - 1) * a.rpad];
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        if (c0 + u < a.nchunks) lse_merge(M, L, v[u].x, v[u].y);
    }
    a.stats[(size_t)head * a.rpad + row] = (row < a.R && L > 0.f) ? make_float2(M, 1.f / L) : make_float2(0.f, 0.f);
  }
}

// Pass 2: column sums of the normalised window attention, value norms, c.
template <typename T, int D, int NRB, int RW>
__global__ __launch_bounds__(kThreads) void score_colsum_kernel(ScoreArgs a) {
  constexpr int NCH = Row<T, D>::kNch;
  constexpr int EPC = Elem<T>::kPerChunk;
  constexpr int TS = 4 / RW;
  constexpr int ROWS = RW * NRB * 16;
  const int chunk = blockIdx.x;
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int half = wave % RW, stream = wave / RW;
  const int n = a.n, W = a.W;
  const char* Kh = a.K + (size_t)head * n * Row<T, D>::kBytes;
  const char* Vh = a.V + (size_t)head * n * Row<T, D>::kBytes;
  const char* Qh = a.Q + (size_t)head * a.R * Row<T, D>::kBytes;
  const float2* st = a.stats + (size_t)head * a.rpad;
  const int kb = chunk * a.chunk_keys;
  const int ke = min(n, kb + a.chunk_keys);
  const int full_end = min(ke, n - W + 1);

  __shared__ float colacc[RW][kMaxChunkKeys];
  __shared__ float vn_l[RW][kMaxChunkKeys];   // squared-norm partials, one per row half

  for (int rg = 0; rg < a.nrg; ++rg) {
    const int row0 = rg * ROWS + half * NRB * 16;
    Chunk16 q[NRB][NCH];
    load_q<T, D, NRB>(Qh, a.R, row0, col, grp, q);
    float Mr[NRB][4], iL[NRB][4];
    int wi[NRB][4];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = row0 + rb * 16 + grp * 4 + i;
        const float2 v = st[row];
        Mr[rb][i] = -v.x;          // stored negated: exponent = fma(acc, c2, -M)
        iL[rb][i] = v.y;           // 0 for padding rows
        wi[rb][i] = row < a.R ? row % W : -1;
      }
    // each row half reads its share of every V row once: chunks c with c % RW == half
    const bool norms = rg == 0;

    int t = kb + stream * 16;
    Chunk16 kcur[NCH], knxt[NCH];
    if (t < ke) load_tile<T, D>(Kh, t, ke - 1, col, grp, kcur);
    for (; t < ke; t += TS * 16) {
      load_tile<T, D>(Kh, t + TS * 16, ke - 1, col, grp, knxt);
      constexpr int NV = NCH / RW > 0 ? NCH / RW : 1;
      Chunk16 vf[NV];
      if (norms) {
        const int vkey = min(t + col, ke - 1);
#pragma unroll
        for (int c = 0; c < NV; ++c)
          vf[c] = load16(Vh + (size_t)vkey * Row<T, D>::kBytes + ((c * RW + half) * 4 + grp) * 16);
      }
      const bool fast = t + 16 <= full_end;
      const int key = t + col;
      float cs = 0.f;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NCH; ++c) acc = Mma<T>::step(q[rb][c], kcur[c], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = fast_exp2(fmaf(acc[i], a.c2, Mr[rb][i])) * iL[rb][i];
          const bool valid = fast || (key < ke && wi[rb][i] >= 0 && key <= n - W + wi[rb][i]);
          cs += valid ? p : 0.f;
        }
      }
      cs += xor_shfl(cs, 16);
      cs += xor_shfl(cs, 32);
      const int local = key - kb;
      if (grp == 0 && key < ke) colacc[half][local] = (rg == 0 ? 0.f : colacc[half][local]) + cs;
      if (norms) {
        float ss = 0.f;
#pragma unroll
        for (int c = 0; c < NV; ++c)
#pragma unroll
          for (int e = 0; e < EPC; ++e) {
            const float x = Elem<T>::get(vf[c], e);
            ss = fmaf(x, x, ss);
          }
        ss += xor_shfl(ss, 16);
        ss += xor_shfl(ss, 32);
        if (grp == 0 && key < ke) vn_l[half][local] = ss;
      }
#pragma unroll
      for (int c = 0; c < NCH; ++c) kcur[c] = knxt[c];
    }
  }
  __syncthreads();
  for (int k = kb + (int)threadIdx.x; k < ke; k += kThreads) {
    const int local = k - kb;
    float total = colacc[0][local];
#pragma unroll
    for (int h = 1; h < RW; ++h) total += colacc[h][local];
    const float av = total / (float)a.G;
    float ss = vn_l[0][local];
#pragma unroll
    for (int h = 1; h < RW; ++h) ss += vn_l[h][local];
    const float vn = sqrtf(ss);
    const size_t o = (size_t)head * n + k;
    a.attn[o] = av;
    a.vnorm[o] = vn;
    a.cbuf[o] = av * vn;
  }
}

// Centred moving average of width K over the candidate range, zero outside.
__global__ __launch_bounds__(kThreads) void score_pool_kernel(const float* cbuf, float* score, int n, int n_cand,
                                                             int K) {
  const int64_t head = blockIdx.y;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n_cand) return;
  const float* c = cbuf + (size_t)head * n;
  const int h = K / 2;
  float s = 0.f;
  for (int t = -h; t <= h; ++t) {
    const int jj = j + t;
    const float v = c[min(max(jj, 0), n_cand - 1)];   // clamped load, masked below
    s += (jj >= 0 && jj < n_cand) ? v : 0.f;
  }
  score[(size_t)head * n_cand + j] = s / (float)K;
}

template <typename T, int D, int NRB, int RW>
hipError_t launch_t(const Shape& s, const ScorePlan& p, ScoreArgs& a, float* score, int pool_kernel,
                    hipStream_t st) {
  const dim3 blk(kThreads);
  hipLaunchKernelGGL((score_rowstats_kernel<T, D, NRB, RW>), dim3(p.nchunks, (unsigned)s.heads, p.nrg), blk, 0, st,
                     a);
  hipLaunchKernelGGL(score_combine_kernel, dim3((unsigned)s.heads), blk, 0, st, a);
  hipLaunchKernelGGL((score_colsum_kernel<T, D, NRB, RW>), dim3(p.nchunks, (unsigned)s.heads), blk, 0, st, a);
  if (s.n_cand > 0)
    hipLaunchKernelGGL(score_pool_kernel, dim3((s.n_cand + kThreads - 1) / kThreads, (unsigned)s.heads), blk, 0,
                       st, a.cbuf, score, s.n, s.n_cand, pool_kernel);
  return hipGetLastError();
}

// Row blocks per wave (NRB) and waves sharing a tile (RW) for each dtype / head dim.
template <typename T, int D>
hipError_t launch_d(const Shape& s, const ScorePlan& p, ScoreArgs& a, float* score, int pool_kernel,
                    hipStream_t st) {
  switch (p.rows_per_group) {
    case 16: return launch_t<T, D, 1, 1>(s, p, a, score, pool_kernel, st);
    case 32: return launch_t<T, D, 2, 1>(s, p, a, score, pool_kernel, st);
    case 64: return launch_t<T, D, 4, 1>(s, p, a, score, pool_kernel, st);
    case 128: return launch_t<T, D, 4, 2>(s, p, a, score, pool_kernel, st);
    default: return hipErrorInvalidValue;
  }
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

ScorePlan plan_score(const Shape& s, int dtype) {
  ScorePlan p{};
  // up to 128 rows per row group (4 row blocks per wave, two waves per tile);
  // fp32 with d = 128 keeps 32 rows so Q stays within 64 VGPRs per wave
  const int max_rows = (dtype == SELKV_F32 && s.d == 128) ? 32 : 128;
  int rows = 16;
  while (rows < s.R && rows < max_rows) rows <<= 1;
  p.rows_per_group = rows;
  p.nrg = (s.R + rows - 1) / rows;
  p.rpad = p.nrg * rows;

  const int64_t tiles = (s.n + 63) / 64;
  int64_t nchunks = (kTargetBlocks + s.heads - 1) / s.heads;
  if (nchunks > tiles) nchunks = tiles;
  if (nchunks < 1) nchunks = 1;
  int64_t ck = ((s.n + nchunks - 1) / nchunks + 63) / 64 * 64;
  const int64_t n64 = ((int64_t)s.n + 63) / 64 * 64;
  const int64_t min_ck = n64 < kMinChunkKeys ? n64 : kMinChunkKeys;
  if (ck < min_ck) ck = min_ck;
  if (ck > kMaxChunkKeys) ck = kMaxChunkKeys;
  p.chunk_keys = (int)ck;
  p.nchunks = (int)((s.n + ck - 1) / ck);

  p.part_off = 0;
  p.stats_off = align256((size_t)s.heads * p.nchunks * p.rpad * sizeof(float2));
  p.c_off = p.stats_off + align256((size_t)s.heads * p.rpad * sizeof(float2));
  p.bytes = p.c_off + align256((size_t)s.heads * s.n * sizeof(float));
  return p;
}

hipError_t launch_score(const Shape& s, const ScorePlan& p, int dtype, float scale, const void* K, const void* V,
                        const void* Qwin, float* score, float* attn, float* vnorm, int pool_kernel, void* ws,
                        hipStream_t st) {
  ScoreArgs a{};
  a.K = static_cast<const char*>(K);
  a.V = static_cast<const char*>(V);
  a.Q = static_cast<const char*>(Qwin);
  a.attn = attn;
  a.vnorm = vnorm;
  char* w = static_cast<char*>(ws);
  a.part = reinterpret_cast<float2*>(w + p.part_off);
  a.stats = reinterpret_cast<float2*>(w + p.stats_off);
  a.cbuf = reinterpret_cast<float*>(w + p.c_off);
  a.n = s.n;
  a.W = s.W;
  a.R = s.R;
  a.G = s.G;
  a.chunk_keys = p.chunk_keys;
  a.nchunks = p.nchunks;
  a.rpad = p.rpad;
  a.nrg = p.nrg;
  a.c2 = scale * kLog2e;
  if (dtype == SELKV_BF16) {
    if (s.d == 128) return launch_d<bf16_t, 128>(s, p, a, score, pool_kernel, st);
    return launch_d<bf16_t, 64>(s, p, a, score, pool_kernel, st);
  }
  if (s.d == 128) return launch_d<float, 128>(s, p, a, score, pool_kernel, st);
  return launch_d<float, 64>(s, p, a, score, pool_kernel, st);
}

}  // namespace selkv
