// selkv_score: contribution scores of Sec. 3.2 (Eq. 1) from the
// observation-window attention of Sec. 3.1, recomputed on the fly.
//
// For one KV head the window rows are the G*W query rows of its G query
// heads (row r = h*W + i is position n-W+i, causal).  The logits
// scale * Q K^T are produced on MFMA (16x16x32 bf16, or 16x16x4 fp32) with
// Q fragments in registers and K streamed from HBM:
//   pass 1  per (key chunk, row group): online row max / sum of exp  -> ws
//   combine per KV head: merge the chunk partials in chunk order into
//           (-M, 1/L) per row                                        -> ws
//   pass 2  per key chunk: recompute the logits, normalise
//           (2^(x - M) * 1/L), sum the G*W rows of every key column
//           (a_j, divided by G), value norms from V, write attn, vnorm
//   pool    centred K-wide moving average of c = a * ||v|| over
//           [0, n - m_r'), in fp64
// The attention matrix itself is never stored.
//
// bf16 with at most 128 window rows (the shapes of the paper's workloads)
// takes the shared-tile passes further down: one 32-key K tile per step is
// staged in LDS for all four waves (wave w owns rows 32w .. 32w+31), each
// thread keeps four tiles of contiguous 16-byte loads in flight, and pass 1
// keeps a per-row exponent reference that only moves when a logit exceeds
// it by 2^16, so a logit costs one fma, one exp2, one add and a compare.
// Everything else (fp32, more rows) takes the general passes below.
//
// General passes, work split inside a 4-wave workgroup: RW waves share each K tile, each
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

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;          // 4 waves
constexpr int kWaves = kThreads / 64;
constexpr int kMaxChunkKeys = 4096;   // LDS column accumulator bound
constexpr int kColsumStages = 2;       // K/V tiles in registers in pass 2 (loads in flight + 1)
// Pass 1 keeps each row's exponent reference fixed until a logit exceeds it
// by more than this (log2 units); sums of up to 2^kRefSlack stay exact in fp32
// range, and a logit costs one fma, one exp2, one add and one compare.
constexpr float kRefSlack = 16.f;
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
  int n, W, R, G;
  int chunk_keys, nchunks, rpad, nrg;
  int chunk_keys2;   // shared-tile pass 2
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

// Runs body(tile, t) over the 16-key tiles t = t0, t0 + step, ... < ke,
// with load(tile, t) issued STAGES - 1 tiles ahead of use.
template <int STAGES, typename Tile, typename Load, typename Body>
__device__ __forceinline__ void pipeline(int t0, int ke, int step, Load&& load, Body&& body) {
  static_assert(STAGES == 2 || STAGES == 3, "two or three register buffers");
  int t = t0;
  if (t >= ke) return;
  if constexpr (STAGES == 2) {
    Tile ta, tb;
    load(ta, t);
    while (true) {
      load(tb, t + step);
      body(ta, t);
      t += step;
      if (t >= ke) break;
      load(ta, t + step);
      body(tb, t);
      t += step;
      if (t >= ke) break;
    }
  } else {
    Tile ta, tb, tc;
    load(ta, t);
    load(tb, t + step);
    while (true) {
      load(tc, t + 2 * step);
      body(ta, t);
      t += step;
      if (t >= ke) break;
      load(ta, t + 2 * step);
      body(tb, t);
      t += step;
      if (t >= ke) break;
      load(tb, t + 2 * step);
      body(tc, t);
      t += step;
      if (t >= ke) break;
    }
  }
}

template <typename T, int D>
struct KTile {
  Chunk16 k[Row<T, D>::kNch];
};

// K fragments plus this wave's share of the V rows (for the norms).
template <typename T, int D, int NV>
struct KVTile {
  Chunk16 k[Row<T, D>::kNch];
  Chunk16 v[NV];
};

// Whether window row `row` (of R, window W) sees key `key` of an n-key cache.
__device__ __forceinline__ bool row_sees(int row, int key, int R, int W, int n, int ke) {
  return key < ke && row < R && key <= n - W + row % W;
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
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      m[rb][i] = kNegInf;
      s[rb][i] = 0.f;
    }

  const int kb = chunk * a.chunk_keys;
  const int ke = min(n, kb + a.chunk_keys);
  const int full_end = min(ke, n - W + 1);     // keys below this are seen by every row
  const int R = a.R;
  using Tile = KTile<T, D>;
  auto load = [&](Tile& tl, int t) { load_tile<T, D>(Kh, t, ke - 1, col, grp, tl.k); };
  pipeline<2, Tile>(kb + stream * 16, ke, TS * 16, load, [&](const Tile& tl, int t) {
    const bool fast = t + 16 <= full_end;
    f32x4 acc[NRB];
    auto logits = [&]() {
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NCH; ++c) acc[rb] = Mma<T>::step(q[rb][c], tl.k[c], acc[rb]);
      }
    };
    logits();
    if (fast) {
      // common case: every key visible and no logit in the wave more than
      // kRefSlack above its row's reference (acc becomes the exponent)
      bool up = false;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[rb][i] = fmaf(acc[rb][i], a.c2, -m[rb][i]);
          up |= acc[rb][i] > kRefSlack;
        }
      if (!__any(up)) {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) s[rb][i] += fast_exp2(acc[rb][i]);
        return;
      }
      logits();   // rare: recompute the tile for the general update
    }
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool valid = fast || row_sees(row0 + rb * 16 + grp * 4 + i, t + col, R, W, n, ke);
        if (valid) {
          const float x = acc[rb][i] * a.c2;
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
  });

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
    // pass 2 takes p = 2^(x - M) * (1/L): the exponent stays near 0 and 1/L
    // is one correctly rounded division, so no per-row rounding of log2 L
    // (about 1e-6 absolute at L ~ 1e5) enters every probability of the row.
    // Padding rows get (-inf, 0), whose p is then 0.
    const bool live = row < a.R && L > 0.f;
    a.stats[(size_t)head * a.rpad + row] = make_float2(live ? -M : kNegInf, live ? 1.f / L : 0.f);
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
    float off[NRB][4], inv[NRB][4];   // -M and 1/L of each row
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2 sv = st[row0 + rb * 16 + grp * 4 + i];
        off[rb][i] = sv.x;
        inv[rb][i] = sv.y;
      }
    // each row half reads its share of every V row once: chunks c with c % RW == half
    const bool norms = rg == 0;
    const int R = a.R;

    constexpr int NV = NCH / RW > 0 ? NCH / RW : 1;
    using Tile = KVTile<T, D, NV>;
    auto load = [&](Tile& tl, int t) {
      load_tile<T, D>(Kh, t, ke - 1, col, grp, tl.k);
      if (norms) {
        const int vkey = min(t + col, ke - 1);
#pragma unroll
        for (int c = 0; c < NV; ++c)
          tl.v[c] = load16(Vh + (size_t)vkey * Row<T, D>::kBytes + ((c * RW + half) * 4 + grp) * 16);
      }
    };
    pipeline<kColsumStages, Tile>(kb + stream * 16, ke, TS * 16, load, [&](const Tile& tl, int t) {
      const bool fast = t + 16 <= full_end;
      const int key = t + col;
      float cs = 0.f;
      f32x4 acc[NRB];
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NCH; ++c) acc[rb] = Mma<T>::step(q[rb][c], tl.k[c], acc[rb]);
      }
      if (fast) {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) cs = fmaf(fast_exp2(fmaf(acc[rb][i], a.c2, off[rb][i])), inv[rb][i], cs);
      } else {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float p = fast_exp2(fmaf(acc[rb][i], a.c2, off[rb][i]));
            const bool vis = row_sees(row0 + rb * 16 + grp * 4 + i, key, R, W, n, ke);
            cs = fmaf(vis ? p : 0.f, inv[rb][i], cs);
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
            const float x = Elem<T>::get(tl.v[c], e);
            ss = fmaf(x, x, ss);
          }
        ss += xor_shfl(ss, 16);
        ss += xor_shfl(ss, 32);
        if (grp == 0 && key < ke) vn_l[half][local] = ss;
      }
    });
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
    const size_t o = (size_t)head * n + k;
    a.attn[o] = av;
    a.vnorm[o] = sqrtf(ss);
  }
}

// Centred moving average of width K over the candidate range, zero outside,
// of c = a * ||v|| (Eq. 1).  The product of the two fp32 outputs is exact in
// fp64 and the K-term sum and the division are taken there too, so the score
// carries one rounding to fp32 beyond the errors of a and ||v||.  Each
// workgroup stages its kPoolOut outputs' products plus the K - 1 halo values
// in LDS (zeros outside [0, n_cand)), then each output sums its K
// neighbours from LDS in ascending position.
constexpr int kPoolOut = 1024;
constexpr int kPoolMaxK = 1025;

__global__ __launch_bounds__(kThreads) void score_pool_kernel(const float* attn, const float* vnorm, float* score,
                                                             int n, int n_cand, int K) {
  __shared__ double tile[kPoolOut + kPoolMaxK - 1];
  const int64_t head = blockIdx.y;
  const int j0 = blockIdx.x * kPoolOut;
  const int h = K / 2;
  const float* av = attn + (size_t)head * n;
  const float* vn = vnorm + (size_t)head * n;
  if (2 * h < kThreads) {
    // the usual small K: every thread's loads are issued before any is
    // stored, so their latencies overlap (kPoolOut / kThreads + 1 each)
    constexpr int kL = kPoolOut / kThreads + 1;
    float x[kL], y[kL];
#pragma unroll
    for (int u = 0; u < kL; ++u) {
      const int jj = min(max(j0 - h + (int)threadIdx.x + u * kThreads, 0), n_cand - 1);   // clamped, masked below
      x[u] = av[jj];
      y[u] = vn[jj];
    }
#pragma unroll
    for (int u = 0; u < kL; ++u) {
      const int i = threadIdx.x + u * kThreads, jj = j0 - h + i;
      if (i < kPoolOut + 2 * h) tile[i] = (jj >= 0 && jj < n_cand) ? (double)x[u] * (double)y[u] : 0.0;
    }
  } else {
    for (int i = threadIdx.x; i < kPoolOut + 2 * h; i += kThreads) {
      const int jj = j0 - h + i;
      const int jc = min(max(jj, 0), n_cand - 1);   // clamped load, masked below
      const double c = (double)av[jc] * (double)vn[jc];
      tile[i] = (jj >= 0 && jj < n_cand) ? c : 0.0;
    }
  }
  __syncthreads();
  for (int q = threadIdx.x; q < kPoolOut; q += kThreads) {
    const int j = j0 + q;
    if (j < n_cand) {
      double sum = 0.0;
      for (int t = 0; t < K; ++t) sum += tile[q + t];
      score[(size_t)head * n_cand + j] = (float)(sum / (double)K);
    }
  }
}

// ---------------------------------------------------------------------------
// Shared-tile passes (bf16, at most 128 window rows).  The workgroup streams
// its key chunk in 32-key tiles that every wave reads from LDS; each thread
// loads 1/256 of a tile with fully contiguous 16-byte loads and keeps
// kDepth tiles of loads in flight (registers), so a workgroup has 4 * 8 KB
// of HBM reads outstanding instead of one tile per wave.  Wave w owns window
// rows 32w .. 32w + 31 (two 16-row MFMA blocks).  LDS rows are stored with
// their 16-byte chunks XOR-swizzled by the row index, so the 16 lanes that
// read one chunk of 16 different rows hit distinct banks.
constexpr int kTK = 32;        // keys per tile
constexpr int kDepth = 4;      // tiles of loads in flight per thread
constexpr int kTiledRows = 128;
// Pass 2 keeps its per-key outputs in LDS and writes them once at the end:
// a global store inside the loop would make every wait for the oldest tile
// also wait for all younger loads (stores and loads retire out of order).
constexpr int kColsumChunk = 4096;

template <int D>
struct TiledGeo {
  static constexpr int RB = D * 2;                       // bytes per bf16 row
  static constexpr int NCHUNK = RB / 16;                 // 16-byte chunks per row
  static constexpr int NCH = RB / 64;                    // MFMA k-steps per row
  static constexpr int TILE = kTK * RB;                  // bytes per tile
  static constexpr int LPT = TILE / (kThreads * 16);     // 16-byte loads per thread per tile
  static_assert(LPT >= 1 && TILE % (kThreads * 16) == 0, "tile must split evenly over the workgroup");
};

// Thread tid's j-th piece of a tile: row and chunk inside the tile.
template <int D>
__device__ __forceinline__ void piece(int j, int tid, int& row, int& ch) {
  const int off = (j * kThreads + tid) * 16;
  row = off / TiledGeo<D>::RB;
  ch = (off % TiledGeo<D>::RB) / 16;
}

template <int D>
__device__ __forceinline__ void issue_tile(const char* Xh, int t0, int ke, int tid,
                                           Chunk16 (&r)[TiledGeo<D>::LPT]) {
#pragma unroll
  for (int j = 0; j < TiledGeo<D>::LPT; ++j) {
    int row, ch;
    piece<D>(j, tid, row, ch);
    const int key = min(t0 + row, ke - 1);
    r[j] = load16(Xh + (size_t)key * TiledGeo<D>::RB + ch * 16);
  }
}

template <int D>
__device__ __forceinline__ int swz(int row, int ch) {
  return row * TiledGeo<D>::RB + ((ch ^ (row & (TiledGeo<D>::NCHUNK - 1))) * 16);
}

template <int D>
__device__ __forceinline__ void commit_tile(char* stage, int tid, const Chunk16 (&r)[TiledGeo<D>::LPT]) {
#pragma unroll
  for (int j = 0; j < TiledGeo<D>::LPT; ++j) {
    int row, ch;
    piece<D>(j, tid, row, ch);
    store16(stage + swz<D>(row, ch), r[j]);
  }
}

// Logits of this wave's 32 rows against the 16 keys kk*16 .. kk*16+15 of the staged tile.
template <int D>
__device__ __forceinline__ void tile_logits(const char* stage, int kk, int col, int grp,
                                            const Chunk16 (&q)[2][TiledGeo<D>::NCH], f32x4 (&acc)[2]) {
  constexpr int NCH = TiledGeo<D>::NCH;
  Chunk16 bf[NCH];
  const int row = kk * 16 + col;
#pragma unroll
  for (int c = 0; c < NCH; ++c) bf[c] = *reinterpret_cast<const Chunk16*>(stage + swz<D>(row, c * 4 + grp));
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) acc[rb] = Mma<bf16_t>::step(q[rb][c], bf[c], acc[rb]);
  }
}

// Drives the tile pipeline: body(stage, tile) for tile = 0 .. ntiles-1 on
// the staged K tile, with after(tile) called once the tile's body has run
// on every wave.  With WITH_V the same rows of V travel alongside in
// registers (never staged) and vhook(tile, pieces) sees them when the K tile
// is stored.  Register slots are indexed statically (the loop is unrolled by
// kDepth) so the compiler waits only for the oldest tile's loads.
template <int D, bool WITH_V, typename VHook, typename Body, typename After>
__device__ __forceinline__ void tiled_stream(const char* Kh, const char* Vh, int kb, int ke, int tid,
                                             char (*lds)[TiledGeo<D>::TILE], VHook&& vhook, Body&& body,
                                             After&& after) {
  constexpr int LPT = TiledGeo<D>::LPT;
  constexpr int NV = WITH_V ? kDepth : 1;
  const int ntiles = (ke - kb + kTK - 1) / kTK;
  Chunk16 rk[kDepth][LPT];
  Chunk16 rv[NV][LPT];
#pragma unroll
  for (int p = 0; p < kDepth; ++p) {
    issue_tile<D>(Kh, kb + p * kTK, ke, tid, rk[p]);
    if constexpr (WITH_V) issue_tile<D>(Vh, kb + p * kTK, ke, tid, rv[p]);
  }
  commit_tile<D>(lds[0], tid, rk[0]);
  if constexpr (WITH_V) vhook(0, rv[0], true);
  issue_tile<D>(Kh, kb + kDepth * kTK, ke, tid, rk[0]);
  if constexpr (WITH_V) issue_tile<D>(Vh, kb + kDepth * kTK, ke, tid, rv[0]);
  __syncthreads();
  // Loads and LDS stores run unconditionally (past the chunk they re-read
  // its last key and fill stages nobody reads), so the register slots look
  // the same on every trip and the compiler waits only for the oldest slot.
  for (int i = 0; i < ntiles; i += kDepth) {
#pragma unroll
    for (int u = 0; u < kDepth; ++u) {
      const int tile = i + u;
      if (tile > 0 && tile <= ntiles) after(tile - 1);
      const int nu = (u + 1) % kDepth;     // a constant once the loop is unrolled
      // consume the slot (K to LDS, V to norms), then refill it
      commit_tile<D>(lds[(tile + 1) & 1], tid, rk[nu]);
      if constexpr (WITH_V) vhook(tile + 1, rv[nu], tile + 1 < ntiles);
      issue_tile<D>(Kh, kb + (tile + 1 + kDepth) * kTK, ke, tid, rk[nu]);
      if constexpr (WITH_V) issue_tile<D>(Vh, kb + (tile + 1 + kDepth) * kTK, ke, tid, rv[nu]);
      if (tile < ntiles) body(lds[tile & 1], tile);
      __syncthreads();
    }
  }
  const int last = (ntiles + kDepth - 1) / kDepth * kDepth;   // tiles the loop ran
  if (ntiles > 0 && last == ntiles) after(ntiles - 1);
}

template <int D>
__global__ __launch_bounds__(kThreads) void score_rowstats_tiled(ScoreArgs a) {
  using Geo = TiledGeo<D>;
  __shared__ __align__(16) char lds[2][Geo::TILE];
  const int chunk = blockIdx.x;
  const int64_t head = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int n = a.n, W = a.W, R = a.R;
  const char* Kh = a.K + (size_t)head * n * Geo::RB;
  const char* Qh = a.Q + (size_t)head * R * Geo::RB;
  const int row0 = wave * 32;
  const bool active = row0 < R;

  Chunk16 q[2][Geo::NCH];
  load_q<bf16_t, D, 2>(Qh, R, row0, col, grp, q);
  float m[2][4], s[2][4];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      m[rb][i] = kNegInf;
      s[rb][i] = 0.f;
    }
  const int kb = chunk * a.chunk_keys;
  const int ke = min(n, kb + a.chunk_keys);
  const int full_end = min(ke, n - W + 1);

  auto no_vhook = [](int, const Chunk16 (&)[Geo::LPT], bool) {};
  auto no_after = [](int) {};
  tiled_stream<D, false>(Kh, nullptr, kb, ke, tid, lds, no_vhook, [&](const char* stage, int tile) {
    if (!active) return;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int t = kb + tile * kTK + kk * 16;
      if (t >= ke) break;
      f32x4 acc[2];
      tile_logits<D>(stage, kk, col, grp, q, acc);
      const bool fast = t + 16 <= full_end;
      if (fast) {
        bool up = false;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            acc[rb][i] = fmaf(acc[rb][i], a.c2, -m[rb][i]);
            up |= acc[rb][i] > kRefSlack;
          }
        if (!__any(up)) {
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) s[rb][i] += fast_exp2(acc[rb][i]);
          continue;
        }
        tile_logits<D>(stage, kk, col, grp, q, acc);
      }
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (fast || row_sees(row0 + rb * 16 + grp * 4 + i, t + col, R, W, n, ke)) {
            const float x = acc[rb][i] * a.c2;
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
  }, no_after);

#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float m2 = xor_shfl(m[rb][i], off);
        const float s2 = xor_shfl(s[rb][i], off);
        lse_merge(m[rb][i], s[rb][i], m2, s2);
      }
  if (col == 0) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a.part[((size_t)head * a.nchunks + chunk) * a.rpad + row0 + rb * 16 + grp * 4 + i] =
            make_float2(m[rb][i], s[rb][i]);
  }
}

// three workgroups per CU: the register budget is capped at 168 VGPRs
template <int D>
__global__ __launch_bounds__(kThreads, 3) void score_colsum_tiled(ScoreArgs a) {
  using Geo = TiledGeo<D>;
  __shared__ __align__(16) char lds[2][Geo::TILE];
  __shared__ float s_cs[2][kWaves][kTK];   // per-wave column sums of a tile
  __shared__ float s_vn[3][kTK];           // squared value norms of a tile
  __shared__ float s_out[2][kColsumChunk]; // a and ||v|| of the chunk's keys
  const int chunk = blockIdx.x;
  const int64_t head = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int n = a.n, W = a.W, R = a.R;
  const char* Kh = a.K + (size_t)head * n * Geo::RB;
  const char* Vh = a.V + (size_t)head * n * Geo::RB;
  const char* Qh = a.Q + (size_t)head * R * Geo::RB;
  const float2* st = a.stats + (size_t)head * a.rpad;
  const int row0 = wave * 32;
  const bool active = row0 < R;

  Chunk16 q[2][Geo::NCH];
  load_q<bf16_t, D, 2>(Qh, R, row0, col, grp, q);
  // -M of each of the lane's rows in registers; 1/L read from LDS where it
  // is used (four consecutive rows per 16-byte read), which keeps the
  // kernel within the register budget of three workgroups per CU
  __shared__ __align__(16) float s_inv[kTiledRows];
  float off[2][4];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) off[rb][i] = st[row0 + rb * 16 + grp * 4 + i].x;
  if (tid < kTiledRows) s_inv[tid] = st[tid].y;   // visible after the stream's first barrier
  const int kb = chunk * a.chunk_keys2;
  const int ke = min(n, kb + a.chunk_keys2);
  const int full_end = min(ke, n - W + 1);
  const float invG = 1.f / (float)a.G;

  // squared value norms: each thread's pieces of a V tile (four bf16 pairs,
  // each squared and summed by one fp32-accumulating dot2), summed over the
  // NCHUNK consecutive threads that hold one row (fixed order)
  auto vnorms = [&](int tile, const Chunk16 (&v)[Geo::LPT], bool live) {
#pragma unroll
    for (int j = 0; j < Geo::LPT; ++j) {
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 x = __builtin_bit_cast(bf16x2, v[j].w[e]);
        ss = __builtin_amdgcn_fdot2_f32_bf16(x, x, ss, false);
      }
#pragma unroll
      for (int o = Geo::NCHUNK / 2; o >= 1; o >>= 1) ss += xor_shfl(ss, o);
      int row, ch;
      piece<D>(j, tid, row, ch);
      if (live && ch == 0) s_vn[tile % 3][row] = ss;
    }
  };

  tiled_stream<D, true>(Kh, Vh, kb, ke, tid, lds, vnorms, [&](const char* stage, int tile) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int t = kb + tile * kTK + kk * 16;
      float cs = 0.f;
      if (active && t < ke) {
        f32x4 acc[2];
        tile_logits<D>(stage, kk, col, grp, q, acc);
        float4 inv[2];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) inv[rb] = *reinterpret_cast<const float4*>(&s_inv[row0 + rb * 16 + grp * 4]);
        if (t + 16 <= full_end) {
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) cs = fmaf(fast_exp2(fmaf(acc[rb][i], a.c2, off[rb][i])), inv[rb][i], cs);
        } else {
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float p = fast_exp2(fmaf(acc[rb][i], a.c2, off[rb][i]));
              const bool vis = row_sees(row0 + rb * 16 + grp * 4 + i, t + col, R, W, n, ke);
              cs = fmaf(vis ? p : 0.f, inv[rb][i], cs);
            }
        }
        cs += xor_shfl(cs, 16);
        cs += xor_shfl(cs, 32);
      }
      if (grp == 0) s_cs[tile & 1][wave][kk * 16 + col] = cs;
    }
  }, [&](int tile) {
    if (tid < kTK) {
      float total = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) total += s_cs[tile & 1][w][tid];
      s_out[0][tile * kTK + tid] = total * invG;
      s_out[1][tile * kTK + tid] = sqrtf(s_vn[tile % 3][tid]);
    }
  });
  __syncthreads();
  for (int k = kb + tid; k < ke; k += kThreads) {
    const size_t o = (size_t)head * n + k;
    a.attn[o] = s_out[0][k - kb];
    a.vnorm[o] = s_out[1][k - kb];
  }
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
    hipLaunchKernelGGL(score_pool_kernel, dim3((s.n_cand + kPoolOut - 1) / kPoolOut, (unsigned)s.heads), blk, 0,
                       st, a.attn, a.vnorm, score, s.n, s.n_cand, pool_kernel);
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

template <int D>
hipError_t launch_tiled(const Shape& s, const ScorePlan& p, ScoreArgs& a, float* score, int pool_kernel,
                        hipStream_t st) {
  const dim3 blk(kThreads);
  hipLaunchKernelGGL(score_rowstats_tiled<D>, dim3(p.nchunks, (unsigned)s.heads), blk, 0, st, a);
  hipLaunchKernelGGL(score_combine_kernel, dim3((unsigned)s.heads), blk, 0, st, a);
  hipLaunchKernelGGL(score_colsum_tiled<D>, dim3(p.nchunks2, (unsigned)s.heads), blk, 0, st, a);
  if (s.n_cand > 0)
    hipLaunchKernelGGL(score_pool_kernel, dim3((s.n_cand + kPoolOut - 1) / kPoolOut, (unsigned)s.heads), blk, 0,
                       st, a.attn, a.vnorm, score, s.n, s.n_cand, pool_kernel);
  return hipGetLastError();
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

ScorePlan plan_score(const Shape& s, int dtype) {
  ScorePlan p{};
  if (dtype == SELKV_BF16 && s.R <= kTiledRows) {
    // shared-tile passes: one row group of 128 (rows past R are padding),
    // chunks of whole 32-key tiles, about kTargetBlocks workgroups
    p.tiled = 1;
    p.rows_per_group = kTiledRows;
    p.nrg = 1;
    p.rpad = kTiledRows;
    const int64_t tiles = (s.n + kTK - 1) / kTK;
    int64_t nchunks = (kTargetBlocks + s.heads - 1) / s.heads;
    if (nchunks > tiles) nchunks = tiles;
    if (nchunks < 1) nchunks = 1;
    int64_t ck = ((s.n + nchunks - 1) / nchunks + kTK - 1) / kTK * kTK;
    const int64_t nt = tiles * kTK;
    const int64_t min_ck = nt < kMinChunkKeys ? nt : kMinChunkKeys;
    if (ck < min_ck) ck = min_ck;
    p.chunk_keys = (int)ck;
    p.nchunks = (int)((s.n + ck - 1) / ck);
    p.chunk_keys2 = (int)(nt < kColsumChunk ? nt : kColsumChunk);
    p.nchunks2 = (int)((s.n + p.chunk_keys2 - 1) / p.chunk_keys2);
    p.part_off = 0;
    p.stats_off = align256((size_t)s.heads * p.nchunks * p.rpad * sizeof(float2));
    p.bytes = p.stats_off + align256((size_t)s.heads * p.rpad * sizeof(float2));
    return p;
  }
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
  p.bytes = p.stats_off + align256((size_t)s.heads * p.rpad * sizeof(float2));
  return p;
}

namespace {

ScoreArgs make_args(const Shape& s, const ScorePlan& p, float scale, const void* K, const void* V, const void* Qwin,
                    float* attn, float* vnorm, void* ws) {
  ScoreArgs a{};
  a.K = static_cast<const char*>(K);
  a.V = static_cast<const char*>(V);
  a.Q = static_cast<const char*>(Qwin);
  a.attn = attn;
  a.vnorm = vnorm;
  char* w = static_cast<char*>(ws);
  a.part = reinterpret_cast<float2*>(w + p.part_off);
  a.stats = reinterpret_cast<float2*>(w + p.stats_off);
  a.n = s.n;
  a.W = s.W;
  a.R = s.R;
  a.G = s.G;
  a.chunk_keys = p.chunk_keys;
  a.nchunks = p.nchunks;
  a.chunk_keys2 = p.chunk_keys2;
  a.rpad = p.rpad;
  a.nrg = p.nrg;
  a.c2 = scale * kLog2e;
  return a;
}

template <typename T, int D>
void launch_rowstats_general(const Shape& s, const ScorePlan& p, const ScoreArgs& a, hipStream_t st) {
  const dim3 grid(p.nchunks, (unsigned)s.heads, p.nrg), blk(kThreads);
  switch (p.rows_per_group) {
    case 16: hipLaunchKernelGGL((score_rowstats_kernel<T, D, 1, 1>), grid, blk, 0, st, a); break;
    case 32: hipLaunchKernelGGL((score_rowstats_kernel<T, D, 2, 1>), grid, blk, 0, st, a); break;
    case 64: hipLaunchKernelGGL((score_rowstats_kernel<T, D, 4, 1>), grid, blk, 0, st, a); break;
    default: hipLaunchKernelGGL((score_rowstats_kernel<T, D, 4, 2>), grid, blk, 0, st, a); break;
  }
}

}  // namespace

hipError_t launch_row_stats(const Shape& s, const ScorePlan& p, int dtype, float scale, const void* K,
                            const void* Qwin, void* ws, hipStream_t st) {
  const ScoreArgs a = make_args(s, p, scale, K, nullptr, Qwin, nullptr, nullptr, ws);
  if (dtype == SELKV_BF16 && p.tiled) {
    if (s.d == 128) hipLaunchKernelGGL(score_rowstats_tiled<128>, dim3(p.nchunks, (unsigned)s.heads), dim3(kThreads),
                                       0, st, a);
    else hipLaunchKernelGGL(score_rowstats_tiled<64>, dim3(p.nchunks, (unsigned)s.heads), dim3(kThreads), 0, st, a);
  } else if (dtype == SELKV_BF16) {
    if (s.d == 128) launch_rowstats_general<bf16_t, 128>(s, p, a, st);
    else launch_rowstats_general<bf16_t, 64>(s, p, a, st);
  } else {
    if (s.d == 128) launch_rowstats_general<float, 128>(s, p, a, st);
    else launch_rowstats_general<float, 64>(s, p, a, st);
  }
  hipLaunchKernelGGL(score_combine_kernel, dim3((unsigned)s.heads), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_score(const Shape& s, const ScorePlan& p, int dtype, float scale, const void* K, const void* V,
                        const void* Qwin, float* score, float* attn, float* vnorm, int pool_kernel, void* ws,
                        hipStream_t st) {
  ScoreArgs a = make_args(s, p, scale, K, V, Qwin, attn, vnorm, ws);
  if (dtype == SELKV_BF16 && p.tiled) {
    if (s.d == 128) return launch_tiled<128>(s, p, a, score, pool_kernel, st);
    return launch_tiled<64>(s, p, a, score, pool_kernel, st);
  }
  if (dtype == SELKV_BF16) {
    if (s.d == 128) return launch_d<bf16_t, 128>(s, p, a, score, pool_kernel, st);
    return launch_d<bf16_t, 64>(s, p, a, score, pool_kernel, st);
  }
  if (s.d == 128) return launch_d<float, 128>(s, p, a, score, pool_kernel, st);
  return launch_d<float, 64>(s, p, a, score, pool_kernel, st);
}

}  // namespace selkv
