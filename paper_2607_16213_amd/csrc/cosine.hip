// Full-cosine routing (the all-pairs alternative of Sec. 3.4) for
// selkv_merge / selkv_bias with SELKV_ROUTE_FULL_COSINE.
//
//   match    per KV head an |E| x |S| x d bf16 (or fp32) MFMA contraction of
//            the evicted value rows against the kept value rows, with the
//            epilogue fused: cos = dot / (||v_j|| ||v_i||) from the fp32 norms,
//            running argmax per evicted row (lowest kept slot on ties), then
//            the gate of Sec. 3.5 from the best cosine.  The |E| x |S| matrix
//            is never written.
//   group    a stable grouping of the evicted tokens by target slot: an LSD
//            radix sort of the target slots carrying the token index (8 bits
//            per pass; block histograms, a scan, ballot-ranked scatter),
//            then every slot's list offset by binary search, so every
//            slot's list ascends.
//   merge    one wave per kept slot: Eq. 5 over its list in a fixed order;
//            keys gathered, values copied bit for bit when nothing is absorbed.
//   bias     one wave per kept slot: Eq. 6 over the same lists.
// All results are independent of scheduling.
#include <algorithm>
#include <cmath>

#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMatchRowBlocks = 4;   // 16-row MFMA blocks of evicted rows per wave

template <typename T, int D>
struct Row {
  static constexpr int kBytes = D * (int)sizeof(T);
  static constexpr int kNch = kBytes / 64;
};

struct MatchArgs {
  const char* V;
  const float* vnorm;
  const int32_t* kept;
  const int32_t* evicted;
  int32_t* target;
  float* gate;
  float* part_best;      // parts > 1: per (head, part, evicted row) best value and slot
  int32_t* part_slot;
  int n, m, gate_mode;
  float tau, inv_temp;
  int parts, part_tiles;   // the kept range split into `parts` runs of part_tiles tiles
  const char* Vk;          // bf16: the kept value rows gathered in slot order, [head][mpad][d]
  const float* ik;         // and their inverse norms, [head][mpad]
  int mpad;
};

// Target and gate of evicted entry e from its best value (dot / ||v_i||) and slot.
__device__ __forceinline__ void write_match(const MatchArgs& a, int64_t head, int e, float best, int slot) {
  const int n = a.n, ne = n - a.m;
  const float vn = a.vnorm[(size_t)head * n + clamp_pos(a.evicted[(size_t)head * ne + e], n)];
  const float cosv = vn > 0.f ? best * (1.f / vn) : 0.f;
  float g;
  if (a.gate_mode == SELKV_GATE_DROP) g = 0.f;
  else if (a.gate_mode == SELKV_GATE_MERGE_ALL) g = 1.f;
  else g = fminf(1.f, fmaxf(0.f, (cosv - a.tau) * a.inv_temp));
  a.target[(size_t)head * ne + e] = slot;
  a.gate[(size_t)head * ne + e] = g;
}

// Evicted rows r0 .. r0+63 of one head against every kept row.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void cosine_match_kernel(MatchArgs a) {
  constexpr int NCH = Row<T, D>::kNch;
  constexpr int RB = Row<T, D>::kBytes;
  constexpr int NRB = kMatchRowBlocks;
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int n = a.n, m = a.m, ne = n - m;
  const int r0 = (blockIdx.x * kWaves + wave) * NRB * 16;
  if (r0 >= ne) return;   // whole wave; no barrier below
  const char* Vh = a.V + (size_t)head * n * RB;
  const float* vnh = a.vnorm + (size_t)head * n;
  const int32_t* kh = a.kept + (size_t)head * m;
  const int32_t* eh = a.evicted + (size_t)head * ne;

  // A operand: evicted value rows (lane row = col), chunks 4c + grp
  Chunk16 q[NRB][NCH];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    const int e = min(r0 + rb * 16 + col, ne - 1);
    const int pos = clamp_pos(eh[e], n);
#pragma unroll
    for (int c = 0; c < NCH; ++c) q[rb][c] = load16(Vh + (size_t)pos * RB + (c * 4 + grp) * 16);
  }
  // inverse norms of the output rows of this lane (rows 4*grp + i of each block)
  float inv_j[NRB][4], best[NRB][4];
  int bidx[NRB][4];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = min(r0 + rb * 16 + grp * 4 + i, ne - 1);
      const float vn = vnh[clamp_pos(eh[e], n)];
      inv_j[rb][i] = vn > 0.f ? 1.f / vn : 0.f;
      best[rb][i] = kNegInf;
      bidx[rb][i] = 0;
    }

  // kept tiles of 16 rows; the next tile's loads are issued before this one is used
  Chunk16 kcur[NCH], knxt[NCH];
  float icur, inxt;
  {
    const int pos = clamp_pos(kh[min(col, m - 1)], n);
#pragma unroll
    for (int c = 0; c < NCH; ++c) kcur[c] = load16(Vh + (size_t)pos * RB + (c * 4 + grp) * 16);
    const float vn = vnh[pos];
    icur = vn > 0.f ? 1.f / vn : 0.f;
  }
  for (int t = 0; t < m; t += 16) {
    {
      const int pos = clamp_pos(kh[min(t + 16 + col, m - 1)], n);
#pragma unroll
      for (int c = 0; c < NCH; ++c) knxt[c] = load16(Vh + (size_t)pos * RB + (c * 4 + grp) * 16);
      const float vn = vnh[pos];
      inxt = vn > 0.f ? 1.f / vn : 0.f;
    }
    const int slot = t + col;
    const bool valid = slot < m;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NCH; ++c) acc = Mma<T>::step(q[rb][c], kcur[c], acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = acc[i] * icur * inv_j[rb][i];
        if (valid && v > best[rb][i]) {   // slots rise along the lane: ties keep the lower slot
          best[rb][i] = v;
          bidx[rb][i] = slot;
        }
      }
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) kcur[c] = knxt[c];
    icur = inxt;
  }

  // merge the 16 lanes (slot subsets) of each row: larger cosine, then lower slot
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float ob = xor_shfl(best[rb][i], off);
        const int oi = xor_shfl(bidx[rb][i], off);
        if (ob > best[rb][i] || (ob == best[rb][i] && oi < bidx[rb][i])) {
          best[rb][i] = ob;
          bidx[rb][i] = oi;
        }
      }
  if (col == 0) {
    int32_t* th = a.target + (size_t)head * ne;
    float* gh = a.gate + (size_t)head * ne;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = r0 + rb * 16 + grp * 4 + i;
        if (e < ne) {
          float g;
          if (a.gate_mode == SELKV_GATE_DROP) g = 0.f;
          else if (a.gate_mode == SELKV_GATE_MERGE_ALL) g = 1.f;
          else g = fminf(1.f, fmaxf(0.f, (best[rb][i] - a.tau) * a.inv_temp));
          th[e] = bidx[rb][i];
          gh[e] = g;
        }
      }
  }
}

// bf16 variant with the kept rows shared through LDS.  The kept value rows
// are first copied in slot order into a contiguous block (gather_kept_kernel,
// with their inverse norms), so the match reads each tile from one base
// address with no index loads.  A workgroup holds 256 evicted rows (64 per
// wave, in registers) and streams the head's kept rows in tiles of 64 through
// two LDS stages that all four waves read.  The tiles go straight into LDS by
// 16-byte LDS-DMA loads (no register staging): a wave's load fills 1 KB of
// LDS in lane order, so each lane loads the kept row and 16-byte chunk whose
// XOR-swizzled place is its own slot.  Only one inverse norm per thread
// passes through registers, which keeps the kernel at three waves per SIMD
// with registers to spare.  The kept tile
// is the MFMA A operand and the evicted rows the B operand, so lane (g, c)
// receives slots 4g .. 4g+3 of a 16-slot block for evicted row c: its four
// candidates for one row.  The running argmax takes their maximum with the
// running best (two max3) and looks up which slot it was only when the best
// improves, which becomes rare along the stream.  It compares
// dot * (1 / ||v_i||) only: the evicted row's own norm does not change its
// argmax and is applied once, to the winner, for the gate.
constexpr int kMT = 64;          // kept rows per tile
constexpr int kMatchTiledRB = 4; // 16-row blocks of evicted rows per wave

template <int D>
struct MGeo {
  static constexpr int RB = D * 2;
  static constexpr int NCHUNK = RB / 16;
  static constexpr int NCH = RB / 64;
  static constexpr int TILE = kMT * RB;
  static constexpr int LPT = TILE / (kThreads * 16);   // LDS-DMA loads per thread per tile
  static_assert(LPT >= 1 && TILE % (kThreads * 16) == 0, "tile must split evenly over the workgroup");
};

template <int D>
__device__ __forceinline__ int mswz(int row, int ch) {
  return row * MGeo<D>::RB + ((ch ^ (row & (MGeo<D>::NCHUNK - 1))) * 16);
}

// The LDS bytes that load j of wave w fills: [(j * kWaves + w) * 1024, + 1024),
// lane L at + 16 L.  Returns the tile row and the (unswizzled) chunk whose
// swizzled place that is.
template <int D>
__device__ __forceinline__ void dma_piece(int j, int wave, int lane, int& row, int& ch) {
  const int p = (j * kWaves + wave) * 1024 + lane * 16;
  row = p / MGeo<D>::RB;
  ch = ((p % MGeo<D>::RB) / 16) ^ (row & (MGeo<D>::NCHUNK - 1));
}

// Kept value rows of every head copied in slot order into Vk, with 1 / ||v||
// per row (0 for a zero row), for the bf16 match.  Rows m .. mpad - 1 repeat
// row m - 1, so the match's tiles past the last kept slot need no mask.
template <int D>
__global__ __launch_bounds__(kThreads) void gather_kept_kernel(const char* V, const float* vnorm, const int32_t* kept,
                                                               char* Vk, float* ik, int n, int m, int mpad) {
  constexpr int RB = D * 2, NCHUNK = RB / 16;
  const int64_t head = blockIdx.y;
  const int64_t idx = blockIdx.x * (int64_t)kThreads + threadIdx.x;
  const int slot = (int)(idx / NCHUNK), ch = (int)(idx % NCHUNK);
  if (slot >= mpad) return;
  const int pos = clamp_pos(kept[(size_t)head * m + min(slot, m - 1)], n);
  store16(Vk + ((size_t)head * mpad + slot) * RB + ch * 16, load16(V + ((size_t)head * n + pos) * RB + ch * 16));
  if (ch == 0) {
    const float rn = vnorm[(size_t)head * n + pos];
    ik[(size_t)head * mpad + slot] = rn > 0.f ? 1.f / rn : 0.f;
  }
}

template <int D>
__global__ __launch_bounds__(kThreads, 3) void cosine_match_tiled(MatchArgs a) {
  using Geo = MGeo<D>;
  constexpr int NCH = Geo::NCH, LPT = Geo::LPT, NRB = kMatchTiledRB;
  // two stages as separate arrays, addressed statically (the tile loop is
  // unrolled by two), so that reading one stage never waits for the loads
  // still filling the other
  __shared__ __align__(16) char lds0[Geo::TILE], lds1[Geo::TILE];
  __shared__ __align__(16) float s_inv0[kMT], s_inv1[kMT];   // 1 / ||v_i|| of the tile's kept rows
  const int64_t head = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int n = a.n, m = a.m, ne = n - m;
  // workgroup x: evicted row block x / parts against the kept tiles of run x % parts
  const int part = blockIdx.x % a.parts;
  const int r0 = ((blockIdx.x / a.parts) * kWaves + wave) * NRB * 16;
  const bool active = r0 < ne;
  const int t_begin = part * a.part_tiles;
  const int t_end = min((m + kMT - 1) / kMT, t_begin + a.part_tiles);
  const char* Vh = a.V + (size_t)head * n * Geo::RB;
  const int32_t* eh = a.evicted + (size_t)head * ne;

  Chunk16 q[NRB][NCH];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    const int pos = clamp_pos(eh[min(r0 + rb * 16 + col, ne - 1)], n);
#pragma unroll
    for (int c = 0; c < NCH; ++c) q[rb][c] = load16(Vh + (size_t)pos * Geo::RB + (c * 4 + grp) * 16);
  }
  float best[NRB];   // evicted row rb*16 + col, over the slots 4g .. 4g+3 of every block
  int bidx[NRB];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    best[rb] = kNegInf;
    bidx[rb] = 0;
  }

  const int ntiles = max(0, t_end - t_begin);   // tiles of this run; tile t is kept tile t_begin + t
  const char* Vkh = a.Vk + (size_t)head * a.mpad * Geo::RB;
  const float* ikh = a.ik + (size_t)head * a.mpad;
  float rn = 0.f;   // the inverse norm of slot tid & (kMT - 1) of the tile in flight
  // Past the run a trip reads the next run's kept rows (true slots, which
  // that run reports as well); past the last kept slot the gathered block
  // repeats row m - 1 under higher slot numbers: equal values, and ties keep
  // the lower slot, so nothing needs masking and every trip issues the same
  // loads.  The block holds two tiles beyond the last (mpad rows), which
  // covers the trip an odd tile count adds and the load it issues ahead.
  auto issue_tile = [&](int tile, char* stage) {
    const char* tb = Vkh + (size_t)(t_begin + tile) * kMT * Geo::RB;
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      int row, ch;
      dma_piece<D>(j, wave, lane, row, ch);
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(tb + row * Geo::RB + ch * 16),
                                       (__attribute__((address_space(3))) void*)(stage + (j * kWaves + wave) * 1024),
                                       16, 0, 0);
    }
    rn = ikh[(t_begin + tile) * kMT + (tid & (kMT - 1))];
  };
  auto commit_norm = [&](float* sinv) {
    if (tid < kMT) sinv[tid] = rn;
  };
  // value = dot * (1 / ||v_i||)
  // the MFMAs of column block kk + 1 are issued before the epilogue of block
  // kk, so the matrix core and the VALU work on independent data
  auto mfma_block = [&](const char* stage, int kk, f32x4 (&acc)[NRB]) {
    const int row = kk * 16 + col;
    Chunk16 bf[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) bf[c] = *reinterpret_cast<const Chunk16*>(stage + mswz<D>(row, c * 4 + grp));
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NCH; ++c) acc[rb] = Mma<bf16_t>::step(bf[c], q[rb][c], acc[rb]);
    }
  };
  auto epilogue = [&](const float* sinv, int tile, int kk, const f32x4 (&acc)[NRB]) {
    const int s0 = kk * 16 + grp * 4;
    const f32x4 inv = *reinterpret_cast<const f32x4*>(sinv + s0);
    const int slot0 = (t_begin + tile) * kMT + s0;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      const float v0 = acc[rb][0] * inv[0];
      const float v1 = acc[rb][1] * inv[1];
      const float v2 = acc[rb][2] * inv[2];
      const float v3 = acc[rb][3] * inv[3];
      const float mx = fmaxf(fmaxf(best[rb], v0), fmaxf(fmaxf(v1, v2), v3));
      // slots rise along the stream: only a strictly larger value moves the
      // best, and the lowest of the four slots holding it is taken
      if (mx > best[rb]) {   // the lowest of the four equal to mx: one find-first-set on their flags
        const uint32_t eq = (v0 == mx ? 1u : 0u) | (v1 == mx ? 2u : 0u) | (v2 == mx ? 4u : 0u) | 8u;
        bidx[rb] = slot0 + (int)__builtin_ctz(eq);
        best[rb] = mx;
      }
    }
  };
  auto body = [&](const char* stage, const float* sinv, int tile) {
    f32x4 acc[2][NRB];
    mfma_block(stage, 0, acc[0]);
#pragma unroll
    for (int kk = 0; kk < kMT / 16; ++kk) {
      if (kk + 1 < kMT / 16) mfma_block(stage, kk + 1, acc[(kk + 1) & 1]);
      epilogue(sinv, tile, kk, acc[kk & 1]);
    }
  };
  // trip t: the other stage was released by the last barrier, so tile t+1 is
  // gathered into it while tile t is used; the barrier at the end waits for
  // every load of the trip, issued a whole tile body earlier
  auto trip = [&](int cur, char* Lc, float* ic, char* Ln, float* in_, int t) {
    issue_tile(t + 1, Ln);
    body(Lc, ic, t);
    commit_norm(in_);
    __syncthreads();
  };

  issue_tile(0, lds0);
  commit_norm(s_inv0);
  __syncthreads();
  // two trips per pass; an odd tile count runs one trip past the run (see
  // issue_tile: its slots need no mask)
  for (int t = 0; t < ntiles; t += 2) {
    trip(0, lds0, s_inv0, lds1, s_inv1, t);
    trip(1, lds1, s_inv1, lds0, s_inv0, t + 1);
  }

  if (!active) return;
  // merge the four lane groups (slot subsets) of each row: larger value, then lower slot
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int off = 16; off < 64; off <<= 1) {
      const float ob = xor_shfl(best[rb], off);
      const int oi = xor_shfl(bidx[rb], off);
      if (ob > best[rb] || (ob == best[rb] && oi < bidx[rb])) {
        best[rb] = ob;
        bidx[rb] = oi;
      }
    }
  if (grp == 0) {
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      const int e = r0 + rb * 16 + col;
      if (e < ne) {
        if (a.parts == 1) {
          write_match(a, head, e, best[rb], bidx[rb]);
        } else {
          const size_t o = ((size_t)head * a.parts + part) * ne + e;
          a.part_best[o] = best[rb];
          a.part_slot[o] = bidx[rb];
        }
      }
    }
  }
}

// The runs' results of every evicted row, merged in run (= slot) order: a
// strictly larger value replaces the best, so equal values keep the lower slot.
__global__ __launch_bounds__(kThreads) void match_parts_kernel(MatchArgs a) {
  const int64_t head = blockIdx.y;
  const int ne = a.n - a.m;
  const int e = blockIdx.x * kThreads + threadIdx.x;
  if (e >= ne) return;
  float best = kNegInf;
  int slot = 0;
  for (int p = 0; p < a.parts; ++p) {
    const size_t o = ((size_t)head * a.parts + p) * ne + e;
    const float v = a.part_best[o];
    if (v > best) {
      best = v;
      slot = a.part_slot[o];
    }
  }
  write_match(a, head, e, best, slot);
}


// In place: cnt[head][0..m] becomes the exclusive prefix sum (cnt[m] = total).
// Rounds of 1024 x kScanRun entries: each thread loads its kScanRun
// consecutive entries at once and scans them in order, the workgroup scans
// the thread totals, so a round costs one load latency.
constexpr int kScanRun = 8;

__global__ __launch_bounds__(1024) void group_scan_kernel(int32_t* cnt, int m) {
  const int64_t head = blockIdx.x;
  int32_t* c = cnt + (size_t)head * (m + 1);
  __shared__ int s_w[16];
  __shared__ int s_run;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) s_run = 0;
  __syncthreads();
  for (int base = 0; base <= m; base += 1024 * kScanRun) {
    const int i0 = base + tid * kScanRun;
    int v[kScanRun];
#pragma unroll
    for (int r = 0; r < kScanRun; ++r) v[r] = (i0 + r < m) ? c[i0 + r] : 0;
    int t = 0;
#pragma unroll
    for (int r = 0; r < kScanRun; ++r) {   // exclusive within the thread's run
      const int x = v[r];
      v[r] = t;
      t += x;
    }
    const int incl = wave_inclusive_scan(t, lane);
    if (lane == 63) s_w[wave] = incl;
    __syncthreads();
    int woff = 0;
    for (int w = 0; w < wave; ++w) woff += s_w[w];
    int total = 0;
    for (int w = 0; w < 16; ++w) total += s_w[w];
    const int run = s_run;
    const int pre = run + woff + incl - t;
#pragma unroll
    for (int r = 0; r < kScanRun; ++r)
      if (i0 + r <= m) c[i0 + r] = pre + v[r];
    __syncthreads();
    if (tid == 0) s_run = run + total;
    __syncthreads();
  }
}

// Stable grouping of the evicted tokens by target slot as an LSD radix sort
// of the keys (target slot, or m for a token routed nowhere) carrying the
// token index, 8 key bits per pass.  Each pass: a digit histogram per block
// of kSortBlock tokens (digit-major table), the exclusive scan of the table
// per head, and a scatter in which each block ranks its tokens stably: wave
// w takes the block's tokens w*512 .. w*512+511 in eight rounds of 64; a
// token's rank among equal digits in its round comes from ballots, the
// wave's running count per digit lives in LDS (a wave's LDS accesses stay in
// program order), and the waves' counts are prefixed in wave order.  Equal
// keys therefore keep ascending token order, so every slot's list ascends.
// Then off[s] = the first sorted position whose key is >= s (binary search).
constexpr int kSortWaveTok = 512;                   // tokens per wave per block
constexpr int kSortBlock = kWaves * kSortWaveTok;   // tokens per block
constexpr int kBins = 256;                          // 8-bit digits

__device__ __forceinline__ int sort_key(const int32_t* keys_in, const int32_t* th, int e, int m) {
  if (keys_in) return keys_in[e];
  const int t = th[e];
  return (t >= 0 && t < m) ? t : m;
}

// keys_in == nullptr: the first pass, keys from the targets, values = token index
__global__ __launch_bounds__(kThreads) void sort_hist_kernel(const int32_t* keys_in, const int32_t* target,
                                                             int32_t* table, int ne, int m, int shift, int nblk) {
  __shared__ int hist[kBins];
  const int64_t head = blockIdx.y;
  const int blk = blockIdx.x, tid = threadIdx.x;
  const int32_t* kin = keys_in ? keys_in + (size_t)head * ne : nullptr;
  const int32_t* th = target + (size_t)head * ne;
  for (int d = tid; d < kBins; d += kThreads) hist[d] = 0;
  __syncthreads();
  for (int k = 0; k < kSortBlock / kThreads; ++k) {
    const int e = blk * kSortBlock + k * kThreads + tid;
    if (e < ne) atomicAdd(&hist[(sort_key(kin, th, e, m) >> shift) & (kBins - 1)], 1);
  }
  __syncthreads();
  int32_t* tab = table + (size_t)head * (kBins * nblk + 1);
  for (int d = tid; d < kBins; d += kThreads) tab[(size_t)d * nblk + blk] = hist[d];
}

__global__ __launch_bounds__(kThreads) void sort_scatter_kernel(const int32_t* keys_in, const int32_t* vals_in,
                                                                const int32_t* target, const int32_t* table,
                                                                int32_t* keys_out, int32_t* vals_out, int ne, int m,
                                                                int shift, int nblk) {
  constexpr int R = kSortWaveTok / 64;
  __shared__ int wcnt[kWaves][kBins];
  const int64_t head = blockIdx.y;
  const int blk = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int32_t* kin = keys_in ? keys_in + (size_t)head * ne : nullptr;
  const int32_t* vin = vals_in ? vals_in + (size_t)head * ne : nullptr;
  const int32_t* th = target + (size_t)head * ne;
  for (int d = tid; d < kWaves * kBins; d += kThreads) wcnt[d / kBins][d % kBins] = 0;
  __syncthreads();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int key[R], val[R], rnk[R];
  const int base = blk * kSortBlock + wave * kSortWaveTok;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int e = base + r * 64 + lane;
    const bool valid = e < ne;
    const int ec = valid ? e : ne - 1;
    key[r] = sort_key(kin, th, ec, m);
    val[r] = vin ? vin[ec] : ec;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const bool valid = base + r * 64 + lane < ne;
    const int d = (key[r] >> shift) & (kBins - 1);
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {                  // lanes holding the same digit
      const bool one = (d >> bit) & 1;
      const uint64_t ones = __ballot(valid && one);
      peers &= one ? ones : ~ones;
    }
    if (!valid) peers = 0ull;
    const int before = wcnt[wave][d];
    rnk[r] = before + __popcll(peers & below);
    const bool last = valid && ((peers >> lane) >> 1) == 0ull;    // highest lane of its digit
    if (last) wcnt[wave][d] = before + __popcll(peers);
  }
  __syncthreads();
  // per digit: the counts of the waves before each wave
  for (int d = tid; d < kBins; d += kThreads) {
    int run = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int c = wcnt[w][d];
      wcnt[w][d] = run;
      run += c;
    }
  }
  __syncthreads();
  const int32_t* tab = table + (size_t)head * (kBins * nblk + 1);
  int32_t* ko = keys_out + (size_t)head * ne;
  int32_t* vo = vals_out + (size_t)head * ne;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (base + r * 64 + lane < ne) {
      const int d = (key[r] >> shift) & (kBins - 1);
      const int dst = tab[(size_t)d * nblk + blk] + wcnt[wave][d] + rnk[r];
      ko[dst] = key[r];
      vo[dst] = val[r];
    }
  }
}

// off[head][s] for s = 0 .. m: the first position of the sorted keys that is >= s.
__global__ __launch_bounds__(kThreads) void sort_offsets_kernel(const int32_t* keys, int32_t* off, int ne, int m) {
  const int64_t head = blockIdx.y;
  const int s = blockIdx.x * kThreads + threadIdx.x;
  if (s > m) return;
  const int32_t* k = keys + (size_t)head * ne;
  int lo = 0, hi = ne;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (k[mid] < s) lo = mid + 1;
    else hi = mid;
  }
  off[(size_t)head * (m + 1) + s] = lo;
}

// The listed tokens' positions and Eq. 5 weights g_j * a_j, in list order:
// gathered once here so the merge reads them without a chain of dependent
// lookups (token index -> position -> attention) per slot.
__global__ __launch_bounds__(kThreads) void group_payload_kernel(const int32_t* list, const int32_t* evicted,
                                                                 const float* gate, const float* attn,
                                                                 int32_t* lpos, float* lw, int n, int ne) {
  const int64_t head = blockIdx.y;
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= ne) return;
  const size_t o = (size_t)head * ne + i;
  const int e = (int)min((uint32_t)list[o], (uint32_t)(ne - 1));
  const int jp = clamp_pos(evicted[(size_t)head * ne + e], n);
  lpos[o] = jp;
  lw[o] = weight_rn(gate[(size_t)head * ne + e], attn[(size_t)head * n + jp]);
}

struct GroupMergeArgs {
  const char* K;
  const char* V;
  const float* attn;
  const int32_t* kept;
  const int32_t* off;
  const int32_t* lpos;   // per list entry: the token's position
  const float* lw;       // and its weight g * a
  char* K_out;
  char* V_out;
  float* bias;
  int n, m;
  float alpha;
  int raw;   // bias mode: write wsum / a_s (R - 1) instead of alpha * ln R
};

// Eq. 5 (and the Eq. 6 bias when `bias` is set) per kept slot, kSlotsPerWave
// consecutive slots per wave: their lists are contiguous in the sorted order,
// so the wave walks the combined range [off[s0], off[s0 + kSlotsPerWave]) in
// chunks of 64 entries.  Entry p of the range (counted from its start) goes to
// lane group p % 4, which adds it to its running sums of the entry's slot;
// the four lane groups' sums of a slot combine as (g0 + g1) + (g2 + g3), and
// lane group k writes slot s0 + k.  A slot's sums are thus formed in one
// fixed order, the same in the values pass and the bias pass, and a long list
// still spreads over all four lane groups.
// MK (values mode only): keys merged with the value weights instead of gathered
constexpr int kSlotsPerWave = 4;   // one per lane group

template <typename T, int D, bool VALUES, bool MK>
__global__ __launch_bounds__(kThreads) void group_merge_kernel(GroupMergeArgs a) {
  constexpr int E = Slice<T, D>::kElems;
  constexpr int RB = D * (int)sizeof(T);
  constexpr int SPW = kSlotsPerWave;
  constexpr int EK = MK ? E : 1;
  const int64_t head = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int s0 = (blockIdx.x * kWaves + wave) * SPW;
  const int n = a.n, m = a.m, ne = n - m;
  if (s0 >= m) return;
  const int32_t* kh = a.kept + (size_t)head * m;
  const int32_t* oh = a.off + (size_t)head * (m + 1);
  const int32_t* ph = a.lpos + (size_t)head * ne;
  const float* wh = a.lw + (size_t)head * ne;
  const float* ah = a.attn + (size_t)head * n;
  // list bounds of the wave's slots; slots past m have empty lists, and with
  // nothing evicted there are no lists (the grouping wrote no offsets)
  int L[SPW + 1];
#pragma unroll
  for (int k = 0; k <= SPW; ++k) L[k] = ne > 0 ? oh[min(s0 + k, m)] : 0;
  // lane group grp owns slot s0 + grp: its rows are loaded ahead of the walk
  const int my = s0 + grp;
  const int pos = clamp_pos(kh[min(my, m - 1)], n);
  RawSlice<T, D> kr, vr;
  if constexpr (VALUES) {
    kr.load(a.K + ((size_t)head * n + pos) * RB, col);
    vr.load(a.V + ((size_t)head * n + pos) * RB, col);
  }
  const float a_s = ah[pos];

  float acc[SPW][VALUES ? E : 1], kacc[SPW][EK], wsum[SPW];
#pragma unroll
  for (int k = 0; k < SPW; ++k) {
#pragma unroll
    for (int e = 0; e < (VALUES ? E : 1); ++e) acc[k][e] = 0.f;
#pragma unroll
    for (int e = 0; e < EK; ++e) kacc[k][e] = 0.f;
    wsum[k] = 0.f;
  }
  for (int lb = L[0]; lb < L[SPW]; lb += 64) {
    // lane-parallel metadata of up to 64 entries: position, weight, slot
    const int li = lb + lane;
    int jp = 0, sk = 0;
    float w = 0.f;
    if (li < L[SPW]) {
      jp = ph[li];
      w = wh[li];
#pragma unroll
      for (int k = 1; k < SPW; ++k) sk += li >= L[k] ? 1 : 0;
    }
    const int cnt = min(64, L[SPW] - lb);
    constexpr int kBatch = 4;
    for (int ib0 = 0; ib0 < cnt; ib0 += 4 * kBatch) {
      int jj[kBatch], kk[kBatch];
      float wv[kBatch];
      RawSlice<T, D> vv[VALUES ? kBatch : 1], kre[MK ? kBatch : 1];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = ib0 + 4 * u + grp;
        const int src = i < cnt ? i : 0;
        // the shuffles run on every lane: a shuffle under a lane-dependent
        // condition would read inactive source lanes
        jj[u] = __shfl(jp, src, 64);
        wv[u] = __shfl(w, src, 64);
        kk[u] = __shfl(sk, src, 64);
      }
      if constexpr (VALUES) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) vv[u].load(a.V + ((size_t)head * n + jj[u]) * RB, col);
      }
      if constexpr (MK) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) kre[u].load(a.K + ((size_t)head * n + jj[u]) * RB, col);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (ib0 + 4 * u + grp < cnt) {
#pragma unroll
          for (int k = 0; k < SPW; ++k) {
            const bool hit = kk[u] == k;
            if constexpr (VALUES) {
#pragma unroll
              for (int e = 0; e < E; ++e) acc[k][e] = hit ? fmaf(wv[u], vv[u].get(e), acc[k][e]) : acc[k][e];
            }
            if constexpr (MK) {
#pragma unroll
              for (int e = 0; e < E; ++e) kacc[k][e] = hit ? fmaf(wv[u], kre[u].get(e), kacc[k][e]) : kacc[k][e];
            }
            wsum[k] = hit ? wsum[k] + wv[u] : wsum[k];
          }
        }
      }
    }
  }
  // (g0 + g1) + (g2 + g3) on every lane, then lane group grp keeps its slot's sums
  float mw = 0.f, mv[VALUES ? E : 1], mk[EK];
#pragma unroll
  for (int e = 0; e < (VALUES ? E : 1); ++e) mv[e] = 0.f;
#pragma unroll
  for (int e = 0; e < EK; ++e) mk[e] = 0.f;
#pragma unroll
  for (int k = 0; k < SPW; ++k) {
    wsum[k] += xor_shfl(wsum[k], 16);
    wsum[k] += xor_shfl(wsum[k], 32);
    mw = grp == k ? wsum[k] : mw;
    if constexpr (VALUES) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        acc[k][e] += xor_shfl(acc[k][e], 16);
        acc[k][e] += xor_shfl(acc[k][e], 32);
        mv[e] = grp == k ? acc[k][e] : mv[e];
      }
    }
    if constexpr (MK) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        kacc[k][e] += xor_shfl(kacc[k][e], 16);
        kacc[k][e] += xor_shfl(kacc[k][e], 32);
        mk[e] = grp == k ? kacc[k][e] : mk[e];
      }
    }
  }
  if (my >= m) return;
  // the Eq. 6 bias of the slot from the same absorbed mass (fused call, or the bias pass)
  if (a.bias != nullptr && col == 0) a.bias[(size_t)head * m + my] = ratio_bias(mw, a_s, a.alpha, a.raw != 0);
  if constexpr (VALUES) {
    if (mw > 0.f) {
      const float den = a_s + mw;
      RawSlice<T, D> ov;
#pragma unroll
      for (int e = 0; e < E; ++e) ov.put(e, fmaf(a_s, vr.get(e), mv[e]) / den);
      ov.store(a.V_out + ((size_t)head * m + my) * RB, col);
      if constexpr (MK) {
        RawSlice<T, D> ok;
#pragma unroll
        for (int e = 0; e < E; ++e) ok.put(e, fmaf(a_s, kr.get(e), mk[e]) / den);
        ok.store(a.K_out + ((size_t)head * m + my) * RB, col);
      } else {
        kr.store(a.K_out + ((size_t)head * m + my) * RB, col);
      }
    } else {
      kr.store(a.K_out + ((size_t)head * m + my) * RB, col);
      vr.store(a.V_out + ((size_t)head * m + my) * RB, col);
    }
  }
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

namespace {

// Runs the kept range of the bf16 match is split into.  A match workgroup
// (one per 256 evicted rows) is long-lived and three fit on each of the 256
// CUs, so with one run per row block the last round of workgroups can leave
// most CUs idle: the run count doubles until the launch holds at least six
// rounds of workgroups (each run keeping at least 8 tiles).  It stays a power
// of two because consecutive workgroups go to the eight XCDs in turn: with a
// run count dividing eight, every XCD serves one run, so its L2 holds half
// or a quarter of a head's kept rows instead of all of them.  On one
// 102400-token layer (8 heads) 2 runs take 3.37 ms, 4 runs 3.40 ms, and 3 or
// 6 runs, whose workgroups of one run spread over every XCD, 3.5 - 3.6 ms.
// A run past the last tile (possible when the split is fine) does no work
// and reports -inf, which the merge of the runs skips.
int match_parts(const Shape& s) {
  const int64_t ne = s.n - s.m;
  if (ne <= 0) return 1;
  const int64_t row_wgs = (ne + kWaves * kMatchTiledRB * 16 - 1) / (kWaves * kMatchTiledRB * 16) * s.heads;
  const int64_t cap = std::max<int64_t>(1, ((int64_t)s.m + kMT - 1) / kMT / 8);   // runs of at least 8 tiles
  const int64_t slots = 256 * 3;
  int64_t p = 1;
  while (2 * p <= cap && row_wgs * p < 6 * slots) p *= 2;
  return (int)p;
}

}  // namespace

int sort_passes(int m) {
  int bits = 1;
  while ((1ll << bits) < (int64_t)m + 1) ++bits;      // keys 0 .. m
  return (bits + 7) / 8;
}

GroupPlan plan_group(const Shape& s, int dtype) {
  GroupPlan p{};
  const size_t ne = (size_t)(s.n - s.m);
  const size_t nel = ne > 0 ? ne : 1;
  const int nblk = (int)((nel + kSortBlock - 1) / kSortBlock);
  p.off_off = 0;
  p.table_off = align256((size_t)s.heads * (s.m + 1) * sizeof(int32_t));
  p.keys_off[0] = p.table_off + align256((size_t)s.heads * ((size_t)kBins * nblk + 1) * sizeof(int32_t));
  p.vals_off[0] = p.keys_off[0] + align256(nel * (size_t)s.heads * sizeof(int32_t));
  p.keys_off[1] = p.vals_off[0] + align256(nel * (size_t)s.heads * sizeof(int32_t));
  p.vals_off[1] = p.keys_off[1] + align256(nel * (size_t)s.heads * sizeof(int32_t));
  p.bytes = p.vals_off[1] + align256(nel * (size_t)s.heads * sizeof(int32_t));
  p.passes = sort_passes(s.m);
  p.list_off = p.vals_off[(p.passes - 1) & 1];    // the last pass's values
  // the match's scratch (per-run results; bf16: the gathered kept rows and
  // their inverse norms) comes first and is consumed before the grouping starts
  const int parts = match_parts(s);
  p.match_parts = parts;
  size_t match_bytes = 0;
  if (parts > 1) {
    p.match_slot_off = align256((size_t)s.heads * parts * ne * sizeof(float));
    match_bytes = p.match_slot_off + align256((size_t)s.heads * parts * ne * sizeof(int32_t));
  }
  if (dtype == SELKV_BF16 && ne > 0) {
    // two tiles past the last: the trip an odd run adds and the load it issues ahead
    p.match_mpad = ((s.m + kMT - 1) / kMT + 2) * kMT;
    p.match_vk_off = match_bytes;
    p.match_ik_off = p.match_vk_off + align256((size_t)s.heads * p.match_mpad * s.d * 2);
    match_bytes = p.match_ik_off + align256((size_t)s.heads * p.match_mpad * sizeof(float));
  }
  p.bytes = std::max(p.bytes, match_bytes);
  return p;
}

hipError_t launch_cosine_match(const Shape& s, const GroupPlan& gp, int dtype, int gate_mode, float tau, float temp,
                               const void* V, const float* vnorm, const int32_t* kept, const int32_t* evicted,
                               int32_t* target, float* gate, void* ws, hipStream_t st) {
  const int ne = s.n - s.m;
  if (ne <= 0) return hipSuccess;
  MatchArgs a{};
  a.V = static_cast<const char*>(V);
  a.vnorm = vnorm;
  a.kept = kept;
  a.evicted = evicted;
  a.target = target;
  a.gate = gate;
  a.n = s.n;
  a.m = s.m;
  a.gate_mode = gate_mode;
  a.tau = tau;
  a.inv_temp = 1.f / temp;
  a.parts = 1;
  a.part_tiles = (s.m + kMT - 1) / kMT;
  if (dtype == SELKV_BF16) {
    const int rows_per_block = kWaves * kMatchTiledRB * 16;
    const int row_blocks = (ne + rows_per_block - 1) / rows_per_block;
    a.parts = gp.match_parts;
    a.part_tiles = (a.part_tiles + a.parts - 1) / a.parts;
    a.part_best = reinterpret_cast<float*>(ws);
    a.part_slot = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + gp.match_slot_off);
    a.mpad = gp.match_mpad;
    char* vk = static_cast<char*>(ws) + gp.match_vk_off;
    float* ik = reinterpret_cast<float*>(static_cast<char*>(ws) + gp.match_ik_off);
    a.Vk = vk;
    a.ik = ik;
    const int64_t gthreads = (int64_t)a.mpad * (s.d * 2 / 16);
    const dim3 ggrid((unsigned)((gthreads + kThreads - 1) / kThreads), (unsigned)s.heads);
    if (s.d == 128)
      hipLaunchKernelGGL((gather_kept_kernel<128>), ggrid, dim3(kThreads), 0, st, a.V, vnorm, kept, vk, ik, s.n, s.m,
                         a.mpad);
    else
      hipLaunchKernelGGL((gather_kept_kernel<64>), ggrid, dim3(kThreads), 0, st, a.V, vnorm, kept, vk, ik, s.n, s.m,
                         a.mpad);
    const dim3 grid((unsigned)(row_blocks * a.parts), (unsigned)s.heads);
    if (s.d == 128) hipLaunchKernelGGL((cosine_match_tiled<128>), grid, dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((cosine_match_tiled<64>), grid, dim3(kThreads), 0, st, a);
    if (a.parts > 1)
      hipLaunchKernelGGL(match_parts_kernel, dim3((ne + kThreads - 1) / kThreads, (unsigned)s.heads), dim3(kThreads),
                         0, st, a);
  } else {
    const int rows_per_block = kWaves * kMatchRowBlocks * 16;
    const dim3 grid((ne + rows_per_block - 1) / rows_per_block, (unsigned)s.heads);
    if (s.d == 128) hipLaunchKernelGGL((cosine_match_kernel<float, 128>), grid, dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((cosine_match_kernel<float, 64>), grid, dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_group(const Shape& s, const GroupPlan& p, const int32_t* target, void* ws, hipStream_t st) {
  const int ne = s.n - s.m;
  if (ne <= 0) return hipSuccess;
  char* w = static_cast<char*>(ws);
  int32_t* off = reinterpret_cast<int32_t*>(w + p.off_off);
  int32_t* table = reinterpret_cast<int32_t*>(w + p.table_off);
  const int nblk = (ne + kSortBlock - 1) / kSortBlock;
  const dim3 grid((unsigned)nblk, (unsigned)s.heads);
  const int32_t* kin = nullptr;
  const int32_t* vin = nullptr;
  for (int pass = 0; pass < p.passes; ++pass) {
    int32_t* kout = reinterpret_cast<int32_t*>(w + p.keys_off[pass & 1]);
    int32_t* vout = reinterpret_cast<int32_t*>(w + p.vals_off[pass & 1]);
    hipLaunchKernelGGL(sort_hist_kernel, grid, dim3(kThreads), 0, st, kin, target, table, ne, s.m, 8 * pass, nblk);
    hipLaunchKernelGGL(group_scan_kernel, dim3((unsigned)s.heads), dim3(1024), 0, st, table, kBins * nblk);
    hipLaunchKernelGGL(sort_scatter_kernel, grid, dim3(kThreads), 0, st, kin, vin, target, table, kout, vout, ne,
                       s.m, 8 * pass, nblk);
    kin = kout;
    vin = vout;
  }
  hipLaunchKernelGGL(sort_offsets_kernel, dim3((unsigned)((s.m + 1 + kThreads - 1) / kThreads), (unsigned)s.heads),
                     dim3(kThreads), 0, st, kin, off, ne, s.m);
  return hipGetLastError();
}

hipError_t launch_group_merge(const Shape& s, const GroupPlan& p, int dtype, const void* K, const void* V,
                              const float* attn, const int32_t* kept, const int32_t* evicted, const float* gate,
                              void* ws, void* K_out, void* V_out, float* bias, float alpha, bool raw,
                              bool merge_keys, hipStream_t st) {
  char* w = static_cast<char*>(ws);
  GroupMergeArgs a{};
  a.K = static_cast<const char*>(K);
  a.V = static_cast<const char*>(V);
  a.attn = attn;
  a.kept = kept;
  a.off = reinterpret_cast<const int32_t*>(w + p.off_off);
  // the payload goes to the sort buffers the last pass read (free once it ran)
  int32_t* lpos = reinterpret_cast<int32_t*>(w + p.vals_off[p.passes & 1]);
  float* lw = reinterpret_cast<float*>(w + p.keys_off[p.passes & 1]);
  a.lpos = lpos;
  a.lw = lw;
  const int ne = s.n - s.m;
  if (ne > 0)
    hipLaunchKernelGGL(group_payload_kernel, dim3((unsigned)((ne + kThreads - 1) / kThreads), (unsigned)s.heads),
                       dim3(kThreads), 0, st, reinterpret_cast<const int32_t*>(w + p.list_off), evicted, gate, attn,
                       lpos, lw, s.n, ne);
  a.K_out = static_cast<char*>(K_out);
  a.V_out = static_cast<char*>(V_out);
  a.bias = bias;
  a.n = s.n;
  a.m = s.m;
  a.alpha = alpha;
  a.raw = raw ? 1 : 0;
  const int waves = (s.m + kSlotsPerWave - 1) / kSlotsPerWave;
  const dim3 grid((waves + kWaves - 1) / kWaves, (unsigned)s.heads);
  const bool values = V_out != nullptr;   // else the bias pass alone
#define SELKV_GM(T, D)                                                                                     \
  do {                                                                                                     \
    if (values && merge_keys)                                                                              \
      hipLaunchKernelGGL((group_merge_kernel<T, D, true, true>), grid, dim3(kThreads), 0, st, a);          \
    else if (values)                                                                                       \
      hipLaunchKernelGGL((group_merge_kernel<T, D, true, false>), grid, dim3(kThreads), 0, st, a);         \
    else                                                                                                   \
      hipLaunchKernelGGL((group_merge_kernel<T, D, false, false>), grid, dim3(kThreads), 0, st, a);        \
  } while (0)
  if (dtype == SELKV_BF16) {
    if (s.d == 128) SELKV_GM(bf16_t, 128);
    else SELKV_GM(bf16_t, 64);
  } else {
    if (s.d == 128) SELKV_GM(float, 128);
    else SELKV_GM(float, 64);
  }
#undef SELKV_GM
  return hipGetLastError();
}

}  // namespace selkv
