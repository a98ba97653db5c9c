// selkv_rope_reposition: RoPE repositioning of Eq. 7 on the compressed keys.
//
// Kept slot s of a head holds the key of original position kept[s]; Eq. 7
// undoes its rotation at kept[s] and applies the one at s.  Rotations about
// the same planes compose, so each dimension pair (j, j + d/2) turns once, by
// (s - kept[s]) * theta^(-2j/d) radians.  That angle can reach 1e5 rad, so it
// is formed in fp64 in whole turns (radians / 2 pi) and only the fraction of
// a turn is kept; the hardware sine and cosine take their argument in turns,
// so that fraction goes to them directly as fp32 (no further range
// reduction, no division).  One thread owns the 16-byte chunk c of the low
// half of a row and the matching chunk of the high half; the row is
// rewritten in place.
#include "common.hpp"
#include "internal.hpp"

namespace selkv {
namespace {

constexpr int kThreads = 256;

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void rope_reposition_kernel(const int32_t* kept, char* K_out, int64_t rows,
                                                                   int m, double theta) {
  constexpr int EPC = Elem<T>::kPerChunk;          // elements per 16-byte chunk
  constexpr int HALF = D / 2;
  constexpr int TPR = HALF / EPC;                  // threads per row
  constexpr int RB = D * (int)sizeof(T);
  // turns per position of pair j: theta^(-2j/d) / (2 pi)
  constexpr double kInvTwoPi = 0.15915494309189533576888376337251;
  __shared__ double turns_per_pos[HALF];
  for (int j = threadIdx.x; j < HALF; j += kThreads) turns_per_pos[j] = pow(theta, -2.0 * j / D) * kInvTwoPi;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t row = t / TPR;
  const int c = (int)(t % TPR);
  if (row >= rows) return;
  const int s = (int)(row % m);
  const double delta = (double)s - (double)kept[row];
  if (delta == 0.0) return;                         // already at its slot
  char* base = K_out + row * RB;
  Chunk16 lo = load16(base + c * 16), hi = load16(base + HALF * sizeof(T) + c * 16);
#pragma unroll
  for (int e = 0; e < EPC; ++e) {
    const int j = c * EPC + e;
    const double turns = delta * turns_per_pos[j];
    const float frac = (float)(turns - floor(turns));   // [0, 1]: the angle modulo one turn
    const float sn = __builtin_amdgcn_sinf(frac), cs = __builtin_amdgcn_cosf(frac);
    const float x1 = Elem<T>::get(lo, e), x2 = Elem<T>::get(hi, e);
    Elem<T>::put(lo, e, x1 * cs - x2 * sn);
    Elem<T>::put(hi, e, x2 * cs + x1 * sn);
  }
  store16(base + c * 16, lo);
  store16(base + HALF * sizeof(T) + c * 16, hi);
}

template <typename T, int D>
hipError_t launch_t(const Shape& s, const int32_t* kept, void* K_out, double theta, hipStream_t st) {
  constexpr int TPR = (D / 2) / Elem<T>::kPerChunk;
  const int64_t rows = s.heads * s.m;
  const int64_t threads = rows * TPR;
  hipLaunchKernelGGL((rope_reposition_kernel<T, D>), dim3((unsigned)((threads + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, st, kept, static_cast<char*>(K_out), rows, s.m, theta);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rope_reposition(const Shape& s, int dtype, const int32_t* kept, void* K_out, double theta,
                                  hipStream_t st) {
  if (dtype == SELKV_BF16) {
    if (s.d == 128) return launch_t<bf16_t, 128>(s, kept, K_out, theta, st);
    return launch_t<bf16_t, 64>(s, kept, K_out, theta, st);
  }
  if (s.d == 128) return launch_t<float, 128>(s, kept, K_out, theta, st);
  return launch_t<float, 64>(s, kept, K_out, theta, st);
}

}  // namespace selkv
