// Device helpers shared by the SelKV kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace selkv {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// bf16 storage is kept as raw 16-bit patterns.
typedef uint16_t bf16_t;

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round-to-nearest-even fp32 -> bf16 (NaN stays NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

// A 16-byte chunk of a row in storage type T, as raw 32-bit words.
struct Chunk16 {
  uint32_t w[4];
};

__device__ __forceinline__ Chunk16 load16(const void* p) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  Chunk16 c;
  c.w[0] = v.x; c.w[1] = v.y; c.w[2] = v.z; c.w[3] = v.w;
  return c;
}

__device__ __forceinline__ void store16(void* p, const Chunk16& c) {
  *reinterpret_cast<uint4*>(p) = make_uint4(c.w[0], c.w[1], c.w[2], c.w[3]);
}

__device__ __forceinline__ Chunk16 zero16() {
  Chunk16 c;
  c.w[0] = c.w[1] = c.w[2] = c.w[3] = 0u;
  return c;
}

// Elements per 16-byte chunk and their conversion to fp32.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kPerChunk = 4;
  __device__ static __forceinline__ float get(const Chunk16& c, int e) { return __uint_as_float(c.w[e]); }
  __device__ static __forceinline__ void put(Chunk16& c, int e, float x) { c.w[e] = __float_as_uint(x); }
};
template <> struct Elem<bf16_t> {
  static constexpr int kPerChunk = 8;
  __device__ static __forceinline__ float get(const Chunk16& c, int e) {
    const uint32_t w = c.w[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  __device__ static __forceinline__ void put(Chunk16& c, int e, float x) {
    const uint32_t h = f32_to_bf16(x);
    uint32_t& w = c.w[e >> 1];
    w = (e & 1) ? ((w & 0x0000ffffu) | (h << 16)) : ((w & 0xffff0000u) | h);
  }
};

// One 16x16 fp32 tile update D += A * B from 16-byte chunks holding the
// lane's A and B fragments (16x16x32 bf16 MFMA, or four 16x16x4 fp32 MFMAs).
template <typename T> struct Mma;
template <> struct Mma<bf16_t> {
  __device__ static __forceinline__ f32x4 step(const Chunk16& a, const Chunk16& b, f32x4 acc) {
    const bf16x8 av = __builtin_bit_cast(bf16x8, a);
    const bf16x8 bv = __builtin_bit_cast(bf16x8, b);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  __device__ static __forceinline__ f32x4 step(const Chunk16& a, const Chunk16& b, f32x4 acc) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w[e]), __uint_as_float(b.w[e]), acc, 0, 0, 0);
    return acc;
  }
};

// A lane's slice of one row when 16 lanes share the row: d/16 elements of T.
template <typename T, int D>
struct Slice {
  static constexpr int kElems = D / 16;
  static constexpr int kBytes = kElems * (int)sizeof(T);   // 8, 16 or 32
};

// Raw slice kept in registers until used (no conversion on load).
template <typename T, int D>
struct RawSlice {
  static constexpr int kBytes = Slice<T, D>::kBytes;
  uint32_t w[kBytes / 4];
  __device__ __forceinline__ void load(const char* row, int col) {
    const char* p = row + col * kBytes;
    if constexpr (kBytes >= 16) {
#pragma unroll
      for (int c = 0; c < kBytes / 16; ++c) {
        const uint4 v = *reinterpret_cast<const uint4*>(p + c * 16);
        w[4 * c] = v.x; w[4 * c + 1] = v.y; w[4 * c + 2] = v.z; w[4 * c + 3] = v.w;
      }
    } else {
      const uint2 v = *reinterpret_cast<const uint2*>(p);
      w[0] = v.x; w[1] = v.y;
    }
  }
  __device__ __forceinline__ void store(char* row, int col) const {
    char* p = row + col * kBytes;
    if constexpr (kBytes >= 16) {
#pragma unroll
      for (int c = 0; c < kBytes / 16; ++c)
        *reinterpret_cast<uint4*>(p + c * 16) = make_uint4(w[4 * c], w[4 * c + 1], w[4 * c + 2], w[4 * c + 3]);
    } else {
      *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
    }
  }
  __device__ __forceinline__ float get(int e) const {
    if constexpr (sizeof(T) == 4) {
      return __uint_as_float(w[e]);
    } else {
      const uint32_t x = w[e >> 1];
      return __uint_as_float((e & 1) ? (x & 0xffff0000u) : (x << 16));
    }
  }
  __device__ __forceinline__ void put(int e, float f) {
    if constexpr (sizeof(T) == 4) {
      w[e] = __float_as_uint(f);
    } else {
      const uint32_t h = f32_to_bf16(f);
      uint32_t& x = w[e >> 1];
      x = (e & 1) ? ((x & 0x0000ffffu) | (h << 16)) : ((x & 0xffff0000u) | h);
    }
  }
};

// A token position read from a kept / evicted list, clamped into [0, n): a
// list that breaks its contract (say, not produced by selkv_select) gives
// wrong results but never an access outside the cache.
__device__ __forceinline__ int clamp_pos(int32_t p, int n) {
  return (int)min((uint32_t)p, (uint32_t)(n - 1));
}

// A value every lane of the wave holds alike, moved to a scalar register.
__device__ __forceinline__ float uniform(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

__device__ __forceinline__ float xor_shfl(float v, int mask) { return __shfl_xor(v, mask, 64); }
__device__ __forceinline__ int xor_shfl(int v, int mask) { return __shfl_xor(v, mask, 64); }

// Lane i of a 16-lane row reads lane (i + n) mod 16 of the same row (DPP row_ror).
template <int N>
__device__ __forceinline__ float row_ror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x120 + N, 0xf, 0xf, false));
}

// Sum over the 16 lanes of a lane group (lanes 16q .. 16q+15) with DPP row
// rotations; every lane of the group ends with the bitwise-same total.
__device__ __forceinline__ float sum16(float v) {
  v += row_ror<8>(v);
  v += row_ror<4>(v);
  v += row_ror<2>(v);
  v += row_ror<1>(v);
  return v;
}

// A merge weight g * a rounded on its own: the product is never fused into
// the sum it feeds, so the merge and the bias kernels add the same values.
__device__ __forceinline__ float weight_rn(float g, float a) {
#pragma clang fp contract(off)
  return g * a;
}

// Absorbed-mass sums in the merge kernels' order.  A kept slot's weights
// g * a (Eq. 5) are accumulated by lane group: group q (lanes 16q .. 16q+15)
// adds entries q, q + 4, q + 8, ... of the slot's segment in turn, and the
// four group sums combine as (s0 + s1) + (s2 + s3).  The bias kernels form
// the same sums from a one-entry-per-lane layout with the two helpers below,
// so the R of Eq. 6 they compute is bit for bit the one the merge divides by.
// seg_sum_add: adds a 64-entry chunk of the segment (lane i holds entry i of
// the chunk, 0 past the segment's end; chunks start at multiples of 64 from
// the segment start) to the running group sum s, which lane l holds for
// group l & 3.  seg_sum_total: the combined sum, on every lane.
__device__ __forceinline__ float seg_sum_add(float s, float c, int lane) {
#pragma unroll
  for (int t = 0; t < 16; ++t) s += __shfl(c, 4 * t + (lane & 3), 64);
  return s;
}

__device__ __forceinline__ float seg_sum_total(float s) {
  return (__shfl(s, 0, 64) + __shfl(s, 1, 64)) + (__shfl(s, 2, 64) + __shfl(s, 3, 64));
}

// alpha * ln R with R = 1 + absorbed / a (Eq. 6), exactly 0 when nothing was
// absorbed; raw: R - 1 itself, which the union mode averages over heads first.
__device__ __forceinline__ float ratio_bias(float absorbed, float a, float alpha, bool raw) {
  return absorbed > 0.f ? (raw ? absorbed / a : alpha * log1pf(absorbed / a)) : 0.f;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_inclusive_scan(int v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(v, off, 64);
    if (lane >= off) v += u;
  }
  return v;
}

}  // namespace selkv
