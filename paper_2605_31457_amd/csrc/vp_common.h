// Device-side helpers shared by the VisionPulse HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace vp {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// float -> bfloat16 bits, round to nearest even (NaN kept quiet)
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// cross-lane max / sum over the four lanes that share lane % 16 (lanes l, l^16, l^32, l^48)
__device__ __forceinline__ float max_over_quads(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}
__device__ __forceinline__ float sum_over_quads(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

// Walks the visual segments of one sequence in position order, clipping each
// segment to [previous end, L) so that ranks stay consistent and in range for
// any device layout. `rank` is the visual rank of position `st`.
struct SegWalker {
  const int32_t* seg;
  int nseg;
  int L;
  int s;
  int st;
  int en;
  int rank;

  __device__ __forceinline__ void start(const int32_t* seg_, int nseg_, int L_) {
    seg = seg_;
    nseg = nseg_ < 0 ? 0 : nseg_;
    L = L_;
    s = -1;
    st = 0;
    en = 0;
    rank = 0;
    next();
  }
  __device__ __forceinline__ void next() {
    rank += en - st;
    const int prev = en;
    ++s;
    if (s < nseg) {
      const long a = seg[2 * s];
      const long n = seg[2 * s + 1];
      long lo = a > prev ? a : prev;
      lo = lo < 0 ? 0 : (lo > L ? L : lo);
      long hi = a + (n > 0 ? n : 0);
      hi = hi < lo ? lo : (hi > L ? L : hi);
      st = static_cast<int>(lo);
      en = static_cast<int>(hi);
    } else {
      st = L;
      en = L;
    }
  }
  // move to the first segment whose end lies beyond p
  __device__ __forceinline__ void seek(int p) {
    while (s < nseg && en <= p) next();
  }
  __device__ __forceinline__ bool contains(int p) const { return s < nseg && st <= p && p < en; }
  // total visual tokens (walks to the end; call on a copy)
  __device__ __forceinline__ int total() {
    while (s < nseg) next();
    return rank;
  }
};

__device__ __forceinline__ int clamp_len(int L, int cap) { return L < 0 ? 0 : (L > cap ? cap : L); }

// visual-token count of sequence b under the clipping rules of SegWalker
__device__ __forceinline__ int count_visual(const int32_t* seg_off, const int32_t* seg, int b, int L) {
  SegWalker w;
  const int o0 = seg_off[b];
  w.start(seg + 2 * static_cast<long>(o0), seg_off[b + 1] - o0, L);
  return w.total();
}

}  // namespace vp
