// Device-side helpers shared by the VisionPulse HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "vp_internal.h"

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

// Cross-lane all-reduce inside aligned groups of `width` lanes (a power of two
// <= 64, uniform): butterflies on the DPP network (quad permutes, half-row and
// row mirrors), then a swizzle across 16 lanes and a permute across 32.
template <typename Op>
__device__ __forceinline__ uint32_t group_allreduce_u32(uint32_t v, int width, Op op) {
  auto dpp = [](uint32_t x, int ctrl) -> uint32_t {
    switch (ctrl) {
      case 0xB1: return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0xB1, 0xf, 0xf, false));
      case 0x4E: return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x4E, 0xf, 0xf, false));
      case 0x141: return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x141, 0xf, 0xf, false));
      default: return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x140, 0xf, 0xf, false));
    }
  };
  if (width > 1) v = op(v, dpp(v, 0xB1));   // quad_perm [1,0,3,2]: lane ^ 1
  if (width > 2) v = op(v, dpp(v, 0x4E));   // quad_perm [2,3,0,1]: lane ^ 2
  if (width > 4) v = op(v, dpp(v, 0x141));  // row_half_mirror: the other quad of 8
  if (width > 8) v = op(v, dpp(v, 0x140));  // row_mirror: the other half of 16
  if (width > 16) v = op(v, static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(v), 0x401F)));  // lane ^ 16
  if (width > 32) v = op(v, static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), 32)));
  return v;
}
__device__ __forceinline__ float group_max_f32(float v, int width) {
  return __uint_as_float(group_allreduce_u32(__float_as_uint(v), width, [](uint32_t a, uint32_t b) {
    return __float_as_uint(fmaxf(__uint_as_float(a), __uint_as_float(b)));
  }));
}
// double sums: the two halves travel separately, the add happens in double
__device__ __forceinline__ double group_sum_f64(double v, int width) {
  auto step = [&](auto mov) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = mov(static_cast<uint32_t>(u)), hi = mov(static_cast<uint32_t>(u >> 32));
    v += __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
  };
  if (width > 1) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0xB1, 0xf, 0xf, false)); });
  if (width > 2) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x4E, 0xf, 0xf, false)); });
  if (width > 4) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x141, 0xf, 0xf, false)); });
  if (width > 8) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x140, 0xf, 0xf, false)); });
  if (width > 16) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(x), 0x401F)); });
  if (width > 32) step([](uint32_t x) { return static_cast<uint32_t>(__shfl_xor(static_cast<int>(x), 32)); });
  return v;
}
__device__ __forceinline__ double group_max_f64(double v, int width) {
  auto step = [&](auto mov) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = mov(static_cast<uint32_t>(u)), hi = mov(static_cast<uint32_t>(u >> 32));
    const double o = __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
    v = o > v ? o : v;
  };
  if (width > 1) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0xB1, 0xf, 0xf, false)); });
  if (width > 2) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x4E, 0xf, 0xf, false)); });
  if (width > 4) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x141, 0xf, 0xf, false)); });
  if (width > 8) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x140, 0xf, 0xf, false)); });
  if (width > 16) step([](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(x), 0x401F)); });
  if (width > 32) step([](uint32_t x) { return static_cast<uint32_t>(__shfl_xor(static_cast<int>(x), 32)); });
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
    nseg = nseg_ < 0 ? 0 : (nseg_ > 256 ? 256 : nseg_);  // at most 256 segments are read
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

constexpr int kMaxSegs = 256;  // visual segments read per sequence

// The visual segments of one sequence in LDS, clipped exactly as SegWalker
// clips them: segment s covers positions [st[s], en[s]) and visual ranks
// [rk[s], rk[s + 1]); rk[n] is the sequence's visual count.
struct alignas(16) SegTable {
  int st[kMaxSegs];
  int en[kMaxSegs];
  int rk[kMaxSegs + 1];
  int n;
};

// Fills `t` with one wave (lane = 0..63, every lane calls) in two rounds of
// independent loads instead of one dependent load per segment. SegWalker's
// clipping unrolls to prefix scans: with a_s = clamp(start_s, 0, L) and
// e_s = clamp(start_s + max(len_s, 0), 0, L),
//   en_s = max(0, max_{s' <= s} max(a_s', e_s')),  st_s = max(a_s, en_{s-1}).
// The caller synchronises before reading `t`.
__device__ __forceinline__ void load_segments(SegTable& t, const int32_t* seg, int nseg, int L, int lane) {
  constexpr int PER = kMaxSegs / 64;
  nseg = nseg < 0 ? 0 : (nseg > kMaxSegs ? kMaxSegs : nseg);
  int a[PER], m[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int s = PER * lane + j;
    a[j] = 0;
    m[j] = 0;
    if (s < nseg) {
      const long st = seg[2 * s];
      const long ln = seg[2 * s + 1];
      const long e = st + (ln > 0 ? ln : 0);
      a[j] = static_cast<int>(st < 0 ? 0 : (st > L ? L : st));
      const int ce = static_cast<int>(e < 0 ? 0 : (e > L ? L : e));
      m[j] = a[j] > ce ? a[j] : ce;
    }
  }
  // exclusive prefix max of the lane maxima
  int lm = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) lm = m[j] > lm ? m[j] : lm;
  int incl = lm;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(incl, off);
    if (lane >= off) incl = v > incl ? v : incl;
  }
  int prev = __shfl_up(incl, 1);
  prev = lane == 0 ? 0 : prev;
  int st[PER], en[PER], len = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    st[j] = a[j] > prev ? a[j] : prev;
    en[j] = m[j] > prev ? m[j] : prev;
    prev = en[j];
    if (PER * lane + j < nseg) len += en[j] - st[j];
  }
  // exclusive prefix sum of the lane lengths
  int rinc = len;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(rinc, off);
    if (lane >= off) rinc += v;
  }
  int r = rinc - len;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int s = PER * lane + j;
    if (s < nseg) {
      t.st[s] = st[j];
      t.en[s] = en[j];
      t.rk[s] = r;
      r += en[j] - st[j];
    }
  }
  if (lane == 63) t.rk[nseg] = rinc;
  if (lane == 0) t.n = nseg;
}

static_assert(sizeof(SegTable) == kSegTableBytes, "segment table size");

// position of visual rank r (0 <= r < t.rk[t.n]): binary search on the ranks
__device__ __forceinline__ int rank_to_pos(const SegTable& t, int r) {
  int lo = 0, hi = t.n;  // invariant: rk[lo] <= r < rk[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (t.rk[mid] <= r) lo = mid;
    else hi = mid;
  }
  return t.st[lo] + (r - t.rk[lo]);
}

// visual-token count of sequence b under the clipping rules of SegWalker
__device__ __forceinline__ int count_visual(const int32_t* seg_off, const int32_t* seg, int b, int L) {
  SegWalker w;
  const int o0 = seg_off[b];
  w.start(seg + 2 * static_cast<long>(o0), seg_off[b + 1] - o0, L);
  return w.total();
}

}  // namespace vp
