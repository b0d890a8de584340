// Block-level building blocks shared by the per-sequence kernels: the mass
// reduction (Eq. (5)/(6) with the head mean and head max of Sec. 4.3), the
// Eq. (2) score of one visual token, and the Eq. (3) top-k selection.
#pragma once

#include "vp_common.h"
#include "vp_internal.h"

namespace vp {

// ---------------------------------------------------------------------------
// mass reduction
// ---------------------------------------------------------------------------
constexpr int kMassThreads = 512;  // threads that take part in reduce_mass

// Merges the per-part statistics of sequence b (visual and text rows, kept
// apart by the context pass) for every head onto the head's maximum, in
// double with fixed-order reductions. Threads 0..kMassThreads-1 of the block
// call it (all of them; others may skip it but must reach the same barriers).
// Every head gets a group of `lph` lanes (a power of two, lph * Hq <= 512 when
// possible) that strides over the parts.
// Writes m^{vis}_{t,h}, the per-head (max, Eq. (2) normaliser) to a.head and,
// when hm/hinv are given, to LDS as (max, 1/normaliser); returns (in thread 0)
// M_vis,max and writes (M_vis, M_vis,max) to a.mass_seq.
// s_mass: kMassThreads doubles of LDS. Contains two block barriers.
__device__ __forceinline__ float reduce_mass(const MassArgs& a, int b, int tid, double* s_mass, float* hm,
                                             float* hinv) {
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int nv = parts_used(L, a.nparts);
  int lph = 64;
  while (lph > 1 && lph * a.Hq > kMassThreads) lph >>= 1;
  const int hpr = kMassThreads / lph;  // heads per round
  const int sub = tid % lph;
  const bool member = tid < kMassThreads;
  double msum = 0.0, mmax = 0.0;
  for (int h0 = 0; h0 < a.Hq; h0 += hpr) {
    const int h = h0 + tid / lph;
    const bool on = member && h < a.Hq;
    // per part: [0] visual {m, Ls, Lm, -}, [1] text {m, l, Lm, Ls}
    const float4* st =
        reinterpret_cast<const float4*>(a.stats + (static_cast<size_t>(b) * a.Hq + (on ? h : 0)) * a.nparts * 8);
    // four parts per lane per round, loaded before use (clamped indices keep
    // every load in bounds; selects, not branches, drop the extra ones)
    constexpr int U = 4;
    float m = kNegInf;
    if (on) {
      for (int c0 = sub; c0 < nv; c0 += U * lph) {
        float x[2 * U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int c = min(c0 + u * lph, nv - 1);
          x[2 * u] = st[2 * c].x;
          x[2 * u + 1] = st[2 * c + 1].x;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (c0 + u * lph < nv) m = fmaxf(m, fmaxf(x[2 * u], x[2 * u + 1]));
      }
    }
    for (int off = 1; off < lph; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
    double Ls = 0.0, Lm = 0.0, Vm = 0.0;
    if (on) {
      for (int c0 = sub; c0 < nv; c0 += U * lph) {
        float4 v[U], t[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int c = min(c0 + u * lph, nv - 1);
          v[u] = st[2 * c];
          t[u] = st[2 * c + 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const bool ok = c0 + u * lph < nv;
          const bool okv = ok && v[u].x != kNegInf;
          const bool okt = ok && t[u].x != kNegInf;
          const float dv = okv ? v[u].x - m : 0.f;
          const float dt = okt ? t[u].x - m : 0.f;
          const double fm = okv ? static_cast<double>(fast_exp2(dv * a.inv_tau_m)) : 0.0;
          const double fs = okv ? static_cast<double>(fast_exp2(dv * a.inv_tau_s)) : 0.0;
          const double gm = okt ? static_cast<double>(fast_exp2(dt * a.inv_tau_m)) : 0.0;
          const double gs = okt ? static_cast<double>(fast_exp2(dt * a.inv_tau_s)) : 0.0;
          Ls += fs * v[u].y;
          Lm += fm * v[u].z;
          Vm += fm * v[u].z;
          Ls += gs * t[u].w;
          Lm += gm * t[u].z;
        }
      }
    }
    for (int off = 1; off < lph; off <<= 1) {
      Ls += __shfl_xor(Ls, off);
      Lm += __shfl_xor(Lm, off);
      Vm += __shfl_xor(Vm, off);
    }
    const double mass = Lm > 0.0 ? Vm / Lm : 0.0;
    if (on && sub == 0) {
      const float ls = static_cast<float>(Ls);
      a.mass_head[static_cast<size_t>(b) * a.Hq + h] = static_cast<float>(mass);
      *reinterpret_cast<float2*>(a.head + (static_cast<size_t>(b) * a.Hq + h) * 2) = make_float2(m, ls);
      if (hm) {
        hm[h] = m;
        hinv[h] = ls > 0.f ? 1.0f / ls : 0.f;
      }
      s_mass[tid / lph] = mass;
    }
    __syncthreads();
    if (tid == 0) {
      const int nh = min(hpr, a.Hq - h0);
      for (int i = 0; i < nh; ++i) {
        msum += s_mass[i];
        mmax = s_mass[i] > mmax ? s_mass[i] : mmax;
      }
    }
    __syncthreads();
  }
  float mx = 0.f;
  if (tid == 0) {
    mx = static_cast<float>(mmax);
    a.mass_seq[2 * b + 0] = static_cast<float>(msum / a.Hq);
    a.mass_seq[2 * b + 1] = mx;
  }
  return mx;
}

// ---------------------------------------------------------------------------
// Eq. (2) score of the visual token at cache position pos of sequence b:
// S = (1/Hq) sum_h 2^((z_h - m_h) / tau_score) / Ls_h from the spilled logits,
// with 32 loads in flight at a time. hm/hinv: per-head max and 1/Ls.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float token_score(const MassArgs& a, int b, int pos, const float* hm, const float* hinv) {
  const float* z = a.zs + static_cast<size_t>(b) * a.Hq * a.zs_stride + pos;
  constexpr int kBatch = 32;
  float s = 0.f;
  for (int h0 = 0; h0 < a.Hq; h0 += kBatch) {
    float zz[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) zz[j] = z[static_cast<size_t>(min(h0 + j, a.Hq - 1)) * a.zs_stride];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      if (h0 + j < a.Hq) s += fast_exp2((zz[j] - hm[h0 + j]) * a.inv_tau_s) * hinv[h0 + j];
  }
  return s / static_cast<float>(a.Hq);
}

// ---------------------------------------------------------------------------
// Eq. (3) selection by one 1024-thread block
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kDigitBits = 13;
constexpr int kBins = 1 << kDigitBits;
constexpr int kBinsPerThread = kBins / kSelThreads;
// counters are stored with one pad word after every kBinsPerThread, so a
// thread's own run of counters starts on a different bank for every lane
constexpr int kHistWords = kBins + kBins / kBinsPerThread;
__device__ __forceinline__ int hslot(int bin) { return bin + bin / kBinsPerThread; }

// order-preserving map of a float to a 32-bit key
__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// number of set bits of `mask` below this lane
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

struct SelectShared {
  uint32_t hist[kHistWords];
  int wcnt[kSelWaves];
  int gt[kSelWaves];
  int eq[kSelWaves];
  uint32_t wmin[kSelWaves];
  uint32_t wmax[kSelWaves];
  uint32_t digit;
  int above;
};

// Block min/max of per-thread (kmin, kmax); contains one barrier.
__device__ __forceinline__ void block_key_range(SelectShared& sh, uint32_t& kmin, uint32_t& kmax, int lane,
                                                int wid) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    kmin = min(kmin, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmin), off)));
    kmax = max(kmax, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmax), off)));
  }
  if (lane == 0) {
    sh.wmin[wid] = kmin;
    sh.wmax[wid] = kmax;
  }
  __syncthreads();
  kmin = sh.wmin[0];
  kmax = sh.wmax[0];
  for (int v = 1; v < kSelWaves; ++v) {
    kmin = min(kmin, sh.wmin[v]);
    kmax = max(kmax, sh.wmax[v]);
  }
}

// Radix select of the k-th largest of n keys (key_at(i)), 0 < k < n, whose
// range is [kmin, kmax]: each pass histograms the surviving candidates on the
// next 13 bits of (key - lo) into 8192 counters; a block suffix scan finds the
// digit holding the k-th largest key and the live range shrinks to it. Digits
// are relative to the live range, so clustered scores still spread over many
// counters. Returns the k-th largest key T; `need` becomes the number of keys
// equal to T that are kept. sh.hist must be zero on entry (it is zero on exit).
// Three barriers per pass; the owner of a counter clears it while scanning.
template <typename KeyAt>
__device__ __forceinline__ uint32_t radix_select(SelectShared& sh, KeyAt key_at, int n, int& need, uint32_t kmin,
                                                 uint32_t kmax, int tid, int lane, int wid) {
  uint32_t lo = kmin;
  uint32_t span = kmax - kmin;  // candidates: lo <= key <= lo + span
  int shift = span == 0 ? 0 : max(0, 32 - __clz(static_cast<int>(span)) - kDigitBits);
  while (span != 0) {
    for (int i = tid; i < n; i += kSelThreads) {
      const uint32_t u = key_at(i);
      if (u >= lo && u - lo <= span) atomicAdd(&sh.hist[hslot(static_cast<int>((u - lo) >> shift))], 1u);
    }
    __syncthreads();
    // thread t owns bins kBins-1-8t .. kBins-8-8t (descending): read and clear
    // them, then a block inclusive scan of the per-thread totals
    int c[kBinsPerThread];
    int local = 0;
#pragma unroll
    for (int j = 0; j < kBinsPerThread; ++j) {
      const int bin = kBins - 1 - kBinsPerThread * tid - j;
      c[j] = static_cast<int>(sh.hist[hslot(bin)]);
      sh.hist[hslot(bin)] = 0;
      local += c[j];
    }
    int incl = local;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    if (lane == 63) sh.wcnt[wid] = incl;
    __syncthreads();
    for (int v = 0; v < wid; ++v) incl += sh.wcnt[v];
    const int excl = incl - local;
    if (excl < need && need <= incl) {
      int acc = excl;
#pragma unroll
      for (int j = 0; j < kBinsPerThread; ++j) {
        if (acc < need && need <= acc + c[j]) {
          sh.digit = static_cast<uint32_t>(kBins - 1 - kBinsPerThread * tid - j);
          sh.above = acc;
        }
        acc += c[j];
      }
    }
    __syncthreads();
    const uint32_t d = sh.digit;
    need -= sh.above;
    lo += d << shift;
    const uint32_t width = (shift >= 32 ? 0xffffffffu : ((1u << shift) - 1u));
    span = min(span - (d << shift), width);
    if (shift == 0) break;
    shift = max(0, shift - kDigitBits);
  }
  return lo;
}

// Ordered compaction: writes the positions of the k selected visual ranks
// (every key > T and the first `need` keys == T; with take_all every key) in
// ascending order to out[0..k). Wave w owns a contiguous block of ranks; a
// first sweep counts, one block scan gives every wave its offsets, a second
// sweep writes. One barrier.
template <typename KeyAt>
__device__ __forceinline__ void ordered_compaction(SelectShared& sh, const SegTable& tab, KeyAt key_at, int n, int k,
                                                   int need, uint32_t T, bool take_all, int32_t* out, int lane,
                                                   int wid) {
  const int per = ((n + kSelWaves * 64 - 1) / (kSelWaves * 64)) * 64;
  const int r0 = min(n, wid * per), r1 = min(n, r0 + per);
  int cgt = 0, ceq = 0;
  if (!take_all) {
    for (int base = r0; base < r1; base += 64) {
      const int i = base + lane;
      const uint32_t u = i < r1 ? key_at(i) : 0u;
      cgt += __popcll(__ballot(i < r1 && u > T));
      ceq += __popcll(__ballot(i < r1 && u == T));
    }
  }
  if (lane == 0) {
    sh.gt[wid] = cgt;
    sh.eq[wid] = ceq;
  }
  __syncthreads();
  int gt_run = 0, eq_run = 0;  // keys > T / == T at ranks below the current chunk
  for (int v = 0; v < wid; ++v) {
    gt_run += sh.gt[v];
    eq_run += sh.eq[v];
  }
  for (int base = r0; base < r1; base += 64) {
    const int i = base + lane;
    const bool in = i < r1;
    const uint32_t u = (in && !take_all) ? key_at(i) : 0u;
    const bool gt = in && (take_all || u > T);
    const bool eq = in && !take_all && u == T;
    const uint64_t bgt = __ballot(gt);
    const uint64_t beq = __ballot(eq);
    const int g_b = gt_run + lanes_below(bgt);
    const int e_b = eq_run + lanes_below(beq);
    if (gt || (eq && e_b < need)) {
      const int o = g_b + min(need, e_b);
      if (o < k) out[o] = rank_to_pos(tab, i);
    }
    gt_run += __popcll(bgt);
    eq_run += __popcll(beq);
  }
}

}  // namespace vp
