// Block-level building blocks shared by the per-sequence kernels: the mass
// reduction (Eq. (5)/(6) with the head mean and head max of Sec. 4.3), the
// Eq. (2) score of one visual token, and the Eq. (3) top-k selection.
#pragma once

#include "vp_common.h"
#include "vp_internal.h"

namespace vp {

// ---------------------------------------------------------------------------
// Per-head reduction of the context pass's statistics (Eq. (5)/(6), with the
// head mean and head max of Sec. 4.3, and the Eq. (2) normaliser)
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 1024;  // threads of every per-sequence block below
constexpr int kSelWaves = kSelThreads / 64;

// Per-head results in LDS (dynamic shared memory, Hq entries each; see
// head_lds_bytes): the head's maximum logit (log2 domain), the reciprocal
// of its Eq. (2) normaliser and its visual mass m^vis_{t,h}; then the head mean
// M_vis and head max M_vis,max as fp32.
struct HeadLds {
  float* hm;
  float* hinv;
  double* mass;
  float* mseq;  // [0] M_vis, [1] M_vis,max
};
__host__ __device__ inline int head_lds_bytes(int Hq) {
  return ((2 * Hq * 4 + 7) / 8) * 8 + Hq * 8 + 16;
}
__device__ __forceinline__ HeadLds head_lds(unsigned char* base, int Hq) {
  HeadLds h;
  h.hm = reinterpret_cast<float*>(base);
  h.hinv = h.hm + Hq;
  h.mass = reinterpret_cast<double*>(base + ((2 * Hq * 4 + 7) / 8) * 8);
  h.mseq = reinterpret_cast<float*>(h.mass + Hq);
  return h;
}

// Lanes that share one head in reduce_heads: the fewest (a power of two) whose
// four parts each cover the part capacity, at most 64 and at most
// kSelThreads / Hq.
__device__ __forceinline__ int lanes_per_head(int Hq, int nparts) {
  int l = 1;
  while (l < 64 && 4 * l < nparts && 2 * l * Hq <= kSelThreads) l <<= 1;
  return l;
}

// Merges the per-part statistics of query qt of sequence b (visual and text
// rows, kept apart by the context pass) for every head of selection row u of
// the query (heads [u Hq/U, (u+1) Hq/U)) onto the head's maximum, in
// double with fixed-order reductions, by a kSelThreads block (every thread
// calls it; two block barriers). Every head gets a group of lanes (a power of
// two, lanes_per_head of the row's head count; one round of heads since Hq <= kSelThreads) that
// strides over the parts and reduces on the DPP network. When the part capacity allows, each lane's (up to four) parts are
// requested at entry at addresses that do not depend on the sequence length,
// `between()` runs while they are in flight (the caller's other independent
// loads), and the maximum and the sums then come from registers; more parts
// take two sweeps with the same arithmetic order. The head mean and head max
// over the row's heads are summed by one wave in a fixed order.
// L is the sequence's clamped length. Fills `hs` (by head index) for the row's heads; with
// `write_out` also writes their m^vis_{t,h} (mass_head), per-head (max, Eq. (2)
// normaliser) (head) and the row's (M_vis, M_vis,max) (mass_seq).
namespace detail {
constexpr int kPartsPerLane = 4;
// parts c0, c0 + step, ... of one head (slots past `cap` read as empty parts)
__device__ __forceinline__ void load_parts(float4 (&v)[kPartsPerLane], float4 (&t)[kPartsPerLane], const float4* st,
                                           bool on, int c0, int step, int cap) {
  const float4 empty = make_float4(kNegInf, 0.f, 0.f, 0.f);
#pragma unroll
  for (int u = 0; u < kPartsPerLane; ++u) {
    const int c = c0 + u * step;
    const bool ok = on && c < cap;
    const int cc = ok ? c : 0;  // part 0 always exists; its duplicate loads share one line
    const float4 x = st[2 * cc];
    const float4 y = st[2 * cc + 1];
    v[u] = ok ? x : empty;
    t[u] = ok ? y : empty;
  }
}
__device__ __forceinline__ float max_parts(float m, const float4 (&v)[kPartsPerLane],
                                           const float4 (&t)[kPartsPerLane], bool on, int c0, int step, int nv) {
#pragma unroll
  for (int u = 0; u < kPartsPerLane; ++u)
    if (on && c0 + u * step < nv) m = fmaxf(m, fmaxf(v[u].x, t[u].x));
  return m;
}
// Eq. (2) normaliser Ls, Eq. (6) denominator Lm and Eq. (5) numerator Vm of
// the parts, rescaled to the head maximum m (double accumulation)
__device__ __forceinline__ void sum_parts(double& Ls, double& Lm, double& Vm, const float4 (&v)[kPartsPerLane],
                                          const float4 (&t)[kPartsPerLane], bool on, int c0, int step, int nv,
                                          float m, float inv_tau_m, float inv_tau_s) {
#pragma unroll
  for (int u = 0; u < kPartsPerLane; ++u) {
    const bool ok = on && c0 + u * step < nv;
    const bool okv = ok && v[u].x != kNegInf;
    const bool okt = ok && t[u].x != kNegInf;
    const float dv = okv ? v[u].x - m : 0.f;
    const float dt = okt ? t[u].x - m : 0.f;
    const double fm = okv ? static_cast<double>(fast_exp2(dv * inv_tau_m)) : 0.0;
    const double fs = okv ? static_cast<double>(fast_exp2(dv * inv_tau_s)) : 0.0;
    const double gm = okt ? static_cast<double>(fast_exp2(dt * inv_tau_m)) : 0.0;
    const double gs = okt ? static_cast<double>(fast_exp2(dt * inv_tau_s)) : 0.0;
    Ls += fs * (okv ? v[u].y : 0.f);
    Lm += fm * (okv ? v[u].z : 0.f);
    Vm += fm * (okv ? v[u].z : 0.f);
    Ls += gs * (okt ? t[u].w : 0.f);
    Lm += gm * (okt ? t[u].z : 0.f);
  }
}
}  // namespace detail

// With `early_on` (uniform over the block), `early()` runs after `between()` and
// a block barrier, before the reduction's arithmetic: loads it issues fly while
// the statistics are reduced.
template <typename Between, typename Early>
__device__ __forceinline__ void reduce_heads(const MassArgs& a, int b, int qt, int u, int L, int tid,
                                             const HeadLds& hs, bool write_out, Between between, bool early_on,
                                             Early early) {
  using namespace detail;
  const int Hu = a.Hq / a.U;  // heads of the row
  const int h0 = u * Hu;
  const int lph = lanes_per_head(Hu, a.nparts);
  // Only the waves that hold a head's lanes reduce; the others go straight to
  // the barrier. Every wave of a 1024-thread block shares its SIMD with three
  // others, so idle waves issuing the same instructions would slow the
  // working ones down (the address arithmetic and the double sums).
  const bool busy = (tid >> 6) < (Hu * lph + 63) / 64;  // uniform over the wave
  constexpr int U = kPartsPerLane;
  const bool one_round = a.nparts <= U * lph;
  int sub = 0, h = h0;
  bool on = false;
  size_t vh = 0;
  const float4* st = nullptr;
  float4 v[U], t[U];
  if (busy) {
    sub = tid % lph;
    on = tid / lph < Hu;
    h = h0 + (on ? tid / lph : 0);
    // the head's statistics and merged results sit at its virtual head for query qt
    vh = static_cast<size_t>(b) * a.T * a.Hq + vhead(h, qt, a.G, a.T);
    // per part: [0] visual {m, Ls, Lm, -}, [1] text {m, l, Lm, Ls}
    st = reinterpret_cast<const float4*>(a.stats + vh * a.nparts * 8);
    if (one_round) load_parts(v, t, st, on, sub, lph, a.nparts);
  }
  between();
  if (early_on) {
    __syncthreads();
    early();
  }
  if (busy) {
    const int nv = parts_used(L, a.nparts);
    float m = kNegInf;
    double Ls = 0.0, Lm = 0.0, Vm = 0.0;
    if (one_round) {
      m = max_parts(m, v, t, on, sub, lph, nv);
      m = group_max_f32(m, lph);
      sum_parts(Ls, Lm, Vm, v, t, on, sub, lph, nv, m, a.inv_tau_m, a.inv_tau_s);
    } else {
      for (int c0 = sub; c0 < nv; c0 += U * lph) {
        load_parts(v, t, st, on, c0, lph, nv);
        m = max_parts(m, v, t, on, c0, lph, nv);
      }
      m = group_max_f32(m, lph);
      for (int c0 = sub; c0 < nv; c0 += U * lph) {
        load_parts(v, t, st, on, c0, lph, nv);
        sum_parts(Ls, Lm, Vm, v, t, on, c0, lph, nv, m, a.inv_tau_m, a.inv_tau_s);
      }
    }
    Ls = group_sum_f64(Ls, lph);
    Lm = group_sum_f64(Lm, lph);
    Vm = group_sum_f64(Vm, lph);
    if (on && sub == 0) {
      const double mass = Lm > 0.0 ? Vm / Lm : 0.0;
      const float ls = static_cast<float>(Ls);
      hs.hm[h] = m;
      hs.hinv[h] = ls > 0.f ? 1.0f / ls : 0.f;
      hs.mass[h] = mass;
      if (write_out) {
        a.mass_head[(static_cast<size_t>(b) * a.T + qt) * a.Hq + h] = static_cast<float>(mass);
        *reinterpret_cast<float2*>(a.head + vh * 2) = make_float2(m, ls);
      }
    }
  }
  __syncthreads();
  // head mean and head max of the row: lane j takes heads h0 + j, h0 + j + 64,
  // ... in order, then a fixed butterfly
  if (tid < 64) {
    double msum = 0.0, mmax = 0.0;
    for (int hh = h0 + tid; hh < h0 + Hu; hh += 64) {
      msum += hs.mass[hh];
      mmax = hs.mass[hh] > mmax ? hs.mass[hh] : mmax;
    }
    msum = group_sum_f64(msum, 64);
    mmax = group_max_f64(mmax, 64);
    if (tid == 0) {
      const float mv = static_cast<float>(msum / Hu);
      const float mx = static_cast<float>(mmax);
      hs.mseq[0] = mv;
      hs.mseq[1] = mx;
      if (write_out) {
        const size_t row = (static_cast<size_t>(b) * a.T + qt) * a.U + u;
        a.mass_seq[2 * row + 0] = mv;
        a.mass_seq[2 * row + 1] = mx;
      }
    }
  }
  __syncthreads();
}

// One head's term of the Eq. (2) score of a visual token: s + 2^((z - m)/tau) / Ls,
// with z the token's logit and m, 1/Ls the head's maximum and normaliser
// (explicit fma, so every kernel that scores rounds the same way).
__device__ __forceinline__ float score_term(float s, float z, float hm, float hinv, float inv_tau) {
  return fmaf(fast_exp2((z - hm) * inv_tau), hinv, s);
}

// Summation order of the Eq. (2) head sum, shared by every kernel that scores:
// over the Gu = Hkv/U KV groups g0 .. g0 + Gu - 1 of a selection row, lane slot l
// of ng = min(64, Gu rounded up to a power of two) sums, in order, the KV groups
// g0 + l, g0 + l + ng, ..., each group's G heads in head order, from zero; the
// lane sums are then added in lane order and the total divided by the row's
// head count Hq/U.
__host__ __device__ inline int score_lanes(int Hkv) {
  int ng = 1;
  while (ng < 64 && ng < Hkv) ng <<= 1;
  return ng;
}

// one KV group's spill row for one token (GP floats, 16-byte aligned)
template <int GP>
__device__ __forceinline__ void load_group_row(const float* row, float (&z)[GP]) {
#pragma unroll
  for (int q = 0; q < GP / 4; ++q) {
    const float4 v = reinterpret_cast<const float4*>(row)[q];
    z[4 * q] = v.x;
    z[4 * q + 1] = v.y;
    z[4 * q + 2] = v.z;
    z[4 * q + 3] = v.w;
  }
}
// p plus the score terms of the G heads of query t in a loaded spill row (the
// query's heads are columns o .. o + G - 1, o = t*G); hm/hinv point at the
// group's first head
template <int GP>
__device__ __forceinline__ float group_terms_of(float p, const float (&z)[GP], int G, int o, const float* hm,
                                                const float* hinv, float inv_tau) {
#pragma unroll
  for (int j = 0; j < GP; ++j)
    if (j >= o && j < o + G) p = score_term(p, z[j], hm[j - o], hinv[j - o], inv_tau);
  return p;
}
// the same, loading the row
template <int GP>
__device__ __forceinline__ float group_terms(float p, const float* row, int G, int o, const float* hm,
                                             const float* hinv, float inv_tau) {
  float z[GP];
  load_group_row<GP>(row, z);
  return group_terms_of<GP>(p, z, G, o, hm, hinv, inv_tau);
}

// ---------------------------------------------------------------------------
// Eq. (2) score of the visual token at cache position pos of sequence b for
// query t's selection row u, by one thread (the same order as the select kernel's lanes):
// S = (1/Hu) sum_h 2^((z_h - m_h) / tau_score) / Ls_h over the row's heads,
// from the spilled logits. hm/hinv: per-head max and 1/Ls (by head index).
// ---------------------------------------------------------------------------
template <int GP>
__device__ __forceinline__ float token_score_gp(const MassArgs& a, int b, int t, int u, int pos, const float* hm,
                                                const float* hinv) {
  const float* zb = a.zs + static_cast<size_t>(b) * a.Hkv * a.zs_rows * GP + static_cast<size_t>(pos) * GP;
  const int Gu = a.Hkv / a.U;
  const int g0 = u * Gu;
  const int ng = score_lanes(Gu);
  float total = 0.f;
  for (int l = 0; l < ng; ++l) {
    float p = 0.f;
    for (int g = g0 + l; g < g0 + Gu; g += ng)
      p = group_terms<GP>(p, zb + static_cast<size_t>(g) * a.zs_rows * GP, a.G, t * a.G, hm + g * a.G,
                          hinv + g * a.G, a.inv_tau_s);
    total = l == 0 ? p : total + p;
  }
  return total / static_cast<float>(a.Hq / a.U);
}
__device__ __forceinline__ float token_score(const MassArgs& a, int b, int t, int u, int pos, const float* hm,
                                             const float* hinv) {
  return a.zs_gp == 8 ? token_score_gp<8>(a, b, t, u, pos, hm, hinv) : token_score_gp<16>(a, b, t, u, pos, hm, hinv);
}

// ---------------------------------------------------------------------------
// Eq. (3) selection by one 1024-thread block
// ---------------------------------------------------------------------------
constexpr int kDigitBits = 13;
constexpr int kBins = 1 << kDigitBits;
constexpr int kBinsPerThread = kBins / kSelThreads;
// counters are stored with one pad word after every kBinsPerThread, so a
// thread's own run of counters starts on a different bank for every lane
constexpr int kHistWords = kBins + kBins / kBinsPerThread;
__device__ __forceinline__ int hslot(int bin) { return bin + bin / kBinsPerThread; }

// Inclusive prefix sum over the 64 lanes of a wave on the DPP network: shifts
// by 1, 2, 4, 8 inside each 16-lane row, then the row totals carried into the
// later rows by the lane-15 and lane-31 broadcasts.
__device__ __forceinline__ int wave_incl_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1 and 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2 and 3
  return v;
}

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
  alignas(16) int wcnt[kSelWaves];
  alignas(16) int gt[kSelWaves];
  alignas(16) int eq[kSelWaves];
  alignas(16) uint32_t wmin[kSelWaves];
  alignas(16) uint32_t wmax[kSelWaves];
  uint32_t digit;
  int above;
  int dcount;
};

// The kSelWaves per-wave values of an LDS array in registers (four 16-byte reads)
__device__ __forceinline__ void wave_values(const int* arr, int (&v)[kSelWaves]) {
#pragma unroll
  for (int j = 0; j < kSelWaves / 4; ++j) {
    const int4 x = reinterpret_cast<const int4*>(arr)[j];
    v[4 * j] = x.x;
    v[4 * j + 1] = x.y;
    v[4 * j + 2] = x.z;
    v[4 * j + 3] = x.w;
  }
}
// sum of the per-wave values of waves below `wid`
__device__ __forceinline__ int waves_below(const int* arr, int wid) {
  int v[kSelWaves];
  wave_values(arr, v);
  int s = 0;
#pragma unroll
  for (int j = 0; j < kSelWaves; ++j) s += j < wid ? v[j] : 0;
  return s;
}

// Block min/max of per-thread (kmin, kmax); contains one barrier.
__device__ __forceinline__ void block_key_range(SelectShared& sh, uint32_t& kmin, uint32_t& kmax, int lane,
                                                int wid) {
  kmin = __ockl_wfred_min_u32(kmin);
  kmax = __ockl_wfred_max_u32(kmax);
  if (lane == 0) {
    sh.wmin[wid] = kmin;
    sh.wmax[wid] = kmax;
  }
  __syncthreads();
  int lo[kSelWaves], hi[kSelWaves];
  wave_values(reinterpret_cast<const int*>(sh.wmin), lo);
  wave_values(reinterpret_cast<const int*>(sh.wmax), hi);
#pragma unroll
  for (int v = 0; v < kSelWaves; ++v) {
    kmin = min(kmin, static_cast<uint32_t>(lo[v]));
    kmax = max(kmax, static_cast<uint32_t>(hi[v]));
  }
}

// Radix select of the k-th largest of n keys (key_at(i)), 0 < k < n, whose
// range is [kmin, kmax]: each pass histograms the surviving candidates on the
// next 13 bits of (key - lo) into 8192 counters; a block suffix scan finds the
// digit holding the k-th largest key and the live range shrinks to it. Digits
// are relative to the live range, so clustered scores still spread over many
// counters. When every candidate of that digit is kept (its count equals the
// number still needed) the selection is complete: the kept keys are exactly
// those >= the digit's lower bound. Returns T with `need` such that the kept
// keys are every key > T and the first `need` keys equal to T (need = 0 after
// an early finish). sh.hist must be zero on entry (it is zero on exit).
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
    int incl = wave_incl_sum(local);
    if (lane == 63) sh.wcnt[wid] = incl;
    __syncthreads();
    incl += waves_below(sh.wcnt, wid);
    const int excl = incl - local;
    if (excl < need && need <= incl) {
      int acc = excl;
#pragma unroll
      for (int j = 0; j < kBinsPerThread; ++j) {
        if (acc < need && need <= acc + c[j]) {
          sh.digit = static_cast<uint32_t>(kBins - 1 - kBinsPerThread * tid - j);
          sh.above = acc;
          sh.dcount = c[j];
        }
        acc += c[j];
      }
    }
    __syncthreads();
    const uint32_t d = sh.digit;
    need -= sh.above;
    lo += d << shift;
    if (sh.dcount == need && lo > 0u) {  // the whole digit is kept
      need = 0;
      return lo - 1u;
    }
    const uint32_t width = (shift >= 32 ? 0xffffffffu : ((1u << shift) - 1u));
    span = min(span - (d << shift), width);
    if (shift == 0) break;
    shift = max(0, shift - kDigitBits);
  }
  return lo;
}

// Ordered compaction: writes the positions of the k selected visual ranks
// (every key > T and the first `need` keys == T; with take_all every key) in
// ascending order to out[0..k). Wave w owns a contiguous block of ranks. A
// first sweep counts its keys > T and == T per lane (no cross-lane work in the
// loop), one block scan gives every wave its offsets, a second sweep finds the
// kept ranks 64 at a time (ballots, four chunks per step so the LDS reads
// overlap) and stages them in LDS (the radix counters, free by then); a last
// pass turns ranks into cache positions and writes them out, so the
// segment-table search runs once per kept token. When k exceeds the staging
// room the second sweep writes positions directly. Three barriers.
template <typename KeyAt>
__device__ __forceinline__ void ordered_compaction(SelectShared& sh, const SegTable& tab, KeyAt key_at, int n, int k,
                                                   int need, uint32_t T, bool take_all, int32_t* out, int lane,
                                                   int wid) {
  const int per = ((n + kSelWaves * 64 - 1) / (kSelWaves * 64)) * 64;
  const int r0 = min(n, wid * per), r1 = min(n, r0 + per);
  int cgt = 0, ceq = 0;
  if (!take_all) {
    for (int i = r0 + lane; i < r1; i += 64) {
      const uint32_t u = key_at(i);
      cgt += u > T ? 1 : 0;
      ceq += u == T ? 1 : 0;
    }
    cgt = __ockl_wfred_add_i32(cgt);
    ceq = __ockl_wfred_add_i32(ceq);
  } else {
    cgt = r1 - r0;
  }
  if (lane == 0) {
    sh.gt[wid] = cgt;
    sh.eq[wid] = ceq;
  }
  __syncthreads();
  int gt_run = 0, eq_run = 0;  // keys > T / == T at ranks below the current chunk
  gt_run = waves_below(sh.gt, wid);
  eq_run = waves_below(sh.eq, wid);
  const bool staged = k <= kHistWords;
  uint32_t* stage = sh.hist;
  constexpr int Q = 4;  // chunks of 64 ranks per step
  for (int base = r0; base < r1; base += Q * 64) {
    uint32_t u[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int i = base + q * 64 + lane;
      u[q] = (i < r1 && !take_all) ? key_at(i) : 0u;
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int i = base + q * 64 + lane;
      const bool in = i < r1;
      const bool gt = in && (take_all || u[q] > T);
      const bool eq = in && !take_all && u[q] == T;
      const uint64_t bgt = __ballot(gt);
      const uint64_t beq = __ballot(eq);
      const int g_b = gt_run + lanes_below(bgt);
      const int e_b = eq_run + lanes_below(beq);
      if (gt || (eq && e_b < need)) {
        const int o = g_b + min(need, e_b);
        if (o < k) {
          if (staged) stage[o] = static_cast<uint32_t>(i);
          else out[o] = rank_to_pos(tab, i);
        }
      }
      gt_run += __popcll(bgt);
      eq_run += __popcll(beq);
    }
  }
  if (staged) {
    __syncthreads();
    for (int o = wid * 64 + lane; o < k; o += kSelThreads) out[o] = rank_to_pos(tab, static_cast<int>(stage[o]));
  }
}


}  // namespace vp
