// Eq. (3): Top-K_t selection of visual tokens by score (Sec. 4.2).
//
// One 1024-thread work-group (16 waves) per sequence:
//  1. the scores are mapped to order-preserving 32-bit keys, staged once in LDS
//     (when they fit) while the block finds their min and max;
//  2. radix select over the key range [min, max]: each pass histograms the
//     surviving candidates on the next 11 bits of (key - lo) into 2048 LDS
//     counters, a block-wide suffix scan finds the digit holding the k-th
//     largest key, and the candidate range shrinks to that digit. Digits are
//     taken relative to the live range, so scores that share an exponent still
//     spread over many counters. The result is the k-th largest key T and the
//     number `need` of keys equal to T that are kept;
//  3. one ordered sweep in rank (= position) order keeps every key > T and the
//     first `need` keys == T (ties go to the lower position), compacting with
//     wave ballots and mbcnt so the kept positions come out ascending.
#include "vp_common.h"
#include "vp_internal.h"

namespace vp {
namespace {

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// number of set bits of `mask` below this lane
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kDigitBits = 11;
constexpr int kBins = 1 << kDigitBits;

__global__ __launch_bounds__(kThreads) void topk_kernel(const TopkArgs a, int lds_keys) {
  extern __shared__ uint32_t s_keys[];
  __shared__ uint32_t hist[kBins];
  __shared__ int s_wcnt[2][kWaves];
  __shared__ uint32_t s_wmin[kWaves], s_wmax[kWaves];
  __shared__ int s_nv;
  __shared__ uint32_t s_digit;
  __shared__ int s_above;

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int o0 = a.seg_off[b];
  const int nseg = a.seg_off[b + 1] - o0;
  const int32_t* seg = a.seg + 2 * static_cast<long>(o0);
  if (tid == 0) {
    SegWalker w;
    w.start(seg, nseg, L);
    const int nv = w.total();
    s_nv = nv < a.max_vis ? nv : a.max_vis;
  }
  __syncthreads();
  const int n = s_nv;
  int k = a.k[b];
  k = k < 0 ? 0 : k;
  k = k > n ? n : k;
  k = k > a.k_cap ? a.k_cap : k;
  int32_t* out = a.vis_idx + static_cast<size_t>(b) * a.k_cap;
  for (int i = k + tid; i < a.k_cap; i += kThreads) out[i] = -1;
  if (k == 0) return;
  const float* sc = a.scores + static_cast<size_t>(b) * a.max_vis;
  const bool in_lds = n <= lds_keys;
  const bool take_all = k >= n;

  // ---- 1. stage keys, find their range ----
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  for (int i = tid; i < n; i += kThreads) {
    const uint32_t u = order_key(sc[i]);
    if (in_lds) s_keys[i] = u;
    kmin = min(kmin, u);
    kmax = max(kmax, u);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    kmin = min(kmin, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmin), off)));
    kmax = max(kmax, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmax), off)));
  }
  if (lane == 0) {
    s_wmin[wid] = kmin;
    s_wmax[wid] = kmax;
  }
  __syncthreads();
  kmin = s_wmin[0];
  kmax = s_wmax[0];
  for (int v = 1; v < kWaves; ++v) {
    kmin = min(kmin, s_wmin[v]);
    kmax = max(kmax, s_wmax[v]);
  }
  auto key_at = [&](int i) -> uint32_t { return in_lds ? s_keys[i] : order_key(sc[i]); };

  // ---- 2. radix select of the k-th largest key over the live range ----
  uint32_t lo = kmin;
  uint32_t span = kmax - kmin;  // candidates: lo <= key <= lo + span
  int need = k;
  if (!take_all) {
    int shift = span == 0 ? 0 : max(0, 32 - __clz(static_cast<int>(span)) - kDigitBits);
    while (span != 0) {
      for (int i = tid; i < kBins; i += kThreads) hist[i] = 0;
      __syncthreads();
      for (int i = tid; i < n; i += kThreads) {
        const uint32_t u = key_at(i);
        if (u >= lo && u - lo <= span) atomicAdd(&hist[(u - lo) >> shift], 1u);
      }
      __syncthreads();
      // thread t owns bins kBins-1-2t and kBins-2-2t (descending); block inclusive scan
      const int d0 = kBins - 1 - 2 * tid, d1 = d0 - 1;
      const int c0 = static_cast<int>(hist[d0]), c1 = static_cast<int>(hist[d1]);
      const int local = c0 + c1;
      int incl = local;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
      }
      if (lane == 63) s_wcnt[0][wid] = incl;
      __syncthreads();
      for (int v = 0; v < wid; ++v) incl += s_wcnt[0][v];
      const int excl = incl - local;
      if (excl < need && need <= incl) {
        if (excl + c0 >= need) {
          s_digit = static_cast<uint32_t>(d0);
          s_above = excl;
        } else {
          s_digit = static_cast<uint32_t>(d1);
          s_above = excl + c0;
        }
      }
      __syncthreads();
      const uint32_t d = s_digit;
      need -= s_above;
      lo += d << shift;
      const uint32_t width = (shift >= 32 ? 0xffffffffu : ((1u << shift) - 1u));
      span = min(span - (d << shift), width);
      __syncthreads();
      if (shift == 0) break;
      shift = max(0, shift - kDigitBits);
    }
  }
  const uint32_t T = lo;  // with take_all every key is kept

  // ---- 3. ordered compaction ----
  SegWalker w;  // per-thread rank -> position walker (ranks visited in increasing order)
  w.start(seg, nseg, L);
  int base = 0, eq_seen = 0;
  for (int start = 0; start < n; start += kThreads) {
    const int i = start + tid;
    const bool in = i < n;
    const uint32_t u = in ? key_at(i) : 0u;
    const bool gt = in && (take_all || u > T);
    const bool eq = in && !take_all && u == T;
    const uint64_t beq = __ballot(eq);
    if (lane == 0) s_wcnt[0][wid] = __popcll(beq);
    __syncthreads();
    int eq_before = eq_seen + lanes_below(beq), eq_tot = 0;
    for (int v = 0; v < kWaves; ++v) {
      const int c = s_wcnt[0][v];
      eq_before += v < wid ? c : 0;
      eq_tot += c;
    }
    const bool sel = gt || (eq && eq_before < need);
    const uint64_t bsel = __ballot(sel);
    if (lane == 0) s_wcnt[1][wid] = __popcll(bsel);
    __syncthreads();
    int o = base + lanes_below(bsel), sel_tot = 0;
    for (int v = 0; v < kWaves; ++v) {
      const int c = s_wcnt[1][v];
      o += v < wid ? c : 0;
      sel_tot += c;
    }
    if (sel && o < k) {
      while (w.s < w.nseg && w.rank + (w.en - w.st) <= i) w.next();
      out[o] = w.st + (i - w.rank);
    }
    base += sel_tot;
    eq_seen += eq_tot;
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_topk(const TopkArgs& a, hipStream_t st) {
  // dynamic LDS left for staged keys after the kernel's static arrays
  int dev = 0, max_lds = 65536;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    max_lds = 65536;
  const int stat = static_cast<int>(sizeof(uint32_t)) * (kBins + 4 * kWaves + 4) + 64;
  const int keys = min(max(0, (max_lds - stat) / 4), a.max_vis);
  hipLaunchKernelGGL(topk_kernel, dim3(a.B), dim3(kThreads), static_cast<size_t>(keys) * 4, st, a, keys);
  return hipGetLastError();
}

}  // namespace vp
