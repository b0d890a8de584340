// Eq. (3): Top-K_t selection of visual tokens by score (Sec. 4.2).
//
// One 1024-thread work-group (16 waves) per sequence:
//  1. wave 0 loads the sequence's segment table into LDS while the block maps
//     the scores to order-preserving 32-bit keys, stages them in LDS (when
//     they fit) and finds their min and max;
//  2. radix select over the key range [min, max]: each pass histograms the
//     surviving candidates on the next 11 bits of (key - lo) into 2048 LDS
//     counters, a block-wide suffix scan finds the digit holding the k-th
//     largest key, and the candidate range shrinks to that digit. Digits are
//     taken relative to the live range, so scores that share an exponent still
//     spread over many counters. The result is the k-th largest key T and the
//     number `need` of keys equal to T that are kept;
//  3. ordered compaction: wave w owns a contiguous block of ranks (= position
//     order). A first sweep counts its keys > T and == T with ballots; one
//     block scan of those counts gives every wave its offsets; a second sweep
//     keeps every key > T and the first `need` keys == T (ties go to the lower
//     position) and writes positions in ascending order. No block barrier runs
//     inside the sweeps.
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
  __shared__ SegTable tab;
  __shared__ int s_wcnt[kWaves];
  __shared__ int s_gt[kWaves], s_eq[kWaves];
  __shared__ uint32_t s_wmin[kWaves], s_wmax[kWaves];
  __shared__ uint32_t s_digit;
  __shared__ int s_above;

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int o0 = a.seg_off[b];
  if (wid == 0) load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, lane);
  __syncthreads();
  const int n = min(tab.rk[tab.n], a.max_vis);
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
  auto key_at = [&](int i) -> uint32_t { return in_lds ? s_keys[i] : order_key(sc[i]); };

  uint32_t T = 0u;
  int need = k;
  if (!take_all) {
    // ---- 1. stage keys, find their range ----
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    constexpr int kBatch = 8;  // loads in flight per thread
    for (int base = 0; base < n; base += kBatch * kThreads) {
      float v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int i = base + j * kThreads + tid;
        v[j] = i < n ? sc[i] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int i = base + j * kThreads + tid;
        if (i < n) {
          const uint32_t u = order_key(v[j]);
          if (in_lds) s_keys[i] = u;
          kmin = min(kmin, u);
          kmax = max(kmax, u);
        }
      }
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

    // ---- 2. radix select of the k-th largest key over the live range ----
    uint32_t lo = kmin;
    uint32_t span = kmax - kmin;  // candidates: lo <= key <= lo + span
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
      if (lane == 63) s_wcnt[wid] = incl;
      __syncthreads();
      for (int v = 0; v < wid; ++v) incl += s_wcnt[v];
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
    T = lo;
  }

  // ---- 3. ordered compaction: wave w owns ranks [r0, r1) ----
  const int per = ((n + kWaves * 64 - 1) / (kWaves * 64)) * 64;
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
    s_gt[wid] = cgt;
    s_eq[wid] = ceq;
  }
  __syncthreads();
  int gt_run = 0, eq_run = 0;  // keys > T / == T at ranks below the current chunk
  for (int v = 0; v < wid; ++v) {
    gt_run += s_gt[v];
    eq_run += s_eq[v];
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

}  // namespace

hipError_t launch_topk(const TopkArgs& a, hipStream_t st) {
  // dynamic LDS left for staged keys after the kernel's static arrays (one GPU
  // model per process is assumed: the figure is computed once)
  static const int lds_room = [] {
    int dev = 0, max_lds = 65536;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      max_lds = 65536;
    hipFuncAttributes attr;
    const int stat = hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(topk_kernel)) == hipSuccess
                         ? static_cast<int>(attr.sharedSizeBytes)
                         : 16384;
    return max(0, max_lds - stat - 64);
  }();
  const int keys = min(lds_room / 4, a.max_vis);
  hipLaunchKernelGGL(topk_kernel, dim3(a.B), dim3(kThreads), static_cast<size_t>(keys) * 4, st, a, keys);
  return hipGetLastError();
}

}  // namespace vp
