// Eq. (3): Top-K_t selection of visual tokens by score (Sec. 4.2).
//
// One 1024-thread work-group (16 waves) per selection row (a sequence, or one
// query or KV group of it; the row's sequence gives the visual tokens):
//  1. wave 0 loads the sequence's segment table into LDS while the block maps
//     the scores to order-preserving 32-bit keys, stages them in LDS (when
//     they fit) and finds their min and max;
//  2. radix select over the key range [min, max]: each pass histograms the
//     surviving candidates on the next 13 bits of (key - lo) into 8192 LDS
//     counters, a block-wide suffix scan finds the digit holding the k-th
//     largest key, and the candidate range shrinks to that digit. Digits are
//     taken relative to the live range, so scores that share an exponent still
//     spread over many counters, and score ranges of up to 2^26 key steps
//     resolve in two passes. Each pass has three barriers: the owner of a
//     counter clears it while scanning. The result is the k-th largest key T
//     and the number `need` of keys equal to T that are kept;
//  3. ordered compaction: wave w owns a contiguous block of ranks (= position
//     order). A first sweep counts its keys > T and == T with ballots; one
//     block scan of those counts gives every wave its offsets; a second sweep
//     keeps every key > T and the first `need` keys == T (ties go to the lower
//     position) and writes positions in ascending order. No block barrier runs
//     inside the sweeps.
#include "vp_blocks.h"

namespace vp {
namespace {

__global__ __launch_bounds__(kSelThreads) void topk_kernel(const TopkArgs a, int lds_keys) {
  extern __shared__ uint32_t s_keys[];
  __shared__ SelectShared sh;
  __shared__ SegTable tab;

  const int row = blockIdx.x;  // selection row of sequence b
  const int b = row / a.R;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int L = vis_len(clamp_len(a.seq_len[b], a.max_seq_len), a.T);
  const int o0 = a.seg_off[b];
  if (wid == 0) load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, lane);
  __syncthreads();
  const int n = min(tab.rk[tab.n], a.max_vis);
  int k;
  if (a.mass_seq) {
    k = budget_rule(static_cast<double>(a.mass_seq[2 * row + 1]), tab.rk[tab.n], a.r_lo_bp, a.r_hi_bp, a.clamp);
    if (tid == 0) a.k_out[row] = k;
  } else {
    k = a.k[row];
  }
  k = k < 0 ? 0 : k;
  k = k > n ? n : k;
  k = k > a.k_cap ? a.k_cap : k;
  int32_t* out = a.vis_idx + static_cast<size_t>(row) * a.k_cap;
  for (int i = k + tid; i < a.k_cap; i += kSelThreads) out[i] = -1;
  if (k == 0) return;
  const float* sc = a.scores + static_cast<size_t>(row) * a.max_vis;
  const bool in_lds = n <= lds_keys;
  const bool take_all = k >= n;
  auto key_at = [&](int i) -> uint32_t { return in_lds ? s_keys[i] : order_key(sc[i]); };

  uint32_t T = 0u;
  int need = k;
  if (!take_all) {
    // ---- 1. stage keys, find their range ----
    for (int i = tid; i < kHistWords; i += kSelThreads) sh.hist[i] = 0;
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    constexpr int kBatch = 8;  // loads in flight per thread
    for (int base = 0; base < n; base += kBatch * kSelThreads) {
      float v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int i = base + j * kSelThreads + tid;
        v[j] = i < n ? sc[i] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int i = base + j * kSelThreads + tid;
        if (i < n) {
          const uint32_t u = order_key(v[j]);
          if (in_lds) s_keys[i] = u;
          kmin = min(kmin, u);
          kmax = max(kmax, u);
        }
      }
    }
    block_key_range(sh, kmin, kmax, lane, wid);
    // ---- 2. radix select of the k-th largest key ----
    T = radix_select(sh, key_at, n, need, kmin, kmax, tid, lane, wid);
  }
  // ---- 3. ordered compaction ----
  ordered_compaction(sh, tab, key_at, n, k, need, T, take_all, out, lane, wid);
}

// ---------------------------------------------------------------------------
// Top-p budget: the smallest number of visual tokens, in the Eq. (3) order,
// whose scores sum to at least p. A radix descent like the one above, driven by
// score mass instead of count: each pass histograms the live keys' counts and
// their masses (exact 2^-40 fixed point, each score rounded down, 64-bit sums)
// over 2048 digits, and a block scan from the top digit finds where the
// cumulative mass crosses the remaining target. At the last digit every live
// key is one value T, and the tokens at T needed to close the gap are a
// division away.
// ---------------------------------------------------------------------------
constexpr int kPBits = 11;
constexpr int kPBins = 1 << kPBits;
constexpr double kFix = 1099511627776.0;  // 2^40

__device__ __forceinline__ float key_float(uint32_t u) {
  return __uint_as_float((u & 0x80000000u) ? (u ^ 0x80000000u) : ~u);
}
__device__ __forceinline__ uint64_t fixed_mass(uint32_t u) {
  const float f = key_float(u);
  return f > 0.f ? static_cast<uint64_t>(static_cast<double>(f) * kFix) : 0ull;  // rounds down
}

__global__ __launch_bounds__(kSelThreads) void top_p_kernel(const TopPArgs a, int lds_keys) {
  extern __shared__ uint32_t s_keys[];
  __shared__ uint32_t s_cnt[kPBins];
  __shared__ unsigned long long s_mass[kPBins];
  __shared__ SegTable tab;
  __shared__ unsigned long long s_wm[kSelWaves];
  __shared__ int s_wc[kSelWaves];
  __shared__ uint32_t s_wmin[kSelWaves], s_wmax[kSelWaves];
  __shared__ uint32_t s_digit;
  __shared__ unsigned long long s_above_m;
  __shared__ int s_above_c;

  const int row = blockIdx.x;  // selection row of sequence b
  const int b = row / a.R;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int L = vis_len(clamp_len(a.seq_len[b], a.max_seq_len), a.T);
  const int o0 = a.seg_off[b];
  if (wid == 0) load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, lane);
  __syncthreads();
  const int n = min(tab.rk[tab.n], a.max_vis);
  if (!(a.p > 0.f) || n == 0) {
    if (tid == 0) a.k[row] = 0;
    return;
  }
  const float* sc = a.scores + static_cast<size_t>(row) * a.max_vis;
  const bool in_lds = n <= lds_keys;
  auto key_at = [&](int i) -> uint32_t { return in_lds ? s_keys[i] : order_key(sc[i]); };
  // target in fixed point, rounded up: sum >= p  <=>  fixed sum >= ceil(p 2^40)
  const uint64_t target = static_cast<uint64_t>(ceil(static_cast<double>(a.p) * kFix));

  // ---- stage keys; total mass and key range ----
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  unsigned long long tot = 0;
  constexpr int kBatch = 8;  // loads in flight per thread
  for (int base = 0; base < n; base += kBatch * kSelThreads) {
    float v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) v[j] = sc[min(base + j * kSelThreads + tid, n - 1)];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * kSelThreads + tid;
      if (i < n) {
        const uint32_t u = order_key(v[j]);
        if (in_lds) s_keys[i] = u;
        kmin = min(kmin, u);
        kmax = max(kmax, u);
        tot += fixed_mass(u);
      }
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    kmin = min(kmin, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmin), off)));
    kmax = max(kmax, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmax), off)));
    tot += __shfl_xor(tot, off);
  }
  if (lane == 0) {
    s_wmin[wid] = kmin;
    s_wmax[wid] = kmax;
    s_wm[wid] = tot;
  }
  for (int i = tid; i < kPBins; i += kSelThreads) {
    s_cnt[i] = 0;
    s_mass[i] = 0;
  }
  __syncthreads();
  kmin = s_wmin[0];
  kmax = s_wmax[0];
  tot = 0;
  for (int v = 0; v < kSelWaves; ++v) {
    kmin = min(kmin, s_wmin[v]);
    kmax = max(kmax, s_wmax[v]);
    tot += s_wm[v];
  }
  if (tot < target) {  // every visual token together stays below p
    if (tid == 0) a.k[row] = n;
    return;
  }

  // ---- descent by mass ----
  uint32_t lo = kmin;
  uint32_t span = kmax - kmin;
  uint64_t need = target;  // mass still to collect from keys in [lo, lo + span]
  int above = 0;           // tokens already counted (keys above the live range)
  int shift = span == 0 ? 0 : max(0, 32 - __clz(static_cast<int>(span)) - kPBits);
  while (true) {
    if (span != 0) {
      for (int i = tid; i < n; i += kSelThreads) {
        const uint32_t u = key_at(i);
        if (u >= lo && u - lo <= span) {
          const int d = static_cast<int>((u - lo) >> shift);
          atomicAdd(&s_cnt[d], 1u);
          atomicAdd(&s_mass[d], static_cast<unsigned long long>(fixed_mass(u)));
        }
      }
      __syncthreads();
      // thread t owns digits kPBins-1-2t, kPBins-2-2t (descending)
      const int d0 = kPBins - 1 - 2 * tid, d1 = d0 - 1;
      const unsigned long long m0 = s_mass[d0], m1 = s_mass[d1];
      const int c0 = static_cast<int>(s_cnt[d0]), c1 = static_cast<int>(s_cnt[d1]);
      s_mass[d0] = 0;
      s_mass[d1] = 0;
      s_cnt[d0] = 0;
      s_cnt[d1] = 0;
      unsigned long long im = m0 + m1;
      int ic = c0 + c1;
      const unsigned long long lm = im;
      const int lc = ic;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const unsigned long long vm = __shfl_up(im, off);
        const int vc = __shfl_up(ic, off);
        if (lane >= off) {
          im += vm;
          ic += vc;
        }
      }
      if (lane == 63) {
        s_wm[wid] = im;
        s_wc[wid] = ic;
      }
      __syncthreads();
      for (int v = 0; v < wid; ++v) {
        im += s_wm[v];
        ic += s_wc[v];
      }
      const unsigned long long em = im - lm;
      const int ec = ic - lc;
      if (em < need && need <= im) {
        if (em + m0 >= need) {
          s_digit = static_cast<uint32_t>(d0);
          s_above_m = em;
          s_above_c = ec;
        } else {
          s_digit = static_cast<uint32_t>(d1);
          s_above_m = em + m0;
          s_above_c = ec + c0;
        }
      }
      __syncthreads();
      const uint32_t d = s_digit;
      need -= s_above_m;
      above += s_above_c;
      lo += d << shift;
      const uint32_t width = (shift >= 32 ? 0xffffffffu : ((1u << shift) - 1u));
      span = min(span - (d << shift), width);
      if (shift != 0) {
        shift = max(0, shift - kPBits);
        continue;
      }
    }
    break;
  }
  // every live key is lo now; each carries the same mass
  if (tid == 0) {
    const uint64_t m = fixed_mass(lo);
    const uint64_t j = m > 0 ? (need + m - 1) / m : 0;
    a.k[row] = min(n, above + static_cast<int>(j));
  }
}

}  // namespace

hipError_t launch_top_p(const TopPArgs& a, hipStream_t st) {
  static const int lds_room = [] {
    int dev = 0, max_lds = 65536;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      max_lds = 65536;
    hipFuncAttributes attr;
    const int stat = hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(top_p_kernel)) == hipSuccess
                         ? static_cast<int>(attr.sharedSizeBytes)
                         : 48 * 1024;
    return max(0, max_lds - stat - 64);
  }();
  const int keys = min(lds_room / 4, a.max_vis);
  hipLaunchKernelGGL(top_p_kernel, dim3(a.B * a.R), dim3(kSelThreads), static_cast<size_t>(keys) * 4, st, a, keys);
  return hipGetLastError();
}

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
                         : 48 * 1024;
    return max(0, max_lds - stat - 64);
  }();
  const int keys = min(lds_room / 4, a.max_vis);
  hipLaunchKernelGGL(topk_kernel, dim3(a.B * a.R), dim3(kSelThreads), static_cast<size_t>(keys) * 4, st, a, keys);
  return hipGetLastError();
}

}  // namespace vp
