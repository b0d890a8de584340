// Eq. (3): Top-K_t selection of visual tokens by score (Sec. 4.2).
//
// One 1024-thread work-group (16 waves) per sequence:
//  1. radix select on order-preserving 32-bit keys of the float scores, 8 bits
//     per pass from the top: each pass histograms the keys that match the
//     prefix found so far (LDS counters), one wave finds the digit holding the
//     k-th largest key with a wave prefix scan; after 4 passes the k-th largest
//     key T and the number `need` of keys equal to T to keep are known;
//  2. one ordered sweep over the scores in rank (= position) order keeps every
//     key > T and the first `need` keys == T (ties go to the lower position),
//     compacting with wave ballots and mbcnt so the kept positions come out
//     ascending.
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

__global__ __launch_bounds__(kThreads) void topk_kernel(const TopkArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ int s_wcnt[2][kWaves];
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

  // ---- 1. radix select of the k-th largest key ----
  const bool take_all = k >= n;
  uint32_t prefix = 0, pmask = 0;
  int need = k;
  if (!take_all) {
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < n; i += kThreads) {
        const uint32_t u = order_key(sc[i]);
        if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (wid == 0) {
        // lane l owns digits 255-4l .. 252-4l (descending); inclusive scan of counts over lanes
        int cnt[4];
        int local = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          cnt[e] = static_cast<int>(hist[255 - 4 * lane - e]);
          local += cnt[e];
        }
        int incl = local;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const int v = __shfl_up(incl, off);
          if (lane >= off) incl += v;
        }
        int c = incl - local;  // keys with a larger digit than this lane's first
        if (c < need && need <= incl) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (c + cnt[e] >= need) {
              s_digit = static_cast<uint32_t>(255 - 4 * lane - e);
              s_above = c;
              break;
            }
            c += cnt[e];
          }
        }
      }
      __syncthreads();
      need -= s_above;
      prefix |= s_digit << shift;
      pmask |= 255u << shift;
      __syncthreads();
    }
  }
  const uint32_t T = prefix;

  // ---- 2. ordered compaction ----
  SegWalker w;  // per-thread rank -> position walker (ranks visited in increasing order)
  w.start(seg, nseg, L);
  int base = 0, eq_seen = 0;
  for (int start = 0; start < n; start += kThreads) {
    const int i = start + tid;
    const bool in = i < n;
    const uint32_t u = in ? order_key(sc[i]) : 0u;
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
  hipLaunchKernelGGL(topk_kernel, dim3(a.B), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace vp
