// Eq. (3): Top-K_t selection of visual tokens by score (Sec. 4.2).
//
// One 1024-thread work-group (16 waves) per sequence:
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

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int o0 = a.seg_off[b];
  if (wid == 0) load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, lane);
  __syncthreads();
  const int n = min(tab.rk[tab.n], a.max_vis);
  int k;
  if (a.mass_seq) {
    k = budget_rule(static_cast<double>(a.mass_seq[2 * b + 1]), tab.rk[tab.n], a.r_lo_bp, a.r_hi_bp, a.clamp);
    if (tid == 0) a.k_out[b] = k;
  } else {
    k = a.k[b];
  }
  k = k < 0 ? 0 : k;
  k = k > n ? n : k;
  k = k > a.k_cap ? a.k_cap : k;
  int32_t* out = a.vis_idx + static_cast<size_t>(b) * a.k_cap;
  for (int i = k + tid; i < a.k_cap; i += kSelThreads) out[i] = -1;
  if (k == 0) return;
  const float* sc = a.scores + static_cast<size_t>(b) * a.max_vis;
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
                         : 48 * 1024;
    return max(0, max_lds - stat - 64);
  }();
  const int keys = min(lds_room / 4, a.max_vis);
  hipLaunchKernelGGL(topk_kernel, dim3(a.B), dim3(kSelThreads), static_cast<size_t>(keys) * 4, st, a, keys);
  return hipGetLastError();
}

}  // namespace vp
