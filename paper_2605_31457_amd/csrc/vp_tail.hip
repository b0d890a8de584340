// The tail of one decode step for one sequence, in a single 1024-thread
// work-group: Eq. (5)/(6) mass reduction with the head mean and head max
// (Sec. 4.3), the Eq. (7) budget with the Sec. 5.2 clamp, the Eq. (2) score of
// every visual token and the Eq. (3) top-k. It replaces four launches (mass
// reduction, scores, budget, top-k) when a sequence's keys fit in LDS, which
// matters where the step is bound by launch and memory latency (small batches).
// Results equal those of the four separate kernels: the same reductions in the
// same order.
#include "vp_blocks.h"

namespace vp {
namespace {

__global__ __launch_bounds__(kSelThreads) void tail_kernel(const TailArgs t, int lds_keys) {
  extern __shared__ uint32_t s_keys[];
  __shared__ SelectShared sh;
  __shared__ SegTable tab;
  __shared__ double s_mass[kMassThreads];
  __shared__ float s_hm[kTailMaxHeads], s_hinv[kTailMaxHeads];
  __shared__ int s_k;

  const MassArgs& a = t.m;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int o0 = a.seg_off[b];
  if (wid == 0) load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, lane);
  for (int i = tid; i < kHistWords; i += kSelThreads) sh.hist[i] = 0;

  // ---- mass reduction (its barriers also publish the segment table) ----
  const float mmax = reduce_mass(a, b, tid, s_mass, s_hm, s_hinv);
  if (tid == 0) {
    const int kb = budget_rule(static_cast<double>(mmax), tab.rk[tab.n], t.r_lo_bp, t.r_hi_bp, t.clamp);
    t.k[b] = kb;
    s_k = kb;
  }
  __syncthreads();
  const int n = min(tab.rk[tab.n], a.max_vis);
  int k = s_k;
  k = k > n ? n : k;
  k = k > t.k_cap ? t.k_cap : k;
  int32_t* out = t.vis_idx + static_cast<size_t>(b) * t.k_cap;
  for (int i = k + tid; i < t.k_cap; i += kSelThreads) out[i] = -1;

  // ---- scores of every visual rank (2 tokens x 16 heads of loads in flight:
  // one round trip per 2048 tokens and 16 heads) ----
  const bool in_lds = n <= lds_keys;  // the launch guarantees it
  float* sc = a.scores + static_cast<size_t>(b) * a.max_vis;
  const float* zb = a.zs + static_cast<size_t>(b) * a.Hq * a.zs_stride;
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  constexpr int TB = 2, HB = 16;
  for (int base = 0; base < n; base += TB * kSelThreads) {
    int pos[TB];
    bool ok[TB];
    float s[TB];
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int i = base + j * kSelThreads + tid;
      ok[j] = i < n;
      pos[j] = ok[j] ? rank_to_pos(tab, i) : 0;
      s[j] = 0.f;
    }
    for (int h0 = 0; h0 < a.Hq; h0 += HB) {
      float zz[TB][HB];
#pragma unroll
      for (int j = 0; j < TB; ++j)
#pragma unroll
        for (int hh = 0; hh < HB; ++hh)
          zz[j][hh] = zb[static_cast<uint32_t>(min(h0 + hh, a.Hq - 1) * a.zs_stride + pos[j])];  // in bounds
      // heads past Hq add exactly 0 (selects, not branches, so the loads above
      // stay in one batch)
#pragma unroll
      for (int j = 0; j < TB; ++j)
#pragma unroll
        for (int hh = 0; hh < HB; ++hh) {
          const int h = min(h0 + hh, a.Hq - 1);
          const bool v = h0 + hh < a.Hq;
          const float d = v ? zz[j][hh] - s_hm[h] : 0.f;
          s[j] += fast_exp2(d * a.inv_tau_s) * (v ? s_hinv[h] : 0.f);
        }
    }
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      if (ok[j]) {
        const int i = base + j * kSelThreads + tid;
        const float S = s[j] / static_cast<float>(a.Hq);
        sc[i] = S;
        const uint32_t u = order_key(S);
        if (in_lds) s_keys[i] = u;
        kmin = min(kmin, u);
        kmax = max(kmax, u);
      }
    }
  }
  if (k == 0) return;
  auto key_at = [&](int i) -> uint32_t { return s_keys[i]; };

  // ---- top-k ----
  const bool take_all = k >= n;
  uint32_t T = 0u;
  int need = k;
  block_key_range(sh, kmin, kmax, lane, wid);
  if (!take_all) T = radix_select(sh, key_at, n, need, kmin, kmax, tid, lane, wid);
  ordered_compaction(sh, tab, key_at, n, k, need, T, take_all, out, lane, wid);
}

// dynamic LDS left for keys after the kernel's static arrays (one GPU model per
// process is assumed: the figure is computed once)
int tail_key_room() {
  static const int room = [] {
    int dev = 0, max_lds = 65536;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      max_lds = 65536;
    hipFuncAttributes attr;
    const int stat = hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(tail_kernel)) == hipSuccess
                         ? static_cast<int>(attr.sharedSizeBytes)
                         : 64 * 1024;
    return max(0, max_lds - stat - 64) / 4;
  }();
  return room;
}

}  // namespace

bool tail_fits(int n_q_heads, int max_vis) { return n_q_heads <= kTailMaxHeads && max_vis <= tail_key_room(); }

hipError_t launch_tail(const TailArgs& t, hipStream_t st) {
  const int keys = min(tail_key_room(), t.m.max_vis);
  if (t.m.max_vis > keys || t.m.Hq > kTailMaxHeads) return hipErrorInvalidValue;
  hipLaunchKernelGGL(tail_kernel, dim3(t.m.B), dim3(kSelThreads), static_cast<size_t>(keys) * 4, st, t, keys);
  return hipGetLastError();
}

}  // namespace vp
