// Everything of one decode step between the context pass and the kept-row
// pass, in one launch: the Eq. (5)/(6) mass reduction with the head mean and
// head max (Sec. 4.3), the Eq. (2) score of every visual token (Sec. 4.2), the
// Eq. (7) budget with the Sec. 5.2 clamp and the Eq. (3) top-k.
//
// grid = (chunks, B*T*U), 1024 threads per work-group, one row of work-groups per
// selection row (b, t, u): query t of the sequence (U = 1), or one KV group of
// it (U = Hkv).
// Work-group c of row (b, u) reduces the per-part statistics of the row's heads
// (every work-group of the row does, so none waits for another), scores the
// visual ranks [c * chunk, (c + 1) * chunk) from the spilled logits and writes
// them. With one chunk per row the same work-group selects (its keys in LDS,
// or, beyond the LDS room, re-read from its own score stores); with several, each work-group publishes its scores (device-scope
// atomic stores, coherent across the XCDs) and, once they have completed,
// counts itself in on the row's arrival counter (zeroed by the context pass of
// the same step); the last to arrive reads every score of the row back with
// device-scope loads and selects. No work-group ever waits for another.
//
// Latency: the statistics and the segment table (built by the context pass)
// are requested at once at entry; the spilled logits of a thread's tokens (all heads) are one
// batch of loads; the selection is the LDS radix select of vp_blocks.h.
// Results equal those of the separate kernels (mass_finalize_kernel,
// scores_kernel, budget rule, topk_kernel): the same device functions in the
// same order.
#include <type_traits>

#include "vp_blocks.h"

namespace vp {
namespace {

// The scores are the only data that crosses work-groups: they are stored and
// re-read as device-scope atomics, which are coherent across the XCDs' L2
// caches, so a work-group counts in once its own stores have completed, with no
// L2 write-back (a release per work-group serialised at ~0.15 us per
// work-group on each XCD: 4.9 us of arrival at the 16-sequence batch), and the
// last one reads them back with no L2 invalidation.
__device__ __forceinline__ void store_score(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_score(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// GP: floats per spill row (the query group padded to 8 or 16)
template <int GP>
__global__ __launch_bounds__(kSelThreads) void select_kernel(const SelectArgs t, int lds_keys) {
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
  __shared__ SelectShared sh;
  __shared__ SegTable tab;
  __shared__ int s_last;

  const MassArgs& a = t.m;
  const int c = blockIdx.x;
  const int row = blockIdx.y;
  const int b = row / (a.T * a.U);
  const int qt = (row / a.U) % a.T;  // query of the row
  const int u = row % a.U;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const HeadLds hs = head_lds(dyn, a.Hq);
  uint32_t* s_keys = reinterpret_cast<uint32_t*>(dyn + head_lds_bytes(a.Hq));

  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  // the Eq. (2) scoring layout (below): ng lanes per token, lane l takes the
  // row's KV groups g0 + l, g0 + l + ng, ...
  const int Gu = a.Hkv / a.U;
  const int g0 = u * Gu;
  const int ng = score_lanes(Gu);
  const int l = tid & (ng - 1);
  const float* zb = a.zs + static_cast<size_t>(b) * a.Hkv * a.zs_rows * GP;
  // the first scoring round's position and spill row of this lane's first
  // KV group, requested as soon as the segment table is in LDS, when a chunk
  // is a single round (latency-bound; with more rounds the extra barrier
  // costs as much as the round it hides)
  const bool early = t.chunk <= kSelThreads / ng;
  int pos0 = 0;
  bool pre = false;
  float z0[GP];

  // ---- per-head statistics; the segment table is copied in while the
  // statistics are in flight (a barrier publishes it, then the first round of
  // spill rows is requested and flies while the statistics are reduced) ----
  reduce_heads(a, b, qt, u, L, tid, hs, c == 0, [&] {
    // the context pass left the clipped table in the workspace: one 16-byte
    // load for every fourth thread, spread over the waves so that no wave
    // waits on more than its own statistics and one load
    constexpr int kWords = static_cast<int>(sizeof(SegTable) / 16);
    static_assert(4 * kWords <= kSelThreads, "segment table copy");
    if ((tid & 3) == 0 && (tid >> 2) < kWords) {
      const uint4* src = reinterpret_cast<const uint4*>(static_cast<const SegTable*>(t.segtab) + b);
      reinterpret_cast<uint4*>(&tab)[tid >> 2] = src[tid >> 2];
    }
  }, early, [&] {
    const int nv = min(tab.rk[tab.n], a.max_vis);
    const int q0 = min(nv, c * t.chunk);
    const int i = q0 + tid / ng;
    if (i < min(nv, q0 + t.chunk) && l < Gu) {
      pos0 = rank_to_pos(tab, i);
      load_group_row<GP>(zb + (static_cast<size_t>(g0 + l) * a.zs_rows + pos0) * GP, z0);
      pre = true;
    }
  });
  // the radix counters are first used after the key-range barrier: cleared
  // here, while the spilled logits below are in flight
  for (int i = tid; i < kHistWords; i += kSelThreads) sh.hist[i] = 0;
  const int nvis = tab.rk[tab.n];
  const int n = min(nvis, a.max_vis);
  const bool single = t.nchunks == 1;
  const bool in_lds = n <= lds_keys;
  float* sc = a.scores + static_cast<size_t>(row) * a.max_vis;

  // ---- Eq. (2) scores of this chunk's visual ranks: ng lanes per token, lane
  // l takes the row's KV groups g0 + l, g0 + l + ng, ... (a 16-byte-aligned
  // spill row each), the lane sums are added in lane order ----
  const int tpw = kSelThreads / ng;  // tokens per round
  const int r0 = min(n, c * t.chunk);
  const int r1 = min(n, r0 + t.chunk);
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  // one round of tokens; with kPre the lane's first KV group comes from the
  // row requested during the head reduction
  auto score_round = [&](int base, auto pre_tag) {
    constexpr bool kPre = decltype(pre_tag)::value;
    const int i = base + tid / ng;
    const bool ok = i < r1;
    const bool use = kPre && pre;
    const int pos = use ? pos0 : (ok ? rank_to_pos(tab, i) : 0);
    float p = 0.f;
    for (int g = g0 + l; g < g0 + Gu; g += ng) {
      if (use && g == g0 + l)
        p = group_terms_of<GP>(p, z0, a.G, qt * a.G, hs.hm + g * a.G, hs.hinv + g * a.G, a.inv_tau_s);
      else
        p = group_terms<GP>(p, zb + (static_cast<size_t>(g) * a.zs_rows + pos) * GP, a.G, qt * a.G,
                            hs.hm + g * a.G, hs.hinv + g * a.G, a.inv_tau_s);
    }
    float total = p;
    for (int j = 1; j < ng; ++j) total = total + __shfl(p, (lane & ~(ng - 1)) + j);
    if (ok && l == 0) {
      const float S = total / static_cast<float>(a.Hq / a.U);
      store_score(sc + i, S);
      const uint32_t u = order_key(S);
      if (single && in_lds) s_keys[i] = u;
      kmin = min(kmin, u);
      kmax = max(kmax, u);
    }
  };
  int base = r0;
  if (early && base < r1) {
    score_round(base, std::true_type{});
    base += tpw;
  }
  for (; base < r1; base += tpw) score_round(base, std::false_type{});

  if (single && !in_lds) {
    // one work-group, keys beyond its LDS room: the radix select reads the
    // scores back from memory (device-scope loads, like the multi-chunk path).
    // Every wave waits for its own score stores to complete; the barrier in
    // block_key_range then puts them before any wave's reads.
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  }
  if (!single) {
    // publish this chunk's scores and count in; the last work-group of the
    // row selects. Every wave waits for its own score stores to complete
    // (device-coherent once acknowledged), the barrier then puts all of them
    // before thread 0's count-in; the last arrival reads the scores with
    // device-scope loads after the second barrier.
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    __syncthreads();
    if (tid == 0) {
      const bool last = __hip_atomic_fetch_add(t.sync + row, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                        static_cast<unsigned>(t.nchunks - 1);
      s_last = last;
    }
    __syncthreads();
    if (!s_last) return;
    kmin = 0xffffffffu;
    kmax = 0u;
    constexpr int kBatch = 8;  // loads in flight per thread
    for (int base = 0; base < n; base += kBatch * kSelThreads) {
      float v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) v[j] = load_score(sc + min(base + j * kSelThreads + tid, n - 1));
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
  }

  // ---- Eq. (7) budget, then Eq. (3) selection ----
  const int kb = budget_rule(static_cast<double>(hs.mseq[1]), nvis, t.r_lo_bp, t.r_hi_bp, t.clamp);
  if (tid == 0) t.k[row] = kb;
  int k = kb > n ? n : kb;
  k = k > t.k_cap ? t.k_cap : k;
  int32_t* out = t.vis_idx + static_cast<size_t>(row) * t.k_cap;
  for (int i = k + tid; i < t.k_cap; i += kSelThreads) out[i] = -1;
  if (k == 0) return;
  auto key_at = [&](int i) -> uint32_t { return in_lds ? s_keys[i] : order_key(load_score(sc + i)); };
  const bool take_all = k >= n;
  uint32_t T = 0u;
  int need = k;
  block_key_range(sh, kmin, kmax, lane, wid);
  if (!take_all) T = radix_select(sh, key_at, n, need, kmin, kmax, tid, lane, wid);
  ordered_compaction(sh, tab, key_at, n, k, need, T, take_all, out, lane, wid);
}

// LDS per work-group beyond the kernel's static arrays, and the keys it leaves
// room for (one GPU model per process is assumed: computed once)
template <int GP>
int key_room(int Hq) {
  static const int stat = [] {
    hipFuncAttributes attr;
    return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(select_kernel<GP>)) == hipSuccess
               ? static_cast<int>(attr.sharedSizeBytes)
               : 48 * 1024;
  }();
  static const int max_lds = [] {
    int dev = 0, v = 65536;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      v = 65536;
    return v;
  }();
  return max(0, max_lds - stat - head_lds_bytes(Hq) - 64) / 4;
}

template <int GP>
hipError_t launch_gp(const SelectArgs& t, hipStream_t st) {
  const int room = key_room<GP>(t.m.Hq);
  // keys of up to `room` visual ranks stay in LDS; a row with more reads its
  // scores back from memory during the selection
  const int keys = min(room, t.m.max_vis);
  const size_t dyn = static_cast<size_t>(head_lds_bytes(t.m.Hq)) + static_cast<size_t>(keys) * 4;
  hipLaunchKernelGGL((select_kernel<GP>), dim3(t.nchunks, t.m.B * t.m.T * t.m.U), dim3(kSelThreads), dyn, st, t,
                     keys);
  return hipGetLastError();
}

}  // namespace

int select_tokens_per_round(int n_kv_heads, int rows_per_seq) {
  return kSelThreads / score_lanes(n_kv_heads / rows_per_seq);
}

hipError_t launch_select(const SelectArgs& t, hipStream_t st) {
  if (t.m.Hq > kMaxSelectHeads || t.nchunks < 1 || t.chunk < 1) return hipErrorInvalidValue;
  return t.m.zs_gp == 8 ? launch_gp<8>(t, st) : launch_gp<16>(t, st);
}

}  // namespace vp
