// Reductions after the context pass: Eq. (5)/(6) masses with the head mean and
// head max (Sec. 4.3), Eq. (2) scores (Sec. 4.2), and the Eq. (7) budget with
// the Sec. 5.2 clamp.
#include "vp_blocks.h"

namespace vp {
namespace {

// One work-group per selection row (b, t, u): the per-part statistics merged
// per head of the row, then the row's head mean and head max (reduce_heads, as
// in the select kernel).
__global__ __launch_bounds__(kSelThreads) void mass_finalize_kernel(const MassArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
  const int row = blockIdx.x;
  const int b = row / (a.T * a.U);
  const int t = (row / a.U) % a.T;
  const int u = row % a.U;
  reduce_heads(a, b, t, u, clamp_len(a.seq_len[b], a.max_seq_len), threadIdx.x, head_lds(dyn, a.Hq), true, [] {}, false, [] {});
}

// S_i of Eq. (2) for every visual rank i of every selection row.
// grid = (ceil(max_vis / 256), B*T*U); consecutive threads take consecutive ranks,
// whose logits sit at consecutive cache positions inside a segment.
__global__ __launch_bounds__(256) void scores_kernel(const MassArgs a) {
  extern __shared__ float sh[];  // [Hq] max, [Hq] 1/Ls
  float* s_m = sh;
  float* s_inv = sh + a.Hq;
  __shared__ SegTable tab;
  const int row = blockIdx.y;
  const int b = row / (a.T * a.U);
  const int t = (row / a.U) % a.T;
  const int u = row % a.U;
  const int tid = threadIdx.x;
  const int L = vis_len(clamp_len(a.seq_len[b], a.max_seq_len), a.T);
  const int o0 = a.seg_off[b];
  if (tid < 64) load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, tid);
  const int Hu = a.Hq / a.U;
  for (int h = u * Hu + tid; h < (u + 1) * Hu; h += blockDim.x) {
    const size_t vh = static_cast<size_t>(b) * a.T * a.Hq + vhead(h, t, a.G, a.T);
    const float2 hs = *reinterpret_cast<const float2*>(a.head + vh * 2);
    s_m[h] = hs.x;
    s_inv[h] = hs.y > 0.f ? 1.0f / hs.y : 0.f;
  }
  __syncthreads();
  const int nv = min(tab.rk[tab.n], a.max_vis);
  const int i = blockIdx.x * blockDim.x + tid;
  if (i >= nv) return;
  a.scores[static_cast<size_t>(row) * a.max_vis + i] = token_score(a, b, t, u, rank_to_pos(tab, i), s_m, s_inv);
}

// one wave per selection row: the visual count from the segment table, then Eq. (7)
__global__ __launch_bounds__(64) void budget_kernel(const BudgetArgs a) {
  __shared__ SegTable tab;
  const int row = blockIdx.x;
  const int b = row / a.R;
  const int lane = threadIdx.x;
  const int L = vis_len(clamp_len(a.seq_len[b], a.max_seq_len), a.T);
  const int o0 = a.seg_off[b];
  load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, lane);
  __syncthreads();
  if (lane == 0)
    a.k[row] = budget_rule(static_cast<double>(a.mass_seq[2 * row + 1]), tab.rk[tab.n], a.r_lo_bp, a.r_hi_bp, a.clamp);
}

}  // namespace

hipError_t launch_mass_finalize(const MassArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(mass_finalize_kernel, dim3(a.B * a.T * a.U), dim3(kSelThreads), head_lds_bytes(a.Hq), st, a);
  return hipGetLastError();
}

hipError_t launch_scores(const MassArgs& a, hipStream_t st) {
  const dim3 grid((a.max_vis + 255) / 256, a.B * a.T * a.U);
  hipLaunchKernelGGL(scores_kernel, grid, dim3(256), 2 * a.Hq * sizeof(float), st, a);
  return hipGetLastError();
}

hipError_t launch_budget(const BudgetArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(budget_kernel, dim3(a.B * a.R), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace vp
