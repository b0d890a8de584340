// Reductions after the context pass: Eq. (5)/(6) masses with the head mean and
// head max (Sec. 4.3), Eq. (2) scores (Sec. 4.2), and the Eq. (7) budget with
// the Sec. 5.2 clamp.
#include "vp_common.h"
#include "vp_internal.h"

namespace vp {
namespace {

// One work-group per sequence, one wave per head (lanes over parts): merges
// the per-part statistics of every head (visual rows and text rows are kept
// apart by the context pass; max-shifted sums, combined in double with
// fixed-order wave reductions), writes m^{vis}_{t,h}, the head mean M_vis and
// head max M_vis,max, and the per-head (max, score normaliser) the scores
// kernel needs.
__global__ __launch_bounds__(256) void mass_finalize_kernel(const MassArgs a) {
  constexpr int kWaves = 4;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int nv = parts_used(L, a.nparts);
  double msum = 0.0;
  double mmax = 0.0;
  for (int h = wid; h < a.Hq; h += kWaves) {
    // per part: [0] visual {m, Ls, Lm, -}, [1] text {m, l, Lm, Ls}
    const float4* st = reinterpret_cast<const float4*>(a.stats + (static_cast<size_t>(b) * a.Hq + h) * a.nparts * 8);
    float m = kNegInf;
    for (int c = lane; c < nv; c += 64) m = fmaxf(m, fmaxf(st[2 * c].x, st[2 * c + 1].x));
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    double Ls = 0.0, Lm = 0.0, Vm = 0.0;
    for (int c = lane; c < nv; c += 64) {
      const float4 v = st[2 * c];
      const float4 t = st[2 * c + 1];
      if (v.x != kNegInf) {
        const double fm = fast_exp2((v.x - m) * a.inv_tau_m);
        Ls += static_cast<double>(fast_exp2((v.x - m) * a.inv_tau_s)) * v.y;
        Lm += fm * v.z;
        Vm += fm * v.z;
      }
      if (t.x != kNegInf) {
        Ls += static_cast<double>(fast_exp2((t.x - m) * a.inv_tau_s)) * t.w;
        Lm += static_cast<double>(fast_exp2((t.x - m) * a.inv_tau_m)) * t.z;
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      Ls += __shfl_xor(Ls, off);
      Lm += __shfl_xor(Lm, off);
      Vm += __shfl_xor(Vm, off);
    }
    const double mass = Lm > 0.0 ? Vm / Lm : 0.0;
    if (lane == 0) {
      a.mass_head[static_cast<size_t>(b) * a.Hq + h] = static_cast<float>(mass);
      *reinterpret_cast<float2*>(a.head + (static_cast<size_t>(b) * a.Hq + h) * 2) =
          make_float2(m, static_cast<float>(Ls));
    }
    msum += mass;
    mmax = mass > mmax ? mass : mmax;
  }
  __shared__ double s_sum[kWaves];
  __shared__ double s_max[kWaves];
  if (lane == 0) {
    s_sum[wid] = msum;
    s_max[wid] = mmax;
  }
  __syncthreads();
  if (tid == 0) {
    double t = 0.0, mx = 0.0;
    for (int v = 0; v < kWaves; ++v) {
      t += s_sum[v];
      mx = s_max[v] > mx ? s_max[v] : mx;
    }
    a.mass_seq[2 * b + 0] = static_cast<float>(t / a.Hq);
    a.mass_seq[2 * b + 1] = static_cast<float>(mx);
  }
}

// S_i = (1/Hq) sum_h 2^((z_{h,i} - m_h) / tau_score) / Ls_h for every visual rank i.
// grid = (ceil(max_vis / 256), B); consecutive threads take consecutive ranks,
// whose logits sit at consecutive cache positions inside a segment.
__global__ __launch_bounds__(256) void scores_kernel(const MassArgs a) {
  extern __shared__ float sh[];  // [Hq] max, [Hq] 1/Ls
  float* s_m = sh;
  float* s_inv = sh + a.Hq;
  __shared__ int s_nv;
  __shared__ SegWalker s_w;  // walker at the segment holding this block's first rank
  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int rank0 = blockIdx.x * blockDim.x;
  if (tid == 0) {
    const int L = clamp_len(a.seq_len[b], a.max_seq_len);
    const int o0 = a.seg_off[b];
    SegWalker w;
    w.start(a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L);
    SegWalker t = w;
    const int nv = t.total();
    s_nv = nv < a.max_vis ? nv : a.max_vis;
    while (w.s < w.nseg && w.rank + (w.en - w.st) <= rank0) w.next();
    s_w = w;
  }
  for (int h = tid; h < a.Hq; h += blockDim.x) {
    const float* hs = a.head + (static_cast<size_t>(b) * a.Hq + h) * 2;
    s_m[h] = hs[0];
    s_inv[h] = hs[1] > 0.f ? 1.0f / hs[1] : 0.f;
  }
  __syncthreads();
  const int i = rank0 + tid;
  if (i >= s_nv) return;
  SegWalker w = s_w;
  while (w.s < w.nseg && w.rank + (w.en - w.st) <= i) w.next();
  const int pos = w.st + (i - w.rank);
  const float* z = a.zs + static_cast<size_t>(b) * a.Hq * a.zs_stride + pos;
  float s = 0.f;
  for (int h = 0; h < a.Hq; ++h)
    s += fast_exp2((z[static_cast<size_t>(h) * a.zs_stride] - s_m[h]) * a.inv_tau_s) * s_inv[h];
  a.scores[static_cast<size_t>(b) * a.max_vis + i] = s / static_cast<float>(a.Hq);
}

__global__ __launch_bounds__(64) void budget_kernel(const BudgetArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.B) return;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int nv = count_visual(a.seg_off, a.seg, b, L);
  a.k[b] = budget_rule(static_cast<double>(a.mass_seq[2 * b + 1]), nv, a.r_lo_bp, a.r_hi_bp, a.clamp);
}

}  // namespace

hipError_t launch_mass_finalize(const MassArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(mass_finalize_kernel, dim3(a.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_scores(const MassArgs& a, hipStream_t st) {
  const dim3 grid((a.max_vis + 255) / 256, a.B);
  hipLaunchKernelGGL(scores_kernel, grid, dim3(256), 2 * a.Hq * sizeof(float), st, a);
  return hipGetLastError();
}

hipError_t launch_budget(const BudgetArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(budget_kernel, dim3((a.B + 63) / 64), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace vp
