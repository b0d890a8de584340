// Reductions after the context pass: Eq. (5)/(6) masses with the head mean and
// head max (Sec. 4.3), Eq. (2) scores (Sec. 4.2), and the Eq. (7) budget with
// the Sec. 5.2 clamp.
#include "vp_common.h"
#include "vp_internal.h"

namespace vp {
namespace {

constexpr int kFinThreads = 512;

// One work-group per sequence; every head gets a group of `lph` lanes (a power
// of two, lph * Hq <= 512 when possible, so all heads reduce at once) that
// strides over the parts. Merges the per-part statistics of the visual and
// text rows (kept apart by the context pass) onto the head's maximum in
// double, with fixed-order reductions; writes m^{vis}_{t,h}, the per-head
// (max, Eq. (2) normaliser) for the scores, and the head mean M_vis and head
// max M_vis,max of Sec. 4.3.
__global__ __launch_bounds__(kFinThreads) void mass_finalize_kernel(const MassArgs a) {
  __shared__ double s_mass[kFinThreads];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int nv = parts_used(L, a.nparts);
  int lph = 64;
  while (lph > 1 && lph * a.Hq > kFinThreads) lph >>= 1;
  const int hpr = kFinThreads / lph;  // heads per round
  const int sub = tid % lph;
  double msum = 0.0, mmax = 0.0;
  for (int h0 = 0; h0 < a.Hq; h0 += hpr) {
    const int h = h0 + tid / lph;
    const bool on = h < a.Hq;
    // per part: [0] visual {m, Ls, Lm, -}, [1] text {m, l, Lm, Ls}
    const float4* st =
        reinterpret_cast<const float4*>(a.stats + (static_cast<size_t>(b) * a.Hq + (on ? h : 0)) * a.nparts * 8);
    float m = kNegInf;
    if (on) {
#pragma unroll 4
      for (int c = sub; c < nv; c += lph) m = fmaxf(m, fmaxf(st[2 * c].x, st[2 * c + 1].x));
    }
    for (int off = 1; off < lph; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
    double Ls = 0.0, Lm = 0.0, Vm = 0.0;
    if (on) {
#pragma unroll 4
      for (int c = sub; c < nv; c += lph) {
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
    }
    for (int off = 1; off < lph; off <<= 1) {
      Ls += __shfl_xor(Ls, off);
      Lm += __shfl_xor(Lm, off);
      Vm += __shfl_xor(Vm, off);
    }
    const double mass = Lm > 0.0 ? Vm / Lm : 0.0;
    if (on && sub == 0) {
      a.mass_head[static_cast<size_t>(b) * a.Hq + h] = static_cast<float>(mass);
      *reinterpret_cast<float2*>(a.head + (static_cast<size_t>(b) * a.Hq + h) * 2) =
          make_float2(m, static_cast<float>(Ls));
      s_mass[tid / lph] = mass;
    }
    __syncthreads();
    if (tid == 0) {
      const int nh = min(hpr, a.Hq - h0);
      for (int i = 0; i < nh; ++i) {
        msum += s_mass[i];
        mmax = s_mass[i] > mmax ? s_mass[i] : mmax;
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    a.mass_seq[2 * b + 0] = static_cast<float>(msum / a.Hq);
    a.mass_seq[2 * b + 1] = static_cast<float>(mmax);
  }
}

// S_i = (1/Hq) sum_h 2^((z_{h,i} - m_h) / tau_score) / Ls_h for every visual rank i.
// grid = (ceil(max_vis / 256), B); consecutive threads take consecutive ranks,
// whose logits sit at consecutive cache positions inside a segment.
__global__ __launch_bounds__(256) void scores_kernel(const MassArgs a) {
  extern __shared__ float sh[];  // [Hq] max, [Hq] 1/Ls
  float* s_m = sh;
  float* s_inv = sh + a.Hq;
  __shared__ SegTable tab;
  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int o0 = a.seg_off[b];
  if (tid < 64) load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, tid);
  for (int h = tid; h < a.Hq; h += blockDim.x) {
    const float2 hs = *reinterpret_cast<const float2*>(a.head + (static_cast<size_t>(b) * a.Hq + h) * 2);
    s_m[h] = hs.x;
    s_inv[h] = hs.y > 0.f ? 1.0f / hs.y : 0.f;
  }
  __syncthreads();
  const int nv = min(tab.rk[tab.n], a.max_vis);
  const int i = blockIdx.x * blockDim.x + tid;
  if (i >= nv) return;
  const int pos = rank_to_pos(tab, i);
  const float* z = a.zs + static_cast<size_t>(b) * a.Hq * a.zs_stride + pos;
  // the Hq logits of this position, 16 loads in flight at a time
  constexpr int kBatch = 16;
  float s = 0.f;
  for (int h0 = 0; h0 < a.Hq; h0 += kBatch) {
    float zz[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      zz[j] = h0 + j < a.Hq ? z[static_cast<size_t>(h0 + j) * a.zs_stride] : 0.f;
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      if (h0 + j < a.Hq) s += fast_exp2((zz[j] - s_m[h0 + j]) * a.inv_tau_s) * s_inv[h0 + j];
  }
  a.scores[static_cast<size_t>(b) * a.max_vis + i] = s / static_cast<float>(a.Hq);
}

// one wave per sequence: the visual count from the segment table, then Eq. (7)
__global__ __launch_bounds__(64) void budget_kernel(const BudgetArgs a) {
  __shared__ SegTable tab;
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int o0 = a.seg_off[b];
  load_segments(tab, a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L, lane);
  __syncthreads();
  if (lane == 0)
    a.k[b] = budget_rule(static_cast<double>(a.mass_seq[2 * b + 1]), tab.rk[tab.n], a.r_lo_bp, a.r_hi_bp, a.clamp);
}

}  // namespace

hipError_t launch_mass_finalize(const MassArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(mass_finalize_kernel, dim3(a.B), dim3(kFinThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_scores(const MassArgs& a, hipStream_t st) {
  const dim3 grid((a.max_vis + 255) / 256, a.B);
  hipLaunchKernelGGL(scores_kernel, grid, dim3(256), 2 * a.Hq * sizeof(float), st, a);
  return hipGetLastError();
}

hipError_t launch_budget(const BudgetArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(budget_kernel, dim3(a.B), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace vp
