// Split-K reduction of the pruned attention (Sec. 4.1/4.2): merges the text
// partials of the context pass (one per cache chunk) and the kept-row partials
// (one per split of the kept list) of every (sequence, query head):
//   out = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i,  M = max_i m_i,
// over the partials with l_i > 0; an empty context gives zeros.
// grid = (Hq, B), one thread per output dimension.
#include "vp_common.h"
#include "vp_internal.h"

namespace vp {
namespace {

template <int D>
__global__ __launch_bounds__(D) void merge_kernel(const MergeArgs a) {
  __shared__ float s_w[D];   // weight 2^(m_i - M) of each partial of the current block
  __shared__ float s_red[D / 64];
  const int h = blockIdx.x;
  const int b = blockIdx.y;
  const int dim = threadIdx.x;
  const int lane = dim & 63;
  const int wid = dim >> 6;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int nc = (L + a.chunk - 1) / a.chunk;
  int kb = a.kk[b];
  kb = kb < 0 ? 0 : (kb > a.k_cap ? a.k_cap : kb);
  const int ns = L > 0 ? (kb + a.split - 1) / a.split : 0;
  const int np = nc + ns;
  const size_t bh = static_cast<size_t>(b) * a.Hq + h;
  const float* st = a.stats + bh * a.nchunk * 8;
  const float* ks = a.kstats + bh * a.nsplit * 2;
  const float* ac = a.acc + bh * a.nchunk * D + dim;
  const float* ka = a.kacc + bh * a.nsplit * D + dim;
  // (max, sum) of partial i: text chunk i < nc, else kept split i - nc
  auto ml = [&](int i) -> float2 {
    return i < nc ? *reinterpret_cast<const float2*>(st + i * 8 + 4)
                  : *reinterpret_cast<const float2*>(ks + (i - nc) * 2);
  };

  float M = kNegInf;
  for (int i = dim; i < np; i += D) {
    const float2 v = ml(i);
    if (v.y > 0.f) M = fmaxf(M, v.x);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  if (lane == 0) s_red[wid] = M;
  __syncthreads();
  M = s_red[0];
#pragma unroll
  for (int v = 1; v < D / 64; ++v) M = fmaxf(M, s_red[v]);

  float num = 0.f, den = 0.f;
  for (int base = 0; base < np; base += D) {
    __syncthreads();
    {
      const int i = base + dim;
      float wgt = 0.f;
      if (i < np) {
        const float2 v = ml(i);
        wgt = v.y > 0.f ? fast_exp2(v.x - M) : 0.f;
      }
      s_w[dim] = wgt;
    }
    __syncthreads();
    const int cnt = min(D, np - base);
    for (int j = 0; j < cnt; ++j) {
      const float wgt = s_w[j];
      if (wgt == 0.f) continue;
      const int i = base + j;
      const float l = i < nc ? st[i * 8 + 5] : ks[(i - nc) * 2 + 1];
      const float v = i < nc ? ac[static_cast<size_t>(i) * D] : ka[static_cast<size_t>(i - nc) * D];
      den += wgt * l;
      num += wgt * v;
    }
  }
  const float o = den > 0.f ? num / den : 0.f;
  if (a.dtype == VP_BF16)
    static_cast<uint16_t*>(a.out)[bh * D + dim] = f32_to_bf16_bits(o);
  else
    static_cast<float*>(a.out)[bh * D + dim] = o;
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int head_dim, hipStream_t st) {
  const dim3 grid(a.Hq, a.B);
  if (head_dim == 128)
    hipLaunchKernelGGL(merge_kernel<128>, grid, dim3(128), 0, st, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(merge_kernel<64>, grid, dim3(64), 0, st, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace vp
