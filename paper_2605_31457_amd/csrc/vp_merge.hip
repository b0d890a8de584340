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
  const int h = blockIdx.x;
  const int b = blockIdx.y;
  const int dim = threadIdx.x;
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int nc = (L + a.chunk - 1) / a.chunk;
  int kb = a.kk[b];
  kb = kb < 0 ? 0 : (kb > a.k_cap ? a.k_cap : kb);
  const int ns = L > 0 ? (kb + a.split - 1) / a.split : 0;
  const size_t bh = static_cast<size_t>(b) * a.Hq + h;
  const float* st = a.stats + bh * a.nchunk * 8;
  const float* ks = a.kstats + bh * a.nsplit * 2;
  const float* ac = a.acc + bh * a.nchunk * D + dim;
  const float* ka = a.kacc + bh * a.nsplit * D + dim;

  float M = kNegInf;
  for (int c = 0; c < nc; ++c)
    if (st[c * 8 + 5] > 0.f) M = fmaxf(M, st[c * 8 + 4]);
  for (int s = 0; s < ns; ++s)
    if (ks[s * 2 + 1] > 0.f) M = fmaxf(M, ks[s * 2]);

  float num = 0.f, den = 0.f;
  for (int c = 0; c < nc; ++c) {
    const float l = st[c * 8 + 5];
    if (l > 0.f) {
      const float wgt = fast_exp2(st[c * 8 + 4] - M);
      den += wgt * l;
      num += wgt * ac[static_cast<size_t>(c) * D];
    }
  }
  for (int s = 0; s < ns; ++s) {
    const float l = ks[s * 2 + 1];
    if (l > 0.f) {
      const float wgt = fast_exp2(ks[s * 2] - M);
      den += wgt * l;
      num += wgt * ka[static_cast<size_t>(s) * D];
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
