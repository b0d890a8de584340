// Split-K reduction of the pruned attention (Sec. 4.1/4.2): merges the text
// partials of the context pass (one per context-pass part) and the kept-row partials
// (one per split of the kept list) of every (sequence, query, query head):
//   out = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i,  M = max_i m_i,
// over the partials with l_i > 0 (parts and splits with no rows write empty
// ones); an empty context gives zeros.
// grid = (T*Hq, B); 256 threads = (D/4 float4 columns) x R partial lanes, so the
// partials are read in parallel (R at a time, each row as coalesced float4s)
// rather than one after another.
#include "vp_common.h"
#include "vp_internal.h"

namespace vp {
namespace {

constexpr int kMergeThreads = 256;
constexpr int kHeld = 8;  // partials a lane group holds in registers (np <= kHeld * R)

// maximum over the block (every thread gets it)
__device__ __forceinline__ float block_max(float m, float* s_red, int lane, int wid) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if (lane == 0) s_red[wid] = m;
  __syncthreads();
  m = s_red[0];
#pragma unroll
  for (int v = 1; v < kMergeThreads / 64; ++v) m = fmaxf(m, s_red[v]);
  return m;
}

template <int D>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(const MergeArgs a) {
  constexpr int COLS = D / 4;                // float4 columns of a partial
  constexpr int R = kMergeThreads / COLS;    // partials in flight per step
  __shared__ float s_red[kMergeThreads / 64];
  __shared__ float4 s_num[R][COLS];
  __shared__ float s_den[R];
  const int x = blockIdx.x;  // t*Hq + h: query t, head h
  const int qt = x / a.Hq;
  const int h = x - qt * a.Hq;
  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int col = tid % COLS;
  const int r = tid / COLS;
  // every slot holds a partial (parts past the sequence's tiles and splits
  // past its budget hold empty ones), so none of them waits for the length or
  // the budget to be read first
  const int nc = a.nparts;
  const int np = nc + a.nsplit;
  const size_t bh = static_cast<size_t>(b) * a.T * a.Hq + vhead(h, qt, a.G, a.T);  // partials: virtual head
  const size_t ob = static_cast<size_t>(b) * a.T * a.Hq + x;  // out [B][T][Hq][D]
  const float* st = a.stats + bh * a.nparts * 8;
  const float* ks = a.kstats + bh * a.nsplit * 2;
  const float4* ac = reinterpret_cast<const float4*>(a.acc + bh * a.nparts * D) + col;
  const float4* ka = reinterpret_cast<const float4*>(a.kacc + bh * a.nsplit * D) + col;
  // (max, sum) of partial i: text part i < nc, else kept split i - nc
  auto ml = [&](int i) -> float2 {
    return i < nc ? *reinterpret_cast<const float2*>(st + i * 8 + 4)
                  : *reinterpret_cast<const float2*>(ks + (i - nc) * 2);
  };

  float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
  float den = 0.f;
  if (np <= kHeld * R) {
    // every partial of this lane group requested at once, value rows included;
    // the maximum is then reduced and the registers rescaled (one round trip)
    float2 v[kHeld];
    float4 xv[kHeld];
#pragma unroll
    for (int j = 0; j < kHeld; ++j) {
      const int i = r + j * R;
      const bool ok = i < np;
      const int ii = ok ? i : 0;  // an in-bounds slot; its values are not used
      v[j] = ml(ii);
      xv[j] = ii < nc ? ac[static_cast<size_t>(ii) * COLS] : ka[static_cast<size_t>(ii - nc) * COLS];
      if (!ok) v[j] = make_float2(kNegInf, 0.f);
    }
    float M = kNegInf;
#pragma unroll
    for (int j = 0; j < kHeld; ++j)
      if (v[j].y > 0.f) M = fmaxf(M, v[j].x);
    M = block_max(M, s_red, lane, wid);
#pragma unroll
    for (int j = 0; j < kHeld; ++j) {
      if (v[j].y > 0.f) {  // empty partials (and the unused slots) contribute nothing
        const float w = fast_exp2(v[j].x - M);
        den += w * v[j].y;
        num.x += w * xv[j].x;
        num.y += w * xv[j].y;
        num.z += w * xv[j].z;
        num.w += w * xv[j].w;
      }
    }
  } else {
    float M = kNegInf;
    for (int i = tid; i < np; i += kMergeThreads) {
      const float2 v = ml(i);
      if (v.y > 0.f) M = fmaxf(M, v.x);
    }
    M = block_max(M, s_red, lane, wid);
#pragma unroll 4
    for (int i = r; i < np; i += R) {
      const float2 v = ml(i);
      const float w = v.y > 0.f ? fast_exp2(v.x - M) : 0.f;
      const float4 x = i < nc ? ac[static_cast<size_t>(i) * COLS] : ka[static_cast<size_t>(i - nc) * COLS];
      den += w * v.y;
      num.x += w * x.x;
      num.y += w * x.y;
      num.z += w * x.z;
      num.w += w * x.w;
    }
  }
  s_num[r][col] = num;
  if (col == 0) s_den[r] = den;
  __syncthreads();
  if (r == 0) {
    float dd = 0.f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const float4 x = s_num[j][col];
      o.x += x.x;
      o.y += x.y;
      o.z += x.z;
      o.w += x.w;
      dd += s_den[j];
    }
    const float inv = dd > 0.f ? 1.0f / dd : 0.f;
    o.x *= inv;
    o.y *= inv;
    o.z *= inv;
    o.w *= inv;
    if (a.dtype == VP_BF16) {
      uint2 packed;
      packed.x = f32_to_bf16_bits(o.x) | (static_cast<uint32_t>(f32_to_bf16_bits(o.y)) << 16);
      packed.y = f32_to_bf16_bits(o.z) | (static_cast<uint32_t>(f32_to_bf16_bits(o.w)) << 16);
      reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + ob * D)[col] = packed;
    } else {
      reinterpret_cast<float4*>(static_cast<float*>(a.out) + ob * D)[col] = o;
    }
  }
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int head_dim, hipStream_t st) {
  const dim3 grid(a.T * a.Hq, a.B);
  if (head_dim == 128)
    hipLaunchKernelGGL(merge_kernel<128>, grid, dim3(kMergeThreads), 0, st, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(merge_kernel<64>, grid, dim3(kMergeThreads), 0, st, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace vp
