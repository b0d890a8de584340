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

constexpr int kKeptHeld = 8;  // kept rows a lane group holds (k_cap <= kKeptHeld * R)

// four bf16 values (two 32-bit words, low half first) as floats
__device__ __forceinline__ float4 bf16x4_to_f32(uint2 u) {
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xffff0000u));
}

// The kept rows' attention folded into the merge: each kept row of the head's
// selection row is one more "partial" with maximum z (its logit, q.K scaled to
// the log2 domain, summed over the lane group's columns in a fixed butterfly),
// sum 1 and value row V (the weight is 2^(z - M) like a partial's). For small
// steps (a handful of kept work-groups would leave the GPU idle): one launch
// fewer. Every path that merges with the text part from the workspace (the step,
// and vp_sparse_decode_attn given VP_ATTN_TEXT_FROM_WORKSPACE) uses this kernel
// for such steps, so the step and the four calls give the same bits; a layer
// that reads its own text rows keeps its kept pass (there the kept work-groups
// fill the text pass's tail).
// Every kept slot up to k_cap is requested with the budget, the length and the
// text partials; entries past the budget and positions outside [0, L) are skipped.
template <int D>
__global__ __launch_bounds__(kMergeThreads) void merge_kept_kernel(const MergeArgs a) {
  constexpr int COLS = D / 4;
  constexpr int R = kMergeThreads / COLS;
  __shared__ float s_red[kMergeThreads / 64];
  __shared__ float4 s_num[R][COLS];
  __shared__ float s_den[R];
  const int x = blockIdx.x;  // t*Hq + h
  const int qt = x / a.Hq;
  const int h = x - qt * a.Hq;
  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int col = tid % COLS;
  const int r = tid / COLS;
  const int g = h / a.G;
  const int nc = a.nparts;
  const size_t bh = static_cast<size_t>(b) * a.T * a.Hq + vhead(h, qt, a.G, a.T);
  const size_t ob = static_cast<size_t>(b) * a.T * a.Hq + x;
  const float* st = a.stats + bh * a.nparts * 8;
  const float4* ac = reinterpret_cast<const float4*>(a.acc + bh * a.nparts * D) + col;
  const size_t srow = (static_cast<size_t>(b) * a.T + qt) * a.U + g / (a.Hkv / a.U);  // the head's selection row
  const int32_t* kl = a.vis_idx + srow * a.k_cap;
  // first round trip: the text partials, the kept positions, the budget, the
  // length and this lane's four query columns
  const int L = clamp_len(a.seq_len[b], a.max_seq_len);
  const int kb = a.kk[srow];
  const uint2 qu = reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.q) + ob * D)[col];
  const float4 qv = bf16x4_to_f32(qu);
  float2 v[kHeld];
  float4 xv[kHeld];
#pragma unroll
  for (int j = 0; j < kHeld; ++j) {
    const int i = r + j * R;
    const int ii = i < nc ? i : 0;
    v[j] = *reinterpret_cast<const float2*>(st + ii * 8 + 4);
    xv[j] = ac[static_cast<size_t>(ii) * COLS];
    if (i >= nc) v[j] = make_float2(kNegInf, 0.f);
  }
  int pos[kKeptHeld];
#pragma unroll
  for (int j = 0; j < kKeptHeld; ++j) {
    const int i = r + j * R;
    pos[j] = i < a.k_cap ? kl[i] : -1;
  }
  // each kept row's K and V columns (paged caches: after its block id)
  bool okk[kKeptHeld];
  size_t off[kKeptHeld];
#pragma unroll
  for (int j = 0; j < kKeptHeld; ++j) {
    okk[j] = r + j * R < kb && pos[j] >= 0 && pos[j] < L;
    const int p = okk[j] ? pos[j] : 0;
    if (a.block_table) {
      const int blk = a.block_table[static_cast<size_t>(b) * a.nblk + (p >> a.bs_log2)];
      off[j] = static_cast<size_t>(blk) * a.sb + static_cast<size_t>(g) * a.sh +
               static_cast<size_t>(p & ((1 << a.bs_log2) - 1)) * a.ss;
    } else {
      off[j] = static_cast<size_t>(b) * a.sb + static_cast<size_t>(g) * a.sh + static_cast<size_t>(p) * a.ss;
    }
  }
  uint2 ku[kKeptHeld], vu[kKeptHeld];
#pragma unroll
  for (int j = 0; j < kKeptHeld; ++j) {
    ku[j] = reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.K) + off[j])[col];
    vu[j] = reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.V) + off[j])[col];
  }
  float zk[kKeptHeld];
  float4 vk[kKeptHeld];
#pragma unroll
  for (int j = 0; j < kKeptHeld; ++j) {
    const float4 kf = bf16x4_to_f32(ku[j]);
    float z = ((qv.x * kf.x + qv.y * kf.y) + (qv.z * kf.z + qv.w * kf.w));
#pragma unroll
    for (int o = 1; o < COLS; o <<= 1) z += __shfl_xor(z, o);  // the row's COLS column lanes
    zk[j] = okk[j] ? z * a.zscale : kNegInf;
    vk[j] = bf16x4_to_f32(vu[j]);
  }
  float M = kNegInf;
#pragma unroll
  for (int j = 0; j < kHeld; ++j)
    if (v[j].y > 0.f) M = fmaxf(M, v[j].x);
#pragma unroll
  for (int j = 0; j < kKeptHeld; ++j) M = fmaxf(M, zk[j]);
  M = block_max(M, s_red, lane, wid);
  float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
  float den = 0.f;
#pragma unroll
  for (int j = 0; j < kHeld; ++j) {
    if (v[j].y > 0.f) {
      const float w = fast_exp2(v[j].x - M);
      den += w * v[j].y;
      num.x += w * xv[j].x;
      num.y += w * xv[j].y;
      num.z += w * xv[j].z;
      num.w += w * xv[j].w;
    }
  }
#pragma unroll
  for (int j = 0; j < kKeptHeld; ++j) {
    if (zk[j] != kNegInf) {
      const float w = fast_exp2(zk[j] - M);
      den += w;
      num.x += w * vk[j].x;
      num.y += w * vk[j].y;
      num.z += w * vk[j].z;
      num.w += w * vk[j].w;
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
      const float4 y = s_num[j][col];
      o.x += y.x;
      o.y += y.y;
      o.z += y.z;
      o.w += y.w;
      dd += s_den[j];
    }
    const float inv = dd > 0.f ? 1.0f / dd : 0.f;
    uint2 packed;
    packed.x = f32_to_bf16_bits(o.x * inv) | (static_cast<uint32_t>(f32_to_bf16_bits(o.y * inv)) << 16);
    packed.y = f32_to_bf16_bits(o.z * inv) | (static_cast<uint32_t>(f32_to_bf16_bits(o.w * inv)) << 16);
    reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + ob * D)[col] = packed;
  }
}

}  // namespace

int merge_kept_max_parts(int head_dim) { return kHeld * (kMergeThreads / (head_dim / 4)); }
int merge_kept_max_rows(int head_dim) { return kKeptHeld * (kMergeThreads / (head_dim / 4)); }

hipError_t launch_merge_kept(const MergeArgs& a, int head_dim, hipStream_t st) {
  const dim3 grid(a.T * a.Hq, a.B);
  if (head_dim == 128)
    hipLaunchKernelGGL(merge_kept_kernel<128>, grid, dim3(kMergeThreads), 0, st, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(merge_kept_kernel<64>, grid, dim3(kMergeThreads), 0, st, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

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
