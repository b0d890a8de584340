// One streaming pass over a sequence's KV cache for one KV head: the kernel
// behind vp_visual_mass (Eq. (2), (5), (6)) and the attention partials of
// vp_sparse_decode_attn (Sec. 4.1/4.2).
//
// Work decomposition: one 64-lane wave per work-group; grid = (parts, Hkv, B).
// A part is a chunk of `chunk` consecutive cache positions (context pass) or
// `split` consecutive entries of the kept-index list (kept pass). The wave walks
// its part in tiles of 64 rows (two 32-row sub-tiles) and issues all of a
// tile's HBM reads at once: key rows into registers, value rows straight into
// LDS with global_load_lds_dwordx4 (no registers held), so each wave keeps up
// to 32 KB in flight.
//
// Per tile the grouped query heads of this KV head (G <= 16, padded to 16) are
// scored against the 32 key rows with matrix-core instructions:
//   C'[token][head] = K_tile[token][:] . q[head][:]
// bf16: v_mfma_f32_16x16x32_bf16 (two 16-row halves x d/32 k-steps);
// fp32: v_mfma_f32_16x16x4_f32. Key rows are loaded straight from HBM into the
// A-operand registers (16 B per lane, 4 lanes cover 64 contiguous bytes of a
// row). The output leaves lane l with head l%16 and tokens 16*half + 4*(l/16) + r.
//
// Statistics, all in the log2 domain z = Z * log2(e) with a running maximum
// shared by the four lanes of a head:
//   Ls = sum_j 2^((z_j - m)/tau_score)   (normaliser of the Eq. (2) attention)
//   Lm = sum_j 2^((z_j - m)/tau_mass)    (denominator of Eq. (6))
//   Vm = sum_{j visual} 2^((z_j - m)/tau_mass)   (numerator of Eq. (5))
// Visual logits are spilled to the workspace (rank order) for the scores,
// which need the global (m, Ls) of every head.
//
// Attention partial (text rows of the context pass, or the gathered kept rows):
//   (m_t, l_t, acc[d]) with p_j = 2^(z_j - m_t), acc = sum_j p_j V_j.
// The value product runs on the matrix cores as out^T[dim][head] += V^T P^T:
// the V rows sit in LDS in groups of 1 KB (one DMA instruction each) padded to
// 1152 bytes, so the four lane groups of the transposed read fall in different
// bank windows; P comes straight from the score registers, so the accumulator
// keeps lane l on head l%16 and the rescaling factor stays lane-local.
#include "vp_common.h"
#include "vp_internal.h"

#ifndef VP_ATTEND_WAVES
#define VP_ATTEND_WAVES 2
#endif

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

namespace vp {
namespace {

template <int DT, int D>
struct Cfg {
  static constexpr bool BF = DT == VP_BF16;
  static constexpr int ESZ = BF ? 2 : 4;
  static constexpr int ROWB = D * ESZ;                      // bytes per K/V row
  static constexpr int KLD_HALF = ROWB / 64;                // 16-byte K loads per lane per 16-row half
  static constexpr int KLD = 2 * KLD_HALF;                  // per 32-row sub-tile
  static constexpr int LANES_PER_ROW = ROWB / 16;           // 16-byte pieces per row
  static constexpr int RPI = 64 / LANES_PER_ROW;            // rows per 1 KB LDS-DMA instruction
  static constexpr int GSTR = 1024 + 128;                   // LDS bytes per DMA group (padded)
  static constexpr int SUB_GROUPS = 32 / RPI;               // DMA instructions per sub-tile
  static constexpr int SUB_BYTES = SUB_GROUPS * GSTR;       // LDS bytes per sub-tile
  static constexpr int ACC_N = BF ? (D / 64) * 4 : D / 16;  // f32x4 accumulators
  // LDS offset of row r of a sub-tile
  static __device__ __forceinline__ int row_off(int r) { return (r / RPI) * GSTR + (r % RPI) * ROWB; }
};

template <int DT, int D>
struct QFrag;

template <int D>
struct QFrag<VP_BF16, D> {
  bf16x8 v[D / 32];
};
template <int D>
struct QFrag<VP_F32, D> {
  float v[D / 4];
};

// q row of head h as the B operand (k-slot (a4, i) of step s <-> dim s*32 + 8*a4 + i
// for bf16; dim (D/4)*a4 + s for fp32)
template <int DT, int D>
__device__ __forceinline__ void load_q(QFrag<DT, D>& f, const void* qrow, bool valid, int a4) {
  if constexpr (DT == VP_BF16) {
    const uint4* p = reinterpret_cast<const uint4*>(qrow);
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      uint4 u = valid ? p[4 * s + a4] : make_uint4(0, 0, 0, 0);
      f.v[s] = __builtin_bit_cast(bf16x8, u);
    }
  } else {
    const float4* p = reinterpret_cast<const float4*>(qrow);
#pragma unroll
    for (int s4 = 0; s4 < D / 16; ++s4) {
      float4 u = valid ? p[(D / 16) * a4 + s4] : make_float4(0.f, 0.f, 0.f, 0.f);
      f.v[4 * s4 + 0] = u.x;
      f.v[4 * s4 + 1] = u.y;
      f.v[4 * s4 + 2] = u.z;
      f.v[4 * s4 + 3] = u.w;
    }
  }
}

// 16-byte piece j of this lane's share of a key row (same dim mapping as load_q)
template <int DT, int D>
__device__ __forceinline__ int kpiece(int a4, int j) {
  if constexpr (DT == VP_BF16)
    return 4 * j + a4;
  else
    return (D / 16) * a4 + j;
}

// C'[token n16 of a 16-row half][head] from the lane's preloaded key pieces
template <int DT, int D>
__device__ __forceinline__ f32x4 score_half(const uint4* kr, const QFrag<DT, D>& q) {
  f32x4 c = {0.f, 0.f, 0.f, 0.f};
  if constexpr (DT == VP_BF16) {
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[s]), q.v[s], c, 0, 0, 0);
  } else {
#pragma unroll
    for (int s4 = 0; s4 < D / 16; ++s4) {
      const float4 u = __builtin_bit_cast(float4, kr[s4]);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(u.x, q.v[4 * s4 + 0], c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(u.y, q.v[4 * s4 + 1], c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(u.z, q.v[4 * s4 + 2], c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(u.w, q.v[4 * s4 + 3], c, 0, 0, 0);
    }
  }
  return c;
}

// sub-tile-relative token held by lane slot (a4, i) of the value product: the
// score registers of lane l hold tokens 4*a4 + r (half 0) and 16 + 4*a4 + r (half 1)
__device__ __forceinline__ int pv_token(int a4, int i) { return i < 4 ? 4 * a4 + i : 16 + 4 * a4 + (i - 4); }

template <int DT, int D, int N>
__device__ __forceinline__ void value_product(f32x4 (&acc)[N], const unsigned char* vlds, const float (&p)[8],
                                              int a4, int n16) {
  using C = Cfg<DT, D>;
  if constexpr (DT == VP_BF16) {
    // P^T operand: slot (a4, i) <-> token pv_token(a4, i), head n16
    bf16x8 pf;
#pragma unroll
    for (int i = 0; i < 8; ++i) pf[i] = static_cast<__bf16>(p[i]);
#pragma unroll
    for (int u = 0; u < D / 64; ++u) {
      uint2 w[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        w[i] = *reinterpret_cast<const uint2*>(vlds + C::row_off(pv_token(a4, i)) + 128 * u + 8 * n16);
      // A operand of MFMA (u, e): row n16 <-> dim 64u + 4*n16 + e, slot i <-> token pv_token(a4, i)
      uint32_t lo0[4], hi0[4], lo1[4], hi1[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        lo0[j] = __builtin_amdgcn_perm(w[2 * j + 1].x, w[2 * j].x, 0x05040100u);
        hi0[j] = __builtin_amdgcn_perm(w[2 * j + 1].x, w[2 * j].x, 0x07060302u);
        lo1[j] = __builtin_amdgcn_perm(w[2 * j + 1].y, w[2 * j].y, 0x05040100u);
        hi1[j] = __builtin_amdgcn_perm(w[2 * j + 1].y, w[2 * j].y, 0x07060302u);
      }
      const bf16x8 a0 = __builtin_bit_cast(bf16x8, make_uint4(lo0[0], lo0[1], lo0[2], lo0[3]));
      const bf16x8 a1 = __builtin_bit_cast(bf16x8, make_uint4(hi0[0], hi0[1], hi0[2], hi0[3]));
      const bf16x8 a2 = __builtin_bit_cast(bf16x8, make_uint4(lo1[0], lo1[1], lo1[2], lo1[3]));
      const bf16x8 a3 = __builtin_bit_cast(bf16x8, make_uint4(hi1[0], hi1[1], hi1[2], hi1[3]));
      acc[4 * u + 0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, pf, acc[4 * u + 0], 0, 0, 0);
      acc[4 * u + 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, pf, acc[4 * u + 1], 0, 0, 0);
      acc[4 * u + 2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, pf, acc[4 * u + 2], 0, 0, 0);
      acc[4 * u + 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, pf, acc[4 * u + 3], 0, 0, 0);
    }
  } else {
    // k-step s covers tokens pv_token(a4, s) (one per lane group); row n16 <-> dim 16*dt + n16
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const unsigned char* row = vlds + C::row_off(pv_token(a4, s));
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const float v = *reinterpret_cast<const float*>(row + 4 * (16 * dt + n16));
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(v, p[s], acc[dt], 0, 0, 0);
      }
    }
  }
}

// store the lane's accumulator slice (head n16) of a (D)-float partial row
template <int DT, int D, int N>
__device__ __forceinline__ void store_acc(float* dst, const f32x4 (&acc)[N], int a4) {
  if constexpr (DT == VP_BF16) {
    // acc[4u + e][r] holds dim 64u + 16*a4 + 4r + e
#pragma unroll
    for (int u = 0; u < D / 64; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float4 o = make_float4(acc[4 * u + 0][r], acc[4 * u + 1][r], acc[4 * u + 2][r], acc[4 * u + 3][r]);
        *reinterpret_cast<float4*>(dst + 64 * u + 16 * a4 + 4 * r) = o;
      }
  } else {
    // acc[dt][r] holds dim 16*dt + 4*a4 + r
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      *reinterpret_cast<float4*>(dst + 16 * dt + 4 * a4) = make_float4(acc[dt][0], acc[dt][1], acc[dt][2], acc[dt][3]);
  }
}

enum TileClass : int { TILE_TEXT = 0, TILE_VIS = 1, TILE_MIXED = 2 };

// class of tile [t0, t_end) given a walker already seeked to t0
__device__ __forceinline__ int classify(const SegWalker& w, int t0, int t_end) {
  if (w.s < w.nseg && w.st < t_end) return (w.st <= t0 && w.en >= t_end) ? TILE_VIS : TILE_MIXED;
  return TILE_TEXT;
}

struct Sub {
  int t0;       // first row of the 32-row sub-tile (cache position, or index into the kept list)
  int cls;      // TileClass (context pass)
  SegWalker w;  // segment walker positioned at t0 (context pass)
};

// All per-wave state of one part; the member functions are force-inlined so the
// key registers never leave the register file.
template <int DT, int D, int MODE>
struct Pass {
  using C = Cfg<DT, D>;
  static constexpr bool KEPT = MODE == MODE_KEPT;
  static constexpr bool SCORE = (MODE & MODE_SCORE) != 0 && !KEPT;
  static constexpr bool ATTN = KEPT || (MODE & MODE_TEXT) != 0;
  static constexpr bool SKIP_VIS = MODE == MODE_TEXT;  // text-only pass never touches visual rows

  const AttendArgs& a;
  unsigned char* vlds;
  int lane, n16, a4, L, r0, r1, h;
  bool hv;
  const int32_t* kept;
  const char* Kb;
  const char* Vb;
  size_t rstride;
  float* zrow;
  QFrag<DT, D> qf;
  float m_all, Ls, Lm, Vm, m_t, l_t;
  f32x4 acc[C::ACC_N];

  __device__ __forceinline__ Pass(const AttendArgs& a_, unsigned char* vlds_) : a(a_), vlds(vlds_) {}

  // cache position of part row t (clamped to a readable row; validity is tracked separately)
  __device__ __forceinline__ int row_pos(int t) const {
    if constexpr (KEPT) {
      const int p = t < r1 ? kept[t] : 0;
      return (p < 0 || p >= L) ? 0 : p;
    } else {
      return t < L ? t : L - 1;
    }
  }

  __device__ __forceinline__ bool active(const Sub& s) const {
    return s.t0 < r1 && !(SKIP_VIS && s.cls == TILE_VIS);
  }
  __device__ __forceinline__ bool needs_v(const Sub& s) const { return ATTN && (KEPT || s.cls != TILE_VIS); }

  __device__ __forceinline__ Sub sub_at(const Sub& prev, int t0) const {
    Sub n = prev;
    n.t0 = t0;
    n.cls = TILE_TEXT;
    if constexpr (!KEPT) {
      if (t0 < r1) {
        n.w.seek(t0);
        n.cls = classify(n.w, t0, min(t0 + 32, r1));
      }
    }
    return n;
  }

  // this lane's key pieces of sub-tile s, into registers
  __device__ __forceinline__ void load_k(uint4 (&kr)[C::KLD], const Sub& s) const {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const uint4* row = reinterpret_cast<const uint4*>(Kb + row_pos(s.t0 + 16 * hf + n16) * rstride);
#pragma unroll
      for (int j = 0; j < C::KLD_HALF; ++j) kr[hf * C::KLD_HALF + j] = row[kpiece<DT, D>(a4, j)];
    }
  }
  // the 32 value rows of sub-tile s, HBM -> LDS directly (lane l of DMA group j
  // carries 16 bytes of row j*RPI + l/LANES_PER_ROW)
  __device__ __forceinline__ void dma_v(const Sub& s, unsigned char* lbase) const {
    const int rr = lane / C::LANES_PER_ROW;
    const int col = lane % C::LANES_PER_ROW;
#pragma unroll
    for (int j = 0; j < C::SUB_GROUPS; ++j) {
      const char* src = Vb + row_pos(s.t0 + j * C::RPI + rr) * rstride + 16 * col;
      __builtin_amdgcn_global_load_lds((global_void*)(src), (lds_void*)(lbase + j * C::GSTR), 16, 0, 0);
    }
  }

  __device__ __forceinline__ void process(const Sub& tile, const uint4 (&kr)[C::KLD], const unsigned char* vsub) {
    const int t0 = tile.t0;
    const int cls = tile.cls;
    const int t_end = min(t0 + 32, r1);
    // ---- scores of the 32 rows against the query group ----
    const f32x4 c0 = score_half<DT, D>(kr, qf);
    const f32x4 c1 = score_half<DT, D>(kr + C::KLD_HALF, qf);

    float z[8];
    bool valid[8], vis[8];
    int rank[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int tt = 16 * (i >> 2) + 4 * a4 + (i & 3);
      z[i] = (i < 4 ? c0[i & 3] : c1[i & 3]) * a.zscale;
      vis[i] = false;
      rank[i] = 0;
      if constexpr (KEPT) {
        const int t = t0 + tt;
        bool ok = t < r1;
        if (ok) {
          const int p = kept[t];
          ok = p >= 0 && p < L;
        }
        valid[i] = ok;
      } else {
        valid[i] = t0 + tt < t_end;
      }
    }
    if constexpr (!KEPT) {
      if (cls == TILE_VIS) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          vis[i] = true;
          rank[i] = tile.w.rank + (t0 + 16 * (i >> 2) + 4 * a4 + (i & 3) - tile.w.st);
        }
      } else if (cls == TILE_MIXED) {
        SegWalker lw = tile.w;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int p = t0 + 16 * (i >> 2) + 4 * a4 + (i & 3);
          if (p < t_end) {
            lw.seek(p);
            vis[i] = lw.contains(p);
            rank[i] = lw.rank + (p - lw.st);
          }
        }
      }
    }

    // ---- Eq. (5)/(6) and Eq. (2) statistics ----
    if constexpr (SCORE) {
      float tmax = kNegInf;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (valid[i]) tmax = fmaxf(tmax, z[i]);
      tmax = max_over_quads(tmax);
      const float mn = fmaxf(m_all, tmax);
      const float als = fast_exp2((m_all - mn) * a.inv_tau_s);
      const float alm = fast_exp2((m_all - mn) * a.inv_tau_m);
      float ts = 0.f, tm = 0.f, tv = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float d = valid[i] ? z[i] - mn : kNegInf;
        const float es = fast_exp2(d * a.inv_tau_s);
        const float em = fast_exp2(d * a.inv_tau_m);
        ts += es;
        tm += em;
        tv += vis[i] ? em : 0.f;
      }
      Ls = Ls * als + ts;
      Lm = Lm * alm + tm;
      Vm = Vm * alm + tv;
      m_all = mn;
      if (hv) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (valid[i] && vis[i] && rank[i] < a.max_vis) zrow[rank[i]] = z[i];
      }
    }

    // ---- attention partial over text rows (context pass) or kept rows ----
    if constexpr (ATTN) {
      if (needs_v(tile)) {
        float zt[8];
        float tmax = kNegInf;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          zt[i] = (valid[i] && !vis[i]) ? z[i] : kNegInf;
          tmax = fmaxf(tmax, zt[i]);
        }
        tmax = max_over_quads(tmax);
        if (tmax != kNegInf) {
          const float mn = fmaxf(m_t, tmax);
          const float al = fast_exp2(m_t - mn);
          float p[8];
          float ps = 0.f;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            p[i] = fast_exp2(zt[i] - mn);
            ps += p[i];
          }
          l_t = l_t * al + ps;
          m_t = mn;
#pragma unroll
          for (int i = 0; i < C::ACC_N; ++i) acc[i] *= al;
          // the value rows were written to LDS by the DMA: wait for every
          // outstanding vector-memory operation, then read them transposed
          __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
          value_product<DT, D, C::ACC_N>(acc, vsub, p, a4, n16);
        }
      }
    }
  }
};

template <int DT, int D, int MODE>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(VP_ATTEND_WAVES))) void attend_kernel(
    const AttendArgs a) {
  using C = Cfg<DT, D>;
  using P = Pass<DT, D, MODE>;
  __shared__ __attribute__((aligned(16))) unsigned char vlds[P::ATTN ? 2 * C::SUB_BYTES : 16];

  P s(a, vlds);
  s.lane = threadIdx.x;
  s.n16 = s.lane & 15;
  s.a4 = s.lane >> 4;
  const int b = blockIdx.z;
  const int g = blockIdx.y;
  const int part = blockIdx.x;
  s.L = clamp_len(a.seq_len[b], a.max_seq_len);
  s.kept = nullptr;
  if constexpr (P::KEPT) {
    if (s.L == 0) return;
    int kb = a.kk[b];
    kb = kb < 0 ? 0 : (kb > a.k_cap ? a.k_cap : kb);
    s.r0 = part * a.split;
    s.r1 = min(s.r0 + a.split, kb);
    s.kept = a.vis_idx + static_cast<size_t>(b) * a.k_cap;
  } else {
    s.r0 = part * a.chunk;
    s.r1 = min(s.r0 + a.chunk, s.L);
  }
  if (s.r0 >= s.r1) return;

  s.h = g * a.G + s.n16;
  s.hv = s.n16 < a.G;
  s.Kb = static_cast<const char*>(a.K) + (static_cast<size_t>(b) * a.sb + static_cast<size_t>(g) * a.sh) * C::ESZ;
  s.Vb = P::ATTN ? static_cast<const char*>(a.V) +
                       (static_cast<size_t>(b) * a.sb + static_cast<size_t>(g) * a.sh) * C::ESZ
                 : nullptr;
  s.rstride = static_cast<size_t>(a.ss) * C::ESZ;
  load_q<DT, D>(s.qf,
                static_cast<const char*>(a.q) + (static_cast<size_t>(b) * a.Hq + (s.hv ? s.h : 0)) * C::ROWB,
                s.hv, s.a4);
  s.m_all = kNegInf;
  s.Ls = s.Lm = s.Vm = 0.f;
  s.m_t = kNegInf;
  s.l_t = 0.f;
#pragma unroll
  for (int i = 0; i < C::ACC_N; ++i) s.acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  s.zrow = P::SCORE ? a.zs + (static_cast<size_t>(b) * a.Hq + (s.hv ? s.h : 0)) * a.max_vis : nullptr;

  Sub s0;
  s0.t0 = s.r0;
  s0.cls = TILE_TEXT;
  if constexpr (!P::KEPT) {
    const int o0 = a.seg_off[b];
    s0.w.start(a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, s.L);
  }
  s0 = s.sub_at(s0, s.r0);

  uint4 k0[C::KLD], k1[C::KLD];
  unsigned char* v0 = vlds;
  unsigned char* v1 = vlds + C::SUB_BYTES;
  // 64-row tiles: every read of the tile is issued before any of it is used
  while (s0.t0 < s.r1) {
    const Sub s1 = s.sub_at(s0, s0.t0 + 32);
    const bool act0 = s.active(s0), act1 = s.active(s1);
    if constexpr (P::ATTN) __syncthreads();  // the previous tile's LDS reads are done
    if (act0) s.load_k(k0, s0);
    if (act1) s.load_k(k1, s1);
    if constexpr (P::ATTN) {
      if (act0 && s.needs_v(s0)) s.dma_v(s0, v0);
      if (act1 && s.needs_v(s1)) s.dma_v(s1, v1);
    }
    if (act0) s.process(s0, k0, v0);
    if (act1) s.process(s1, k1, v1);
    s0 = s.sub_at(s1, s1.t0 + 32);
  }

  // ---- write this part's partials ----
  if constexpr (P::SCORE) {
    const float s_ls = sum_over_quads(s.Ls);
    const float s_lm = sum_over_quads(s.Lm);
    const float s_vm = sum_over_quads(s.Vm);
    if (s.hv && s.a4 == 0) {
      float* st = a.stats + ((static_cast<size_t>(b) * a.Hq + s.h) * a.nchunk + part) * 8;
      *reinterpret_cast<float4*>(st) = make_float4(s.m_all, s_ls, s_lm, s_vm);
    }
  }
  if constexpr (P::ATTN) {
    const float s_lt = sum_over_quads(s.l_t);
    if (s.hv) {
      float* dst;
      if constexpr (P::KEPT) {
        const size_t row = (static_cast<size_t>(b) * a.Hq + s.h) * a.nsplit + part;
        dst = a.kacc + row * D;
        if (s.a4 == 0) *reinterpret_cast<float2*>(a.kstats + row * 2) = make_float2(s.m_t, s_lt);
      } else {
        const size_t row = (static_cast<size_t>(b) * a.Hq + s.h) * a.nchunk + part;
        dst = a.acc + row * D;
        if (s.a4 == 0) *reinterpret_cast<float2*>(a.stats + row * 8 + 4) = make_float2(s.m_t, s_lt);
      }
      store_acc<DT, D, C::ACC_N>(dst, s.acc, s.a4);
    }
  }
}

template <int DT, int D>
hipError_t launch_dd(const AttendArgs& a, int mode, hipStream_t st) {
  const dim3 grid(mode == MODE_KEPT ? a.nsplit : a.nchunk, a.Hkv, a.B);
  const dim3 block(64);
  switch (mode) {
    case MODE_SCORE:
      hipLaunchKernelGGL((attend_kernel<DT, D, MODE_SCORE>), grid, block, 0, st, a);
      break;
    case MODE_TEXT:
      hipLaunchKernelGGL((attend_kernel<DT, D, MODE_TEXT>), grid, block, 0, st, a);
      break;
    case MODE_SCORE_TEXT:
      hipLaunchKernelGGL((attend_kernel<DT, D, MODE_SCORE_TEXT>), grid, block, 0, st, a);
      break;
    case MODE_KEPT:
      hipLaunchKernelGGL((attend_kernel<DT, D, MODE_KEPT>), grid, block, 0, st, a);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attend(const AttendArgs& a, int mode, int dtype, int head_dim, hipStream_t st) {
  if (dtype == VP_BF16) {
    if (head_dim == 128) return launch_dd<VP_BF16, 128>(a, mode, st);
    if (head_dim == 64) return launch_dd<VP_BF16, 64>(a, mode, st);
  } else if (dtype == VP_F32) {
    if (head_dim == 128) return launch_dd<VP_F32, 128>(a, mode, st);
    if (head_dim == 64) return launch_dd<VP_F32, 64>(a, mode, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace vp
