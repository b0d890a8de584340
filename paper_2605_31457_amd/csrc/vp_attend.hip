// One streaming pass over a sequence's KV cache for one KV head: the kernel
// behind vp_visual_mass (Eq. (2), (5), (6)) and the attention partials of
// vp_sparse_decode_attn (Sec. 4.1/4.2).
//
// Work decomposition: one 64-lane wave per work-group; grid = (parts, Hkv, B)
// (kept pass: (splits, Hkv * T, B), one row of work-groups per query).
// In the context pass part p of `nparts` takes the 32-row tiles p, p + nparts,
// p + 2 nparts, ... of the cache (a cyclic deal: every part, and so every XCD,
// sees the sequence's own mix of visual and text rows); in the kept pass a part
// is `split` consecutive entries of the kept-index list.
//
// Three roles share this kernel:
//   visual pass  visual rows only: Eq. (5)/(6) and Eq. (2) statistics and the
//                logit spill (the only large write of the step);
//   text pass    text rows only: the same statistics and/or the attention
//                partial over text K/V, with no large writes, so its reads
//                stream without write traffic mixed in;
//   kept pass    gathered kept visual rows: the attention partial.
//
// Memory path. Every K and V row of a tile is copied HBM -> LDS with
// global_load_lds_dwordx4 (non-temporal): one instruction moves whole rows (1 KB contiguous
// per instruction for 256-byte rows), the access pattern that streams at full
// HBM rate on gfx950 (the matrix-core operand layout, 16 rows x 64 B per load,
// streams about 25% slower). All of a tile's copies are issued before any of
// it is used, so no registers are held by data in flight. Inside LDS a row's
// 16-byte pieces are XOR-swizzled by the row index (slot = piece ^ row), which
// keeps the operand reads below free of bank conflicts.
//
// Per 32-row sub-tile the query rows of this KV head -- its G grouped heads for
// each of the sequence's T queries, T*G <= 16, padded to 16 -- are scored
// against the key rows on the matrix cores (with several queries per sequence
// the K/V rows are read once for all of them; query t sees the positions
// before L - T + 1 + t):
//   C'[token][head] = K_tile[token][:] . q[head][:]
// bf16: v_mfma_f32_16x16x32_bf16 (two 16-row halves x d/32 k-steps);
// fp32: v_mfma_f32_16x16x4_f32. Lane l then holds head l%16 for tokens
// 16*half + 4*(l/16) + r.
//
// Statistics, all in the log2 domain z = Z * log2(e), each over the rows of its
// pass relative to a running maximum m (lane-local in the visual pass, shared
// by the four lanes of a head in the text pass):
//   Ls = sum_j 2^((z_j - m)/tau_score)   (normaliser of the Eq. (2) attention)
//   Lm = sum_j 2^((z_j - m)/tau_mass)    (Eq. (6) denominator; over the visual
//                                         rows alone it is the Eq. (5) numerator)
// A maximum is raised only when a logit exceeds it by more than a margin that
// keeps every weight below 2^64, so rescaling is rare.
// Visual logits are spilled to the workspace for the scores, which need the
// global (m, Ls) of every head. The spill holds one plane per (sequence, KV
// group) with a row of zs_gp floats (the group's heads, padded to 8 or 16) per
// cache position; a full visual sub-tile is transposed through a small LDS
// stage so that its 32 rows leave as one contiguous 1-2 KB store (whole lines:
// partial-line writes would compete with the streaming reads for the L1's
// outstanding-request slots), and the scores read each (token, group) row with
// 16-byte loads.
//
// Attention partial (text rows of the context pass, or the gathered kept rows):
//   (m_t, l_t, acc[d]) with p_j = 2^(z_j - m_t), acc = sum_j p_j V_j.
// The value product runs on the matrix cores as out^T[dim][head] += V^T P^T:
// V is read transposed from LDS, P comes straight from the score registers, so
// the accumulator keeps lane l on head l%16 and the rescaling factor is lane-local.
#include "vp_common.h"
#include "vp_internal.h"

#include <hip/hip_ext.h>

#ifndef VP_ATTEND_WAVES
#define VP_ATTEND_WAVES 2  // bf16 passes that read V
#endif
#ifndef VP_ATTEND_WAVES_LEAN
#define VP_ATTEND_WAVES_LEAN 4  // bf16 passes that read only K
#endif
#ifndef VP_TILE_SUBS
#define VP_TILE_SUBS 1  // 32-row sub-tiles whose copies are issued together (context pass)
#endif
#ifndef VP_KEPT_SUBS
#define VP_KEPT_SUBS 1  // same for the kept pass
#endif

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// Cache policy of the K/V row copies: non-temporal (the "nt" bit). Every row is
// used once per step, and streaming it without cache allocation measured ~13%
// faster on the text pass (5.4 -> 6.1 TB/s on the 64 x 32k batch).
constexpr int kCopyPolicy = 2;

// s_waitcnt immediates (gfx9 encoding: vmcnt [3:0]+[15:14], expcnt [6:4], lgkmcnt [11:8])
constexpr int kWaitLgkm0 = 0xC07F;  // lgkmcnt(0), others unconstrained
constexpr int kWaitVm0 = 0x0F70;    // vmcnt(0), others unconstrained
// buffer resource word 3 for raw (untyped) dword access: 32-bit data format
constexpr int kRawBufferWord3 = 0x00020000;
// cache policy of the full-tile spill stores: sc1 (device scope) in the visual
// pass launched alone (64 x 32k batch: visual pass 230 -> 226 us; non-temporal
// stores: 242), the default in the one-launch context pass (sc1 there: 72B-class
// decode loop 84.0 -> 84.6 us per step)
constexpr int spill_policy(int mode) { return (mode & vp::MODE_ONE_LAUNCH) ? 0 : 16; }

namespace vp {
namespace {

// waves per SIMD the register allocation is sized for (one wave per work-group)
constexpr int attend_waves(int dt, int mode) {
  return dt != VP_BF16 ? 1
                       : ((base_mode(mode) == MODE_VIS || base_mode(mode) == MODE_TEXT_STATS)
                              ? VP_ATTEND_WAVES_LEAN
                              : VP_ATTEND_WAVES);
}

// LDS floor per work-group: 20 KB keeps the bf16 passes that read V at 8
// resident work-groups per CU (their 160 registers would allow 10 with 16 KB);
// measured ~8% faster on the text pass of the 64 x 32k batch.
#ifndef VP_LDS_FLOOR_TEXT
#define VP_LDS_FLOOR_TEXT 20480  // bytes; bf16 passes that read V
#endif
#ifndef VP_LDS_FLOOR_VIS
#define VP_LDS_FLOOR_VIS 0  // bytes; bf16 K-only passes
#endif
constexpr int max_i(int x, int y) { return x > y ? x : y; }
constexpr int lds_floor(int dt, int mode) {
  return dt != VP_BF16 ? 0
                       : ((base_mode(mode) == MODE_VIS || base_mode(mode) == MODE_TEXT_STATS)
                              ? VP_LDS_FLOOR_VIS
                              : VP_LDS_FLOOR_TEXT);
}

template <int DT, int D>
struct Cfg {
  static constexpr bool BF = DT == VP_BF16;
  static constexpr int ESZ = BF ? 2 : 4;
  static constexpr int ROWB = D * ESZ;                      // bytes per K/V row
  static constexpr int PIECES = ROWB / 16;                  // 16-byte pieces per row
  static constexpr int RPI = 64 / PIECES;                   // rows per 1 KB copy instruction
  static constexpr int SUB_ROWS_BYTES = 32 * ROWB;          // one 32-row block of K or V
  static constexpr int STAGE_BYTES = 16 * 32 * 4;           // logits of 16 heads x 32 rows
  static constexpr int COPIES = 32 / RPI;                   // copy instructions per block
  static constexpr int ACC_N = BF ? (D / 64) * 4 : D / 16;  // f32x4 accumulators
  // LDS byte offset of 16-byte piece p of row r inside a block
  static __device__ __forceinline__ int at(int r, int p) { return r * ROWB + 16 * (p ^ (r & (PIECES - 1))); }
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

// C'[token n16 of 16-row half hf][head] from the key block in LDS (same dim
// mapping as load_q)
template <int DT, int D>
__device__ __forceinline__ f32x4 score_half(const unsigned char* kb, int hf, const QFrag<DT, D>& q, int a4,
                                            int n16) {
  using C = Cfg<DT, D>;
  const int r = 16 * hf + n16;
  f32x4 c = {0.f, 0.f, 0.f, 0.f};
  if constexpr (DT == VP_BF16) {
    uint4 k[D / 32];
#pragma unroll
    for (int s = 0; s < D / 32; ++s) k[s] = *reinterpret_cast<const uint4*>(kb + C::at(r, 4 * s + a4));
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, k[s]), q.v[s], c, 0, 0, 0);
  } else {
    float4 k[D / 16];
#pragma unroll
    for (int s4 = 0; s4 < D / 16; ++s4) k[s4] = *reinterpret_cast<const float4*>(kb + C::at(r, (D / 16) * a4 + s4));
#pragma unroll
    for (int s4 = 0; s4 < D / 16; ++s4) {
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(k[s4].x, q.v[4 * s4 + 0], c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(k[s4].y, q.v[4 * s4 + 1], c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(k[s4].z, q.v[4 * s4 + 2], c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(k[s4].w, q.v[4 * s4 + 3], c, 0, 0, 0);
    }
  }
  return c;
}

// sub-tile-relative token held by lane slot (a4, i) of the value product: the
// score registers of lane l hold tokens 4*a4 + r (half 0) and 16 + 4*a4 + r (half 1)
__device__ __forceinline__ int pv_token(int a4, int i) { return i < 4 ? 4 * a4 + i : 16 + 4 * a4 + (i - 4); }

template <int DT, int D, int N>
__device__ __forceinline__ void value_product(f32x4 (&acc)[N], const unsigned char* vb, const float (&p)[8],
                                              int a4, int n16) {
  using C = Cfg<DT, D>;
  if constexpr (DT == VP_BF16) {
    // P^T operand: slot (a4, i) <-> token pv_token(a4, i), head n16
    bf16x8 pf;
#pragma unroll
    for (int i = 0; i < 8; ++i) pf[i] = static_cast<__bf16>(p[i]);
#pragma unroll
    for (int u = 0; u < D / 64; ++u) {
      // lane n16 takes dims 64u + 4*n16 .. +3 = 8 bytes in piece 8u + n16/2
      uint2 w[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        w[i] = *reinterpret_cast<const uint2*>(vb + C::at(pv_token(a4, i), 8 * u + (n16 >> 1)) + 8 * (n16 & 1));
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
      const int t = pv_token(a4, s);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const int dim = 16 * dt + n16;
        const float v = *reinterpret_cast<const float*>(vb + C::at(t, dim >> 2) + 4 * (dim & 3));
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
  int kp;       // kept pass: lane r < 32 holds the cache position of row t0 + r (-1 past the list)
  int blk;      // paged caches: lane r < 32 holds the physical block of row t0 + r
  SegWalker w;  // segment walker positioned at t0 (context pass)
};

// All per-wave state of one part; member functions are force-inlined.
template <int DT, int D, int MODE>
struct Pass {
  using C = Cfg<DT, D>;
  static constexpr int BASE = base_mode(MODE);
  static constexpr bool PAGED = (MODE & MODE_PAGED) != 0;        // rows through the block table
  static constexpr bool KEPT = BASE == MODE_KEPT;
  static constexpr bool ZSPILL = KEPT && (MODE & MODE_ZSPILL) != 0;  // kept logits from the spill
  static constexpr bool VIS = BASE == MODE_VIS;                  // visual rows: statistics + spill
  static constexpr bool TSTATS = (BASE & MODE_TEXT_STATS) != 0;  // text rows: statistics
  static constexpr bool ATTN = KEPT || (BASE & MODE_TEXT_ATTN) != 0;
  static constexpr bool TEXT = !KEPT && !VIS;                    // a text-row pass

  const AttendArgs& a;
  int lane, n16, a4, L, r0, r1, step, h;  // rows [r0, r1) in tiles `step` apart; h: virtual head
  int L0, lim;  // rows from L0 on are the queries' own; this lane's query sees rows < lim
  bool hv;
  const int32_t* kept;
  const char* Kb;
  const char* Vb;
  size_t rstride;
  const int32_t* bt;  // paged caches: this sequence's block table (else null)
  size_t bstride;     // paged caches: bytes per physical block
  int bmask;          // paged caches: rows per block - 1
  float* zbase;  // spill plane of this KV group: row p holds the logits of its heads at position p
                 // (kept pass from the spill: offset to the query's first head)
  __amdgpu_buffer_rsrc_t zrsrc;  // visual pass: the same plane as a buffer (its full-tile stores)
  QFrag<DT, D> qf;
  // visual pass: lane-local reference and sums (merged over a head's 4 lanes at the end)
  float m_v, Ls_v, Lm_v;
  // text / kept pass: reference shared by a head's 4 lanes, sums and value partial
  float m_t, l_t, Lm_t, Ls_t;
  f32x4 acc[C::ACC_N];

  __device__ __forceinline__ explicit Pass(const AttendArgs& a_) : a(a_) {}

  // cache position of row r of sub-tile s (clamped to a readable row; validity is tracked separately)
  __device__ __forceinline__ int row_pos(const Sub& s, int r) const {
    if constexpr (KEPT) {
      const int p = __shfl(s.kp, r);
      return (p < 0 || p >= L) ? 0 : p;
    } else {
      const int t = s.t0 + r;
      return t < L ? t : L - 1;
    }
  }

  // does this pass have rows in sub-tile s
  __device__ __forceinline__ bool active(const Sub& s) const {
    if (s.t0 >= r1) return false;
    if constexpr (VIS) return s.cls != TILE_TEXT;
    if constexpr (TEXT) return s.cls != TILE_VIS;
    return true;
  }
  __device__ __forceinline__ bool needs_v(const Sub& s) const { return ATTN; }

  __device__ __forceinline__ Sub sub_at(const Sub& prev, int t0, int kp_loaded = -2) const {
    Sub n = prev;
    n.t0 = t0;
    n.cls = TILE_TEXT;
    if constexpr (KEPT) {
      // one coalesced load of the tile's kept positions (issued a tile ahead;
      // the first tile's come in as kp_loaded, requested before the budget)
      const int t = t0 + lane;
      n.kp = (lane < 32 && t < r1) ? (kp_loaded != -2 ? kp_loaded : kept[t]) : -1;
    } else {
      if (t0 < r1) {
        n.w.seek(t0);
        n.cls = classify(n.w, t0, min(t0 + 32, r1));
      }
    }
    if constexpr (PAGED) {
      // the physical block of each of the tile's rows (the row that row_pos
      // will read: clipped positions included)
      if (lane < 32) {
        int p;
        if constexpr (KEPT) p = (n.kp < 0 || n.kp >= L) ? 0 : n.kp;
        else p = min(t0 + lane, L - 1);
        n.blk = bt[p >> __builtin_ctz(static_cast<unsigned>(bmask + 1))];
      }
    }
    return n;
  }

  // kept pass from the spill: the logits of this lane's 8 rows (head n16 of
  // the query), requested with the tile's V rows; rows past the list read
  // position 0 and are masked like their V rows
  __device__ __forceinline__ void load_spill(const Sub& s, float (&z)[8]) const {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int p = __shfl(s.kp, 16 * (i >> 2) + 4 * a4 + (i & 3));
      const int pp = (p < 0 || p >= L) ? 0 : p;
      z[i] = hv ? zbase[static_cast<size_t>(pp) * a.zs_gp + n16] : 0.f;
    }
  }

  // byte offsets (from the head's base) of what lane l copies in copy j: row
  // j*RPI + l/PIECES, 16-byte piece (l%PIECES) ^ (row & (PIECES-1)) (the swizzle)
  __device__ __forceinline__ void row_offsets(const Sub& s, size_t (&off)[C::COPIES]) const {
    const int rr = lane / C::PIECES;
    const int slot = lane % C::PIECES;
#pragma unroll
    for (int j = 0; j < C::COPIES; ++j) {
      const int r = j * C::RPI + rr;
      const int piece = slot ^ (r & (C::PIECES - 1));
      const int pos = row_pos(s, r);
      if constexpr (PAGED) {
        const int blk = __shfl(s.blk, r);
        off[j] = static_cast<size_t>(blk) * bstride + static_cast<size_t>(pos & bmask) * rstride + 16 * piece;
      } else {
        off[j] = static_cast<size_t>(pos) * rstride + 16 * piece;
      }
    }
  }

  // the 32 rows of a sub-tile from `src` (K or V of this head) into an LDS block
  __device__ __forceinline__ void copy_rows(const char* src, const size_t (&off)[C::COPIES],
                                            unsigned char* block) const {
#pragma unroll
    for (int j = 0; j < C::COPIES; ++j)
      __builtin_amdgcn_global_load_lds((global_void*)(src + off[j]), (lds_void*)(block + 1024 * j), 16, 0,
                                       kCopyPolicy);
  }

  __device__ __forceinline__ void process(const Sub& tile, const unsigned char* kblk, const unsigned char* vblk,
                                         float* stage, const float (&zk)[8]) {
    const int t0 = tile.t0;
    const int cls = tile.cls;
    const int t_end = min(t0 + 32, r1);
    // ---- scores of the 32 rows against the query group ----
    float z[8];
    if constexpr (ZSPILL) {
      // the visual pass computed these logits with the same products (the
      // same operands and instructions give the same bits)
#pragma unroll
      for (int i = 0; i < 8; ++i) z[i] = zk[i];
    } else {
      const f32x4 c0 = score_half<DT, D>(kblk, 0, qf, a4, n16);
      const f32x4 c1 = score_half<DT, D>(kblk, 1, qf, a4, n16);
#pragma unroll
      for (int i = 0; i < 8; ++i) z[i] = (i < 4 ? c0[i & 3] : c1[i & 3]) * a.zscale;
    }

    // value i of this lane is row t0 + 16*(i/4) + 4*a4 + i%4; bit i of the masks
    unsigned valid = 0xffu, vis = 0u;
    if constexpr (KEPT) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int p = __shfl(tile.kp, 16 * (i >> 2) + 4 * a4 + (i & 3));  // -1 past the list
        valid &= (p >= 0 && p < L) ? 0xffu : ~(1u << i);
      }
    } else {
      if (t_end - t0 < 32) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (t0 + 16 * (i >> 2) + 4 * a4 + (i & 3) >= t_end) valid &= ~(1u << i);
      }
      if (t_end > L0) {
        // several queries: the rows after a query's own position are hidden from it
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (t0 + 16 * (i >> 2) + 4 * a4 + (i & 3) >= lim) valid &= ~(1u << i);
      }
      if (cls == TILE_VIS) {
        vis = valid;
      } else if (cls == TILE_MIXED) {
        SegWalker lw = tile.w;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int p = t0 + 16 * (i >> 2) + 4 * a4 + (i & 3);
          if (p < t_end) {
            lw.seek(p);
            if (lw.contains(p)) vis |= 1u << i;
          }
        }
      }
    }

    if constexpr (VIS) {
      // ---- Eq. (5)/(6) and Eq. (2) statistics over visual rows ----
      float lmax = kNegInf;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (vis & (1u << i)) lmax = fmaxf(lmax, z[i]);
      const bool up = lmax > m_v + a.thr_s;  // per lane; rare after the first tile
      if (__builtin_amdgcn_ballot_w64(up)) {
        Ls_v *= up ? fast_exp2((m_v - lmax) * a.inv_tau_s) : 1.f;
        Lm_v *= up ? fast_exp2((m_v - lmax) * a.inv_tau_m) : 1.f;
        m_v = up ? lmax : m_v;
      }
      float ts = 0.f, tm = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float d = (vis & (1u << i)) ? z[i] - m_v : kNegInf;
        ts += fast_exp2(d * a.inv_tau_s);
        tm += fast_exp2(d * a.inv_tau_m);
      }
      Ls_v += ts;
      Lm_v += tm;
      // visual logits: spill rows of zs_gp floats (this KV group's heads) by position
      if (cls == TILE_VIS && t_end - t0 == 32) {
        // transpose through the stage (row = token, zs_gp heads): lane (a4, n16)
        // holds head n16 for tokens 16*(i/4) + 4*a4 + i%4; then the 32 rows go
        // out as one contiguous block of 32 * zs_gp floats, 16 bytes per lane
        const int gp = a.zs_gp;
        if (n16 < gp) {
#pragma unroll
          for (int i = 0; i < 8; ++i) stage[(16 * (i >> 2) + 4 * a4 + (i & 3)) * gp + n16] = z[i];
        }
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        const u32x4* src = reinterpret_cast<const u32x4*>(stage);
        const int soff = t0 * gp * 4;
        __builtin_amdgcn_raw_buffer_store_b128(src[lane], zrsrc, lane * 16, soff, spill_policy(MODE));
        if (gp > 8)
          __builtin_amdgcn_raw_buffer_store_b128(src[64 + lane], zrsrc, 1024 + lane * 16, soff, spill_policy(MODE));
      } else if (hv && vis) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (vis & (1u << i)) zbase[static_cast<size_t>(t0 + 16 * (i >> 2) + 4 * a4 + (i & 3)) * a.zs_gp + n16] = z[i];
      }
    } else {
      // ---- text rows (or kept rows): attention weights, statistics, value product ----
      const unsigned att = valid & ~vis;
      float lmax = kNegInf;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (att & (1u << i)) lmax = fmaxf(lmax, z[i]);
      if (__builtin_amdgcn_ballot_w64(lmax > m_t + a.thr_t)) {
        // the four lanes of a head share the reference (their weights meet in one MFMA)
        const float tm = max_over_quads(lmax);
        const bool up = tm > m_t + a.thr_t;
        const float d = m_t - tm;
        const float al = up ? fast_exp2(d) : 1.f;
        l_t *= al;
        if constexpr (TSTATS) {
          Lm_t *= up ? fast_exp2(d * a.inv_tau_m) : 1.f;
          Ls_t *= up ? fast_exp2(d * a.inv_tau_s) : 1.f;
        }
        if constexpr (ATTN) {
#pragma unroll
          for (int i = 0; i < C::ACC_N; ++i) acc[i] *= al;
        }
        m_t = up ? tm : m_t;
      }
      float p[8];
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        p[i] = (att & (1u << i)) ? fast_exp2(z[i] - m_t) : 0.f;
        ps += p[i];
      }
      l_t += ps;
      if constexpr (TSTATS) {
        float tm = 0.f, ts = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float d = (att & (1u << i)) ? z[i] - m_t : kNegInf;
          tm += fast_exp2(d * a.inv_tau_m);
          if (!a.tau_s_one) ts += fast_exp2(d * a.inv_tau_s);
        }
        Lm_t += tm;
        Ls_t += ts;
      }
      if constexpr (ATTN) {
        if (__builtin_amdgcn_ballot_w64(att != 0u)) value_product<DT, D, C::ACC_N>(acc, vblk, p, a4, n16);
      }
    }
  }
};

// LDS layout of one pass: per sub-tile a K block, a V block (passes that read
// V) and a logit stage (visual pass); the total also sets how many work-groups
// stay resident per CU
template <int DT, int D, int MODE>
struct PassLds {
  using C = Cfg<DT, D>;
  using P = Pass<DT, D, MODE>;
  static constexpr int NSUB = P::KEPT ? VP_KEPT_SUBS : VP_TILE_SUBS;
  static constexpr int VB = P::ATTN ? C::SUB_ROWS_BYTES : 0;
  static constexpr int SB = P::VIS ? C::STAGE_BYTES : 0;
  static constexpr int SUB = C::SUB_ROWS_BYTES + VB + SB;
  static constexpr int BYTES = max_i(NSUB * SUB, lds_floor(DT, MODE));
};

// The work of one work-group (part `part` of KV head g of sequence b; in the
// kept pass gy = g*T + t also names the query t whose kept list it reads).
template <int DT, int D, int MODE>
__device__ __forceinline__ void attend_body(const AttendArgs& a, unsigned char* lds, int part, int gy, int b) {
  using C = Cfg<DT, D>;
  using P = Pass<DT, D, MODE>;
  using Q = PassLds<DT, D, MODE>;
  constexpr int NSUB = Q::NSUB;
  constexpr int VB = Q::VB;
  constexpr int SUB = Q::SUB;

  P s(a);
  s.lane = threadIdx.x;
  s.n16 = s.lane & 15;
  s.a4 = s.lane >> 4;
  s.L = clamp_len(a.seq_len[b], a.max_seq_len);
  s.kept = nullptr;
  const int qk = P::KEPT ? gy % a.T : 0;  // kept pass: the query
  const int g = P::KEPT ? gy / a.T : gy;   // KV head
  // lane row n16 <-> virtual head vh of this KV head: query vh / G, head g*G + vh % G
  const int vh = P::KEPT ? qk * a.G + s.n16 : s.n16;
  s.hv = s.n16 < (P::KEPT ? a.G : a.T * a.G);
  const int tq = s.hv ? vh / a.G : 0;
  s.h = g * a.T * a.G + vh;
  int kp0 = -2;  // kept pass: the first tile's kept positions, requested with the budget
  if constexpr (P::KEPT) {
    // the selection row of query qk that KV head g belongs to
    const size_t row = (static_cast<size_t>(b) * a.T + qk) * a.U + g / (a.Hkv / a.U);
    s.kept = a.vis_idx + row * a.k_cap;
    s.r0 = part * a.split;
    const int t = s.r0 + s.lane;
    kp0 = (s.lane < 32 && t < a.k_cap) ? s.kept[t] : -1;  // entries past the budget are masked below
    int kb = a.kk[row];
    kb = kb < 0 ? 0 : (kb > a.k_cap ? a.k_cap : kb);
    s.r1 = s.L == 0 ? s.r0 : min(s.r0 + a.split, kb);
    s.step = 32;
  } else {
    s.r0 = 32 * part;
    s.r1 = s.L;
    s.step = 32 * a.nparts;
  }
  // the query rows load while the length and the budget arrive
  const size_t qrow = s.hv ? (static_cast<size_t>(b) * a.T + tq) * a.Hq + g * a.G + (vh - tq * a.G) : 0;
  load_q<DT, D>(s.qf, static_cast<const char*>(a.q) + qrow * C::ROWB, s.hv, s.a4);
  if (s.r0 >= s.r1) {
    // no rows: an empty partial (max -inf, sum 0), so that the merge can read
    // every part's slot without first learning the length and the budget
    if constexpr (P::ATTN) {
      if (s.hv && s.a4 == 0) {
        if constexpr (P::KEPT) {
          const size_t row = (static_cast<size_t>(b) * a.T * a.Hq + s.h) * a.nsplit + part;
          *reinterpret_cast<float2*>(a.kstats + row * 2) = make_float2(kNegInf, 0.f);
        } else {
          const size_t row = (static_cast<size_t>(b) * a.T * a.Hq + s.h) * a.nparts + part;
          if constexpr (P::TSTATS)
            *reinterpret_cast<float4*>(a.stats + row * 8 + 4) = make_float4(kNegInf, 0.f, 0.f, 0.f);
          else
            *reinterpret_cast<float2*>(a.stats + row * 8 + 4) = make_float2(kNegInf, 0.f);
        }
      }
    }
    return;
  }

  s.L0 = s.L - a.T + 1;
  s.lim = s.L0 + tq;
  // contiguous caches: sequence b's rows from its base; paged caches: rows of
  // physical blocks (the block offset is added per row)
  constexpr bool paged = P::PAGED;
  const size_t seq_off = paged ? 0 : static_cast<size_t>(b) * a.sb;
  s.Kb = static_cast<const char*>(a.K) + (seq_off + static_cast<size_t>(g) * a.sh) * C::ESZ;
  s.Vb = P::ATTN ? static_cast<const char*>(a.V) + (seq_off + static_cast<size_t>(g) * a.sh) * C::ESZ : nullptr;
  s.rstride = static_cast<size_t>(a.ss) * C::ESZ;
  s.bt = paged ? a.block_table + static_cast<size_t>(b) * a.nblk : nullptr;
  s.bstride = static_cast<size_t>(a.sb) * C::ESZ;
  s.bmask = paged ? (1 << a.bs_log2) - 1 : 0;
  s.m_v = kNegInf;
  s.Ls_v = s.Lm_v = 0.f;
  s.m_t = kNegInf;
  s.l_t = s.Lm_t = s.Ls_t = 0.f;
#pragma unroll
  for (int i = 0; i < C::ACC_N; ++i) s.acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (P::VIS) {
    // the plane (zs_rows * zs_gp floats) as a raw buffer: offsets past it are dropped
    const size_t plane = static_cast<size_t>(a.zs_rows) * a.zs_gp * 4;
    s.zrsrc = __builtin_amdgcn_make_buffer_rsrc(
        a.zs + (static_cast<size_t>(b) * a.Hkv + g) * a.zs_rows * static_cast<size_t>(a.zs_gp), 0,
        static_cast<int>(plane < 0x7fffffffu ? plane : 0x7fffffffu), kRawBufferWord3);
  }
  s.zbase = (P::VIS || P::ZSPILL)
                ? a.zs + (static_cast<size_t>(b) * a.Hkv + g) * a.zs_rows * static_cast<size_t>(a.zs_gp) + qk * a.G
                : nullptr;

  Sub cur;
  cur.t0 = s.r0;
  cur.cls = TILE_TEXT;
  if constexpr (!P::KEPT) {
    const int o0 = a.seg_off[b];
    cur.w.start(a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, vis_len(s.L, a.T));
  }
  cur = s.sub_at(cur, s.r0, kp0);

  // tiles of NSUB sub-tiles: all copies of a tile are issued before any of it is used
  while (cur.t0 < s.r1) {
    Sub sub[NSUB];
    bool act[NSUB];
    sub[0] = cur;
#pragma unroll
    for (int i = 1; i < NSUB; ++i) sub[i] = s.sub_at(sub[i - 1], sub[i - 1].t0 + s.step);
#pragma unroll
    for (int i = 0; i < NSUB; ++i) act[i] = s.active(sub[i]);
    // The work-group is a single wave, so ordering needs counters, not barriers
    // (a barrier's release fence would also wait for the logit stores of the
    // previous tile). LDS reads of the previous tile must have returned before
    // the copies overwrite it:
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    float zk[NSUB][8];
#pragma unroll
    for (int i = 0; i < NSUB; ++i) {
      if (act[i]) {
        unsigned char* blk = lds + i * SUB;
        size_t off[C::COPIES];
        s.row_offsets(sub[i], off);
        if constexpr (!P::ZSPILL) s.copy_rows(s.Kb, off, blk);
        if (s.needs_v(sub[i])) s.copy_rows(s.Vb, off, blk + C::SUB_ROWS_BYTES);
        if constexpr (P::ZSPILL) s.load_spill(sub[i], zk[i]);
      }
    }
    // the next tile's kept positions / segment state load while these copies fly
    cur = s.sub_at(sub[NSUB - 1], sub[NSUB - 1].t0 + s.step);
    // the copies have landed in LDS once the vector-memory counter drains
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
#pragma unroll
    for (int i = 0; i < NSUB; ++i)
      if (act[i])
        s.process(sub[i], lds + i * SUB, lds + i * SUB + C::SUB_ROWS_BYTES,
                  reinterpret_cast<float*>(lds + i * SUB + C::SUB_ROWS_BYTES + VB), zk[i]);
  }

  // ---- write this part's partials ----
  if constexpr (P::VIS) {
    // merge the four lanes' statistics onto their common maximum
    const float M = max_over_quads(s.m_v);
    const bool any = s.m_v != kNegInf;
    const float fs = any ? fast_exp2((s.m_v - M) * a.inv_tau_s) : 0.f;
    const float fm = any ? fast_exp2((s.m_v - M) * a.inv_tau_m) : 0.f;
    const float s_ls = sum_over_quads(s.Ls_v * fs);
    const float s_lm = sum_over_quads(s.Lm_v * fm);
    if (s.hv && s.a4 == 0) {
      float* st = a.stats + ((static_cast<size_t>(b) * a.T * a.Hq + s.h) * a.nparts + part) * 8;
      *reinterpret_cast<float4*>(st) = make_float4(M, s_ls, s_lm, 0.f);
    }
  } else {
    const float s_lt = sum_over_quads(s.l_t);
    const float s_lm = P::TSTATS ? sum_over_quads(s.Lm_t) : 0.f;
    const float s_ls = P::TSTATS ? (a.tau_s_one ? s_lt : sum_over_quads(s.Ls_t)) : 0.f;
    if (s.hv) {
      if constexpr (P::KEPT) {
        const size_t row = (static_cast<size_t>(b) * a.T * a.Hq + s.h) * a.nsplit + part;
        if (s.a4 == 0) *reinterpret_cast<float2*>(a.kstats + row * 2) = make_float2(s.m_t, s_lt);
        store_acc<DT, D, C::ACC_N>(a.kacc + row * D, s.acc, s.a4);
      } else {
        const size_t row = (static_cast<size_t>(b) * a.T * a.Hq + s.h) * a.nparts + part;
        if (s.a4 == 0) {
          if constexpr (P::TSTATS)
            *reinterpret_cast<float4*>(a.stats + row * 8 + 4) = make_float4(s.m_t, s_lt, s_lm, s_ls);
          else
            *reinterpret_cast<float2*>(a.stats + row * 8 + 4) = make_float2(s.m_t, s_lt);
        }
        if constexpr (P::ATTN) store_acc<DT, D, C::ACC_N>(a.acc + row * D, s.acc, s.a4);
      }
    }
  }
}

// The extra work-group of a launch with the visual role (x = its last index,
// KV head 0): a new step's arrival counters of the sequence's T*U selection
// rows at zero, and the sequence's clipped segment table (positions and visual
// ranks) for the select kernel.
__device__ __forceinline__ void step_setup(const AttendArgs& a, int g, int b) {
  if (g != 0) return;
  const int lane = threadIdx.x;
  if (a.sync)
    for (int i = lane; i < a.T * a.U; i += 64) a.sync[static_cast<size_t>(b) * a.T * a.U + i] = 0u;
  if (a.segtab) {
    const int L = vis_len(clamp_len(a.seq_len[b], a.max_seq_len), a.T);
    const int o0 = a.seg_off[b];
    load_segments(static_cast<SegTable*>(a.segtab)[b], a.seg + 2 * static_cast<long>(o0), a.seg_off[b + 1] - o0, L,
                  lane);
  }
}

template <int DT, int D, int MODE>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(attend_waves(DT, MODE)))) void attend_kernel(
    const AttendArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[PassLds<DT, D, MODE>::BYTES];
  if (base_mode(MODE) == MODE_VIS && static_cast<int>(blockIdx.x) == a.nparts) {
    step_setup(a, blockIdx.y, blockIdx.z);
    return;
  }
  attend_body<DT, D, MODE>(a, lds, blockIdx.x, blockIdx.y, blockIdx.z);
}

// Both context passes in one launch (grid.x = 2 parts + 1): work-group 2p takes
// the text role of part p, 2p + 1 its visual role, the last one the step setup.
// Used up to mid-size caches, where launch latency and load balance, not the
// visual spill's interference with the text stream, bound the step.
template <int DT, int D, int PG>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(attend_waves(DT, MODE_TEXT_BOTH)))) void
attend_dual_kernel(const AttendArgs a) {
  constexpr int VIS = MODE_VIS | MODE_ONE_LAUNCH | PG;
  constexpr int TEXT = MODE_TEXT_BOTH | MODE_ONE_LAUNCH | PG;
  constexpr int BYTES = max_i(PassLds<DT, D, VIS>::BYTES, PassLds<DT, D, TEXT>::BYTES);
  __shared__ __attribute__((aligned(1024))) unsigned char lds[BYTES];
  const int x = blockIdx.x;
  // the roles alternate, so every CU gets a mix of visual (K, spill) and text
  // (K and V) work-groups (measured 86.5 -> 84.8 us at the 16-sequence ragged batch)
  if (x < 2 * a.nparts) {
    if (x & 1) attend_body<DT, D, VIS>(a, lds, x >> 1, blockIdx.y, blockIdx.z);
    else attend_body<DT, D, TEXT>(a, lds, x >> 1, blockIdx.y, blockIdx.z);
  } else {
    step_setup(a, blockIdx.y, blockIdx.z);
  }
}

// A later layer's text attention pass and kept pass in one launch (their rows
// are disjoint and the kept list is the anchor layer's, known before the
// launch): grid.x = P text parts + T*splits kept work-groups per (KV head,
// sequence); each work-group does what it does in its own launch, so the
// partials are the same bits, and the kept work-groups fill the text pass's tail.
template <int DT, int D, int PG>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(attend_waves(DT, MODE_TEXT_ATTN)))) void
attend_text_kept_kernel(const AttendArgs a) {
  constexpr int TEXT = MODE_TEXT_ATTN | PG;
  constexpr int KEPT = MODE_KEPT | PG;
  constexpr int BYTES = max_i(PassLds<DT, D, TEXT>::BYTES, PassLds<DT, D, KEPT>::BYTES);
  __shared__ __attribute__((aligned(1024))) unsigned char lds[BYTES];
  const int x = blockIdx.x;
  if (x < a.nparts) {
    attend_body<DT, D, TEXT>(a, lds, x, blockIdx.y, blockIdx.z);
  } else {
    const int j = x - a.nparts;
    const int t = j / a.nsplit;
    attend_body<DT, D, KEPT>(a, lds, j - t * a.nsplit, blockIdx.y * a.T + t, blockIdx.z);
  }
}

// Launches one pass. With events given, they are attached to the launch itself
// (hipExtLaunchKernel): they time the kernel's execution alone, as a profiler does.
template <typename K>
hipError_t launch_one(K kernel, dim3 grid, const AttendArgs& a, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  if (ev0 || ev1) {
    void* args[1] = {const_cast<AttendArgs*>(&a)};
    return hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, dim3(64), args, 0, st, ev0, ev1, 0);
  }
  hipLaunchKernelGGL(kernel, grid, dim3(64), 0, st, a);
  return hipGetLastError();
}

template <int DT, int D, int PG>
hipError_t launch_dd(const AttendArgs& a, int mode, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  // launches with the visual role carry one more work-group per sequence (step_setup)
  const bool kept = (mode & ~MODE_ZSPILL) == MODE_KEPT;
  int gx = a.nparts;
  if (kept) gx = a.nsplit;
  else if (mode == MODE_DUAL) gx = 2 * a.nparts + 1;
  else if (mode == MODE_VIS) gx = a.nparts + 1;
  else if (mode == MODE_TEXT_KEPT) gx = a.nparts + a.T * a.nsplit;  // text parts, then kept splits
  const dim3 grid(gx, kept ? a.Hkv * a.T : a.Hkv, a.B);
  switch (mode) {
    case MODE_TEXT_KEPT: return launch_one(attend_text_kept_kernel<DT, D, PG>, grid, a, st, ev0, ev1);
    case MODE_DUAL: return launch_one(attend_dual_kernel<DT, D, PG>, grid, a, st, ev0, ev1);
    case MODE_VIS: return launch_one(attend_kernel<DT, D, MODE_VIS | PG>, grid, a, st, ev0, ev1);
    case MODE_TEXT_STATS: return launch_one(attend_kernel<DT, D, MODE_TEXT_STATS | PG>, grid, a, st, ev0, ev1);
    case MODE_TEXT_ATTN: return launch_one(attend_kernel<DT, D, MODE_TEXT_ATTN | PG>, grid, a, st, ev0, ev1);
    case MODE_TEXT_BOTH: return launch_one(attend_kernel<DT, D, MODE_TEXT_BOTH | PG>, grid, a, st, ev0, ev1);
    case MODE_KEPT: return launch_one(attend_kernel<DT, D, MODE_KEPT | PG>, grid, a, st, ev0, ev1);
    case MODE_KEPT | MODE_ZSPILL:
      return launch_one(attend_kernel<DT, D, MODE_KEPT | MODE_ZSPILL | PG>, grid, a, st, ev0, ev1);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attend(const AttendArgs& a, int mode, int dtype, int head_dim, hipStream_t st, hipEvent_t ev0,
                         hipEvent_t ev1) {
  const bool paged = a.bs_log2 >= 0;
  if (dtype == VP_BF16) {
    if (head_dim == 128)
      return paged ? launch_dd<VP_BF16, 128, MODE_PAGED>(a, mode, st, ev0, ev1) : launch_dd<VP_BF16, 128, 0>(a, mode, st, ev0, ev1);
    if (head_dim == 64)
      return paged ? launch_dd<VP_BF16, 64, MODE_PAGED>(a, mode, st, ev0, ev1) : launch_dd<VP_BF16, 64, 0>(a, mode, st, ev0, ev1);
  } else if (dtype == VP_F32) {
    if (head_dim == 128)
      return paged ? launch_dd<VP_F32, 128, MODE_PAGED>(a, mode, st, ev0, ev1) : launch_dd<VP_F32, 128, 0>(a, mode, st, ev0, ev1);
    if (head_dim == 64)
      return paged ? launch_dd<VP_F32, 64, MODE_PAGED>(a, mode, st, ev0, ev1) : launch_dd<VP_F32, 64, 0>(a, mode, st, ev0, ev1);
  }
  return hipErrorInvalidValue;
}

}  // namespace vp
