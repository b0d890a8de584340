// Host/device interface between the C ABI (vp_api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "visionpulse.h"

namespace vp {

constexpr int kMaxHq_ = 1024;  // query heads supported
// bytes of one sequence's segment table (SegTable: 256 starts, 256 ends, 257 ranks, count; 16-byte aligned)
constexpr size_t kSegTableBytes = 3088;

// Several queries per sequence (T >= 1): the T*G query rows that read one KV
// head are "virtual heads" of that KV head, in the order (query t, head j of
// the group), so one pass over a KV head's rows serves all of them. Per-head
// workspace arrays are indexed by virtual head: b*T*Hq + g*T*G + t*G + j.
__host__ __device__ inline int vhead(int h, int t, int G, int T) { return (h / G) * (T * G) + t * G + h % G; }
// positions visible as visual to the queries of a sequence of length L: the
// last T - 1 positions are the other queries' tokens (text)
__host__ __device__ inline int vis_len(int L, int T) { return L - T + 1 > 0 ? L - T + 1 : 0; }

// Work decomposition and workspace carving, a pure function of the shape.
struct Plan {
  int nparts;   // context-pass work-groups per (sequence, KV head); part p takes
                // the 32-row tiles p, p + nparts, p + 2 nparts, ...
  int split;    // kept rows per kept-pass work-group (multiple of 32)
  int nsplit;   // ceil(k_cap / split)
  bool text_kept_one_launch;  // a later layer's text and kept passes fit one resident round together
  bool merge_kept;            // the step folds the kept rows into the merge (no kept pass)
  int zs_rows;    // rows per spill plane: max_seq_len rounded up to 32
  int zs_gp;      // floats per spill row: the query group padded to 8 or 16
  size_t zs;      // float [B][Hkv][zs_rows][zs_gp]  visual logits (log2 domain) by cache position
  size_t stats;   // float [B][T*Hq][nparts][8] per-part statistics (by virtual head): visual rows
                  //   {m_v, Ls_v, Lm_v, -}, text rows {m_t, l_t, Lm_t, Ls_t}
  size_t acc;     // float [B][T*Hq][nparts][d] per-part text value partials
  size_t head;    // float [B][T*Hq][2]         merged (max, score normaliser)
  size_t kstats;  // float [B][T*Hq][nsplit][2] kept-row (max, sum)
  size_t kacc;    // float [B][T*Hq][nsplit][d] kept-row value partials
  size_t sync;    // uint32 [B][T][U]           select-kernel arrival counters (per selection row)
  size_t segtab;  // SegTable [B]               clipped segment tables (positions, ranks)
  int sel_chunk;  // visual ranks scored per select work-group
  int sel_chunks; // select work-groups per selection row
  size_t total;
};

Plan make_plan(const vp_shape& s);
// both context passes in one launch (VP_PLAN_ONE_CONTEXT_LAUNCH)
bool use_dual(const vp_shape* s);
// queries per sequence, and selection rows per query: one, or one per KV group
int queries(const vp_shape& s);
int rows_per_query(const vp_shape& s);
int rows_per_seq(const vp_shape& s);

// Passes over the cache. The visual pass is the only one that writes a large
// output (the logit spill); keeping it apart from the text pass keeps writes out
// of the text pass's read stream.
enum Mode : int {
  MODE_VIS = 1,         // visual rows: Eq. (5)/(6) statistics + logit spill
  MODE_TEXT_STATS = 2,  // text rows: Eq. (6)/(2) normaliser statistics
  MODE_TEXT_ATTN = 4,   // text rows: attention partial (reads V)
  MODE_TEXT_BOTH = 6,
  MODE_KEPT = 8,        // kept visual rows: attention partial
  MODE_DUAL = 16,       // visual pass and text pass (statistics + attention) in one launch
  MODE_PAGED = 32,      // flag: K and V rows addressed through a block table (paged caches)
  MODE_ZSPILL = 64,     // flag (kept pass): the kept rows' logits come from the visual pass's
                        // spill of the same step instead of their K rows (V rows only are read)
  MODE_ONE_LAUNCH = 128, // flag: a role of the one-launch context pass (attend_dual_kernel)
  MODE_TEXT_KEPT = 256   // launch of a later layer: the text attention pass and the kept pass together
};
constexpr int base_mode(int mode) { return mode & ~(MODE_PAGED | MODE_ZSPILL | MODE_ONE_LAUNCH); }

struct AttendArgs {
  const void* q;
  const void* K;
  const void* V;
  int64_t sb, sh, ss;   // KV strides (elements); paged caches: sb is the block stride
  const int32_t* block_table;  // paged caches: [B][nblk] physical blocks (else null)
  int bs_log2;          // paged caches: log2 of the rows per block; -1: contiguous
  int nblk;             // row stride of block_table
  const int32_t* seq_len;
  const int32_t* seg_off;
  const int32_t* seg;
  int B, Hq, Hkv, G, max_seq_len, max_vis;
  int T;                // queries per sequence (q, out: [B][T][Hq][d])
  int U;                // selection rows per query: 1, or Hkv (one per KV group)
  float zscale;         // sm_scale * log2(e)
  float inv_tau_m;      // 1 / tau_mass
  float inv_tau_s;      // 1 / tau_score
  float thr_s;          // raise a running maximum of the statistics only past this margin (log2 units)
  float thr_t;          // same for the attention partial
  int tau_s_one;        // tau_score == 1: the attention weight doubles as the score weight
  int nparts;
  int zs_rows, zs_gp;
  float* zs;
  float* stats;
  float* acc;
  const int32_t* vis_idx;
  const int32_t* kk;
  int k_cap, split, nsplit;
  float* kstats;
  float* kacc;
  uint32_t* sync;       // [B][T][U] arrival counters of the select kernel (may be null)
  void* segtab;         // [B] segment tables (SegTable) for the select kernel (may be null)
};

// context-pass parts that hold at least one tile of a sequence of length L
__host__ __device__ inline int parts_used(int L, int nparts) {
  const int tiles = (L + 31) / 32;
  return tiles < nparts ? tiles : nparts;
}

// ev0 / ev1 (optional): events attached to the launch, timing the kernel alone
hipError_t launch_attend(const AttendArgs& a, int mode, int dtype, int head_dim, hipStream_t st,
                         hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

struct MassArgs {
  const int32_t* seq_len;
  const int32_t* seg_off;
  const int32_t* seg;
  int B, Hq, Hkv, G, max_seq_len, max_vis, nparts, zs_rows, zs_gp;
  int T;  // queries per sequence
  int U;  // selection rows per query (1 or Hkv); row (b*T + t)*U + u covers query t's
          // heads [u Hq/U, (u+1) Hq/U) and KV groups [u Hkv/U, (u+1) Hkv/U)
  float inv_tau_m, inv_tau_s;
  const float* stats;
  const float* zs;
  float* head;
  float* mass_head;
  float* mass_seq;
  float* scores;
};

hipError_t launch_mass_finalize(const MassArgs& a, hipStream_t st);
hipError_t launch_scores(const MassArgs& a, hipStream_t st);

// Everything between the context pass and the kept-row pass of a decode step
// (mass reduction, scores, budget, top-k) in one launch: grid (nchunks, B*T*U).
constexpr int kMaxSelectHeads = 1024;
struct SelectArgs {
  MassArgs m;
  int r_lo_bp, r_hi_bp, clamp;
  int k_cap;
  int32_t* k;
  int32_t* vis_idx;
  int chunk;       // visual ranks scored per work-group
  int nchunks;     // work-groups per selection row
  uint32_t* sync;  // [B*T*U] arrival counters (nchunks > 1), zeroed by the context pass
  const void* segtab;  // [B] segment tables written by the context pass
};

// visual ranks one select work-group scores per round (1024 lanes over the
// lanes per token of the score order)
int select_tokens_per_round(int n_kv_heads, int rows_per_seq);
hipError_t launch_select(const SelectArgs& t, hipStream_t st);

struct BudgetArgs {
  const int32_t* seq_len;
  const int32_t* seg_off;
  const int32_t* seg;
  int B, R, T, max_seq_len;  // R: selection rows per sequence (T*U); row b*R + r
  int r_lo_bp, r_hi_bp, clamp;
  const float* mass_seq;
  int32_t* k;
};

hipError_t launch_budget(const BudgetArgs& a, hipStream_t st);

struct TopkArgs {
  const int32_t* seq_len;
  const int32_t* seg_off;
  const int32_t* seg;
  int B, R, T, max_seq_len, max_vis, k_cap;  // R: selection rows per sequence
  const float* scores;
  const int32_t* k;
  int32_t* vis_idx;
  // optional: when mass_seq is set, k[b] is not read but computed by Eq. (7)
  // from mass_seq (the budget of vp_budget) and written to k_out
  const float* mass_seq;
  int32_t* k_out;
  int r_lo_bp, r_hi_bp, clamp;
};

hipError_t launch_topk(const TopkArgs& a, hipStream_t st);

struct TopPArgs {
  const int32_t* seq_len;
  const int32_t* seg_off;
  const int32_t* seg;
  int B, R, T, max_seq_len, max_vis;  // R: selection rows per sequence
  float p;
  const float* scores;
  int32_t* k;
};

hipError_t launch_top_p(const TopPArgs& a, hipStream_t st);

struct MergeArgs {
  int B, Hq, G, T, nparts, nsplit, dtype;
  const float* stats;
  const float* acc;
  const float* kstats;
  const float* kacc;
  void* out;
  // merge of the kept rows themselves (launch_merge_kept): their positions,
  // the query rows and the kept K and V rows
  const int32_t* seq_len;
  const int32_t* vis_idx;  // [B*T*U][k_cap]
  const int32_t* kk;       // [B*T*U] budgets
  int max_seq_len, Hkv, U, k_cap;
  const void* q;
  const void* K;
  const void* V;
  int64_t sb, sh, ss;  // K/V strides (elements); paged caches: sb is the block stride
  const int32_t* block_table;  // paged caches: [B][nblk] physical blocks (else null)
  int bs_log2, nblk;           // paged caches: log2 of the rows per block, table row stride
  float zscale;        // sm_scale * log2(e)
};

hipError_t launch_merge(const MergeArgs& a, int head_dim, hipStream_t st);
// The kept rows' attention folded into the merge, for small steps (plan.merge_kept):
// bf16 caches.
hipError_t launch_merge_kept(const MergeArgs& a, int head_dim, hipStream_t st);
// capacities of launch_merge_kept's single batch: text parts and kept rows per head
int merge_kept_max_parts(int head_dim);
int merge_kept_max_rows(int head_dim);

// one read of `bytes` (a multiple of 16 KiB) at src: mode 0 vector loads, 1 LDS copies
hipError_t launch_stream_read(const void* src, size_t bytes, int mode, uint32_t* sink, hipStream_t st);

// kept-row budget helpers shared by host validation and the budget kernel
__host__ __device__ inline int ceil_bp(long n, int bp) { return static_cast<int>((static_cast<long>(bp) * n + 9999) / 10000); }
__host__ __device__ inline int floor_bp(long n, int bp) { return static_cast<int>((static_cast<long>(bp) * n) / 10000); }

// Eq. (7) with the Sec. 5.2 clamp; m is the head-max visual mass
__host__ __device__ inline int budget_rule(double m, int n_vis, int r_lo_bp, int r_hi_bp, int clamp) {
  if (n_vis <= 0) return 0;
  if (!(m >= 0.0)) m = 0.0;  // NaN or negative mass -> no visual mass
  const double x = m * static_cast<double>(n_vis);
  long k = x >= static_cast<double>(n_vis) ? n_vis : static_cast<long>(ceil(x));
  if (clamp) {
    const int lo = ceil_bp(n_vis, r_lo_bp);
    int hi = floor_bp(n_vis, r_hi_bp);
    if (hi < lo) hi = lo;
    if (k < lo) k = lo;
    if (k > hi) k = hi;
  }
  if (k > n_vis) k = n_vis;
  if (k < 0) k = 0;
  return static_cast<int>(k);
}

}  // namespace vp
