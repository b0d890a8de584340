// Work decomposition of a step: how many work-groups each launch runs and how
// the workspace is carved, a pure function of the shape (vp_shape). Kept apart
// from the ABI's validation code: these choices, with the kernels, set what
// the passes read and write.
#include "vp_internal.h"

namespace vp {
namespace {
size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }
}  // namespace

// queries per sequence, and selection rows per query: one, or one per KV group
int queries(const vp_shape& s) { return s.n_queries > 1 ? s.n_queries : 1; }
int rows_per_query(const vp_shape& s) { return s.scope == VP_SCOPE_KV_GROUP ? s.n_kv_heads : 1; }
int rows_per_seq(const vp_shape& s) { return queries(s) * rows_per_query(s); }

// Context-pass work-groups of the one launch of both passes: 2048 (1024 parts
// per role) is one resident round (8 work-groups per CU x 256 CUs), so no
// work-group waits for a second round; measured best against 768 to 1280
// parts per role at the ragged 16-sequence batch and the 72B-class loop.
#ifndef VP_TARGET_PARTS
#define VP_TARGET_PARTS 2048
#endif
// The visual and text passes in two launches (large caches) take three
// quarters of that: 6 parts per KV head at the 64 x 32k batch, where 4, 5, 6,
// 7 and 8 parts measured 660, 631, 613.6, 618.5 and 616.5 us per step (the
// visual pass 265 / 238 / 222 / 226 / 225 us; the text pass 328.5 us at 4 parts
// and within 1 us of 325 us at 5 to 8).
#ifndef VP_TWO_LAUNCH_PARTS
#define VP_TWO_LAUNCH_PARTS 1536
#endif
#ifndef VP_MIN_TILES
#define VP_MIN_TILES 2  // 32-row tiles per context-pass part, at least
#endif

// Both context passes in one launch: saves a launch and overlaps the two
// passes' latency chains where the cache is small; kept apart otherwise, so
// the visual pass's logit writes stay out of the text pass's read stream.
// Measured: the 8 x 10.5k batch of the 72B shape (22k tiles) gains 6 us from the
// one launch with half the parts; the 64 x 32k batch (262k tiles) loses 100 us.
#ifndef VP_DUAL_MAX_TILES
#define VP_DUAL_MAX_TILES 32768  // 32-row tiles over the batch and KV heads
#endif
#ifndef VP_DUAL_PART_DIV
#define VP_DUAL_PART_DIV 2  // parts of the one-launch context pass: VP_TARGET_PARTS / this
#endif
bool use_dual(const vp_shape* s) {
  const int64_t tiles = static_cast<int64_t>(s->batch) * s->n_kv_heads * ((s->max_seq_len + 31) / 32);
  return tiles <= static_cast<int64_t>(VP_DUAL_MAX_TILES);
}

#ifndef VP_KEPT_WGS
#define VP_KEPT_WGS 2048  // kept-pass work-groups in one resident round (8 per CU)
#endif

#ifndef VP_MERGE_KEPT_WGS
#define VP_MERGE_KEPT_WGS 64  // kept-pass work-groups at most for the kept rows to be merged directly
#endif

#ifndef VP_SELECT_WGS
#define VP_SELECT_WGS 256  // target work-groups of the select launch: one per CU
#endif

Plan make_plan(const vp_shape& s) {
  Plan p{};
  // Context pass: about VP_TARGET_PARTS one-wave work-groups in all, each
  // with at least two 32-row tiles. Tiles are dealt out cyclically, so every
  // part sees the sequence's own mix of visual and text rows: consecutive
  // work-groups land on different XCDs, and contiguous chunks would hand whole
  // XCDs only visual (K) or only text (K + V) rows.
  const int64_t pairs = static_cast<int64_t>(s.batch) * s.n_kv_heads;
  const int64_t tiles = (s.max_seq_len + 31) / 32;
  // the one-launch context pass runs a visual and a text work-group per part
  const int64_t target = use_dual(&s) ? VP_TARGET_PARTS / VP_DUAL_PART_DIV : VP_TWO_LAUNCH_PARTS;
  int64_t parts = (target + pairs - 1) / pairs;
  if (parts > (tiles + VP_MIN_TILES - 1) / VP_MIN_TILES) parts = (tiles + VP_MIN_TILES - 1) / VP_MIN_TILES;
  if (parts < 1) parts = 1;
  p.nparts = static_cast<int>(parts);
  // Kept pass: the fewest kept rows per work-group (32, 64, 128, ...) that
  // keep the launch within one resident round (VP_KEPT_WGS work-groups), so no
  // work-group waits for a second round (the 64 x 32k batch: 128 rows, 1792
  // work-groups; kept pass and merge 40.2 -> 35.9 us against 64 rows).
#ifdef VP_KEPT_SPLIT
  p.split = VP_KEPT_SPLIT;
#else
  {
    const int64_t heads = static_cast<int64_t>(s.batch) * s.n_kv_heads * queries(s);
    int64_t split = 32;
    while (split < s.k_cap && heads * ((s.k_cap + split - 1) / split) > VP_KEPT_WGS) split *= 2;
    p.split = static_cast<int>(split);
  }
#endif
  p.nsplit = (s.k_cap + p.split - 1) / p.split;
  // A later layer (its own text rows, the anchor's kept list) launches its text
  // and kept passes together when both fit one resident round: the kept
  // work-groups then fill the text pass's tail (8 layers: 131.8 -> 98.6 us at the
  // 1-sequence batch, 381.9 -> 351.9 at the 72B-class loop); beyond one round
  // the text pass is split over two (the 64 x 32k batch: 3081 -> 3663 us).
  p.text_kept_one_launch = static_cast<int64_t>(p.nparts + queries(s) * p.nsplit) * s.n_kv_heads * s.batch <=
                           static_cast<int64_t>(VP_KEPT_WGS);
  // A step whose kept pass would be a handful of work-groups folds the kept
  // rows into the merge (their K and V rows read there): bf16 caches, every
  // text part and kept row in one batch per head.
  p.merge_kept = s.dtype == VP_BF16 &&
                 static_cast<int64_t>(p.nsplit) * queries(s) * s.n_kv_heads * s.batch <= VP_MERGE_KEPT_WGS &&
                 p.nparts <= merge_kept_max_parts(s.head_dim) && s.k_cap <= merge_kept_max_rows(s.head_dim);
  // per-head arrays hold one entry per query row (virtual head): T*Hq per sequence
  const size_t B = s.batch, Hq = static_cast<size_t>(s.n_q_heads) * queries(s), d = s.head_dim;
  p.zs_rows = ((s.max_seq_len + 31) / 32) * 32;
  p.zs_gp = queries(s) * (s.n_q_heads / s.n_kv_heads) <= 8 ? 8 : 16;
  size_t off = 0;
  p.zs = off;
  off = align256(off + B * static_cast<size_t>(s.n_kv_heads) * p.zs_rows * static_cast<size_t>(p.zs_gp) * 4);
  p.stats = off;
  off = align256(off + B * Hq * p.nparts * 8 * 4);
  p.acc = off;
  off = align256(off + B * Hq * p.nparts * d * 4);
  p.head = off;
  off = align256(off + B * Hq * 2 * 4);
  p.kstats = off;
  off = align256(off + B * Hq * p.nsplit * 2 * 4);
  p.kacc = off;
  off = align256(off + B * Hq * p.nsplit * d * 4);
  const size_t rows = B * static_cast<size_t>(rows_per_seq(s));
  p.sync = off;
  off = align256(off + rows * 4);
  p.segtab = off;
  off = align256(off + B * kSegTableBytes);
  p.total = off;
  // Select kernel: chunks of whole rounds (a round scores 1024 / lanes-per-token
  // visual ranks), enough rounds per chunk that the launch has about
  // VP_SELECT_WGS work-groups, so the spilled logits stream through many CUs.
  const int64_t tpr = select_tokens_per_round(s.n_kv_heads, rows_per_query(s));
  const int64_t want = static_cast<int64_t>(rows) * s.max_vis;
  int64_t rounds = (want + tpr * VP_SELECT_WGS - 1) / (tpr * VP_SELECT_WGS);
  if (rounds < 1) rounds = 1;
  const int64_t chunk = tpr * rounds;
  p.sel_chunks = static_cast<int>((s.max_vis + chunk - 1) / chunk);
  p.sel_chunk = p.sel_chunks == 1 ? s.max_vis : static_cast<int>(chunk);
  return p;
}

}  // namespace vp
