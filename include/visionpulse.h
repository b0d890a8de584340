/*
 * visionpulse.h -- C ABI of the VisionPulse per-decode-step path on AMD
 * Instinct MI355X (gfx950).
 *
 * VisionPulse (arXiv 2605.31457) prunes visual tokens at every decoding step:
 * at the anchor layer the current query is scored against the whole KV cache,
 * the tempered attention mass that falls on visual tokens sets a budget k, the
 * k visual tokens with the largest head-averaged attention are kept, and the
 * step's attention runs over the kept visual tokens plus every text token.
 * One step is four calls, in this order, on one stream:
 *
 *   vp_visual_mass         Eq. (5)/(6) mass and Eq. (2) scores     (Sec. 4.2, 4.3)
 *   vp_budget              Eq. (7) budget with the Sec. 5.2 clamp  (Sec. 4.3, 5.2)
 *   vp_select_topk         Eq. (3) Top-K_t selection               (Sec. 4.2)
 *   vp_sparse_decode_attn  attention over kept visual + text KV    (Sec. 4.1, 4.2)
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory.   All tensor arguments are DEVICE pointers owned by the caller; the
 *           library allocates nothing. Scratch memory is the caller's
 *           workspace, sized by vp_workspace_size() (vp_decode_step_static
 *           alone uses the library's own scratch instead, see there).
 * State.    No device state is carried from one call to the next: every call
 *           leaves its results in the caller's buffers. The host side keeps
 *           three things: the detail of the last error, per calling thread
 *           (vp_last_error); per-kernel LDS figures read from the HIP runtime on
 *           first use and cached for the process (one GPU model per process is
 *           assumed); and, per device, the address of vp_decode_step_static's
 *           scratch array. Calls from several threads are safe as long as they
 *           do not share a workspace (or, for vp_decode_step_static, a GPU).
 * Streams.  `stream` is a hipStream_t (NULL = the legacy default stream). Every
 *           call only enqueues kernels on that stream and returns; none
 *           synchronises (vp_validate_layout, a debug helper, excepted). k and
 *           the kept indices stay on the device, so a step never waits for the
 *           host.
 * Shapes.   q and out are [B, T, Hq, d] contiguous (T = 1 by default). K and V caches are addressed as
 *           base + b*kv_stride_b + h*kv_stride_h + s*kv_stride_s (elements) with
 *           the d elements of a row contiguous. Query head h reads KV head
 *           h / (Hq/Hkv) (grouped-query attention).
 * Paged KV. With shape.block_size = P > 0 the caches are paged, as serving
 *           engines keep them: token s of sequence b lives in physical block
 *           blk = block_table[b * ceil(max_seq_len / P) + s / P] at
 *           base + blk*kv_stride_b + h*kv_stride_h + (s % P)*kv_stride_s; P is a
 *           power of two and kv_stride_b is the block stride. Block ids are
 *           trusted like the rest of the layout (they must address blocks of
 *           the caller's K and V).
 * Layout.   Each sequence b holds seq_len[b] cached tokens. Its visual tokens
 *           X_v (Sec. 4.2) are the union of the segments
 *           vis_seg[vis_seg_off[b] .. vis_seg_off[b+1]), each {start, length},
 *           ascending and disjoint inside [0, seq_len[b]); every other position
 *           is text (system prompt, question, generated trace, current token).
 *           A visual token's "rank" is its index among the visual tokens of
 *           its sequence in position order. Device-resident layout contents are
 *           trusted; kernels clip them (seq_len to max_seq_len, segments to the
 *           sequence and to the previous segment's end, ranks to max_vis) so
 *           that malformed layouts cannot cause out-of-bounds accesses.
 * Errors.   Host-checkable problems (null pointers, unsupported shapes, small
 *           workspace, bad parameters) return an error before anything is
 *           enqueued. A failed kernel launch returns VP_ERR_HIP.
 * Scope.    shape.scope chooses where the budget and the kept set live.
 *           VP_SCOPE_SEQUENCE (the paper's method, Sec. 4.2/4.3): one k and one
 *           kept set per sequence, from the mean and max over all Hq query
 *           heads, shared by every head. VP_SCOPE_KV_GROUP (a per-KV-group
 *           variant): each KV group g (query heads g*G .. g*G+G-1, G = Hq/Hkv)
 *           is treated as a sequence of its own: Eq. (5)/(7) take the mean and
 *           max over the group's G heads, Eq. (2) averages over them, and the
 *           group's heads attend over the group's own kept set. Per-query
 *           results are then held in U = Hkv "selection rows" (row u = g),
 *           else U = 1.
 * Queries.  shape.n_queries = T > 1 runs T queries per sequence in one step
 *           (speculative or multi-token decoding; an extension of the paper's
 *           one query per step): the queries are the sequence's last T
 *           positions, query t sees the positions before L - T + 1 + t, and
 *           each is a decode step of its own (own masses, budget, kept set,
 *           output); the positions from L - T + 1 on are text whatever the
 *           segments say. The K/V rows are read once for all T queries.
 *           q and out are then [B, T, Hq, d] and mass_head [B, T, Hq].
 * Rows.     With R = T*U selection rows per sequence, row (b*T + t)*U + u:
 *           mass_seq is [B*R, 2], scores [B*R, max_vis], k [B*R] and vis_idx
 *           [B*R, k_cap] (R = 1 by default: row b).
 * Dtypes.   VP_BF16: q, K, V, out are bfloat16; VP_F32: all float32. Logits,
 *           softmax statistics, masses and scores are float32; accumulation is
 *           float32 (bf16 products are exact in float32).
 */
#ifndef VISIONPULSE_H
#define VISIONPULSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum vp_status {
  VP_OK = 0,
  VP_ERR_NULL = 1,         /* a required pointer is NULL */
  VP_ERR_SHAPE = 2,        /* inconsistent sizes (Hq % Hkv, strides, k_cap ...) */
  VP_ERR_RANGE = 3,        /* a parameter is outside its domain (tau <= 0, bp ...) */
  VP_ERR_DTYPE = 4,        /* dtype is neither VP_F32 nor VP_BF16 */
  VP_ERR_UNSUPPORTED = 5,  /* valid but not implemented (head_dim, group size ...) */
  VP_ERR_WORKSPACE = 6,    /* workspace NULL or smaller than vp_workspace_size() */
  VP_ERR_HIP = 7           /* a HIP runtime call or kernel launch failed */
} vp_status;

typedef enum vp_dtype { VP_F32 = 0, VP_BF16 = 1 } vp_dtype;

/* Where budgets and kept sets live (see "Scope" above). */
typedef enum vp_scope { VP_SCOPE_SEQUENCE = 0, VP_SCOPE_KV_GROUP = 1 } vp_scope;

/* Host-side description of one step's tensors (validated synchronously). */
typedef struct vp_shape {
  int32_t batch;        /* B >= 1 */
  int32_t n_q_heads;    /* Hq >= 1 */
  int32_t n_kv_heads;   /* Hkv >= 1, Hq % Hkv == 0, Hq / Hkv <= 16 */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t dtype;        /* vp_dtype of q, K, V and out */
  int32_t max_seq_len;  /* cache capacity (rows); every seq_len[b] <= max_seq_len <= 2^28 */
  int32_t max_vis;      /* >= N_v of every sequence; row stride of scores; <= 2^28 */
  int32_t max_segs;     /* >= visual segments of any sequence; <= 256 */
  int32_t k_cap;        /* row stride of vis_idx; >= every budget vp_budget can return; <= 2^28 */
  int32_t block_size;   /* 0: contiguous caches; P > 0 (a power of two <= 65536): paged caches of P rows per block */
  int32_t scope;        /* vp_scope: selection rows per sequence R = 1 (VP_SCOPE_SEQUENCE) or Hkv (VP_SCOPE_KV_GROUP) */
  int32_t n_queries;    /* T: queries per sequence (0 is read as 1); T * Hq / Hkv <= 16 */
  int64_t kv_stride_b;  /* elements between sequences in K and V (paged: between physical blocks) */
  int64_t kv_stride_h;  /* elements between KV heads */
  int64_t kv_stride_s;  /* elements between token rows (>= head_dim) */
} vp_shape;

/* Device-resident token layout (Sec. 4.2: X_v = {v_1 .. v_N}; the rest is text). */
typedef struct vp_layout {
  const int32_t* seq_len;      /* [B] cached tokens per sequence */
  const int32_t* vis_seg_off;  /* [B+1] CSR offsets into vis_seg */
  const int32_t* vis_seg;      /* [n_seg][2] {start, length} visual segments */
  const int32_t* block_table;  /* [B][ceil(max_seq_len / block_size)] physical KV blocks (paged caches; else NULL) */
} vp_layout;

/* Method parameters (host-side). */
typedef struct vp_params {
  float tau_mass;   /* tau of Eq. (6) for the mass, > 0 (0.1 for the 5% preset, 0.4 for 10%; App. B.1) */
  float tau_score;  /* temperature of the attention used by the Eq. (2) scores, > 0 (1.0) */
  float sm_scale;   /* logit scale of Z; <= 0 selects 1/sqrt(head_dim) */
  int32_t r_lo_bp;  /* budget clamp lower bound, basis points of N_v (100 = 1%, Sec. 5.2) */
  int32_t r_hi_bp;  /* budget clamp upper bound, basis points of N_v (500 = 5%) */
  int32_t clamp;    /* 1: clamp K_t to [ceil(r_lo N_v), floor(r_hi N_v)]; 0: K_t = ceil(M N_v) */
} vp_params;

/* vp_sparse_decode_attn flags */
#define VP_ATTN_TEXT_FROM_WORKSPACE 1  /* reuse the text-KV partial left by vp_visual_mass (V != NULL) */

/* Human-readable name of a status code (static string). */
const char* vp_status_string(vp_status status);

/* Detail of the most recent error returned on the calling thread ("" if none). */
const char* vp_last_error(void);

/* Bytes of device workspace the calls need for `shape` (at most 256-byte
 * aligned pieces; pass a 256-byte aligned pointer). Pure host computation. */
vp_status vp_workspace_size(const vp_shape* shape, size_t* bytes);

/*
 * vp_visual_mass -- Eq. (6) tempered attention of the current query over the
 * whole cache, Eq. (5) visual mass per head, its head mean and head max
 * (Sec. 4.3), and the Eq. (2) importance score of every visual token (Sec. 4.2).
 *
 *   Z_{h,j}      = sm_scale * <q_h, K_{g(h), j}>                j < seq_len
 *   mass_head    = sum_{j visual} softmax_j(Z_h / tau_mass)      [B, T, Hq]
 *   mass_seq     = {mean_h mass_head, max_h mass_head}           [B*R, 2]
 *   scores[b, i] = (1/Hq) sum_h softmax_j(Z_h / tau_score)_{v_i} [B*R, max_vis], rank order;
 *                  entries i >= N_v of the sequence are not written.
 * (per query t, j < its visible length; VP_SCOPE_KV_GROUP: row per KV group g,
 * with h over the group's G heads and 1/G.)
 *
 * q: [B, Hq, d]; K: cache; V: cache or NULL. When V is non-NULL the same pass
 * over K also accumulates the softmax-weighted text-token values (the text
 * part of the pruned attention) into `workspace`, for a later
 * vp_sparse_decode_attn(..., VP_ATTN_TEXT_FROM_WORKSPACE) with the same
 * q, K, V, layout and workspace. The workspace is used between the kernels of
 * this call and must not be shared by concurrent calls.
 */
vp_status vp_visual_mass(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                         const void* q, const void* K, const void* V,
                         float* mass_head, float* mass_seq, float* scores,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * vp_visual_mass_timed -- vp_visual_mass that also records caller-created HIP
 * events (hipEvent_t) on `stream` around its kernel launches, so a profiler or
 * benchmark can time the kernels with hipEventElapsedTime. events[i],
 * i < n_events (at most VP_MASS_EVENTS; NULL entries are skipped), is recorded
 *   [0] before the visual pass
 *   [1] when the text pass starts executing, [2] when it ends (both attached
 *       to that launch, hipExtLaunchKernel: [1]..[2] is its execution alone)
 *   [3] after the mass reduction    [4] after the scores kernel.
 * (With VP_PLAN_ONE_CONTEXT_LAUNCH and V given, [1]..[2] is the one launch of
 * both passes; see vp_step_plan.)
 * events may be NULL when n_events is 0. Results are identical to
 * vp_visual_mass. VP_ERR_RANGE if n_events is outside [0, VP_MASS_EVENTS].
 */
#define VP_MASS_EVENTS 5
vp_status vp_visual_mass_timed(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                               const void* q, const void* K, const void* V,
                               float* mass_head, float* mass_seq, float* scores,
                               void* workspace, size_t workspace_bytes, void* stream,
                               void* const* events, int32_t n_events);

/*
 * vp_budget -- Eq. (7): K_t = M_vis,max * N_v rounded up, clamped to
 * [ceil(r_lo N_v), floor(r_hi N_v)] (Sec. 5.2; k_hi raised to k_lo if needed)
 * and to [0, N_v]. The product is formed in double from the float mass, so the
 * rounding decision is exact. N_v = 0 gives 0.
 *
 * mass_seq: [B*R, 2] device (column 1 = M_vis,max); k: [B*R] int32 device
 * (one budget per selection row; N_v is the row's sequence's).
 */
vp_status vp_budget(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                    const float* mass_seq, int32_t* k, void* stream);

/*
 * vp_budget_top_p -- the Top-p budget the paper compares the mass rule against
 * (Sec. 5, budgeting strategies): for every sequence, the smallest number of
 * visual tokens, taken in the Eq. (3) order (descending score, ties to the
 * lower position), whose Eq. (2) scores sum to at least p; N_v when all of them
 * sum to less; 0 when p == 0. The sums are exact in 2^-40 fixed point (each
 * fp32 score rounded down), so the count is deterministic. Feed k to
 * vp_select_topk (which clamps it to k_cap).
 *
 * scores: [B*R, max_vis] float (from vp_visual_mass); k: [B*R] int32 device.
 * VP_ERR_RANGE unless 0 <= p <= 1.
 */
vp_status vp_budget_top_p(const vp_shape* shape, const vp_layout* layout, const float* scores, float p,
                          int32_t* k, void* stream);

/*
 * vp_select_topk -- Eq. (3): for every selection row r (of sequence b), the
 * k[r] visual tokens with the largest score, ties to the lower position;
 * written as absolute cache positions in ascending order to
 * vis_idx[r, 0 .. k[r]) and -1 in vis_idx[r, k[r] .. k_cap). k[r] is clamped
 * to [0, min(N_v, k_cap)].
 *
 * scores: [B*R, max_vis] float (from vp_visual_mass); k: [B*R] int32 device;
 * vis_idx: [B*R, k_cap] int32 device.
 */
vp_status vp_select_topk(const vp_shape* shape, const vp_layout* layout,
                         const float* scores, const int32_t* k, int32_t* vis_idx, void* stream);

/*
 * vp_sparse_decode_attn -- the step's attention over the pruned context
 * J_b = {vis_idx[r, 0 .. k[r])} U {text positions of b} (Sec. 4.1/4.2; the
 * dropped visual tokens are absent from the softmax, which is renormalised
 * over J_b at temperature 1), r the selection row of head h (per query t, the
 * text positions of J_b are those query t sees):
 *
 *   out[b, h] = sum_{j in J_b} softmax_{J_b}(Z_{h, j}) V_{g(h), j}      [B, T, Hq, d]
 *
 * An empty J_b yields zeros. Kept indices outside [0, seq_len) or equal to -1
 * are skipped. The kept indices are taken to be distinct visual positions, as
 * vp_select_topk writes them: a repeated index, or a text position, adds that
 * row's term once more (the union above then counts it twice). With flags & VP_ATTN_TEXT_FROM_WORKSPACE the text part is taken
 * from the workspace filled by vp_visual_mass (V non-NULL, same inputs);
 * otherwise this call reads the text K/V itself.
 */
vp_status vp_sparse_decode_attn(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                                const void* q, const void* K, const void* V,
                                const int32_t* vis_idx, const int32_t* k, void* out, int32_t flags,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * vp_decode_step -- one whole decode step (Sec. 4.1-4.3): the results of
 *   vp_visual_mass(V) -> vp_budget -> vp_select_topk
 *     -> vp_sparse_decode_attn(VP_ATTN_TEXT_FROM_WORKSPACE)
 * on the same arguments, in fewer launches: the mass reduction, scores,
 * budget and top-k of every sequence run in one launch (a sequence's visual
 * ranks are scored in chunks on several work-groups, the last chunk to finish
 * selects). All outputs are written as by the four calls (same arithmetic,
 * same reduction order): mass_head [B, T, Hq], mass_seq [B*R, 2],
 * scores [B*R, max_vis], k [B*R], vis_idx [B*R, k_cap], out [B, T, Hq, d]; V is
 * required.
 *
 * events: optional caller-created hipEvent_t recorded on `stream`, i < n_events
 * (at most VP_STEP_EVENTS; NULL entries skipped):
 *   [0] before the visual pass
 *   [1] when the text pass starts executing, [2] when it ends (attached to
 *       that launch: [1]..[2] is its execution alone, as a profiler sees it;
 *       with VP_PLAN_ONE_CONTEXT_LAUNCH, the one launch of both passes)
 *   [3] before the kept-row pass  [4] before the merge  [5] after the merge
 *   (with VP_PLAN_KEPT_IN_MERGE there is no kept-row pass: [3] and [4] both
 *   mark the start of the merge).
 * Errors as for the four calls; VP_ERR_RANGE if n_events is outside
 * [0, VP_STEP_EVENTS]. The workspace must not be shared by concurrent calls.
 */
#define VP_STEP_EVENTS 6
vp_status vp_decode_step(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                         const void* q, const void* K, const void* V,
                         float* mass_head, float* mass_seq, float* scores, int32_t* k, int32_t* vis_idx,
                         void* out, void* workspace, size_t workspace_bytes, void* stream,
                         void* const* events, int32_t n_events);

/*
 * vp_decode_step_static -- vp_decode_step for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops and harnesses that
 * forbid hipMalloc): the same launches and results, bit for bit, with the
 * library's own scratch in place of the caller's workspace. The scratch is a
 * device array of VP_STATIC_SCRATCH_BYTES that every GPU the library runs on
 * holds until the process ends; its address is looked up once per device, on
 * the first call with that device current. This call allocates nothing and
 * records no events. The stream must belong to the current device.
 *
 * The scratch keeps the last call's contents; nothing in it needs to start at
 * zero (every step writes what it later reads). All calls on one GPU share it,
 * so calls that may overlap on one GPU (several streams or threads) race and
 * must be serialised by the caller.
 *
 * Errors: as vp_decode_step; VP_ERR_WORKSPACE, before anything is enqueued,
 * when vp_workspace_size(shape) exceeds VP_STATIC_SCRATCH_BYTES (the 16-sequence
 * 12k-token batch of the 7B shape needs about 29 MiB; 64 sequences of 32k
 * tokens need 268 MiB and must use vp_decode_step); VP_ERR_HIP if the scratch
 * address cannot be obtained.
 */
#define VP_STATIC_SCRATCH_BYTES (32u << 20)
vp_status vp_decode_step_static(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                                const void* q, const void* K, const void* V,
                                float* mass_head, float* mass_seq, float* scores, int32_t* k, int32_t* vis_idx,
                                void* out, void* stream);

/*
 * vp_step_plan -- how vp_visual_mass (with V) and vp_decode_step will launch
 * their kernels for this shape (pure host computation; for profiling and
 * benchmarks). flags is a bit set of
 *   VP_PLAN_ONE_CONTEXT_LAUNCH  the visual and text passes share one launch
 *                               (small and mid-size caches); events [1]..[2]
 *                               then time that whole launch;
 *   VP_PLAN_FUSED_TAIL          vp_decode_step's select launch scores and
 *                               selects each sequence in a single work-group
 *                               (small visual sets; otherwise in chunks, the
 *                               last chunk selecting);
 *   VP_PLAN_KEPT_IN_MERGE       small steps: vp_decode_step and
 *                               vp_sparse_decode_attn(VP_ATTN_TEXT_FROM_WORKSPACE)
 *                               read the kept rows in the merge launch (no kept
 *                               pass); vp_sparse_decode_attn without that flag
 *                               keeps its kept pass, so its output then agrees
 *                               with theirs to rounding, not bit for bit.
 */
#define VP_PLAN_ONE_CONTEXT_LAUNCH 1
#define VP_PLAN_FUSED_TAIL 2
#define VP_PLAN_KEPT_IN_MERGE 4
vp_status vp_step_plan(const vp_shape* shape, const vp_params* params, int32_t* flags);

/*
 * vp_validate_layout -- debug and test helper: synchronises `stream`, copies the
 * device-resident layout to the host and checks what the kernels otherwise
 * trust (they only clip): 0 <= seq_len[b] <= max_seq_len; vis_seg_off
 * non-decreasing from >= 0; at most max_segs segments per sequence, each of
 * length >= 1, ascending, disjoint and inside [0, seq_len[b]); N_v <= max_vis;
 * with paged caches, block ids >= 0 for every block a sequence uses (that an id
 * addresses a block of the caller's caches is not checkable here). Returns
 * VP_ERR_SHAPE naming the first violation (vp_last_error), VP_ERR_HIP if a copy
 * fails. The only call that synchronises; not for the decode loop.
 */
vp_status vp_validate_layout(const vp_shape* shape, const vp_layout* layout, void* stream);

/*
 * vp_stream_read -- measurement helper, not part of the method: enqueues one
 * read of `bytes` of device memory at `src` (16-byte aligned; bytes a positive
 * multiple of 16 KiB), so that a benchmark can time the GPU's streaming-read
 * ceiling next to the decode step. mode 0: 16-byte vector loads into
 * registers; mode 1: the HBM -> LDS row copies the decode-step kernels use.
 * Both are non-temporal. `sink` is a device uint32 the kernel may write (so
 * the loads are kept); its value means nothing. VP_ERR_SHAPE / VP_ERR_RANGE /
 * VP_ERR_NULL for bad arguments.
 */
vp_status vp_stream_read(const void* src, size_t bytes, int32_t mode, uint32_t* sink, void* stream);

/* Host mirror of vp_budget's rule for one sequence (pure; for callers that keep
 * the mass on the host). Returns -1 for invalid parameters. */
int32_t vp_budget_host(double m_max, int32_t n_vis, const vp_params* params);

#ifdef __cplusplus
}
#endif

#endif /* VISIONPULSE_H */
