// C ABI of the VisionPulse decode-step path: argument validation, workspace
// carving and kernel launches on the caller's stream (no allocation, no sync).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "vp_internal.h"

// Scratch memory of vp_decode_step_static: each GPU the library runs on holds
// one copy of this array until the process ends. Host code never uses its name
// as an address (on the host it is only a stand-in for the symbol): the device
// address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[VP_STATIC_SCRATCH_BYTES];

namespace vp {
namespace {

thread_local std::string g_last_error;

vp_status fail(vp_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
vp_status fail(vp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

vp_status hip_fail(hipError_t e, const char* what) {
  return fail(VP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Device address of `scratch` on the current device: looked up on the first
// call for that device (with it current) and kept.
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

vp_status static_scratch(void** ptr) {
  int dev = -1;
  if (hipError_t e = hipGetDevice(&dev)) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(VP_ERR_UNSUPPORTED, "device %d >= %d", dev, kMaxDevices);
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) return hip_fail(e, "hipGetSymbolAddress(scratch)");
      if (!p) return fail(VP_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return VP_OK;
}

constexpr int kMaxGroup = 16;
constexpr int kMaxHq = kMaxHq_;
constexpr int kMaxBatch = 65535;
constexpr int kMaxTokens = 1 << 28;  // bound on max_seq_len, max_vis and k_cap (32-bit index arithmetic)


vp_status check_shape(const vp_shape* s) {
  if (!s) return fail(VP_ERR_NULL, "shape is NULL");
  if (s->dtype != VP_F32 && s->dtype != VP_BF16) return fail(VP_ERR_DTYPE, "dtype %d", s->dtype);
  if (s->batch < 1 || s->batch > kMaxBatch) return fail(VP_ERR_SHAPE, "batch %d outside [1, %d]", s->batch, kMaxBatch);
  if (s->n_q_heads < 1 || s->n_kv_heads < 1) return fail(VP_ERR_SHAPE, "head counts must be >= 1");
  if (s->n_q_heads % s->n_kv_heads != 0)
    return fail(VP_ERR_SHAPE, "n_q_heads %d not a multiple of n_kv_heads %d", s->n_q_heads, s->n_kv_heads);
  if (s->n_q_heads / s->n_kv_heads > kMaxGroup)
    return fail(VP_ERR_UNSUPPORTED, "query group %d > %d", s->n_q_heads / s->n_kv_heads, kMaxGroup);
  if (s->n_q_heads > kMaxHq) return fail(VP_ERR_UNSUPPORTED, "n_q_heads %d > %d", s->n_q_heads, kMaxHq);
  if (s->head_dim != 64 && s->head_dim != 128) return fail(VP_ERR_UNSUPPORTED, "head_dim %d (64 or 128)", s->head_dim);
  if (s->max_seq_len < 1) return fail(VP_ERR_SHAPE, "max_seq_len %d < 1", s->max_seq_len);
  if (s->max_vis < 1) return fail(VP_ERR_SHAPE, "max_vis %d < 1", s->max_vis);
  if (s->max_seq_len > kMaxTokens || s->max_vis > kMaxTokens || s->k_cap > kMaxTokens)
    return fail(VP_ERR_UNSUPPORTED, "max_seq_len, max_vis and k_cap must not exceed %d", kMaxTokens);
  if (s->max_segs < 0 || s->max_segs > 256) return fail(VP_ERR_UNSUPPORTED, "max_segs %d outside [0, 256]", s->max_segs);
  if (s->k_cap < 1) return fail(VP_ERR_SHAPE, "k_cap %d < 1", s->k_cap);
  if (s->block_size < 0 || s->block_size > 65536 || (s->block_size & (s->block_size - 1)) != 0)
    return fail(VP_ERR_SHAPE, "block_size %d: 0 (contiguous) or a power of two <= 65536", s->block_size);
  if (s->scope != VP_SCOPE_SEQUENCE && s->scope != VP_SCOPE_KV_GROUP)
    return fail(VP_ERR_RANGE, "scope %d: VP_SCOPE_SEQUENCE or VP_SCOPE_KV_GROUP", s->scope);
  if (s->n_queries < 0) return fail(VP_ERR_RANGE, "n_queries %d < 0", s->n_queries);
  if (static_cast<int64_t>(queries(*s)) * (s->n_q_heads / s->n_kv_heads) > kMaxGroup)
    return fail(VP_ERR_UNSUPPORTED, "n_queries %d x query group %d > %d rows per KV head", queries(*s),
                s->n_q_heads / s->n_kv_heads, kMaxGroup);
  if (static_cast<int64_t>(s->batch) * rows_per_seq(*s) > kMaxBatch)
    return fail(VP_ERR_UNSUPPORTED, "batch x queries x selection rows %lld > %d",
                static_cast<long long>(s->batch) * rows_per_seq(*s), kMaxBatch);
  const int esz = s->dtype == VP_BF16 ? 2 : 4;
  const int64_t align_elems = 16 / esz;
  if (s->kv_stride_s < s->head_dim) return fail(VP_ERR_SHAPE, "kv_stride_s %lld < head_dim", (long long)s->kv_stride_s);
  if (s->kv_stride_b < 0 || s->kv_stride_h < 0) return fail(VP_ERR_SHAPE, "negative KV stride");
  if (s->kv_stride_s % align_elems || s->kv_stride_h % align_elems || s->kv_stride_b % align_elems)
    return fail(VP_ERR_SHAPE, "KV strides must be multiples of %lld elements (16-byte rows)", (long long)align_elems);
  return VP_OK;
}

vp_status check_params(const vp_params* p) {
  if (!p) return fail(VP_ERR_NULL, "params is NULL");
  if (!(p->tau_mass > 0.f) || !std::isfinite(p->tau_mass)) return fail(VP_ERR_RANGE, "tau_mass must be > 0");
  if (!(p->tau_score > 0.f) || !std::isfinite(p->tau_score)) return fail(VP_ERR_RANGE, "tau_score must be > 0");
  if (!std::isfinite(p->sm_scale)) return fail(VP_ERR_RANGE, "sm_scale not finite");
  if (p->r_lo_bp < 0 || p->r_lo_bp > 10000 || p->r_hi_bp < 0 || p->r_hi_bp > 10000)
    return fail(VP_ERR_RANGE, "retention bounds must lie in [0, 10000] basis points");
  if (p->clamp != 0 && p->clamp != 1) return fail(VP_ERR_RANGE, "clamp must be 0 or 1");
  return VP_OK;
}

vp_status check_layout(const vp_shape* s, const vp_layout* l) {
  if (!l) return fail(VP_ERR_NULL, "layout is NULL");
  if (!l->seq_len || !l->vis_seg_off || !l->vis_seg)
    return fail(VP_ERR_NULL, "layout seq_len / vis_seg_off / vis_seg is NULL");
  if (s->block_size > 0 && !l->block_table) return fail(VP_ERR_NULL, "paged caches (block_size > 0) need a block_table");
  return VP_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

vp_status check_ws(const vp_shape* s, void* ws, size_t bytes, Plan& plan) {
  plan = make_plan(*s);
  if (!ws) return fail(VP_ERR_WORKSPACE, "workspace is NULL");
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return fail(VP_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (bytes < plan.total) return fail(VP_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", bytes, plan.total);
  return VP_OK;
}

float zscale_of(const vp_shape* s, const vp_params* p) {
  const float sm = p->sm_scale > 0.f ? p->sm_scale : 1.0f / std::sqrt(static_cast<float>(s->head_dim));
  return sm * 1.4426950408889634f;  // log2(e)
}

int max_budget(const vp_shape* s, const vp_params* p) {
  if (!p->clamp) return s->max_vis;
  int hi = floor_bp(s->max_vis, p->r_hi_bp);
  const int lo = ceil_bp(s->max_vis, p->r_lo_bp);
  if (hi < lo) hi = lo;
  return hi < s->max_vis ? hi : s->max_vis;
}

AttendArgs attend_args(const vp_shape* s, const vp_layout* l, const vp_params* p, const Plan& plan, char* ws,
                       const void* q, const void* K, const void* V) {
  AttendArgs a{};
  a.q = q;
  a.K = K;
  a.V = V;
  a.sb = s->kv_stride_b;
  a.sh = s->kv_stride_h;
  a.ss = s->kv_stride_s;
  a.bs_log2 = -1;
  a.nblk = 0;
  a.block_table = nullptr;
  if (s->block_size > 0) {
    a.bs_log2 = __builtin_ctz(static_cast<unsigned>(s->block_size));
    a.nblk = (s->max_seq_len + s->block_size - 1) / s->block_size;
    a.block_table = l->block_table;
  }
  a.seq_len = l->seq_len;
  a.seg_off = l->vis_seg_off;
  a.seg = l->vis_seg;
  a.B = s->batch;
  a.Hq = s->n_q_heads;
  a.Hkv = s->n_kv_heads;
  a.G = s->n_q_heads / s->n_kv_heads;
  a.max_seq_len = s->max_seq_len;
  a.max_vis = s->max_vis;
  a.T = queries(*s);
  a.U = rows_per_query(*s);
  a.zscale = zscale_of(s, p);
  a.inv_tau_m = 1.0f / p->tau_mass;
  a.inv_tau_s = 1.0f / p->tau_score;
  // lazy running maxima: a reference is raised only when a logit exceeds it by
  // more than a margin that keeps every tempered weight below 2^64
  a.thr_s = 64.0f / std::max(1.0f, std::max(a.inv_tau_m, a.inv_tau_s));
  a.thr_t = a.thr_s;
  a.tau_s_one = p->tau_score == 1.0f;
  a.nparts = plan.nparts;
  a.zs_rows = plan.zs_rows;
  a.zs_gp = plan.zs_gp;
  a.zs = reinterpret_cast<float*>(ws + plan.zs);
  a.stats = reinterpret_cast<float*>(ws + plan.stats);
  a.acc = reinterpret_cast<float*>(ws + plan.acc);
  a.k_cap = s->k_cap;
  a.split = plan.split;
  a.nsplit = plan.nsplit;
  a.kstats = reinterpret_cast<float*>(ws + plan.kstats);
  a.kacc = reinterpret_cast<float*>(ws + plan.kacc);
  a.sync = reinterpret_cast<uint32_t*>(ws + plan.sync);
  a.segtab = ws + plan.segtab;
  return a;
}

}  // namespace

MassArgs mass_args(const vp_shape* s, const vp_layout* l, const Plan& plan, const AttendArgs& a, char* ws,
                   float* mass_head, float* mass_seq, float* scores) {
  MassArgs m{};
  m.seq_len = l->seq_len;
  m.seg_off = l->vis_seg_off;
  m.seg = l->vis_seg;
  m.B = s->batch;
  m.Hq = s->n_q_heads;
  m.max_seq_len = s->max_seq_len;
  m.max_vis = s->max_vis;
  m.nparts = plan.nparts;
  m.Hkv = s->n_kv_heads;
  m.G = s->n_q_heads / s->n_kv_heads;
  m.T = queries(*s);
  m.U = rows_per_query(*s);
  m.zs_rows = plan.zs_rows;
  m.zs_gp = plan.zs_gp;
  m.inv_tau_m = a.inv_tau_m;
  m.inv_tau_s = a.inv_tau_s;
  m.stats = a.stats;
  m.zs = a.zs;
  m.head = reinterpret_cast<float*>(ws + plan.head);
  m.mass_head = mass_head;
  m.mass_seq = mass_seq;
  m.scores = scores;
  return m;
}

BudgetArgs budget_args(const vp_shape* s, const vp_layout* l, const vp_params* p, const float* mass_seq, int32_t* k) {
  BudgetArgs b{};
  b.seq_len = l->seq_len;
  b.seg_off = l->vis_seg_off;
  b.seg = l->vis_seg;
  b.B = s->batch;
  b.R = rows_per_seq(*s);
  b.T = queries(*s);
  b.max_seq_len = s->max_seq_len;
  b.r_lo_bp = p->r_lo_bp;
  b.r_hi_bp = p->r_hi_bp;
  b.clamp = p->clamp;
  b.mass_seq = mass_seq;
  b.k = k;
  return b;
}

TopkArgs topk_args(const vp_shape* s, const vp_layout* l, const float* scores, const int32_t* k, int32_t* vis_idx) {
  TopkArgs t{};
  t.seq_len = l->seq_len;
  t.seg_off = l->vis_seg_off;
  t.seg = l->vis_seg;
  t.B = s->batch;
  t.R = rows_per_seq(*s);
  t.T = queries(*s);
  t.max_seq_len = s->max_seq_len;
  t.max_vis = s->max_vis;
  t.k_cap = s->k_cap;
  t.scores = scores;
  t.k = k;
  t.vis_idx = vis_idx;
  return t;
}

MergeArgs merge_args(const vp_shape* s, const Plan& plan, const AttendArgs& a, void* out) {
  MergeArgs m{};
  m.B = s->batch;
  m.Hq = s->n_q_heads;
  m.G = s->n_q_heads / s->n_kv_heads;
  m.T = queries(*s);
  m.nparts = plan.nparts;
  m.nsplit = plan.nsplit;
  m.seq_len = a.seq_len;
  m.vis_idx = a.vis_idx;
  m.kk = a.kk;
  m.max_seq_len = s->max_seq_len;
  m.Hkv = s->n_kv_heads;
  m.U = rows_per_query(*s);
  m.k_cap = s->k_cap;
  m.q = a.q;
  m.K = a.K;
  m.V = a.V;
  m.sb = a.sb;
  m.sh = a.sh;
  m.ss = a.ss;
  m.block_table = a.bs_log2 >= 0 ? a.block_table : nullptr;
  m.bs_log2 = a.bs_log2 >= 0 ? a.bs_log2 : 0;
  m.nblk = a.nblk;
  m.zscale = a.zscale;
  m.dtype = s->dtype;
  m.stats = a.stats;
  m.acc = a.acc;
  m.kstats = a.kstats;
  m.kacc = a.kacc;
  m.out = out;
  return m;
}

vp_status check_budget_cap(const vp_shape* s, const vp_params* p) {
  if (s->k_cap < max_budget(s, p))
    return fail(VP_ERR_SHAPE, "k_cap %d < largest budget %d for max_vis %d", s->k_cap, max_budget(s, p), s->max_vis);
  return VP_OK;
}

// Host checks of a whole decode step's arguments (everything but the workspace).
vp_status check_step_args(const vp_shape* shape, const vp_layout* layout, const vp_params* params, const void* q,
                          const void* K, const void* V, const float* mass_head, const float* mass_seq,
                          const float* scores, const int32_t* k, const int32_t* vis_idx, const void* out) {
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_layout(shape, layout)) return e;
  if (vp_status e = check_params(params)) return e;
  if (!q || !K || !V || !mass_head || !mass_seq || !scores || !k || !vis_idx || !out)
    return fail(VP_ERR_NULL, "q, K, V, mass_head, mass_seq, scores, k, vis_idx, out required");
  if (!aligned16(q) || !aligned16(K) || !aligned16(V)) return fail(VP_ERR_SHAPE, "q, K, V must be 16-byte aligned");
  return check_budget_cap(shape, params);
}

// The launches of one decode step (validated arguments; ws holds plan.total bytes):
// the context pass, the select launch, the kept-row pass and the merge.
vp_status launch_step(const vp_shape* shape, const vp_layout* layout, const vp_params* params, const Plan& plan,
                      char* ws, const void* q, const void* K, const void* V, float* mass_head, float* mass_seq,
                      float* scores, int32_t* k, int32_t* vis_idx, void* out, hipStream_t st, void* const* events,
                      int32_t n_events) {
  AttendArgs a = attend_args(shape, layout, params, plan, ws, q, K, V);
  a.vis_idx = vis_idx;
  a.kk = k;
  auto mark = [&](int i) -> hipError_t {
    return (i < n_events && events[i]) ? hipEventRecord(static_cast<hipEvent_t>(events[i]), st) : hipSuccess;
  };
  const int dt = shape->dtype, hd = shape->head_dim;
  // events [1] and [2] ride on the text (or one) context launch: its execution alone
  auto ev = [&](int i) -> hipEvent_t { return i < n_events ? static_cast<hipEvent_t>(events[i]) : nullptr; };
  if (hipError_t e = mark(0)) return hip_fail(e, "event record");
  if (use_dual(shape)) {
    if (hipError_t e = launch_attend(a, MODE_DUAL, dt, hd, st, ev(1), ev(2))) return hip_fail(e, "context pass launch");
  } else {
    if (hipError_t e = launch_attend(a, MODE_VIS, dt, hd, st)) return hip_fail(e, "visual pass launch");
    if (hipError_t e = launch_attend(a, MODE_TEXT_BOTH, dt, hd, st, ev(1), ev(2))) return hip_fail(e, "text pass launch");
  }
  SelectArgs t{};
  t.m = mass_args(shape, layout, plan, a, ws, mass_head, mass_seq, scores);
  t.r_lo_bp = params->r_lo_bp;
  t.r_hi_bp = params->r_hi_bp;
  t.clamp = params->clamp;
  t.k_cap = shape->k_cap;
  t.k = k;
  t.vis_idx = vis_idx;
  t.chunk = plan.sel_chunk;
  t.nchunks = plan.sel_chunks;
  t.sync = a.sync;
  t.segtab = a.segtab;
  if (hipError_t e = launch_select(t, st)) return hip_fail(e, "select launch");
  if (hipError_t e = mark(3)) return hip_fail(e, "event record");
  if (plan.merge_kept) {
    // a small step: the kept rows are merged directly (no kept pass)
    if (hipError_t e = mark(4)) return hip_fail(e, "event record");
    if (hipError_t e = launch_merge_kept(merge_args(shape, plan, a, out), hd, st)) return hip_fail(e, "merge launch");
  } else {
    // the kept rows are visual rows of this step's spill: their logits are read
    // from it, so the kept pass reads V rows only
    if (hipError_t e = launch_attend(a, MODE_KEPT | MODE_ZSPILL, dt, hd, st)) return hip_fail(e, "kept pass launch");
    if (hipError_t e = mark(4)) return hip_fail(e, "event record");
    if (hipError_t e = launch_merge(merge_args(shape, plan, a, out), hd, st)) return hip_fail(e, "merge launch");
  }
  if (hipError_t e = mark(5)) return hip_fail(e, "event record");
  return VP_OK;
}

}  // namespace vp

using namespace vp;

extern "C" {

const char* vp_status_string(vp_status s) {
  switch (s) {
    case VP_OK: return "VP_OK";
    case VP_ERR_NULL: return "VP_ERR_NULL";
    case VP_ERR_SHAPE: return "VP_ERR_SHAPE";
    case VP_ERR_RANGE: return "VP_ERR_RANGE";
    case VP_ERR_DTYPE: return "VP_ERR_DTYPE";
    case VP_ERR_UNSUPPORTED: return "VP_ERR_UNSUPPORTED";
    case VP_ERR_WORKSPACE: return "VP_ERR_WORKSPACE";
    case VP_ERR_HIP: return "VP_ERR_HIP";
  }
  return "VP_ERR_UNKNOWN";
}

const char* vp_last_error(void) { return g_last_error.c_str(); }

vp_status vp_workspace_size(const vp_shape* shape, size_t* bytes) {
  g_last_error.clear();
  if (vp_status e = check_shape(shape)) return e;
  if (!bytes) return fail(VP_ERR_NULL, "bytes is NULL");
  *bytes = make_plan(*shape).total;
  return VP_OK;
}

int32_t vp_budget_host(double m_max, int32_t n_vis, const vp_params* params) {
  if (!params || check_params(params) != VP_OK || n_vis < 0) return -1;
  return budget_rule(m_max, n_vis, params->r_lo_bp, params->r_hi_bp, params->clamp);
}

vp_status vp_visual_mass_timed(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                               const void* q, const void* K, const void* V, float* mass_head, float* mass_seq,
                               float* scores, void* workspace, size_t workspace_bytes, void* stream,
                               void* const* events, int32_t n_events) {
  g_last_error.clear();
  if (n_events < 0 || n_events > VP_MASS_EVENTS) return fail(VP_ERR_RANGE, "n_events %d outside [0, %d]", n_events, VP_MASS_EVENTS);
  if (n_events > 0 && !events) return fail(VP_ERR_NULL, "events is NULL with n_events %d", n_events);
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_layout(shape, layout)) return e;
  if (vp_status e = check_params(params)) return e;
  if (!q || !K || !mass_head || !mass_seq || !scores) return fail(VP_ERR_NULL, "q, K, mass_head, mass_seq, scores required");
  if (!aligned16(q) || !aligned16(K) || (V && !aligned16(V))) return fail(VP_ERR_SHAPE, "q, K, V must be 16-byte aligned");
  Plan plan;
  if (vp_status e = check_ws(shape, workspace, workspace_bytes, plan)) return e;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  AttendArgs a = attend_args(shape, layout, params, plan, ws, q, K, V);
  auto mark = [&](int i) -> hipError_t {
    return (i < n_events && events[i]) ? hipEventRecord(static_cast<hipEvent_t>(events[i]), st) : hipSuccess;
  };
  // events [1] and [2] ride on the text (or one) context launch: its execution alone
  auto ev = [&](int i) -> hipEvent_t { return i < n_events ? static_cast<hipEvent_t>(events[i]) : nullptr; };
  if (hipError_t e = mark(0)) return hip_fail(e, "event record");
  if (V && use_dual(shape)) {
    if (hipError_t e = launch_attend(a, MODE_DUAL, shape->dtype, shape->head_dim, st, ev(1), ev(2)))
      return hip_fail(e, "context pass launch");
  } else {
    if (hipError_t e = launch_attend(a, MODE_VIS, shape->dtype, shape->head_dim, st))
      return hip_fail(e, "visual pass launch");
    if (hipError_t e = launch_attend(a, V ? MODE_TEXT_BOTH : MODE_TEXT_STATS, shape->dtype, shape->head_dim, st, ev(1),
                                     ev(2)))
      return hip_fail(e, "text pass launch");
  }
  const MassArgs m = mass_args(shape, layout, plan, a, ws, mass_head, mass_seq, scores);
  if (hipError_t e = launch_mass_finalize(m, st)) return hip_fail(e, "mass finalize launch");
  if (hipError_t e = mark(3)) return hip_fail(e, "event record");
  if (hipError_t e = launch_scores(m, st)) return hip_fail(e, "scores launch");
  if (hipError_t e = mark(4)) return hip_fail(e, "event record");
  return VP_OK;
}

vp_status vp_visual_mass(const vp_shape* shape, const vp_layout* layout, const vp_params* params, const void* q,
                         const void* K, const void* V, float* mass_head, float* mass_seq, float* scores,
                         void* workspace, size_t workspace_bytes, void* stream) {
  return vp_visual_mass_timed(shape, layout, params, q, K, V, mass_head, mass_seq, scores, workspace,
                              workspace_bytes, stream, nullptr, 0);
}

vp_status vp_budget(const vp_shape* shape, const vp_layout* layout, const vp_params* params, const float* mass_seq,
                    int32_t* k, void* stream) {
  g_last_error.clear();
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_layout(shape, layout)) return e;
  if (vp_status e = check_params(params)) return e;
  if (!mass_seq || !k) return fail(VP_ERR_NULL, "mass_seq and k required");
  if (vp_status e = check_budget_cap(shape, params)) return e;
  if (hipError_t e = launch_budget(budget_args(shape, layout, params, mass_seq, k), static_cast<hipStream_t>(stream)))
    return hip_fail(e, "budget launch");
  return VP_OK;
}

vp_status vp_select_topk(const vp_shape* shape, const vp_layout* layout, const float* scores, const int32_t* k,
                         int32_t* vis_idx, void* stream) {
  g_last_error.clear();
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_layout(shape, layout)) return e;
  if (!scores || !k || !vis_idx) return fail(VP_ERR_NULL, "scores, k, vis_idx required");
  if (hipError_t e = launch_topk(topk_args(shape, layout, scores, k, vis_idx), static_cast<hipStream_t>(stream)))
    return hip_fail(e, "top-k launch");
  return VP_OK;
}

vp_status vp_validate_layout(const vp_shape* shape, const vp_layout* layout, void* stream) {
  g_last_error.clear();
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_layout(shape, layout)) return e;
  const int B = shape->batch;
  // the layout may have been written by work queued on the stream
  if (hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream))) return hip_fail(e, "stream sync");
  std::vector<int32_t> len(B), off(B + 1);
  if (hipError_t e = hipMemcpy(len.data(), layout->seq_len, B * sizeof(int32_t), hipMemcpyDeviceToHost))
    return hip_fail(e, "seq_len copy");
  if (hipError_t e = hipMemcpy(off.data(), layout->vis_seg_off, (B + 1) * sizeof(int32_t), hipMemcpyDeviceToHost))
    return hip_fail(e, "vis_seg_off copy");
  if (off[0] < 0) return fail(VP_ERR_SHAPE, "vis_seg_off[0] = %d < 0", off[0]);
  for (int b = 0; b < B; ++b) {
    if (off[b + 1] < off[b]) return fail(VP_ERR_SHAPE, "vis_seg_off decreases at sequence %d", b);
    if (off[b + 1] - off[b] > shape->max_segs)
      return fail(VP_ERR_SHAPE, "sequence %d: %d segments > max_segs %d", b, off[b + 1] - off[b], shape->max_segs);
  }
  // segments off[0] .. off[B]: at most B * max_segs (<= 16.8M), a bounded host copy
  const size_t nseg = static_cast<size_t>(off[B] - off[0]);
  std::vector<int32_t> seg(2 * nseg + 2);
  if (nseg > 0) {
    if (hipError_t e = hipMemcpy(seg.data(), layout->vis_seg + 2 * static_cast<size_t>(off[0]),
                                 2 * nseg * sizeof(int32_t), hipMemcpyDeviceToHost))
      return hip_fail(e, "vis_seg copy");
  }
  std::vector<int32_t> table;
  int64_t nblk = 0;
  if (shape->block_size > 0) {
    nblk = (shape->max_seq_len + shape->block_size - 1) / shape->block_size;
    table.resize(static_cast<size_t>(B) * nblk);
    if (hipError_t e = hipMemcpy(table.data(), layout->block_table, table.size() * sizeof(int32_t),
                                 hipMemcpyDeviceToHost))
      return hip_fail(e, "block_table copy");
  }
  for (int b = 0; b < B; ++b) {
    const int L = len[b];
    if (L < 0 || L > shape->max_seq_len)
      return fail(VP_ERR_SHAPE, "sequence %d: seq_len %d outside [0, max_seq_len %d]", b, L, shape->max_seq_len);
    int64_t end = 0, nv = 0;
    for (int i = off[b]; i < off[b + 1]; ++i) {
      const size_t j = static_cast<size_t>(i - off[0]);
      const int st = seg[2 * j], ln = seg[2 * j + 1];
      if (ln < 1) return fail(VP_ERR_SHAPE, "sequence %d: segment %d has length %d < 1", b, i - off[b], ln);
      if (st < end)
        return fail(VP_ERR_SHAPE, "sequence %d: segment %d starts at %d, before the previous end %lld", b,
                    i - off[b], st, static_cast<long long>(end));
      if (static_cast<int64_t>(st) + ln > L)
        return fail(VP_ERR_SHAPE, "sequence %d: segment %d [%d, %lld) ends past seq_len %d", b, i - off[b], st,
                    static_cast<long long>(st) + ln, L);
      end = static_cast<int64_t>(st) + ln;
      nv += ln;
    }
    if (nv > shape->max_vis)
      return fail(VP_ERR_SHAPE, "sequence %d: %lld visual tokens > max_vis %d", b, static_cast<long long>(nv),
                  shape->max_vis);
    if (shape->block_size > 0) {
      const int64_t used = (L + shape->block_size - 1) / shape->block_size;
      for (int64_t j = 0; j < used; ++j)
        if (table[b * nblk + j] < 0)
          return fail(VP_ERR_SHAPE, "sequence %d: block_table entry %lld is %d < 0", b, static_cast<long long>(j),
                      table[b * nblk + j]);
    }
  }
  return VP_OK;
}

vp_status vp_stream_read(const void* src, size_t bytes, int32_t mode, uint32_t* sink, void* stream) {
  g_last_error.clear();
  if (!src || !sink) return fail(VP_ERR_NULL, "src and sink required");
  if (!aligned16(src)) return fail(VP_ERR_SHAPE, "src must be 16-byte aligned");
  if (bytes == 0 || bytes % (16u << 10) != 0) return fail(VP_ERR_SHAPE, "bytes %zu: a positive multiple of 16 KiB", bytes);
  if (mode != 0 && mode != 1) return fail(VP_ERR_RANGE, "mode %d: 0 (vector loads) or 1 (LDS copies)", mode);
  if (hipError_t e = launch_stream_read(src, bytes, mode, sink, static_cast<hipStream_t>(stream)))
    return hip_fail(e, "stream read launch");
  return VP_OK;
}

vp_status vp_step_plan(const vp_shape* shape, const vp_params* params, int32_t* flags) {
  g_last_error.clear();
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_params(params)) return e;
  if (!flags) return fail(VP_ERR_NULL, "flags is NULL");
  const Plan plan = make_plan(*shape);
  *flags = (use_dual(shape) ? VP_PLAN_ONE_CONTEXT_LAUNCH : 0) | (plan.sel_chunks == 1 ? VP_PLAN_FUSED_TAIL : 0) |
           (plan.merge_kept ? VP_PLAN_KEPT_IN_MERGE : 0);
  return VP_OK;
}

vp_status vp_budget_top_p(const vp_shape* shape, const vp_layout* layout, const float* scores, float p, int32_t* k,
                          void* stream) {
  g_last_error.clear();
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_layout(shape, layout)) return e;
  if (!scores || !k) return fail(VP_ERR_NULL, "scores and k required");
  if (!(p >= 0.f && p <= 1.f)) return fail(VP_ERR_RANGE, "p %g outside [0, 1]", static_cast<double>(p));
  TopPArgs t{};
  t.seq_len = layout->seq_len;
  t.seg_off = layout->vis_seg_off;
  t.seg = layout->vis_seg;
  t.B = shape->batch;
  t.R = rows_per_seq(*shape);
  t.T = queries(*shape);
  t.max_seq_len = shape->max_seq_len;
  t.max_vis = shape->max_vis;
  t.p = p;
  t.scores = scores;
  t.k = k;
  if (hipError_t e = launch_top_p(t, static_cast<hipStream_t>(stream))) return hip_fail(e, "top-p launch");
  return VP_OK;
}

vp_status vp_sparse_decode_attn(const vp_shape* shape, const vp_layout* layout, const vp_params* params,
                                const void* q, const void* K, const void* V, const int32_t* vis_idx,
                                const int32_t* k, void* out, int32_t flags, void* workspace, size_t workspace_bytes,
                                void* stream) {
  g_last_error.clear();
  if (vp_status e = check_shape(shape)) return e;
  if (vp_status e = check_layout(shape, layout)) return e;
  if (vp_status e = check_params(params)) return e;
  if (!q || !K || !V || !vis_idx || !k || !out) return fail(VP_ERR_NULL, "q, K, V, vis_idx, k, out required");
  if (!aligned16(q) || !aligned16(K) || !aligned16(V)) return fail(VP_ERR_SHAPE, "q, K, V must be 16-byte aligned");
  if (flags & ~VP_ATTN_TEXT_FROM_WORKSPACE) return fail(VP_ERR_RANGE, "unknown flags 0x%x", flags);
  Plan plan;
  if (vp_status e = check_ws(shape, workspace, workspace_bytes, plan)) return e;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  AttendArgs a = attend_args(shape, layout, params, plan, ws, q, K, V);
  a.vis_idx = vis_idx;
  a.kk = k;
  if ((flags & VP_ATTN_TEXT_FROM_WORKSPACE) && plan.merge_kept) {
    // a small step's attention: the kept rows are merged directly, as in
    // vp_decode_step (a layer that reads its own text rows instead runs its
    // kept pass in the text pass's launch, below: faster for later layers)
    if (hipError_t e = launch_merge_kept(merge_args(shape, plan, a, out), shape->head_dim, st))
      return hip_fail(e, "merge launch");
    return VP_OK;
  }
  if (!(flags & VP_ATTN_TEXT_FROM_WORKSPACE) && plan.text_kept_one_launch) {
    // a layer that reads its own text rows: the text and kept passes share one launch
    if (hipError_t e = launch_attend(a, MODE_TEXT_KEPT, shape->dtype, shape->head_dim, st))
      return hip_fail(e, "text and kept pass launch");
  } else {
    if (!(flags & VP_ATTN_TEXT_FROM_WORKSPACE)) {
      if (hipError_t e = launch_attend(a, MODE_TEXT_ATTN, shape->dtype, shape->head_dim, st))
        return hip_fail(e, "text pass launch");
    }
    if (hipError_t e = launch_attend(a, MODE_KEPT, shape->dtype, shape->head_dim, st))
      return hip_fail(e, "kept pass launch");
  }
  if (hipError_t e = launch_merge(merge_args(shape, plan, a, out), shape->head_dim, st))
    return hip_fail(e, "merge launch");
  return VP_OK;
}

vp_status vp_decode_step(const vp_shape* shape, const vp_layout* layout, const vp_params* params, const void* q,
                         const void* K, const void* V, float* mass_head, float* mass_seq, float* scores, int32_t* k,
                         int32_t* vis_idx, void* out, void* workspace, size_t workspace_bytes, void* stream,
                         void* const* events, int32_t n_events) {
  g_last_error.clear();
  if (n_events < 0 || n_events > VP_STEP_EVENTS)
    return fail(VP_ERR_RANGE, "n_events %d outside [0, %d]", n_events, VP_STEP_EVENTS);
  if (n_events > 0 && !events) return fail(VP_ERR_NULL, "events is NULL with n_events %d", n_events);
  if (vp_status e = check_step_args(shape, layout, params, q, K, V, mass_head, mass_seq, scores, k, vis_idx, out))
    return e;
  Plan plan;
  if (vp_status e = check_ws(shape, workspace, workspace_bytes, plan)) return e;
  return launch_step(shape, layout, params, plan, static_cast<char*>(workspace), q, K, V, mass_head, mass_seq, scores,
                     k, vis_idx, out, static_cast<hipStream_t>(stream), events, n_events);
}

vp_status vp_decode_step_static(const vp_shape* shape, const vp_layout* layout, const vp_params* params, const void* q,
                                const void* K, const void* V, float* mass_head, float* mass_seq, float* scores,
                                int32_t* k, int32_t* vis_idx, void* out, void* stream) {
  g_last_error.clear();
  if (vp_status e = check_step_args(shape, layout, params, q, K, V, mass_head, mass_seq, scores, k, vis_idx, out))
    return e;
  const Plan plan = make_plan(*shape);
  if (plan.total > static_cast<size_t>(VP_STATIC_SCRATCH_BYTES))
    return fail(VP_ERR_WORKSPACE,
                "this shape needs %zu bytes of scratch; the static scratch holds %zu (use vp_decode_step with a "
                "workspace of vp_workspace_size bytes)",
                plan.total, static_cast<size_t>(VP_STATIC_SCRATCH_BYTES));
  void* ws = nullptr;
  if (vp_status e = static_scratch(&ws)) return e;
  return launch_step(shape, layout, params, plan, static_cast<char*>(ws), q, K, V, mass_head, mass_seq, scores, k,
                     vis_idx, out, static_cast<hipStream_t>(stream), nullptr, 0);
}

}  // extern "C"
