"""C ABI checks that need no GPU: the library loads, exports every declared
entry point, and rejects bad arguments before launching anything."""
import ctypes
import os
import re

import pytest

from paper_2605_31457_amd import vp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "visionpulse.h")
GOLDEN = os.path.join(ROOT, "tests", "golden")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(vp.LIB_PATH):
        from paper_2605_31457_amd import build
        build.build()
    return vp.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(vp_[a-z_0-9]+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert {"vp_visual_mass", "vp_budget", "vp_select_topk", "vp_sparse_decode_attn",
            "vp_workspace_size", "vp_status_string", "vp_last_error", "vp_budget_host"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def _shape(**kw):
    s = dict(batch=2, n_q_heads=28, n_kv_heads=4, head_dim=128, dtype=vp.VP_BF16, max_seq_len=4096,
             max_vis=1296, max_segs=1, k_cap=64, block_size=0, kv_stride_b=4 * 4096 * 128,
             kv_stride_h=4096 * 128, kv_stride_s=128)
    s.update(kw)
    return vp.vp_shape(**s)


def _params(**kw):
    p = dict(tau_mass=0.1, tau_score=1.0, sm_scale=0.0, r_lo_bp=100, r_hi_bp=500, clamp=1)
    p.update(kw)
    return vp.vp_params(**p)


def test_struct_layout_matches_header(L):
    assert ctypes.sizeof(vp.vp_shape) == 72 and vp.vp_shape.kv_stride_b.offset == 48
    assert ctypes.sizeof(vp.vp_params) == 24 and ctypes.sizeof(vp.vp_layout) == 32
    assert vp.vp_shape.block_size.offset == 36 and vp.vp_layout.block_table.offset == 24
    assert vp.vp_shape.scope.offset == 40 and vp.vp_shape.n_queries.offset == 44


def test_workspace_size_is_pure_and_scales(L):
    a = vp.vp_workspace_size(_shape())
    b = vp.vp_workspace_size(_shape(batch=4))
    assert a > 0 and b > a and a % 256 == 0
    # visual logits (B*Hq*max_vis fp32) are the dominant piece
    assert a >= 2 * 28 * 1296 * 4


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), "VP_ERR_DTYPE"),
    (dict(n_q_heads=30), "VP_ERR_SHAPE"),
    (dict(n_q_heads=68, n_kv_heads=4), "VP_ERR_UNSUPPORTED"),
    (dict(head_dim=96), "VP_ERR_UNSUPPORTED"),
    (dict(batch=0), "VP_ERR_SHAPE"),
    (dict(max_vis=0), "VP_ERR_SHAPE"),
    (dict(k_cap=0), "VP_ERR_SHAPE"),
    (dict(kv_stride_s=64), "VP_ERR_SHAPE"),
    (dict(kv_stride_s=130), "VP_ERR_SHAPE"),
    (dict(block_size=3), "VP_ERR_SHAPE"),
    (dict(block_size=-16), "VP_ERR_SHAPE"),
    (dict(block_size=1 << 17), "VP_ERR_SHAPE"),
    (dict(max_segs=1000), "VP_ERR_UNSUPPORTED"),
    (dict(scope=2), "VP_ERR_RANGE"),
    (dict(scope=-1), "VP_ERR_RANGE"),
    (dict(n_queries=-1), "VP_ERR_RANGE"),
    (dict(n_queries=1 << 30), "VP_ERR_UNSUPPORTED"),
    (dict(max_seq_len=(1 << 28) + 1), "VP_ERR_UNSUPPORTED"),
    (dict(max_vis=(1 << 28) + 1), "VP_ERR_UNSUPPORTED"),
    (dict(n_queries=3), "VP_ERR_UNSUPPORTED"),  # 3 queries x 7 heads > 16 rows per KV head
    (dict(n_queries=17, n_q_heads=4, n_kv_heads=4), "VP_ERR_UNSUPPORTED"),
    (dict(scope=1, batch=20000), "VP_ERR_UNSUPPORTED"),  # 80000 selection rows
])
def test_shape_validation(L, kw, status):
    with pytest.raises(vp.VPError) as e:
        vp.vp_workspace_size(_shape(**kw))
    assert status in str(e.value)


def test_kv_group_scope_sizes_the_arrival_counters(L):
    """One arrival counter per selection row: the workspace grows by at most a
    few 256-byte pieces, never by a per-token amount."""
    a = vp.vp_workspace_size(_shape(batch=64))
    b = vp.vp_workspace_size(_shape(batch=64, scope=vp.VP_SCOPE_KV_GROUP))
    assert a <= b <= a + 1024


def test_queries_scale_the_per_head_workspace(L):
    """T queries: per-head partials for T*Hq query rows; n_queries 0 and 1 agree."""
    one = vp.vp_workspace_size(_shape())
    assert vp.vp_workspace_size(_shape(n_queries=1)) == one
    two = vp.vp_workspace_size(_shape(n_queries=2))
    assert one < two < 2 * one + 4096


def _layout():
    return vp.vp_layout(seq_len=0x1000, vis_seg_off=0x2000, vis_seg=0x3000)


def test_calls_reject_nulls_and_bad_params_before_launch(L):
    s, lay, p = _shape(), _layout(), _params()
    ws_bytes = vp.vp_workspace_size(s)
    fake = 0x10000  # never dereferenced: every case below fails validation first
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_visual_mass(s, lay, p, None, fake, None, fake, fake, fake, fake, ws_bytes, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_WORKSPACE"):
        vp.vp_visual_mass(s, lay, p, fake, fake, None, fake, fake, fake, fake, ws_bytes - 1, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_WORKSPACE"):
        vp.vp_visual_mass(s, lay, p, fake, fake, None, fake, fake, fake, fake + 16, ws_bytes, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
        vp.vp_visual_mass(s, lay, _params(tau_mass=0.0), fake, fake, None, fake, fake, fake, fake, ws_bytes, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
        vp.vp_budget(s, lay, _params(r_hi_bp=20000), fake, fake, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_SHAPE"):
        vp.vp_budget(_shape(k_cap=10), lay, p, fake, fake, 0)  # 5% of 1296 needs 64 rows
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_select_topk(s, lay, fake, None, fake, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_select_topk(s, vp.vp_layout(seq_len=0x1000, vis_seg_off=None, vis_seg=0x3000), fake, fake, fake, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_validate_layout(s, vp.vp_layout(seq_len=None, vis_seg_off=0x2000, vis_seg=0x3000), 0)
    # paged caches need a block table
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_visual_mass(_shape(block_size=32), lay, p, fake, fake, None, fake, fake, fake, fake,
                          vp.vp_workspace_size(_shape(block_size=32)), 0)
    with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
        vp.vp_sparse_decode_attn(s, lay, p, fake, fake, fake, fake, fake, fake, 8, fake, ws_bytes, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_SHAPE"):
        vp.vp_sparse_decode_attn(s, lay, p, fake + 2, fake, fake, fake, fake, fake, 0, fake, ws_bytes, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
        vp.vp_visual_mass_timed(s, lay, p, fake, fake, None, fake, fake, fake, fake, ws_bytes, 0,
                                events=[None] * (vp.VP_MASS_EVENTS + 1))
    rc = L.vp_visual_mass_timed(ctypes.byref(s), ctypes.byref(lay), ctypes.byref(p), fake, fake, None, fake, fake,
                                fake, fake, ws_bytes, None, None, 2)
    assert L.vp_status_string(rc) == b"VP_ERR_NULL"
    assert "workspace" in L.vp_last_error().decode() or L.vp_last_error().decode() != ""


def test_decode_step_rejects_bad_arguments_before_launch(L):
    s, lay, p = _shape(), _layout(), _params()
    ws_bytes = vp.vp_workspace_size(s)
    fake = 0x10000  # never dereferenced: every case below fails validation first

    def step(shape=s, params=p, V=fake, out=fake, ws=fake, nbytes=ws_bytes, events=()):
        vp.vp_decode_step(shape, lay, params, fake, fake, V, fake, fake, fake, fake, fake, out, ws, nbytes, 0,
                          events=events)

    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        step(V=None)  # the step needs V (text attention is fused into the context pass)
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        step(out=None)
    with pytest.raises(vp.VPError, match="VP_ERR_WORKSPACE"):
        step(nbytes=ws_bytes - 1)
    with pytest.raises(vp.VPError, match="VP_ERR_WORKSPACE"):
        step(ws=fake + 16)
    with pytest.raises(vp.VPError, match="VP_ERR_SHAPE"):
        step(shape=_shape(k_cap=10))
    with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
        step(params=_params(tau_score=-1.0))
    with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
        step(events=[None] * (vp.VP_STEP_EVENTS + 1))
    with pytest.raises(vp.VPError, match="VP_ERR_DTYPE"):
        step(shape=_shape(dtype=9))


def test_top_p_rejects_bad_arguments(L):
    s, lay = _shape(), _layout()
    fake = 0x10000
    for p in (-0.1, 1.5, float("nan")):
        with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
            vp.vp_budget_top_p(s, lay, fake, p, fake, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_budget_top_p(s, lay, None, 0.1, fake, 0)


def test_event_array_is_reusable():
    arr, n = vp.event_array([None, None, None])
    assert n == 3 and len(arr) == 3
    assert vp.event_array((arr, n)) == (arr, n)
    assert vp.event_array(()) == (None, 0)


def test_header_constants_match_binding():
    text = open(HEADER).read()
    consts = dict(re.findall(r"#define\s+(VP_[A-Z_]+)\s+(\d+)", text))
    assert int(consts["VP_MASS_EVENTS"]) == vp.VP_MASS_EVENTS
    assert int(consts["VP_STEP_EVENTS"]) == vp.VP_STEP_EVENTS
    assert int(consts["VP_ATTN_TEXT_FROM_WORKSPACE"]) == vp.VP_ATTN_TEXT_FROM_WORKSPACE


def test_header_plan_flags_match_binding():
    text = open(HEADER).read()
    consts = dict(re.findall(r"#define\s+(VP_PLAN_[A-Z_]+)\s+(\d+)", text))
    assert {k: int(v) for k, v in consts.items()} == {
        "VP_PLAN_ONE_CONTEXT_LAUNCH": vp.VP_PLAN_ONE_CONTEXT_LAUNCH, "VP_PLAN_FUSED_TAIL": vp.VP_PLAN_FUSED_TAIL,
        "VP_PLAN_KEPT_IN_MERGE": vp.VP_PLAN_KEPT_IN_MERGE}


def _bench_shape(B, Hq, Hkv, S, n_vis, k_cap, **kw):
    return _shape(batch=B, n_q_heads=Hq, n_kv_heads=Hkv, max_seq_len=S, max_vis=n_vis, max_segs=4, k_cap=k_cap,
                  kv_stride_b=Hkv * S * 128, kv_stride_h=S * 128, **kw)


@pytest.mark.parametrize("name, shape_kw, want", [
    # 1 x 3358 tokens (1296 visual): one context launch, kept rows read in the merge
    ("7b-b1", dict(B=1, Hq=28, Hkv=4, S=3358, n_vis=1296, k_cap=64), 1 | 4),
    # 16 x up to 12288 tokens: one context launch, a kept pass of 448 work-groups
    ("7b-b16", dict(B=16, Hq=28, Hkv=4, S=12288, n_vis=4096, k_cap=204), 1),
    # 64 x 32768 tokens: visual and text passes in two launches, chunked selection
    ("7b-b64-32k", dict(B=64, Hq=28, Hkv=4, S=32768, n_vis=16384, k_cap=819), 0),
    # 8 x 11008 tokens of the 72B-class shape
    ("72b-b8", dict(B=8, Hq=64, Hkv=8, S=11008, n_vis=6400, k_cap=320), 1),
    # fp32 caches never read their kept rows in the merge
    ("7b-b1-f32", dict(B=1, Hq=28, Hkv=4, S=3358, n_vis=1296, k_cap=64, dtype=vp.VP_F32), 1),
    # a kept list longer than the merge holds in one batch
    ("7b-b1-long-list", dict(B=1, Hq=28, Hkv=4, S=3358, n_vis=1296, k_cap=96), 1),
])
def test_step_plan_of_the_benchmark_shapes(L, name, shape_kw, want):
    """vp_step_plan is pure host logic: the launch plans the benchmark shapes take."""
    assert vp.vp_step_plan(_bench_shape(**shape_kw), _params()) == want, name


def test_status_strings(L):
    assert vp.vp_status_string(0) == "VP_OK" and vp.vp_status_string(7) == "VP_ERR_HIP"


def _budget_rows():
    rows = []
    for line in open(os.path.join(GOLDEN, "budget_cases.txt")):
        line = line.split("#")[0].strip()
        if line:
            m, n, lo, hi, c, k = line.split()
            rows.append((float(m), int(n), int(lo), int(hi), int(c), int(k)))
    return rows


@pytest.mark.parametrize("m,n,lo,hi,c,k", _budget_rows())
def test_budget_host_mirror_matches_table(L, m, n, lo, hi, c, k):
    assert vp.vp_budget_host(m, n, _params(r_lo_bp=lo, r_hi_bp=hi, clamp=c)) == k


def test_budget_host_rejects_bad_params(L):
    assert vp.vp_budget_host(0.5, 100, _params(tau_mass=-1.0)) == -1


def test_stream_read_rejects_bad_arguments(L):
    fake = 0x10000
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_stream_read(None, 1 << 20, 0, fake, 0)
    with pytest.raises(vp.VPError, match="VP_ERR_SHAPE"):
        vp.vp_stream_read(fake, (1 << 20) + 16, 0, fake, 0)   # not a multiple of 16 KiB
    with pytest.raises(vp.VPError, match="VP_ERR_SHAPE"):
        vp.vp_stream_read(fake + 8, 1 << 20, 1, fake, 0)       # misaligned
    with pytest.raises(vp.VPError, match="VP_ERR_RANGE"):
        vp.vp_stream_read(fake, 1 << 20, 2, fake, 0)


def test_static_scratch_step_refuses_before_launch(L):
    """vp_decode_step_static checks its arguments, and that the shape's scratch
    fits the library's static array, before touching the GPU."""
    fake = 0x10000
    lay, p = _layout(), _params()
    big = _shape(batch=64, max_seq_len=32768, max_vis=16384, max_segs=4, k_cap=819,
                 kv_stride_b=4 * 32768 * 128, kv_stride_h=32768 * 128)
    assert vp.vp_workspace_size(big) > vp.VP_STATIC_SCRATCH_BYTES
    args = [fake] * 9
    with pytest.raises(vp.VPError, match="VP_ERR_WORKSPACE"):
        vp.vp_decode_step_static(big, lay, p, *args, stream=0)
    with pytest.raises(vp.VPError, match="VP_ERR_NULL"):
        vp.vp_decode_step_static(_shape(), lay, p, fake, fake, None, *([fake] * 6), stream=0)
    with pytest.raises(vp.VPError, match="VP_ERR_SHAPE"):
        vp.vp_decode_step_static(_shape(k_cap=10), lay, p, *args, stream=0)
    m = re.search(r"#define\s+VP_STATIC_SCRATCH_BYTES\s+\((\d+)u << (\d+)\)", open(HEADER).read())
    assert m and vp.VP_STATIC_SCRATCH_BYTES == int(m.group(1)) << int(m.group(2))
