"""Planting makes the reference's discrete decisions robust (no GPU)."""
import numpy as np

from oracle import plant as P
from oracle import vp_oracle as O
from paper_2605_31457_amd import workloads as W


def test_plant_cfg2_gap_and_margin():
    w = W.generate(2)
    p = P.params_of(w)
    res, log = P.plant(w, p)
    r = res[0]
    vis = O.visual_positions(int(w.seq_len[0]), w.segments[0])
    assert P.boundary_gap(r.scores, vis, r.k) >= P.GAP
    assert P.margin_ok(r.M_vis_max, len(vis), p)
    # the stored tensor is what the reference read
    r2 = O.decode_step_sequence(w.q[0], w.K[0], w.V[0], int(w.seq_len[0]), w.segments[0], p)
    assert list(r2.vis_idx) == list(r.vis_idx) and r2.k == r.k


def test_plant_creates_a_gap_where_there_was_none():
    w = W.generate(4, seqs=[0])
    p = P.params_of(w)
    vis = O.visual_positions(int(w.seq_len[0]), w.segments[0])
    r0 = O.decode_step_sequence(w.q[0], w.K[0], w.V[0], int(w.seq_len[0]), w.segments[0], p)
    before = P.boundary_gap(r0.scores, vis, r0.k)
    res, log = P.plant(w, p)
    after = P.boundary_gap(res[0].scores, vis, res[0].k)
    assert after >= P.GAP
    assert before < P.GAP and log[0]["n_edits"] > 0   # this seed needs planting
    assert res[0].k == 819


def test_margin_detects_integer_crossing():
    p = O.OracleParams(clamp=False)
    assert not P.margin_ok(0.5, 256, p)          # 128 exactly: 127.99 vs 128.01
    assert P.margin_ok(0.502, 256, p)


def test_plant_kv_groups_cfg2():
    """Per-KV-group planting: every group's budget margin and score gap hold, and
    the stored tensor is what the reference read."""
    w = W.generate(2)
    p = P.params_of(w)
    res, log = P.plant_kv_groups(w, p)
    r = res[0]
    L = int(w.seq_len[0])
    vis = O.visual_positions(L, w.segments[0])
    assert len(log) == w.Hkv
    for g in range(w.Hkv):
        assert P.boundary_gap(r.scores[g], vis, int(r.k[g])) >= P.GAP
        assert P.margin_ok(r.M_vis_max[g], len(vis), p)
    r2 = O.decode_step_sequence_kv_groups(w.q[0], w.K[0], w.V[0], L, w.segments[0], p, with_output=False)
    assert list(r2.k) == list(r.k)
    assert all(list(a) == list(b) for a, b in zip(r2.vis_idx, r.vis_idx))


def test_plant_queries_cfg2_two_queries():
    """Two queries per sequence: both hold margin and gap at once after planting,
    and each query's reference sees its own prefix."""
    w = W.with_queries(W.generate(2), 2)
    p = P.params_of(w)
    res, ok = P.plant_queries(w, p)
    assert ok[0]
    L = int(w.seq_len[0])
    segs = O.clip_segments(w.segments[0], L - 1)
    vis = O.visual_positions(L - 1, segs)
    for t, r in enumerate(res[0]):
        assert P.margin_ok(r.M_vis_max, len(vis), p)
        assert P.boundary_gap(r.scores, vis, r.k) >= P.GAP
        r2 = O.decode_step_sequence(w.q[0, t], w.K[0], w.V[0], L - 1 + t, segs, p, with_output=False)
        assert r2.k == r.k and list(r2.vis_idx) == list(r.vis_idx)


def test_plant_loop_steps_of_the_72b_decode_loop():
    """Per-step planting of the decode loop (a few steps past the point where the
    drifting query has flattened the scores, so the cut needs planting): after
    each step's planting the reference shows the gap and the margin, the float64
    copy equals the stored rows, and the returned result is what a fresh
    reference evaluation of the stored cache gives."""
    s = W.Cfg5Stream(B=2, steps=48)
    w = s.w
    p = P.params_of(w)
    Kf = [O.as_f64(w.K[b]) for b in range(w.B)]
    Vf = [O.as_f64(w.V[b]) for b in range(w.B)]
    edited = 0
    for t in range(48):
        q, kr, vr, pos = s.step_inputs(t)
        w.K[:, :, pos] = kr
        w.V[:, :, pos] = vr
        for b in range(w.B):
            Kf[b][:, pos] = O.as_f64(kr[b])
            Vf[b][:, pos] = O.as_f64(vr[b])
        if t < 40:
            continue
        for b in range(w.B):
            edits, r = P.plant_loop_step(q[b], w.K[b], Kf[b], w.V[b], Vf[b], pos + 1, w.segments[b], p)
            edited += len(edits)
            vis = O.visual_positions(pos + 1, w.segments[b])
            assert P.boundary_gap(r.scores, vis, r.k) >= P.GAP
            assert P.margin_ok(r.M_vis_max, len(vis), p)
            assert np.array_equal(Kf[b], O.as_f64(w.K[b]))
            fresh = O.decode_step_sequence(q[b], w.K[b], w.V[b], pos + 1, w.segments[b], p)
            assert fresh.k == r.k and np.array_equal(fresh.vis_idx, r.vis_idx)
            np.testing.assert_allclose(fresh.scores, r.scores, rtol=1e-12)
            np.testing.assert_allclose(fresh.out, r.out, rtol=1e-12, atol=1e-15)
    assert edited > 0  # the loop needs planting by then
