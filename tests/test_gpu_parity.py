"""GPU parity: the HIP path through the C ABI against the fp64 reference.

Bars: masses and scores within 1e-5 relative; budgets exact; kept index sets
bit-exact (inputs are planted so that the Eq. (3) cut has a >= 1e-3 relative
score gap and the Eq. (7) rounding has a 1e-4 relative margin); outputs within
bf16 atol 2e-2 / rtol 1e-2 (fp32: 1e-5 / 1e-5).
"""
import numpy as np
import pytest
import torch

from _parity import (ROUNDING_ATOL, ROUNDING_RTOL, assert_step_equals_calls, check_sequence, kept_in_merge,
                     small_workload, tile_batch)
from oracle import plant as P
from oracle import vp_oracle as O
from paper_2605_31457_amd import step as S
from paper_2605_31457_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)


def _run(w, fused=True, **kw):
    ds = S.DeviceStep(w, **kw)
    ds.run(fused=fused)
    return ds, ds.results()


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_config_full(cfg):
    w = W.generate(cfg)
    ref, log = P.plant(w, P.params_of(w))
    _log(f"cfg{cfg}: B={w.B} planted {sum(l['n_edits'] for l in log)} rows; k={[ref[b].k for b in range(w.B)]}")
    for fused in (True, False):
        _log(f"cfg{cfg}: GPU step fused={fused}")
        _, g = _run(w, fused=fused)
        for b in range(w.B):
            check_sequence(f"cfg{cfg} fused={fused}", w, g, b, ref[b])


def test_config4_full_batch():
    """The 64 x 32k multi-image batch at full size, in the benchmark's launch
    configuration. Four generated sequences are planted and checked by the
    reference; the batch repeats them, so every one of the 64 outputs is checked."""
    base = W.generate(4, seqs=[0, 1, 2, 3])
    ref, log = P.plant(base, P.params_of(base))
    w = tile_batch(base, 64)
    _log(f"cfg4: B=64 x 32768, planted {[l['n_edits'] for l in log]}")
    _, g = _run(w)
    for b in range(64):
        check_sequence("cfg4", w, g, b, ref[b % 4], b_src=b % 4)


SMALL = {
    "g4-d64-tails": dict(seed=1, B=3, Hq=8, Hkv=2, d=64, lens=[77, 200, 33],
                         segs=[[(5, 40)], [(0, 64), (100, 50)], [(1, 31)]]),
    "mha-d128": dict(seed=2, B=2, Hq=4, Hkv=4, d=128, lens=[129, 96], segs=[[(10, 100)], [(32, 32), (64, 16)]]),
    "g16-all-visual": dict(seed=3, B=2, Hq=16, Hkv=1, d=128, lens=[300, 257], segs=[[(20, 200)], [(0, 257)]]),
    "g7-many-segments": dict(seed=4, B=2, Hq=28, Hkv=4, d=128, lens=[500, 450],
                             segs=[[(3, 50), (60, 40), (101, 7), (200, 100), (320, 90)],
                                   [(10, 10), (20, 10), (30, 300)]]),
    "f32-d128": dict(seed=5, dtype="f32", B=2, Hq=6, Hkv=2, d=128, lens=[100, 70], segs=[[(0, 60)], [(30, 40)]]),
    "f32-d64-g4": dict(seed=9, dtype="f32", B=2, Hq=4, Hkv=1, d=64, lens=[200, 45], segs=[[(16, 150)], [(0, 40)]]),
    "no-visual": dict(seed=6, B=2, Hq=8, Hkv=2, d=64, lens=[90, 40], segs=[[], [(0, 20)]]),
    "unclamped-tau1": dict(seed=7, B=2, Hq=8, Hkv=2, d=128, lens=[150, 150], segs=[[(10, 100)], [(10, 100)]],
                           tau_mass=1.0, clamp=False),
    "short-seqs": dict(seed=8, B=3, Hq=4, Hkv=1, d=64, lens=[1, 5, 31], segs=[[], [(1, 3)], [(0, 31)]]),
    "capacity-gt-len": dict(seed=10, B=2, Hq=8, Hkv=1, d=128, lens=[70, 130], segs=[[(2, 60)], [(64, 64)]],
                            S_cap=200),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_shapes(name):
    w = small_workload(**SMALL[name])
    ref, _ = P.plant(w, P.params_of(w))
    _log(f"small {name}: k={[ref[b].k for b in range(w.B)]} lens={list(w.seq_len)}")
    for fused in (True, False):
        _, g = _run(w, fused=fused)
        for b in range(w.B):
            check_sequence(f"{name} fused={fused}", w, g, b, ref[b])
    _step_equals_calls(w, g, fused=False)


def _step_equals_calls(w, calls, ds=None, fused=True, **kw):
    """vp_decode_step gives what the four calls give (the same arithmetic and
    reduction order: bit for bit when the calls took the text part from the
    workspace), and so passes the same reference checks."""
    ds = ds or S.DeviceStep(w, **kw)
    ds.decode_step()
    g = ds.results()
    assert_step_equals_calls(g, calls, fused, kept_in_merge(ds))
    return g


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_decode_step_config(cfg):
    w = W.generate(cfg)
    ref, _ = P.plant(w, P.params_of(w))
    _, calls = _run(w)
    g = _step_equals_calls(w, calls)
    for b in range(w.B):
        check_sequence(f"step cfg{cfg}", w, g, b, ref[b])


def test_decode_step_config4_full_batch():
    base = W.generate(4, seqs=[0, 1, 2, 3])
    ref, _ = P.plant(base, P.params_of(base))
    w = tile_batch(base, 64)
    _log("cfg4 decode step: B=64 x 32768")
    ds, calls = _run(w)
    g = _step_equals_calls(w, calls, ds=ds)
    for b in range(64):
        check_sequence("step cfg4", w, g, b, ref[b % 4], b_src=b % 4)


def test_decode_step_many_visual_tokens():
    """40000 visual tokens in one sequence: more keys than one work-group's LDS
    holds, so the step takes the separate kernels and the top-k reads its keys
    from memory."""
    w = small_workload(seed=16, B=1, Hq=4, Hkv=1, d=64, lens=[41000], segs=[[(500, 40000)]])
    ref, _ = P.plant(w, P.params_of(w))
    _log(f"40k visual: k={ref[0].k}")
    _, calls = _run(w)
    check_sequence("40k calls", w, calls, 0, ref[0])
    g = _step_equals_calls(w, calls)
    check_sequence("40k step", w, g, 0, ref[0])


def test_fused_and_unfused_text_paths_agree():
    """The text attention computed inside the mass pass (fused) and by the
    attention call itself (unfused) are separately compiled kernels: discrete
    results are identical, real ones agree to a few fp32 ulps (bf16 output to
    one bf16 ulp). Where the fused path reads the kept rows in the merge, its
    output differs from the kept pass's by that pass's bf16 probabilities."""
    w = W.generate(2)
    ds, a = _run(w, fused=True)
    _, b = _run(w, fused=False)
    for key in ("k", "vis_idx"):
        assert np.array_equal(a[key], b[key]), key
    for key in ("mass_head", "mass_seq", "scores"):
        np.testing.assert_allclose(a[key], b[key], rtol=4e-6, atol=1e-30, err_msg=key)
    if kept_in_merge(ds):
        np.testing.assert_allclose(a["out"], b["out"], rtol=ROUNDING_RTOL, atol=ROUNDING_ATOL)
    else:
        np.testing.assert_allclose(a["out"], b["out"], rtol=8e-3, atol=1e-6)


def test_repeat_runs_are_bitwise_identical():
    w = W.generate(3, B=4)
    ds = S.DeviceStep(w)
    ds.run()
    first = ds.results()
    for _ in range(3):
        ds.run()
        again = ds.results()
        for key in first:
            assert np.array_equal(first[key], again[key]), key


def _repeat_case(name):
    if name == "cfg4-chunked-select":
        # 64 rows of 16384 visual ranks: the select launch scores each row in
        # chunks on several work-groups and the last to arrive selects
        return tile_batch(W.generate(4, seqs=[0, 1, 2, 3]), 64)
    if name == "many-chunks-keys-in-memory":
        # one row of 40000 visual ranks: many chunks, and the selecting
        # work-group reads the keys back from memory (more than its LDS holds)
        return small_workload(seed=16, B=1, Hq=4, Hkv=1, d=64, lens=[41000], segs=[[(500, 40000)]])
    # 256 rows: one work-group per row, keys beyond its LDS read from memory
    base = small_workload(seed=66, B=2, Hq=4, Hkv=1, d=64, lens=[40200, 300], segs=[[(100, 40000)], [(20, 200)]])
    return tile_batch(base, 256)


@pytest.mark.parametrize("name", ["cfg4-chunked-select", "many-chunks-keys-in-memory", "one-group-keys-in-memory"])
def test_repeat_decode_steps_are_bitwise_identical(name):
    """vp_decode_step's select launch hands scores between work-groups through
    device-scope stores and an arrival counter; repeated steps on the same
    inputs must give the same bits every time."""
    w = _repeat_case(name)
    ds = S.DeviceStep(w, max_vis=40000 if name == "one-group-keys-in-memory" else None)
    ds.decode_step()
    first = ds.results()
    for rep in range(4):
        ds.decode_step()
        again = ds.results()
        for key in first:
            assert np.array_equal(first[key], again[key]), f"{name} repeat {rep}: {key}"
    _log(f"repeat {name}: k={list(first['k'][:4])}")


def test_budget_kernel_matches_rule_exactly():
    """vp_budget on given fp32 masses, including products that land exactly on
    an integer, against Eq. (7) + clamp on the same fp32 values widened."""
    n_vis = [256, 1296, 4096, 6400, 16384, 1, 0, 100]
    lens = [max(n, 1) + 10 for n in n_vis]
    segs = [[(5, n)] if n else [] for n in n_vis]
    w = small_workload(seed=11, B=len(n_vis), Hq=4, Hkv=1, d=64, lens=lens, segs=segs, spike=0)
    rng = np.random.default_rng(12)
    for clamp in (True, False):
        w.clamp = clamp
        ds = S.DeviceStep(w, k_cap=max(n_vis))
        for trial in range(20):
            if trial == 0:
                m = np.array([0.5, 0.25, 0.0, 1.0, 0.0625, 0.3, 0.7, 0.125], np.float32)  # exact products
            elif trial == 1:
                m = np.array([0.01, 0.05, 0.02, 0.03, 0.05, 0.01, 1.0, 0.5], np.float32)  # clamp edges
            else:
                m = rng.random(len(n_vis)).astype(np.float32) ** 3
            ms = np.stack([m, m], axis=1)
            ds.mass_seq.copy_(torch.from_numpy(ms))
            ds.budget()
            got = ds.k.cpu().numpy()
            want = [O.budget(float(m[b]), n_vis[b], w.r_lo_bp, w.r_hi_bp, clamp) for b in range(len(n_vis))]
            assert list(got) == want, (clamp, m, got, want)


def test_topk_kernel_matches_sort_with_ties():
    """vp_select_topk on given fp32 scores (many exact ties) against the
    reference selection on the same values: ties go to the lower position."""
    rng = np.random.default_rng(13)
    n_vis = [16384, 4096, 1296, 37, 1, 300]
    segs = [[(16 + 8188 * i, 4096) for i in range(4)], [(0, 4096)], [(14, 1296)], [(3, 10), (20, 27)],
            [(0, 1)], [(0, 100), (150, 100), (300, 100)]]
    lens = [32768, 5000, 3358, 50, 1, 400]
    w = small_workload(seed=14, B=6, Hq=4, Hkv=1, d=64, lens=lens, segs=segs, spike=0)
    ds = S.DeviceStep(w, k_cap=1000, max_vis=16384)
    for trial in range(6):
        sc = np.zeros((6, 16384), np.float32)
        for b, n in enumerate(n_vis):
            if trial % 3 == 0:
                sc[b, :n] = rng.random(n).astype(np.float32)
            elif trial % 3 == 1:
                sc[b, :n] = (np.floor(rng.random(n) * 16) / 16).astype(np.float32)  # heavy ties
            else:
                sc[b, :n] = np.float32(1.0 / 7.0)                                   # all equal
        ks = [rng.integers(0, min(n, 1000) + 1) for n in n_vis]
        ks[0] = 819 if trial < 3 else 1000
        ds.scores.copy_(torch.from_numpy(sc))
        ds.k.copy_(torch.tensor(ks, dtype=torch.int32))
        ds.select_topk()
        got = ds.vis_idx.cpu().numpy()
        for b, n in enumerate(n_vis):
            vis = O.visual_positions(lens[b], segs[b])
            k = min(ks[b], n, 1000)
            want = O.select_top_k(sc[b, :n].astype(np.float64), vis, k)
            assert np.array_equal(got[b, :k], want), (trial, b)
            assert np.all(got[b, k:] == -1)


def test_sparse_attention_on_given_selection():
    """vp_sparse_decode_attn alone, on the reference's own selection, against
    the reference pruned attention (also with k = N_v: dense attention)."""
    w = W.generate(2)
    p = P.params_of(w)
    r = O.decode_step_sequence(w.q[0], w.K[0], w.V[0], int(w.seq_len[0]), w.segments[0], p)
    ds = S.DeviceStep(w, k_cap=1296)
    for k_use, sel in ((r.k, r.vis_idx), (1296, O.visual_positions(3358, w.segments[0]))):
        idx = np.full((1, 1296), -1, np.int32)
        idx[0, :k_use] = sel
        ds.vis_idx.copy_(torch.from_numpy(idx))
        ds.k.copy_(torch.tensor([k_use], dtype=torch.int32))
        ds.sparse_decode_attn(fused=False)
        got = ds.out.float().cpu().numpy()[0]
        rr = O.decode_step_sequence(w.q[0], w.K[0], w.V[0], 3358, w.segments[0], p, k_override=k_use)
        assert np.array_equal(rr.vis_idx, sel)
        np.testing.assert_allclose(got, rr.out, atol=2e-2, rtol=1e-2)


def test_kept_list_entries_that_are_skipped():
    """vp_sparse_decode_attn with the text part from the workspace, on a kept list
    holding -1, positions at or past the sequence length and entries past the
    budget among real kept positions: the skipped entries add nothing, on the
    launch plan of this shape (the kept rows read in the merge at the 1-sequence
    batch, a kept pass otherwise), against the reference attention over the rest."""
    for cfg, B in ((2, None), (3, 4)):
        w = W.generate(cfg, B=B) if B else W.generate(cfg)
        ds = S.DeviceStep(w)
        ds.visual_mass(fused=True)
        G = w.Hq // w.Hkv
        sm = 1.0 / np.sqrt(w.d)
        kc = ds.k_cap
        idx = np.full((w.B, kc), -1, np.int32)
        k = np.zeros(w.B, np.int32)
        want = []
        for b in range(w.B):
            L = int(w.seq_len[b])
            vis = O.visual_positions(L, w.segments[b])
            rng = np.random.default_rng(40 + b)
            take = np.sort(rng.choice(vis, size=min(len(vis), kc // 2), replace=False)).astype(np.int32)
            row = list(take[: len(take) // 2]) + [-1, L, L + 5] + list(take[len(take) // 2:])
            k[b] = min(kc - 2, len(row))
            row = row[: k[b]] + [int(take[0]), int(take[1])]  # entries past the budget: ignored
            idx[b, : len(row)] = row
            kept = np.array([x for x in row[: k[b]] if 0 <= x < L], np.int64)
            J = np.sort(np.concatenate([kept, O.text_positions(L, w.segments[b])]))
            qf = O.as_f64(w.q[b])
            want.append(np.stack([O.pruned_attention(qf[h], w.K[b, h // G], w.V[b, h // G], J, sm)
                                  for h in range(w.Hq)]))
        ds.vis_idx.copy_(torch.from_numpy(idx))
        ds.k.copy_(torch.from_numpy(k))
        ds.sparse_decode_attn(fused=True)
        got = ds.results()["out"]
        plan = S.vp.vp_step_plan(ds.shape, ds.params)
        for b in range(w.B):
            np.testing.assert_allclose(got[b], want[b], atol=2e-2, rtol=1e-2,
                                       err_msg=f"config {cfg} seq {b} (plan flags {plan})")


def _clip_layout(L, segs):
    """The documented reading of an unclean device layout: segments are taken in
    order, each clipped to [end of the previous one, L); lengths < 0 count as 0."""
    out, prev = [], 0
    for a, n in segs:
        lo = max(a, prev)
        lo = 0 if lo < 0 else min(lo, L)
        hi = a + max(n, 0)
        hi = lo if hi < lo else min(hi, L)
        if hi > lo:
            out.append((lo, hi - lo))
        prev = hi
    return out


def test_unclean_device_layout_is_clipped():
    """Overlapping, unsorted, empty, negative and overrunning segments and a
    length beyond capacity give exactly the results of the clipped layout."""
    S_cap = 256
    raw_lens = [300, 200]
    raw_segs = [[(-5, 20), (10, 30), (35, 0), (30, 50), (250, 100)], [(150, -3), (100, 60), (40, 20)]]
    lens = [min(n, S_cap) for n in raw_lens]
    segs = [_clip_layout(L, s) for L, s in zip(lens, raw_segs)]
    assert segs == [[(0, 15), (15, 25), (40, 40), (250, 6)], [(150, 10)]]
    w = small_workload(seed=15, B=2, Hq=8, Hkv=2, d=64, lens=lens, segs=segs, S_cap=S_cap)
    ref, _ = P.plant(w, P.params_of(w))
    ds = S.DeviceStep(w)
    off, seg = W.layout_arrays(raw_segs)
    ds.seq_len = torch.tensor(raw_lens, dtype=torch.int32, device=ds.device)
    ds.seg_off = torch.from_numpy(off).to(ds.device)
    ds.seg = torch.from_numpy(seg.reshape(-1)).to(ds.device)
    ds.layout = S.vp.vp_layout(seq_len=ds.seq_len.data_ptr(), vis_seg_off=ds.seg_off.data_ptr(),
                               vis_seg=ds.seg.data_ptr())
    ds.shape.max_segs = 5
    _log(f"clipped layout: n_vis={[sum(n for _, n in s) for s in segs]} k={[ref[b].k for b in range(2)]}")
    for fused in (True, False):
        ds.run(fused=fused)
        g = ds.results()
        for b in range(2):
            check_sequence(f"clipped fused={fused}", w, g, b, ref[b])


def test_zero_length_sequence_in_a_batch():
    """A sequence of length 0 between two others gets the empty context's
    results (masses 0, budget 0, no kept rows, output 0) from the four calls and
    from the step alike; its neighbours still match the reference, and the step
    equals the four calls (bit for bit but for the attention output of a step
    that reads its kept rows in the merge). Every context-pass part and kept split of
    the empty sequence writes an empty partial, which the merge reads."""
    w = small_workload(seed=21, B=3, Hq=8, Hkv=2, d=64, lens=[120, 40, 90], segs=[[(10, 60)], [(0, 20)], [(0, 40)]])
    ref, _ = P.plant(w, P.params_of(w))
    ds = S.DeviceStep(w)
    ds.seq_len[1] = 0
    got = {}
    for fused in (True, False):
        ds.scores.fill_(-1.0)
        ds.out.fill_(7.0)
        ds.run(fused=fused)
        got[fused] = g = ds.results()
        for b in (0, 2):
            check_sequence(f"zero-length neighbour fused={fused}", w, g, b, ref[b])
        assert np.all(g["mass_head"][1] == 0.0) and np.all(g["mass_seq"][1] == 0.0)
        assert int(g["k"][1]) == 0 and np.all(g["vis_idx"][1] == -1)
        assert np.all(g["scores"][1] == -1.0), "no visual rank: no score is written"
        assert np.all(g["out"][1].astype(np.float32) == 0.0)
    ds.out.fill_(7.0)
    ds.decode_step()
    g = ds.results()
    assert_step_equals_calls(g, got[False], False, kept_in_merge(ds), "zero-length batch")
    assert np.all(g["out"][1].astype(np.float32) == 0.0)


PRESETS = {
    # the 10% retention preset: tau = 0.4, clamp (0.05 N, 0.10 N)
    "retain10": dict(tau_mass=0.4, r_lo_bp=500, r_hi_bp=1000),
    # fixed-ratio budgets: r_lo = r_hi = r gives k = ceil(r N_v)
    "fixed1pct": dict(r_lo_bp=100, r_hi_bp=100),
    "fixed5pct": dict(r_lo_bp=500, r_hi_bp=500),
    # scores at the mass temperature (reading A3's variant)
    "tau_score_0.1": dict(tau_score=0.1),
}


@pytest.mark.parametrize("preset", sorted(PRESETS))
def test_budget_presets(preset):
    """Budget and estimator presets are parameters of the same kernels: the
    10% setting, fixed ratios and tempered scores, on four config-3 sequences."""
    w = W.generate(3, B=4)
    for key, val in PRESETS[preset].items():
        setattr(w, key, val)
    ref, _ = P.plant(w, P.params_of(w))
    _log(f"preset {preset}: k={[ref[b].k for b in range(w.B)]}")
    ds, calls = _run(w)
    for b in range(w.B):
        check_sequence(f"{preset}", w, calls, b, ref[b])
    _step_equals_calls(w, calls, ds=ds)


def test_later_layers_reuse_the_anchor_selection():
    """Layers after the anchor attend over the anchor's kept set on their own KV
    (Sec. 4.1): vp_sparse_decode_attn reading the text part itself, on two other
    layers' caches and queries, against the reference attention over the same
    context. A layout with no visual segments and k = 0 gives dense attention."""
    w = W.generate(2)
    ref, _ = P.plant(w, P.params_of(w))
    ds, g = _run(w)
    check_sequence("anchor", w, g, 0, ref[0])
    sel = g["vis_idx"][0, :int(g["k"][0])]
    for seed in (21, 22):
        wl = W.generate(2, seed=seed)  # another layer: same layout, its own q, K, V
        dl = S.DeviceStep(wl)
        dl.vis_idx.copy_(ds.vis_idx)
        dl.k.copy_(ds.k)
        dl.sparse_decode_attn(fused=False)
        got = dl.results()["out"][0]
        L = int(wl.seq_len[0])
        J = np.sort(np.concatenate([sel, O.text_positions(L, wl.segments[0])]))
        qf = O.as_f64(wl.q[0])
        G = wl.Hq // wl.Hkv
        sm = 1.0 / np.sqrt(wl.d)
        want = np.stack([O.pruned_attention(qf[h], wl.K[0, h // G], wl.V[0, h // G], J, sm) for h in range(wl.Hq)])
        np.testing.assert_allclose(got, want, atol=2e-2, rtol=1e-2, err_msg=f"layer seed {seed}")
        # dense: every cached row attended
        seg_off0 = torch.zeros(2, dtype=torch.int32, device=dl.device)
        seg0 = torch.zeros(2, dtype=torch.int32, device=dl.device)
        dl.layout = S.vp.vp_layout(seq_len=dl.seq_len.data_ptr(), vis_seg_off=seg_off0.data_ptr(),
                                   vis_seg=seg0.data_ptr())
        dl.k.zero_()
        dl.sparse_decode_attn(fused=False)
        got = dl.results()["out"][0]
        J = np.arange(L)
        want = np.stack([O.pruned_attention(qf[h], wl.K[0, h // G], wl.V[0, h // G], J, sm) for h in range(wl.Hq)])
        np.testing.assert_allclose(got, want, atol=2e-2, rtol=1e-2, err_msg=f"dense layer seed {seed}")


def test_later_layer_at_the_64x32k_batch():
    """A later layer at the 64 x 32k batch, where the text and kept passes do not
    fit one resident round together and run as two launches: its outputs against
    the reference attention over the anchor's kept set and the layer's own text
    rows, for the four source sequences and copies of them at the far end of the
    batch."""
    base = W.generate(4, seqs=[0, 1, 2, 3])
    P.plant(base, P.params_of(base))
    w = tile_batch(base, 64)
    ds = S.DeviceStep(w)
    ds.decode_step()
    g = ds.results()
    other = W.generate(4, seqs=[0, 1, 2, 3], seed=33)  # another layer: same layout, its own q, K, V
    wl = tile_batch(other, 64)
    dl = S.DeviceStep(wl)
    dl.vis_idx.copy_(ds.vis_idx)
    dl.k.copy_(ds.k)
    dl.sparse_decode_attn(fused=False)
    got = dl.results()["out"]
    G = wl.Hq // wl.Hkv
    sm = 1.0 / np.sqrt(wl.d)
    for b in (0, 1, 2, 3, 61, 62, 63):
        sel = g["vis_idx"][b, :int(g["k"][b])]
        L = int(wl.seq_len[b])
        J = np.sort(np.concatenate([sel, O.text_positions(L, wl.segments[b])]))
        qf = O.as_f64(wl.q[b])
        want = np.stack([O.pruned_attention(qf[h], wl.K[b, h // G], wl.V[b, h // G], J, sm) for h in range(wl.Hq)])
        np.testing.assert_allclose(got[b], want, atol=2e-2, rtol=1e-2, err_msg=f"later layer, sequence {b}")
    _log("later layer at 64 x 32k: 7 sequences match the reference")


def _prefix_margin(S, vis, p):
    """Distance from p to the nearest prefix sum of S in the Eq. (3) order."""
    csum = np.cumsum(S[np.lexsort((vis, -S))])
    return np.min(np.abs(csum - p)) if len(csum) else np.inf


def test_top_p_budget_kernel():
    """vp_budget_top_p on given fp32 scores (random, tied, dyadic, all equal,
    empty) against the reference Top-p budget on the same values; every p is
    kept at least 1e-7 from any prefix sum (the kernel's fixed-point sums are
    exact to n * 2^-40)."""
    rng = np.random.default_rng(19)
    n_vis = [16384, 4096, 1296, 37, 1, 300, 0]
    segs = [[(16 + 8188 * i, 4096) for i in range(4)], [(0, 4096)], [(14, 1296)], [(3, 10), (20, 27)],
            [(0, 1)], [(0, 100), (150, 100), (300, 100)], []]
    lens = [32768, 5000, 3358, 50, 1, 400, 64]
    w = small_workload(seed=20, B=7, Hq=4, Hkv=1, d=64, lens=lens, segs=segs, spike=0)
    ds = S.DeviceStep(w, k_cap=1000, max_vis=16384)
    checked = 0
    for trial in range(8):
        sc = np.zeros((7, 16384), np.float32)
        for b, n in enumerate(n_vis):
            if trial % 4 == 0:
                x = rng.random(n) ** 3
            elif trial % 4 == 1:
                x = np.floor(rng.random(n) * 8) + 1          # heavy ties
            elif trial % 4 == 2:
                x = np.ones(n)                                 # all equal
            else:
                x = rng.exponential(size=n)
            sc[b, :n] = (x / max(x.sum(), 1e-30) * rng.uniform(0.3, 1.0)).astype(np.float32)
        ds.scores.copy_(torch.from_numpy(sc))
        for p in (0.0, 0.1, 0.37, 0.9, 1.0):
            want = []
            for b, n in enumerate(n_vis):
                vis = O.visual_positions(lens[b], segs[b])
                S64 = sc[b, :n].astype(np.float64)
                if p > 0 and _prefix_margin(S64, vis, p) < 1e-7:
                    want.append(None)      # too close to a prefix sum to be decided in fp32 input
                else:
                    want.append(O.budget_top_p(S64, vis, p))
            S.vp.vp_budget_top_p(ds.shape, ds.layout, ds.scores, p, ds.k)
            got = ds.k.cpu().numpy()
            for b, wv in enumerate(want):
                if wv is not None:
                    assert int(got[b]) == wv, (trial, p, b, int(got[b]), wv)
                    checked += 1
    _log(f"top-p: {checked} budgets checked")
    assert checked > 200


def test_top_p_step_selects_the_reference_set():
    """Scores from the GPU step, the Top-p budget, then the selection: the set
    equals the reference's Top-p selection on the reference scores."""
    w = W.generate(2)
    ref, _ = P.plant(w, P.params_of(w))
    ds, g = _run(w)
    r = ref[0]
    vis = O.visual_positions(int(w.seq_len[0]), w.segments[0])
    ds_k = S.DeviceStep(w, k_cap=len(vis))
    ds_k.scores.copy_(ds.scores)
    checked = 0
    for p in (0.05, 0.1, 0.2, 0.3):
        if _prefix_margin(r.scores, vis, p) < 1e-5:
            continue
        checked += 1
        kp = O.budget_top_p(r.scores, vis, p)
        S.vp.vp_budget_top_p(ds_k.shape, ds_k.layout, ds_k.scores, p, ds_k.k)
        assert int(ds_k.k.cpu()[0]) == kp, p
        ds_k.select_topk()
        idx = ds_k.vis_idx.cpu().numpy()[0]
        want = O.select_top_k(r.scores, vis, kp)
        # the planted gap sits at the Eq. (7) cut; elsewhere compare within rounding
        got = idx[:kp]
        if not np.array_equal(got, want):
            order = np.lexsort((vis, -r.scores))
            cut = r.scores[order[kp - 1]]
            diff = np.setxor1d(got, want)
            assert np.all(np.abs(r.scores[np.searchsorted(vis, diff)] - cut) <= 2e-5 * cut), p
    assert checked >= 2
