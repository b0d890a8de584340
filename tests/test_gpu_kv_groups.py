"""Per-KV-group budgets and kept sets (VP_SCOPE_KV_GROUP) through the C ABI,
against the fp64 reference of the variant (each KV group solved as a sequence
of its own G query heads).

Bars as for the per-sequence path: masses and scores within 1e-5 relative,
budgets exact, kept sets bit-exact on planted inputs (every group's Eq. (3) cut
has a >= 1e-3 relative score gap and its Eq. (7) rounding a 1e-4 margin),
outputs within bf16 atol 2e-2 / rtol 1e-2 (fp32 1e-5). The one-launch step and
the four calls give bit-identical results.
"""
import numpy as np
import pytest

from _parity import assert_step_equals_calls, check_groups, kept_in_merge, small_workload
from oracle import plant as P
from oracle import vp_oracle as O
from paper_2605_31457_amd import step as S
from paper_2605_31457_amd import workloads as W

pytestmark = pytest.mark.gpu

KEYS = ("mass_head", "mass_seq", "scores", "k", "vis_idx", "out")


def _log(msg):
    print(msg, flush=True)


def _step_and_calls(w, **kw):
    """(step results, four-call results); asserts they are bit-identical."""
    ds = S.DeviceStep(w, kv_groups=True, **kw)
    ds.decode_step()
    g = ds.results()
    merged = kept_in_merge(ds)
    for fused in (True, False):
        ds.run(fused=fused)
        assert_step_equals_calls(g, ds.results(), fused, merged)
    return ds, g


def test_kv_groups_config2():
    w = W.generate(2)
    ref, log = P.plant_kv_groups(w, P.params_of(w))
    _log(f"cfg2 per-group: k={list(ref[0].k)}")
    _, g = _step_and_calls(w)
    check_groups("cfg2 groups", w, g, 0, ref[0])


def test_kv_groups_config3_ragged():
    """16 ragged sequences whose visual mass spans 0.01 .. 0.6: per-group
    budgets differ inside a sequence."""
    w = W.generate(3)
    ref, _ = P.plant_kv_groups(w, P.params_of(w))
    ks = np.array([ref[b].k for b in range(w.B)])
    _log(f"cfg3 per-group budgets: {ks.tolist()}")
    assert np.any(ks.max(axis=1) != ks.min(axis=1))  # the variant is not vacuous here
    _, g = _step_and_calls(w)
    for b in range(w.B):
        check_groups("cfg3 groups", w, g, b, ref[b])


def test_kv_groups_config5_shape():
    """Hq = 64, Hkv = 8 (G = 8) on two sequences of the decode-loop workload."""
    w = W.generate(5, seqs=[0, 1])
    ref, _ = P.plant_kv_groups(w, P.params_of(w))
    _, g = _step_and_calls(w)
    for b in range(w.B):
        check_groups("cfg5 groups", w, g, b, ref[b])


SMALL = {
    "mha-g1": dict(seed=21, B=2, Hq=8, Hkv=8, d=64, lens=[300, 257], segs=[[(10, 200)], [(0, 100), (150, 90)]]),
    "g16": dict(seed=22, B=2, Hq=32, Hkv=2, d=128, lens=[400, 96], segs=[[(40, 300)], [(1, 60)]]),
    "f32-ragged": dict(seed=23, dtype="f32", B=3, Hq=12, Hkv=3, d=64, lens=[1, 70, 513],
                       segs=[[], [(5, 50)], [(0, 64), (100, 300), (450, 40)]]),
    "unclamped": dict(seed=24, B=2, Hq=8, Hkv=2, d=128, lens=[640, 800], segs=[[(0, 512)], [(100, 600)]],
                      clamp=False, tau_mass=1.0),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_kv_groups_small_shapes(name):
    w = small_workload(**SMALL[name])
    ref, _ = P.plant_kv_groups(w, P.params_of(w))
    _log(f"{name}: k={[list(ref[b].k) for b in range(w.B)]}")
    _, g = _step_and_calls(w)
    for b in range(w.B):
        check_groups(name, w, g, b, ref[b])


def test_one_kv_head_groups_equal_the_sequence_path():
    """With one KV head the variant is the paper's path: bit-identical outputs."""
    w = small_workload(seed=25, B=2, Hq=8, Hkv=1, d=128, lens=[900, 700], segs=[[(50, 700)], [(0, 600)]])
    a = S.DeviceStep(w)
    a.decode_step()
    ra = a.results()
    b = S.DeviceStep(w, kv_groups=True)
    b.decode_step()
    rb = b.results()
    for key in KEYS:
        want = ra[key]
        got = rb[key].reshape(want.shape)
        assert np.array_equal(got, want), key


def test_kv_groups_paged_caches():
    w = W.generate(2)
    P.plant_kv_groups(w, P.params_of(w))
    flat = S.DeviceStep(w, kv_groups=True)
    flat.decode_step()
    paged = S.DeviceStep(w, kv_groups=True, block_size=32, block_seed=5)
    paged.decode_step()
    a, b = flat.results(), paged.results()
    for key in KEYS:
        assert np.array_equal(a[key], b[key]), key


def test_kv_groups_top_p_rows():
    """vp_budget_top_p per selection row on the GPU step's group scores."""
    w = W.generate(2)
    ref, _ = P.plant_kv_groups(w, P.params_of(w))
    ds, g = _step_and_calls(w)
    vis = O.visual_positions(int(w.seq_len[0]), w.segments[0])
    checked = 0
    for p in (0.1, 0.2, 0.3, 0.5):
        S.vp.vp_budget_top_p(ds.shape, ds.layout, ds.scores, p, ds.k)
        got = ds.k.cpu().numpy()
        for gi in range(w.Hkv):
            S64 = g["scores"][0, gi, :len(vis)].astype(np.float64)
            csum = np.cumsum(S64[np.lexsort((vis, -S64))])
            if np.min(np.abs(csum - p)) < 1e-7:
                continue  # too close to a prefix sum to be decided from fp32 scores
            assert int(got[gi]) == O.budget_top_p(S64, vis, p), (p, gi)
            checked += 1
    assert checked >= 12
