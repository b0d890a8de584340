"""Several queries per sequence (n_queries = T, speculative / multi-token
decoding) through the C ABI, against the fp64 reference: query t is a decode
step of its own over the positions before L - T + 1 + t, with the visual
segments cut at L - T + 1. The K/V rows are read once for all T queries (the
T*G query rows of a KV head share the matrix-core tile).

Bars as for one query: masses and scores within 1e-5 relative, budgets exact,
kept sets bit-exact on inputs planted so that every query holds its score gap
and budget margin at once, outputs within bf16 atol 2e-2 / rtol 1e-2 (fp32
1e-5). The one-launch step and the four calls are bit-identical.
"""
import numpy as np
import pytest

from _parity import assert_step_equals_calls, check_groups, check_sequence, kept_in_merge, small_workload
from oracle import plant as P
from paper_2605_31457_amd import step as S
from paper_2605_31457_amd import workloads as W

pytestmark = pytest.mark.gpu

KEYS = ("mass_head", "mass_seq", "scores", "k", "vis_idx", "out")


def _log(msg):
    print(msg, flush=True)


def _step_and_calls(w, **kw):
    ds = S.DeviceStep(w, **kw)
    ds.decode_step()
    g = ds.results()
    merged = kept_in_merge(ds)
    for fused in (True, False):
        ds.run(fused=fused)
        assert_step_equals_calls(g, ds.results(), fused, merged)
    return ds, g


def _query_view(g, b, t):
    """The results of query t of sequence b as a one-sequence result dict."""
    return {key: g[key][b, t][None] for key in KEYS}


def _check_all(tag, w, g, ref, ok, kv_groups=False):
    T = w.q.shape[1]
    for b in range(w.B):
        assert ok[b], f"{tag}: planting did not hold for sequence {b}"
        for t in range(T):
            check = check_groups if kv_groups else check_sequence
            check(f"{tag} query {t}", w, _query_view(g, b, t), 0, ref[b][t])


@pytest.mark.parametrize("T", [2])
def test_queries_config2(T):
    w = W.with_queries(W.generate(2), T)
    ref, ok = P.plant_queries(w, P.params_of(w))
    _log(f"cfg2 T={T}: k={[r.k for r in ref[0]]}")
    _, g = _step_and_calls(w)
    _check_all(f"cfg2 T={T}", w, g, ref, ok)


def test_queries_config3_ragged():
    w = W.with_queries(W.generate(3), 2)
    ref, ok = P.plant_queries(w, P.params_of(w))
    _, g = _step_and_calls(w)
    _check_all("cfg3 T=2", w, g, ref, ok)


def test_queries_config5_shape():
    """G = 8 and two queries: the 16 query rows of a KV head fill the tile."""
    w = W.with_queries(W.generate(5, seqs=[0, 1]), 2)
    ref, ok = P.plant_queries(w, P.params_of(w))
    _, g = _step_and_calls(w)
    _check_all("cfg5 T=2", w, g, ref, ok)


SMALL = {
    # (workload spec, T)
    "mha-16-queries": (dict(seed=31, B=2, Hq=4, Hkv=4, d=64, lens=[300, 150], segs=[[(10, 200)], [(0, 100)]]), 16),
    "g4-4-queries-f32": (dict(seed=32, dtype="f32", B=3, Hq=8, Hkv=2, d=128, lens=[97, 260, 513],
                              segs=[[(0, 60)], [(5, 100), (120, 80)], [(0, 64), (100, 300), (450, 40)]]), 4),
    # a segment running into the queries' own positions, and a sequence shorter than T
    "into-queries-and-short": (dict(seed=33, B=3, Hq=6, Hkv=2, d=64, lens=[200, 2, 64],
                                    segs=[[(20, 179)], [(0, 2)], [(0, 64)]]), 3),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_queries_small_shapes(name):
    spec, T = SMALL[name]
    w = W.with_queries(small_workload(**spec), T)
    ref, ok = P.plant_queries(w, P.params_of(w))
    _log(f"{name}: k={[[r.k for r in ref[b]] for b in range(w.B)]}")
    _, g = _step_and_calls(w)
    _check_all(name, w, g, ref, ok)


def test_queries_with_kv_group_budgets():
    w = W.with_queries(W.generate(2), 2)
    ref, ok = P.plant_queries(w, P.params_of(w), kv_groups=True)
    _, g = _step_and_calls(w, kv_groups=True)
    _check_all("cfg2 T=2 per KV group", w, g, ref, ok, kv_groups=True)


def test_queries_paged_caches():
    w = W.with_queries(W.generate(2), 2)
    P.plant_queries(w, P.params_of(w))
    flat = S.DeviceStep(w)
    flat.decode_step()
    paged = S.DeviceStep(w, block_size=64, block_seed=9)
    paged.decode_step()
    a, b = flat.results(), paged.results()
    for key in KEYS:
        assert np.array_equal(a[key], b[key]), key
