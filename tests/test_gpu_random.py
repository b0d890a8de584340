"""Seeded random sweep of the option space through vp_decode_step: dtype, head
dim, head shape (G = 1..16), queries per sequence, budget scope, paged caches,
temperature, clamp presets, ragged lengths and segment layouts. Every case is
planted and checked against the fp64 reference at the usual bars (masses and
scores 1e-5 relative, budgets exact, kept sets bit-exact, outputs bf16 2e-2 /
1e-2 or fp32 1e-5), and the one-launch step against the four calls."""
import numpy as np
import pytest

from _parity import assert_step_equals_calls, check_groups, check_sequence, kept_in_merge, small_workload
from oracle import plant as P
from paper_2605_31457_amd import step as S
from paper_2605_31457_amd import workloads as W

pytestmark = pytest.mark.gpu

KEYS = ("mass_head", "mass_seq", "scores", "k", "vis_idx", "out")
N_CASES = 120


def _case(i):
    rng = np.random.default_rng(7100 + i)
    G = int(rng.choice([1, 2, 4, 7, 8, 16]))
    Hkv = int(rng.choice([1, 2, 3, 4, 8])) if G <= 8 else int(rng.choice([1, 2]))
    T = int(rng.choice([t for t in (1, 2, 3, 4) if t * G <= 16]))
    B = int(rng.integers(1, 5))
    lens, segs = [], []
    for _ in range(B):
        L = int(rng.integers(T, 700))
        pos, sg = 0, []
        for _ in range(int(rng.integers(0, 5))):
            st = pos + int(rng.integers(0, 40))
            n = int(rng.integers(1, 200))
            if st + n > L:
                break
            sg.append((st, n))
            pos = st + n
        lens.append(L)
        segs.append(sg)
    preset = [(100, 500), (500, 1000)][int(rng.integers(0, 2))]
    spec = dict(seed=7200 + i, dtype="f32" if rng.random() < 0.2 else "bf16", B=B, Hq=G * Hkv, Hkv=Hkv,
                d=int(rng.choice([64, 128])), lens=lens, segs=segs, tau_mass=float(rng.choice([0.1, 0.4, 1.0])),
                clamp=bool(rng.random() < 0.8), r_lo_bp=preset[0], r_hi_bp=preset[1])
    opts = dict(T=T, kv_groups=bool(rng.random() < 0.4), block_size=int(rng.choice([0, 0, 16, 64])))
    return spec, opts


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_case(i):
    spec, opts = _case(i)
    tag = f"case {i}: {spec['dtype']} d={spec['d']} Hq={spec['Hq']} Hkv={spec['Hkv']} B={spec['B']} {opts}"
    print(tag, flush=True)
    w = W.with_queries(small_workload(**spec), opts["T"])
    ref, ok = P.plant_queries(w, P.params_of(w), kv_groups=opts["kv_groups"])
    if not all(ok.values()):
        pytest.skip(f"{tag}: planting did not hold")
    ds = S.DeviceStep(w, kv_groups=opts["kv_groups"], block_size=opts["block_size"], block_seed=i)
    ds.decode_step()
    g = ds.results()
    ds.run(fused=bool(i % 2))
    assert_step_equals_calls(g, ds.results(), bool(i % 2), kept_in_merge(ds), tag)
    check = check_groups if opts["kv_groups"] else check_sequence
    for b in range(w.B):
        for t in range(opts["T"]):
            view = {key: (g[key][b, t] if opts["T"] > 1 else g[key][b])[None] for key in KEYS}
            check(f"{tag} seq {b} query {t}", w, view, 0, ref[b][t])
