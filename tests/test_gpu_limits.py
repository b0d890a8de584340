"""Parity at the limits the C ABI accepts: 256 visual segments per sequence,
1024 query heads (64 KV heads of 16), a batch of 512 ragged sequences, and a
131072-token cache; every output against the fp64 reference on planted inputs,
and the one-launch step against the four calls."""
import numpy as np
import pytest

from _parity import check_sequence, small_workload, tile_batch
from oracle import plant as P
from paper_2605_31457_amd import step as S

pytestmark = pytest.mark.gpu

KEYS = ("mass_head", "mass_seq", "scores", "k", "vis_idx", "out")


def _log(msg):
    print(msg, flush=True)


def _check(name, w):
    ref, _ = P.plant(w, P.params_of(w))
    ds = S.DeviceStep(w)
    ds.decode_step()
    g = ds.results()
    ds.run(fused=True)
    c = ds.results()
    for key in KEYS:
        assert np.array_equal(g[key], c[key]), f"{name}: {key} step != calls"
    for b in range(w.B):
        check_sequence(name, w, g, b, ref[b])
    return ref


def test_256_segments_per_sequence():
    # 256 segments of 5 tokens with 3-token text gaps, and a sequence with 255
    segs0 = [(8 * i + 2, 5) for i in range(256)]
    segs1 = [(8 * i, 5) for i in range(255)]
    w = small_workload(seed=61, B=2, Hq=8, Hkv=2, d=64, lens=[2100, 2050], segs=[segs0, segs1])
    assert w.max_segs == 256
    ref = _check("256 segments", w)
    _log(f"256 segments: k={[ref[b].k for b in range(w.B)]}")


def test_1024_query_heads():
    w = small_workload(seed=62, B=1, Hq=1024, Hkv=64, d=64, lens=[400], segs=[[(30, 300)]])
    _check("1024 heads", w)


def test_512_ragged_sequences():
    rng = np.random.default_rng(63)
    lens, segs = [], []
    for b in range(512):
        L = int(rng.integers(1, 160))
        n = int(rng.integers(0, L + 1))
        s0 = int(rng.integers(0, L - n + 1))
        lens.append(L)
        segs.append([(s0, n)] if n else [])
    w = small_workload(seed=64, B=512, Hq=4, Hkv=1, d=64, lens=lens, segs=segs)
    _check("512 sequences", w)


def test_131072_token_cache():
    w = small_workload(seed=65, B=1, Hq=4, Hkv=1, d=64, lens=[131072], segs=[[(1000, 60000), (70000, 20000)]])
    ref = _check("131072 tokens", w)
    _log(f"131072 tokens: k={ref[0].k}")


def test_select_keys_beyond_lds_with_one_work_group_per_row():
    """256 selection rows make the select launch score and select each row in a
    single work-group; every other row here holds 40000 visual tokens, more keys
    than that work-group's LDS holds, so its selection reads the scores back from
    memory. Checked against the four calls and the reference."""
    base = small_workload(seed=66, B=2, Hq=4, Hkv=1, d=64, lens=[40200, 300], segs=[[(100, 40000)], [(20, 200)]])
    ref, _ = P.plant(base, P.params_of(base))
    w = tile_batch(base, 256)
    ds = S.DeviceStep(w, max_vis=40000)
    ds.decode_step()
    g = ds.results()
    ds.run(fused=True)
    c = ds.results()
    for key in KEYS:
        assert np.array_equal(g[key], c[key]), f"keys beyond LDS: {key} step != calls"
    for b in range(w.B):
        check_sequence("keys beyond LDS", w, g, b, ref[b % 2], b_src=b % 2)
    _log(f"keys beyond LDS: k={[ref[b].k for b in range(2)]}")
