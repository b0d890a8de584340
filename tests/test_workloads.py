"""The seeded input generator: layouts, determinism, bf16 storage (no GPU)."""
import numpy as np
import pytest

from paper_2605_31457_amd import workloads as W


@pytest.mark.parametrize("cfg,n_vis,L", [(1, 256, 384), (2, 1296, 3358), (4, 16384, 32768), (5, 6400, 10496)])
def test_layouts_partition_the_cache(cfg, n_vis, L):
    lens, segs, S_cap = W._layout(cfg, 2)
    for l, s in zip(lens, segs):
        assert l == L and l <= S_cap
        assert sum(n for _, n in s) == n_vis
        ends = [a + n for a, n in s]
        assert all(a >= 0 for a, _ in s) and all(e <= l for e in ends)
        assert all(ends[i] <= s[i + 1][0] for i in range(len(s) - 1))  # ascending, disjoint


def test_cfg4_has_four_noncontiguous_images_and_16k_text():
    lens, segs, _ = W._layout(4, 1)
    s = segs[0]
    assert len(s) == 4 and all(n == 4096 for _, n in s)
    assert lens[0] - sum(n for _, n in s) == 16384
    assert all(s[i][0] + 4096 < s[i + 1][0] for i in range(3))


def test_cfg3_ragged_text_lengths():
    lens, segs, S_cap = W._layout(3, 16)
    T = np.array(lens) - 4096
    assert T.min() >= 1024 and T.max() <= 8192 and len(set(T.tolist())) > 8
    assert S_cap == 4096 + 8192


def test_generation_is_deterministic_and_subsettable():
    a = W.generate(2)
    b = W.generate(2)
    assert np.array_equal(a.K, b.K) and np.array_equal(a.q, b.q) and np.array_equal(a.V, b.V)
    full = W.generate(3, B=4)
    sub = W.generate(3, B=4, seqs=[2])
    assert np.array_equal(full.K[2], sub.K[0]) and np.array_equal(full.q[2], sub.q[0])
    assert sub.seq_len[0] == full.seq_len[2]
    c = W.generate(2, seed=77)
    assert not np.array_equal(a.K, c.K)


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 3.0e38, 1e-40, 1 + 2 ** -9], dtype=np.float32)
    got = W.bf16_to_f32(W.bf16_round(x))
    want = np.array([1.0, 1.0, 1 + 2 ** -6, -2.5, np.float32(2.9980e38), 0.0, 1.0], dtype=np.float32)
    assert got[0] == 1.0 and got[1] == 1.0 and got[2] == np.float32(1 + 2 ** -6) and got[3] == -2.5
    assert got[6] == 1.0
    # round trip of representable values is exact
    bits = np.arange(0, 0x7F80, 7, dtype=np.uint16)
    assert np.array_equal(W.bf16_round(W.bf16_to_f32(bits)), bits)


def test_spike_count_and_direction():
    w = W.generate(2)
    q = W.bf16_to_f32(w.q[0]).astype(np.float64)
    dirs = W._group_dirs(q, 4)
    K = W.bf16_to_f32(w.K[0]).astype(np.float64)
    proj = np.einsum("gld,gd->gl", K[:, 14:1310], dirs).mean(axis=0)
    # 5% of 1296 visual keys are moved by +3 along q_hat_g; the rest are ~N(0, 0.5^2/4)
    assert int((proj > 1.5).sum()) == round(0.05 * 1296)


def test_cfg5_stream_appends_and_drifts():
    s = W.Cfg5Stream(B=2, steps=8)
    rms = []
    for t in range(8):
        q, kr, vr, pos = s.step_inputs(t)
        assert pos == 10496 + t and q.shape == (2, 64, 128) and kr.shape == (2, 8, 128)
        rms.append(float(np.sqrt((W.bf16_to_f32(q) ** 2).mean())))
    assert rms[7] < rms[0]          # 0.9 decay dominates the 0.1 innovation


def test_with_queries_drift_and_determinism():
    w = W.generate(1)
    a = W.with_queries(w, 3)
    b = W.with_queries(w, 3)
    assert a.q.shape == (w.B, 3, w.Hq, w.d) and a.q.dtype == w.q.dtype
    np.testing.assert_array_equal(a.q, b.q)
    np.testing.assert_array_equal(a.q[:, 0], w.q)          # query 0 is the workload's own
    assert not np.array_equal(a.q[:, 1], a.q[:, 2])
    # the drift keeps consecutive queries close: 0.9 q + 0.1 eps
    c = np.corrcoef(a.q[:, 0].ravel(), a.q[:, 1].ravel())[0, 1]
    assert c > 0.95
