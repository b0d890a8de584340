"""Pins for the fp64 reference: facts fixed by the paper's definitions and by
mathematics, checked without re-typing the reference's own formulas.

Each test names the passage it pins (VisionPulse, arXiv 2605.31457).
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import vp_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_case(rng, Hq=4, Hkv=2, d=8, L=24, segs=((3, 9), (15, 5)), scale=1.0):
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((Hkv, L, d)) * scale
    V = rng.standard_normal((Hkv, L, d))
    return q, K, V, L, [tuple(s) for s in segs]


# ---------------------------------------------------------------------------
# worked example (hand-derived; Eq. (2), (3), (5), (6), (7), pruned attention)
# ---------------------------------------------------------------------------
def test_worked_example_gqa2():
    ex = json.load(open(os.path.join(GOLDEN, "worked_example_gqa2.json")))
    a, b = ex["inputs"]["a"], ex["inputs"]["b"]
    L = ex["inputs"]["seq_len"]
    q = np.array([[1.0, 0.0], [0.0, 1.0]])
    K = np.array([[[math.log(x), math.log(y)] for x, y in zip(a, b)]])
    V = np.array([[[float(j), 1.0] for j in range(L)]])
    p = O.OracleParams(tau_mass=ex["inputs"]["tau_mass"], tau_score=ex["inputs"]["tau_score"],
                       sm_scale=ex["inputs"]["sm_scale"], r_lo_bp=ex["inputs"]["r_lo_bp"],
                       r_hi_bp=ex["inputs"]["r_hi_bp"], clamp=ex["inputs"]["clamp"])
    segs = [tuple(s) for s in ex["inputs"]["segments"]]
    r = O.decode_step_sequence(q, K, V, L, segs, p)
    e = ex["expected"]
    frac = lambda f: f[0] / f[1]
    np.testing.assert_allclose(r.mass_head, [frac(x) for x in e["mass_head"]], rtol=1e-13)
    assert r.M_vis == pytest.approx(frac(e["M_vis"]), rel=1e-13)
    assert r.M_vis_max == pytest.approx(frac(e["M_vis_max"]), rel=1e-13)
    assert r.k == e["k"]
    np.testing.assert_allclose(r.scores, e["scores"], rtol=1e-13)
    assert list(r.vis_idx) == e["vis_idx"]
    want = np.array([[frac(c) for c in row] for row in e["out"]])
    np.testing.assert_allclose(r.out, want, rtol=1e-13)


def test_worked_example_tempered_scores():
    """Eq. (2) at a score temperature of its own (tau_score = 0.5, tau_mass = 0.25):
    hand-derived exact rationals. The fixture is chosen so that scores taken at
    tau_score = 1 or at tau_mass keep a different set, so an oracle that ignores
    or swaps tau_score fails here."""
    ex = json.load(open(os.path.join(GOLDEN, "worked_example_tau_score.json")))
    inp, e = ex["inputs"], ex["expected"]
    a, b, L = inp["a"], inp["b"], inp["seq_len"]
    q = np.array([[1.0, 0.0], [0.0, 1.0]])
    K = np.array([[[math.log(x), math.log(y)] for x, y in zip(a, b)]])
    V = np.array([[[float(j), 1.0] for j in range(L)]])
    p = O.OracleParams(tau_mass=inp["tau_mass"], tau_score=inp["tau_score"], sm_scale=inp["sm_scale"],
                       r_lo_bp=inp["r_lo_bp"], r_hi_bp=inp["r_hi_bp"], clamp=inp["clamp"])
    segs = [tuple(s) for s in inp["segments"]]
    r = O.decode_step_sequence(q, K, V, L, segs, p)
    frac = lambda f: f[0] / f[1]
    np.testing.assert_allclose(r.mass_head, [frac(x) for x in e["mass_head"]], rtol=1e-13)
    assert r.M_vis == pytest.approx(frac(e["M_vis"]), rel=1e-13)
    assert r.M_vis_max == pytest.approx(frac(e["M_vis_max"]), rel=1e-13)
    assert r.k == e["k"]
    np.testing.assert_allclose(r.scores, [frac(x) for x in e["scores"]], rtol=1e-13)
    assert list(r.vis_idx) == e["vis_idx"]
    want = np.array([[frac(c) for c in row] for row in e["out"]])
    np.testing.assert_allclose(r.out, want, rtol=1e-13)
    # the same inputs with the scores at temperature 1 or at tau_mass keep {1, 3}
    for ts in (1.0, inp["tau_mass"]):
        p2 = O.OracleParams(tau_mass=inp["tau_mass"], tau_score=ts, sm_scale=1.0, r_lo_bp=inp["r_lo_bp"],
                            r_hi_bp=inp["r_hi_bp"], clamp=True)
        assert list(O.decode_step_sequence(q, K, V, L, segs, p2).vis_idx) == [1, 3]


# ---------------------------------------------------------------------------
# budget: closed-form table (Eq. (7) + Sec. 5.2 clamp)
# ---------------------------------------------------------------------------
def _budget_rows():
    rows = []
    for line in open(os.path.join(GOLDEN, "budget_cases.txt")):
        line = line.split("#")[0].strip()
        if not line:
            continue
        m, n, lo, hi, c, k = line.split()
        rows.append((float(m), int(n), int(lo), int(hi), bool(int(c)), int(k)))
    return rows


@pytest.mark.parametrize("m,n,lo,hi,c,k", _budget_rows())
def test_budget_table(m, n, lo, hi, c, k):
    assert O.budget(m, n, lo, hi, c) == k


def test_budget_monotone_and_bounded():
    for n in (1, 7, 256, 1296, 4096, 6400, 16384):
        prev = -1
        k_lo, k_hi = O.retention_bounds(n, 100, 500)
        for m in np.linspace(0, 1, 1001):
            k = O.budget(m, n)
            assert k >= prev and k_lo <= k <= k_hi and 0 <= k <= n
            prev = k
        # unclamped: exact inverse of ceil -- k-1 < m*n <= k
        for m in np.linspace(0, 1, 257):
            k = O.budget(m, n, clamp=False)
            assert k - 1 < m * n <= k or (m == 0 and k == 0)


def test_retention_bounds_exact_integers():
    # 5% of 6400 must be exactly 320 and 1% exactly 64 (no float rounding)
    assert O.retention_bounds(6400, 100, 500) == (64, 320)
    assert O.retention_bounds(1296, 100, 500) == (13, 64)
    assert O.retention_bounds(16384, 100, 500) == (164, 819)


# ---------------------------------------------------------------------------
# mass: definition-level invariants (Eq. (5), Eq. (6))
# ---------------------------------------------------------------------------
def test_visual_plus_text_mass_is_one():
    """P1: the tempered softmax of Eq. (6) runs over all tokens, so the visual and
    text masses of a head add to one."""
    rng = np.random.default_rng(1)
    for tau in (0.1, 0.4, 1.0, 3.0):
        q, K, V, L, segs = _rand_case(rng)
        p = O.OracleParams(tau_mass=tau)
        r = O.decode_step_sequence(q, K, V, L, segs, p, keep_logits=True)
        txt = O.text_positions(L, segs)
        m_txt, _, _ = O.visual_mass(r.Z, txt, tau)
        np.testing.assert_allclose(r.mass_head + m_txt, 1.0, rtol=0, atol=1e-14)
        assert 0 <= r.M_vis <= r.M_vis_max <= 1


def test_scores_sum_to_mass_at_equal_temperature():
    """P2: summing Eq. (2) over visual tokens gives the mean over heads of Eq. (5),
    when both use the same (untempered) attention."""
    rng = np.random.default_rng(2)
    q, K, V, L, segs = _rand_case(rng, Hq=6, Hkv=3)
    p = O.OracleParams(tau_mass=1.0, tau_score=1.0, clamp=False)
    r = O.decode_step_sequence(q, K, V, L, segs, p)
    assert r.scores.sum() == pytest.approx(r.M_vis, rel=1e-13)


@pytest.mark.parametrize("tau", [0.1, 0.4, 2.5])
def test_scores_sum_to_mass_at_a_shared_temperature(tau):
    """P2 at a temperature other than one: when Eq. (2) is taken over the
    attention at the mass temperature (tau_score = tau_mass = tau), summing the
    scores over visual tokens gives the mean over heads of the Eq. (5) masses;
    and the visual and text scores of every head add to one, so a score
    normaliser at the wrong temperature breaks the sum."""
    rng = np.random.default_rng(20 + int(10 * tau))
    q, K, V, L, segs = _rand_case(rng, Hq=6, Hkv=3)
    p = O.OracleParams(tau_mass=tau, tau_score=tau, clamp=False)
    r = O.decode_step_sequence(q, K, V, L, segs, p, keep_logits=True)
    assert r.scores.sum() == pytest.approx(r.M_vis, rel=1e-12)
    # the text tokens' scores at the same temperature carry the rest of the mass
    txt = O.text_positions(L, segs)
    assert r.scores.sum() + O.importance_scores(r.Z, txt, tau).sum() == pytest.approx(1.0, rel=1e-13)
    # and at tau_score = 1 the identity fails for these inputs (the temperature matters)
    p1 = O.OracleParams(tau_mass=tau, tau_score=1.0, clamp=False)
    r1 = O.decode_step_sequence(q, K, V, L, segs, p1)
    assert abs(r1.scores.sum() - r.M_vis) > 1e-6


def test_zero_query_uniform_attention():
    """P3: q = 0 makes every logit 0, so every tempered softmax is uniform:
    m_h = N_v / len for any tau, every score is 1/len, and Top-K keeps the
    lowest positions (tie rule)."""
    rng = np.random.default_rng(3)
    q, K, V, L, segs = _rand_case(rng)
    q[:] = 0.0
    n_vis = sum(n for _, n in segs)
    for tau in (0.1, 1.0):
        p = O.OracleParams(tau_mass=tau, r_lo_bp=1000, r_hi_bp=5000)
        r = O.decode_step_sequence(q, K, V, L, segs, p)
        np.testing.assert_allclose(r.mass_head, n_vis / L, rtol=1e-14)
        np.testing.assert_allclose(r.scores, 1.0 / L, rtol=1e-14)
        k = r.k
        assert k == O.budget(n_vis / L, n_vis, 1000, 5000)
        vis = O.visual_positions(L, segs)
        assert list(r.vis_idx) == list(vis[:k])
        # uniform weights over the pruned context: plain mean of its V rows
        J = np.sort(np.concatenate([vis[:k], O.text_positions(L, segs)]))
        for h in range(q.shape[0]):
            np.testing.assert_allclose(r.out[h], V[h // 2][J].mean(axis=0), rtol=1e-12)


def test_temperature_limits():
    """P4: tau -> infinity flattens Eq. (6) (mass -> N_v/len); tau -> 0 puts all
    tempered mass on the arg-max token (mass -> 1 if it is visual, else 0)."""
    rng = np.random.default_rng(4)
    q, K, V, L, segs = _rand_case(rng)
    n_vis = sum(n for _, n in segs)
    vis = set(O.visual_positions(L, segs).tolist())
    r_hot = O.decode_step_sequence(q, K, V, L, segs, O.OracleParams(tau_mass=1e7), keep_logits=True)
    np.testing.assert_allclose(r_hot.mass_head, n_vis / L, rtol=1e-5)
    r_cold = O.decode_step_sequence(q, K, V, L, segs, O.OracleParams(tau_mass=1e-4), keep_logits=True)
    for h in range(q.shape[0]):
        want = 1.0 if int(np.argmax(r_cold.Z[h])) in vis else 0.0
        assert r_cold.mass_head[h] == pytest.approx(want, abs=1e-9)


def test_head_max_is_max_and_mean_is_mean():
    """Eq. (5) mean over heads; the head-max variant of Sec. 4.3 upper-bounds it."""
    rng = np.random.default_rng(5)
    q, K, V, L, segs = _rand_case(rng, Hq=8, Hkv=2)
    r = O.decode_step_sequence(q, K, V, L, segs, O.OracleParams())
    assert r.M_vis_max == max(r.mass_head) and r.M_vis == pytest.approx(sum(r.mass_head) / 8)
    assert r.M_vis <= r.M_vis_max


# ---------------------------------------------------------------------------
# logits and the GQA head mapping
# ---------------------------------------------------------------------------
def test_onehot_logits_are_exact_integers():
    """P10: with one-hot q and K rows and sm_scale = 1, the logit of Eq. (6) is the
    product of the two nonzero entries when they share a coordinate, else 0."""
    d = 8
    q = np.zeros(d); q[3] = 5.0
    K = np.zeros((6, d))
    K[0, 3] = 2.0; K[1, 4] = 7.0; K[2, 3] = -3.0; K[5, 3] = 1.0
    Z = O.logits(q, K, 1.0)
    assert list(Z) == [10.0, 0.0, -15.0, 0.0, 0.0, 5.0]
    assert list(O.logits(q, K, 0.5)) == [5.0, 0.0, -7.5, 0.0, 0.0, 2.5]


def test_gqa_head_to_kv_group_mapping():
    """Query head h reads KV head h // (Hq/Hkv) (reading A4). Group 0 holds a strong
    key at position 3, group 1 at position 5; heads 0,1 must peak at 3 and heads
    2,3 at 5 (a modulo mapping would mix them)."""
    Hq, Hkv, d, L = 4, 2, 4, 8
    q = np.tile(np.array([1.0, 0, 0, 0]), (Hq, 1))
    K = np.zeros((Hkv, L, d))
    K[0, 3, 0] = 20.0
    K[1, 5, 0] = 20.0
    V = np.zeros((Hkv, L, d))
    V[0, 3, 1] = 1.0
    V[1, 5, 2] = 1.0
    r = O.decode_step_sequence(q, K, V, L, [(2, 3)], O.OracleParams(sm_scale=1.0, clamp=False),
                               keep_logits=True)
    assert [int(np.argmax(r.Z[h])) for h in range(Hq)] == [3, 3, 5, 5]
    assert r.out[0, 1] > 0.99 and r.out[1, 1] > 0.99 and r.out[2, 2] > 0.99 and r.out[3, 2] > 0.99
    # heads 0/1 peak inside the visual segment (2..4), heads 2/3 outside it
    assert r.mass_head[0] > 0.99 and r.mass_head[2] < 0.01


# ---------------------------------------------------------------------------
# selection (Eq. (3)) against brute force
# ---------------------------------------------------------------------------
def _brute_top_k(S, pos, k):
    """The unique k-subset whose every member beats every non-member under the
    order (larger S first, then lower position), found by enumeration."""
    n = len(S)
    found = []
    for sub in itertools.combinations(range(n), k):
        inside = set(sub)
        ok = all((S[i] > S[j]) or (S[i] == S[j] and pos[i] < pos[j])
                 for i in inside for j in range(n) if j not in inside)
        if ok:
            found.append(sorted(pos[i] for i in sub))
    assert len(found) == 1
    return found[0]


def test_select_top_k_brute_force():
    """P6: every k on tiny inputs, including exact ties (scores on a coarse grid)."""
    rng = np.random.default_rng(6)
    for trial in range(40):
        n = int(rng.integers(1, 9))
        pos = np.sort(rng.choice(np.arange(40), size=n, replace=False))
        S = np.round(rng.random(n) * 4) / 4 if trial % 2 else rng.random(n)
        for k in range(0, n + 1):
            got = list(O.select_top_k(S, pos, k))
            assert got == (_brute_top_k(S, pos, k) if k else [])


def test_selection_invariant_min_selected_ge_max_rest():
    rng = np.random.default_rng(7)
    q, K, V, L, segs = _rand_case(rng, L=200, segs=((10, 120),), Hq=4, Hkv=1)
    r = O.decode_step_sequence(q, K, V, L, segs, O.OracleParams(clamp=False, tau_mass=1.0))
    vis = O.visual_positions(L, segs)
    sel = np.isin(vis, r.vis_idx)
    assert sel.sum() == r.k
    assert r.scores[sel].min() >= r.scores[~sel].max()


def test_top_p_budget_brute_force_and_closed_forms():
    """Top-p (A18) pinned without reusing its code path: (a) brute force, the
    smallest subset size k such that SOME k tokens reach p is the answer (the
    largest-k-scores subset is the best of any size), on tiny inputs with ties;
    (b) equal scores s give ceil(p / s); (c) p above the total keeps every
    token; p <= 0 keeps none; (d) it is monotone in p."""
    rng = np.random.default_rng(18)
    for trial in range(60):
        n = int(rng.integers(1, 8))
        pos = np.sort(rng.choice(np.arange(30), size=n, replace=False))
        S = np.round(rng.random(n) * 4) / 16 if trial % 2 else rng.random(n) / n
        total = S.sum()
        for p in (0.0, total * 0.3, total * 0.5 + 1e-9, total * 0.999, total * 1.5, 1e-12):
            k = O.budget_top_p(S, pos, p)
            if p <= 0:
                assert k == 0
                continue
            best = [max(S[list(c)].sum() for c in itertools.combinations(range(n), m)) for m in range(1, n + 1)]
            reach = [m + 1 for m, b in enumerate(best) if b >= p]
            assert k == (reach[0] if reach else n), (S, p, k)
    # dyadic scores sum exactly, so the closed form holds without rounding slack
    for s, p, want in ((2.0 ** -7, 10 * 2.0 ** -7, 10), (2.0 ** -6, 0.1, 7), (2.0 ** -5, 0.5, 16),
                       (2.0 ** -10, 2.0 ** -3 + 2.0 ** -11, 129), (2.0 ** -2, 0.9, 4)):
        S = np.full(200, s)
        assert O.budget_top_p(S, np.arange(200), p) == want == min(200, math.ceil(p / s))
    S = rng.random(50) / 100
    ks = [O.budget_top_p(S, np.arange(50), p) for p in np.linspace(0, S.sum() * 1.2, 40)]
    assert ks == sorted(ks) and ks[-1] == 50


# ---------------------------------------------------------------------------
# pruned attention against the library's attention
# ---------------------------------------------------------------------------
def _sdpa(qh, Kg, Vg, scale):
    qt = torch.from_numpy(qh).reshape(1, 1, 1, -1)
    kt = torch.from_numpy(np.ascontiguousarray(Kg)).reshape(1, 1, Kg.shape[0], -1)
    vt = torch.from_numpy(np.ascontiguousarray(Vg)).reshape(1, 1, Vg.shape[0], -1)
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale).reshape(-1).numpy()


def test_keep_all_equals_dense_attention():
    """P7: with every visual token kept the pruned context is the whole cache, so
    the output is ordinary decode attention (torch SDPA, fp64, CPU)."""
    rng = np.random.default_rng(8)
    q, K, V, L, segs = _rand_case(rng, Hq=6, Hkv=2, d=16, L=40, segs=((4, 20),))
    n_vis = 20
    r = O.decode_step_sequence(q, K, V, L, segs, O.OracleParams(), k_override=n_vis)
    for h in range(6):
        want = _sdpa(q[h], K[h // 3], V[h // 3], 1 / 4.0)
        np.testing.assert_allclose(r.out[h], want, rtol=1e-12, atol=1e-13)


def test_no_visual_tokens_and_single_row():
    """P8: N_v = 0 gives k = 0 and dense attention over the text; a context of a
    single row returns that row's value; an empty context returns zeros."""
    rng = np.random.default_rng(9)
    q, K, V, L, _ = _rand_case(rng, Hq=2, Hkv=1, d=8, L=12)
    r = O.decode_step_sequence(q, K, V, L, [], O.OracleParams())
    assert r.k == 0 and len(r.vis_idx) == 0 and r.M_vis == 0.0
    for h in range(2):
        np.testing.assert_allclose(r.out[h], _sdpa(q[h], K[0], V[0], 1 / math.sqrt(8)), rtol=1e-12)
    np.testing.assert_allclose(O.pruned_attention(q[0], K[0], V[0], np.array([7]), 0.3), V[0, 7], rtol=0)
    assert np.all(O.pruned_attention(q[0], K[0], V[0], np.array([], dtype=np.int64), 0.3) == 0)


def test_pruned_attention_subset_equals_sdpa_on_subset():
    """Dropped tokens are absent from the softmax (A12): identical to SDPA run on
    the kept rows only, and independent of the order of J (P9)."""
    rng = np.random.default_rng(10)
    q, K, V, L, segs = _rand_case(rng, Hq=2, Hkv=1, d=8, L=30)
    J = np.array([0, 2, 3, 11, 17, 29])
    out = O.pruned_attention(q[1], K[0], V[0], J, 0.25)
    np.testing.assert_allclose(out, _sdpa(q[1], K[0][J], V[0][J], 0.25), rtol=1e-12)
    out_perm = O.pruned_attention(q[1], K[0], V[0], J[::-1].copy(), 0.25)
    np.testing.assert_allclose(out, out_perm, rtol=1e-13)


def test_common_key_shift_is_invisible():
    """P11: with one query head per KV head, adding c * q_hat to every key adds the
    same constant to all logits of that head, which softmax ignores: masses,
    scores, the budget, the selection and the output are unchanged."""
    rng = np.random.default_rng(11)
    q, K, V, L, segs = _rand_case(rng, Hq=3, Hkv=3, d=8, L=50, segs=((5, 30),))
    p = O.OracleParams(tau_mass=0.4, r_lo_bp=500, r_hi_bp=3000)
    r0 = O.decode_step_sequence(q, K, V, L, segs, p)
    K2 = K.copy()
    for g in range(3):
        K2[g] += 1.7 * q[g] / np.linalg.norm(q[g])
    r1 = O.decode_step_sequence(q, K2, V, L, segs, p)
    np.testing.assert_allclose(r1.mass_head, r0.mass_head, rtol=1e-11)
    np.testing.assert_allclose(r1.scores, r0.scores, rtol=1e-11)
    assert r1.k == r0.k and list(r1.vis_idx) == list(r0.vis_idx)
    np.testing.assert_allclose(r1.out, r0.out, rtol=1e-11)


def test_bf16_decoding_exact():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000, 0x8000, 0x7F80, 0x3C00], dtype=np.uint16)
    want = [1.0, -1.0, 3.140625, 0.0, -0.0, math.inf, 2.0 ** -7]
    got = O.as_f64(bits)
    assert list(got) == want


def test_exact_rational_tiny_case():
    """Cross-check of Eq. (5)/(6)/(2) in exact rational arithmetic: logits ln(w) make
    exp(Z) = w, so tau = 1 attention is w / sum(w) exactly."""
    w = [3, 1, 4, 1, 5, 9, 2, 6]
    L = len(w)
    q = np.array([[1.0]])
    K = np.array([[[math.log(x)] for x in w]])
    V = np.array([[[float(j)] for j in range(L)]])
    segs = [(2, 4)]
    r = O.decode_step_sequence(q, K, V, L, segs, O.OracleParams(tau_mass=1.0, sm_scale=1.0, clamp=False))
    tot = Fraction(sum(w))
    assert r.mass_head[0] == pytest.approx(float(Fraction(sum(w[2:6])) / tot), rel=1e-14)
    np.testing.assert_allclose(r.scores, [float(Fraction(x) / tot) for x in w[2:6]], rtol=1e-14)
    # k = ceil(19/31 * 4) = ceil(2.45) = 3 -> keep positions of 5, 9, 4 -> {2, 4, 5}
    assert r.k == 3 and list(r.vis_idx) == [2, 4, 5]
    J = [0, 1, 2, 4, 5, 6, 7]
    num = sum(Fraction(w[j]) * j for j in J)
    den = sum(Fraction(w[j]) for j in J)
    assert r.out[0, 0] == pytest.approx(float(num / den), rel=1e-14)


# ---------------------------------------------------------------------------
# per-KV-group budgets and kept sets (the variant with one Eq. (7) budget and one
# Eq. (3) set per KV group; its reading of Eq. (2)/(5)/(7) is stated in the
# reference's header)
# ---------------------------------------------------------------------------
def _brute_groups(q, K, V, L, segs, tau_mass, r_lo_bp, r_hi_bp):
    """Pure-Python loops over a tiny case: for each KV group g, the tempered and
    untempered softmax of each of its query heads over every token, the group's
    head mean / head max of the visual mass, k_g = ceil(max * N_v) clamped to
    [ceil(lo N_v), floor(hi N_v)], the group's score average, the top k_g by
    (score desc, position asc) and each head's attention over kept + text."""
    Hq, d = len(q), len(q[0])
    Hkv = len(K)
    G = Hq // Hkv
    vis = [p for s, n in segs for p in range(s, s + n)]
    nv = len(vis)
    res = []
    for g in range(Hkv):
        masses, S = [], [0.0] * nv
        outs = []
        for j in range(G):
            h = g * G + j
            z = [sum(q[h][c] * K[g][t][c] for c in range(d)) / math.sqrt(d) for t in range(L)]
            zt = max(z)
            et = [math.exp((x - zt) / tau_mass) for x in z]
            masses.append(sum(et[p] for p in vis) / sum(et))
            e1 = [math.exp(x - zt) for x in z]
            tot = sum(e1)
            for i, p in enumerate(vis):
                S[i] += e1[p] / tot / G
        mean, mx = sum(masses) / G, max(masses)
        k = math.ceil(mx * nv)
        lo = -((-r_lo_bp * nv) // 10000)
        hi = max((r_hi_bp * nv) // 10000, lo)
        k = min(max(k, lo), hi, nv)
        ranked = sorted(range(nv), key=lambda i: (-S[i], vis[i]))
        kept = sorted(vis[i] for i in ranked[:k])
        J = sorted(set(kept) | (set(range(L)) - set(vis)))
        for j in range(G):
            h = g * G + j
            z = [sum(q[h][c] * K[g][t][c] for c in range(d)) / math.sqrt(d) for t in J]
            zm = max(z)
            e = [math.exp(x - zm) for x in z]
            outs.append([sum(e[i] * V[g][t][c] for i, t in enumerate(J)) / sum(e) for c in range(d)])
        res.append(dict(masses=masses, mean=mean, mx=mx, S=S, k=k, kept=kept, out=outs))
    return res


def test_kv_groups_brute_force_tiny():
    rng = np.random.default_rng(31)
    for trial in range(6):
        Hkv = (1, 2, 3)[trial % 3]
        G = 1 + trial % 2
        q, K, V, L, segs = _rand_case(rng, Hq=Hkv * G, Hkv=Hkv, d=3, L=40, segs=((2, 15), (20, 12)), scale=2.0)
        p = O.OracleParams(tau_mass=0.5, r_lo_bp=500, r_hi_bp=4000)
        r = O.decode_step_sequence_kv_groups(q, K, V, L, segs, p)
        bf = _brute_groups(q.tolist(), K.tolist(), V.tolist(), L, segs, 0.5, 500, 4000)
        for g in range(Hkv):
            np.testing.assert_allclose(r.mass_head[g * G:(g + 1) * G], bf[g]["masses"], rtol=1e-12)
            assert r.M_vis[g] == pytest.approx(bf[g]["mean"], rel=1e-12)
            assert r.M_vis_max[g] == pytest.approx(bf[g]["mx"], rel=1e-12)
            np.testing.assert_allclose(r.scores[g], bf[g]["S"], rtol=1e-12)
            assert r.k[g] == bf[g]["k"]
            assert list(r.vis_idx[g]) == bf[g]["kept"]
            np.testing.assert_allclose(r.out[g * G:(g + 1) * G], bf[g]["out"], rtol=1e-11, atol=1e-13)


def test_kv_groups_aggregate_to_the_sequence_quantities():
    """Equal group sizes: the head mean of Eq. (5) is the mean of the group means,
    the head max is the max of the group maxima, and the Eq. (2) average is the
    mean of the group averages."""
    rng = np.random.default_rng(32)
    q, K, V, L, segs = _rand_case(rng, Hq=12, Hkv=3, d=8, L=60, segs=((5, 30), (40, 10)))
    p = O.OracleParams(clamp=False, tau_mass=0.3)
    r = O.decode_step_sequence(q, K, V, L, segs, p)
    gr = O.decode_step_sequence_kv_groups(q, K, V, L, segs, p)
    np.testing.assert_allclose(gr.mass_head, r.mass_head, rtol=1e-13)
    assert gr.M_vis.mean() == pytest.approx(r.M_vis, rel=1e-13)
    assert gr.M_vis_max.max() == pytest.approx(r.M_vis_max, rel=1e-13)
    np.testing.assert_allclose(gr.scores.mean(axis=0), r.scores, rtol=1e-12)
    # the group whose head attains the sequence head max sets the largest budget
    g_star = int(np.argmax(r.mass_head)) // 4
    assert gr.k[g_star] == r.k == gr.k.max()


def test_kv_groups_replicated_groups_match_the_sequence():
    """Every KV group a copy of the same KV head and the same G query heads: each
    group's budget, kept set and outputs are the per-sequence ones."""
    rng = np.random.default_rng(33)
    q1, K1, V1, L, segs = _rand_case(rng, Hq=2, Hkv=1, d=8, L=80, segs=((10, 50),))
    q = np.tile(q1, (3, 1))
    K = np.tile(K1, (3, 1, 1))
    V = np.tile(V1, (3, 1, 1))
    p = O.OracleParams(r_lo_bp=500, r_hi_bp=3000)
    r = O.decode_step_sequence(q, K, V, L, segs, p)
    gr = O.decode_step_sequence_kv_groups(q, K, V, L, segs, p)
    for g in range(3):
        assert gr.k[g] == r.k and list(gr.vis_idx[g]) == list(r.vis_idx)
        np.testing.assert_allclose(gr.scores[g], r.scores, rtol=1e-12)
    np.testing.assert_allclose(gr.out, r.out, rtol=1e-12)


def test_kv_groups_permuting_groups_permutes_results():
    rng = np.random.default_rng(34)
    q, K, V, L, segs = _rand_case(rng, Hq=6, Hkv=3, d=8, L=70, segs=((0, 20), (30, 25)), scale=1.5)
    p = O.OracleParams(tau_mass=0.2, r_lo_bp=200, r_hi_bp=4000)
    perm = [2, 0, 1]
    qp = np.concatenate([q[2 * g:2 * g + 2] for g in perm])
    a = O.decode_step_sequence_kv_groups(q, K, V, L, segs, p)
    b = O.decode_step_sequence_kv_groups(qp, K[perm], V[perm], L, segs, p)
    assert list(b.k) == [a.k[g] for g in perm]
    assert [list(x) for x in b.vis_idx] == [list(a.vis_idx[g]) for g in perm]
    np.testing.assert_allclose(b.out, np.concatenate([a.out[2 * g:2 * g + 2] for g in perm]), rtol=1e-13)
    # distinct groups really do pick different sets here (the test is not vacuous)
    assert len({tuple(x) for x in a.vis_idx}) > 1


def test_kv_groups_single_group_is_the_sequence_path():
    rng = np.random.default_rng(35)
    q, K, V, L, segs = _rand_case(rng, Hq=4, Hkv=1, d=8, L=50, segs=((5, 30),))
    p = O.OracleParams()
    r = O.decode_step_sequence(q, K, V, L, segs, p)
    gr = O.decode_step_sequence_kv_groups(q, K, V, L, segs, p)
    assert gr.k[0] == r.k and list(gr.vis_idx[0]) == list(r.vis_idx)
    assert gr.M_vis[0] == r.M_vis and gr.M_vis_max[0] == r.M_vis_max
    np.testing.assert_array_equal(gr.out, r.out)


# ---------------------------------------------------------------------------
# several queries per sequence (each query a decode step of its own over the
# positions before it; the reading is stated in the reference's header)
# ---------------------------------------------------------------------------
def _brute_queries(q, K, V, L, segs, tau_mass, r_lo_bp, r_hi_bp):
    """Pure-Python loops: query t sees positions < L - T + 1 + t; positions from
    L - T + 1 on are text whatever the segments say; per query the per-head
    tempered visual mass, head max, budget, head-averaged scores, top-k and
    attention over kept + visible text."""
    T, Hq, d = len(q), len(q[0]), len(q[0][0])
    Hkv = len(K)
    G = Hq // Hkv
    L0 = L - T + 1
    vis = sorted(p for s, n in segs for p in range(s, s + n) if p < L0)
    nv = len(vis)
    res = []
    for t in range(T):
        n = L0 + t
        masses, S = [], [0.0] * nv
        for h in range(Hq):
            z = [sum(q[t][h][c] * K[h // G][j][c] for c in range(d)) / math.sqrt(d) for j in range(n)]
            zt = max(z)
            et = [math.exp((x - zt) / tau_mass) for x in z]
            masses.append(sum(et[p] for p in vis) / sum(et))
            e1 = [math.exp(x - zt) for x in z]
            for i, p in enumerate(vis):
                S[i] += e1[p] / sum(e1) / Hq
        k = math.ceil(max(masses) * nv)
        lo = -((-r_lo_bp * nv) // 10000)
        hi = max((r_hi_bp * nv) // 10000, lo)
        k = min(max(k, lo), hi, nv)
        kept = sorted(vis[i] for i in sorted(range(nv), key=lambda i: (-S[i], vis[i]))[:k])
        J = sorted(set(kept) | (set(range(n)) - set(vis)))
        out = []
        for h in range(Hq):
            z = [sum(q[t][h][c] * K[h // G][j][c] for c in range(d)) / math.sqrt(d) for j in J]
            zm = max(z)
            e = [math.exp(x - zm) for x in z]
            out.append([sum(e[i] * V[h // G][j][c] for i, j in enumerate(J)) / sum(e) for c in range(d)])
        res.append(dict(masses=masses, k=k, S=S, kept=kept, out=out))
    return res


def test_queries_brute_force_tiny():
    rng = np.random.default_rng(41)
    for trial, (T, segs) in enumerate([(3, ((2, 14), (20, 9))), (2, ((0, 10), (25, 15))), (4, ((5, 30),))]):
        # the last segment of the second and third cases runs into the other queries' positions
        L, Hq, Hkv, d = 40, 4, 2, 3
        q = rng.standard_normal((T, Hq, d))
        K = rng.standard_normal((Hkv, L, d)) * 2.0
        V = rng.standard_normal((Hkv, L, d))
        p = O.OracleParams(tau_mass=0.5, r_lo_bp=500, r_hi_bp=4000)
        rs = O.decode_step_queries(q, K, V, L, [tuple(x) for x in segs], p)
        bf = _brute_queries(q.tolist(), K.tolist(), V.tolist(), L, segs, 0.5, 500, 4000)
        for t in range(T):
            np.testing.assert_allclose(rs[t].mass_head, bf[t]["masses"], rtol=1e-12)
            assert rs[t].k == bf[t]["k"]
            np.testing.assert_allclose(rs[t].scores, bf[t]["S"], rtol=1e-12)
            assert list(rs[t].vis_idx) == bf[t]["kept"]
            np.testing.assert_allclose(rs[t].out, bf[t]["out"], rtol=1e-11, atol=1e-13)


def test_queries_single_query_is_the_step():
    rng = np.random.default_rng(42)
    q, K, V, L, segs = _rand_case(rng, Hq=4, Hkv=2, d=8, L=60, segs=((4, 40),))
    p = O.OracleParams()
    r = O.decode_step_sequence(q, K, V, L, segs, p)
    (r1,) = O.decode_step_queries(q[None], K, V, L, segs, p)
    assert r1.k == r.k and list(r1.vis_idx) == list(r.vis_idx)
    np.testing.assert_array_equal(r1.out, r.out)
    np.testing.assert_array_equal(r1.mass_head, r.mass_head)


def test_queries_are_causal():
    """Rows at or after query t's successor positions never change query t's
    results, and do change the later queries'."""
    rng = np.random.default_rng(43)
    T, L, Hq, Hkv, d = 3, 50, 4, 1, 8
    q = rng.standard_normal((T, Hq, d))
    K = rng.standard_normal((Hkv, L, d))
    V = rng.standard_normal((Hkv, L, d))
    p = O.OracleParams(clamp=False, tau_mass=1.0)
    segs = [(3, 30)]
    a = O.decode_step_queries(q, K, V, L, segs, p)
    K2, V2 = K.copy(), V.copy()
    K2[:, L - 1] += 3.0   # the last query's own row
    V2[:, L - 1] -= 2.0
    b = O.decode_step_queries(q, K2, V2, L, segs, p)
    for t in range(T - 1):
        np.testing.assert_array_equal(a[t].out, b[t].out)
        np.testing.assert_array_equal(a[t].mass_head, b[t].mass_head)
    assert not np.allclose(a[T - 1].out, b[T - 1].out)
    assert not np.allclose(a[T - 1].mass_head, b[T - 1].mass_head)


def test_queries_shorter_than_the_batch_of_queries():
    """A sequence of 2 tokens with 4 queries: the first two queries see nothing
    (zero output, no budget), the others see 1 and 2 text tokens."""
    rng = np.random.default_rng(44)
    q = rng.standard_normal((4, 2, 4))
    K = rng.standard_normal((1, 2, 4))
    V = rng.standard_normal((1, 2, 4))
    rs = O.decode_step_queries(q, K, V, 2, [(0, 2)], O.OracleParams())
    assert [r.k for r in rs] == [0, 0, 0, 0]
    np.testing.assert_array_equal(rs[0].out, 0.0)
    np.testing.assert_array_equal(rs[1].out, 0.0)
    np.testing.assert_allclose(rs[2].out, np.tile(V[0, 0], (2, 1)), rtol=1e-15)
