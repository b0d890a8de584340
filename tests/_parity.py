"""Shared helpers for the GPU parity tests (imported by test modules only)."""
from __future__ import annotations

import numpy as np

from oracle import vp_oracle as O
from paper_2605_31457_amd import workloads as W

# Tolerances. Masses: fp32 within 1e-5 relative; an absolute floor of 1e-30
# covers fp32 exp2 underflow (terms below 2^-126 of the head maximum, at most
# 2^15 of them). Scores: same derivation. Outputs: bf16 atol 2e-2 / rtol 1e-2;
# fp32 1e-5 / 1e-5.
MASS_RTOL, MASS_ATOL = 1e-5, 1e-30
OUT_TOL = {"bf16": (2e-2, 1e-2), "f32": (1e-5, 1e-5)}


STEP_KEYS = ("mass_head", "mass_seq", "scores", "k", "vis_idx", "out")
# The attention output of the kept pass against the merge that reads the kept
# rows itself: the pass rounds its probabilities to bf16 for the matrix cores
# (relative error 2^-9 each), the merge keeps them in fp32. The output moves by
# at most 2^-9 times the weighted mean of |V| (under 2e-3 for V drawn from
# N(0, 1) or narrower, as every workload here does), plus two bf16 units in the
# last place of the output itself.
ROUNDING_RTOL, ROUNDING_ATOL = 2.0 ** -7, 2e-3


def kept_in_merge(ds) -> bool:
    """Small steps read the kept rows in the merge launch (VP_PLAN_KEPT_IN_MERGE)."""
    from paper_2605_31457_amd import vp
    return bool(vp.vp_step_plan(ds.shape, ds.params) & vp.VP_PLAN_KEPT_IN_MERGE)


def assert_step_equals_calls(step, calls, fused, kept_merged, ctx=""):
    """vp_decode_step against the four calls. With the text part taken from the
    workspace (fused) every output is the same bits (the same arithmetic, the
    header's promise). Without it vp_sparse_decode_attn runs its kept pass, while
    a small step (VP_PLAN_KEPT_IN_MERGE) reads the kept rows in the merge: its
    attention output then agrees to rounding, everything else bit for bit."""
    for key in STEP_KEYS:
        if key == "out" and not fused and kept_merged:
            np.testing.assert_allclose(step[key], calls[key], rtol=ROUNDING_RTOL, atol=ROUNDING_ATOL,
                                       err_msg=f"{ctx}: out (step against the calls without the workspace text part)")
        else:
            assert np.array_equal(step[key], calls[key]), \
                f"{ctx}: {key} differs between the step and the calls (fused={fused})"


def check_sequence(tag, w, gpu, b, r: O.SequenceResult, b_src=None):
    """Compare GPU outputs of sequence b with the reference result r."""
    ctx = f"{tag} seq {b}" + (f" (source {b_src})" if b_src is not None else "")
    np.testing.assert_allclose(gpu["mass_head"][b], r.mass_head, rtol=MASS_RTOL, atol=MASS_ATOL,
                               err_msg=f"{ctx}: mass_head")
    np.testing.assert_allclose(gpu["mass_seq"][b], [r.M_vis, r.M_vis_max], rtol=MASS_RTOL, atol=MASS_ATOL,
                               err_msg=f"{ctx}: M_vis / M_vis_max")
    nv = len(r.scores)
    np.testing.assert_allclose(gpu["scores"][b, :nv], r.scores, rtol=MASS_RTOL, atol=MASS_ATOL,
                               err_msg=f"{ctx}: scores")
    assert int(gpu["k"][b]) == r.k, f"{ctx}: k {int(gpu['k'][b])} != {r.k}"
    idx = gpu["vis_idx"][b]
    assert np.array_equal(idx[:r.k], r.vis_idx), f"{ctx}: kept index set differs"
    assert np.all(idx[r.k:] == -1), f"{ctx}: padding"
    atol, rtol = OUT_TOL[w.dtype]
    np.testing.assert_allclose(gpu["out"][b], r.out, atol=atol, rtol=rtol, err_msg=f"{ctx}: out")


def tile_batch(w: W.Workload, B: int) -> W.Workload:
    """Batch of B sequences built by repeating w's sequences (b -> b % w.B)."""
    src = [b % w.B for b in range(B)]
    return W.Workload(name=w.name + f"-tiled{B}", dtype=w.dtype, B=B, Hq=w.Hq, Hkv=w.Hkv, d=w.d, S_cap=w.S_cap,
                      seq_len=w.seq_len[src].copy(), segments=[list(w.segments[s]) for s in src],
                      q=w.q[src], K=w.K[src], V=w.V[src], tau_mass=w.tau_mass, tau_score=w.tau_score,
                      r_lo_bp=w.r_lo_bp, r_hi_bp=w.r_hi_bp, clamp=w.clamp, meta=dict(w.meta, tiled_from=src))


def small_workload(seed, B, Hq, Hkv, d, lens, segs, dtype="bf16", S_cap=None, spike=3.0, tau_mass=0.1,
                   r_lo_bp=100, r_hi_bp=500, clamp=True, kv_scale=0.5):
    """A small seeded workload with arbitrary layout (ragged lengths, any segments)."""
    rng = np.random.default_rng(seed)
    S_cap = S_cap or max(max(lens), 1)
    f32 = dtype == "f32"
    st = np.float32 if f32 else np.uint16
    q = np.zeros((B, Hq, d), st)
    K = np.zeros((B, Hkv, S_cap, d), st)
    V = np.zeros((B, Hkv, S_cap, d), st)
    for b in range(B):
        qb = rng.standard_normal((Hq, d)).astype(np.float32)
        Kb = (rng.standard_normal((Hkv, S_cap, d)) * kv_scale).astype(np.float32)
        Vb = (rng.standard_normal((Hkv, S_cap, d)) * kv_scale).astype(np.float32)
        dirs = W._group_dirs(qb, Hkv)
        vis = [p for s, n in segs[b] for p in range(s, s + n)]
        if vis and spike:
            sp = rng.choice(vis, size=max(1, len(vis) // 20), replace=False)
            Kb[:, sp, :] += np.float32(spike) * dirs[:, None, :]
        if f32:
            q[b], K[b], V[b] = qb, Kb, Vb
        else:
            q[b], K[b], V[b] = W.bf16_round(qb), W.bf16_round(Kb), W.bf16_round(Vb)
    return W.Workload(name=f"small-{seed}", dtype=dtype, B=B, Hq=Hq, Hkv=Hkv, d=d, S_cap=S_cap,
                      seq_len=np.array(lens, np.int32), segments=[list(s) for s in segs], q=q, K=K, V=V,
                      tau_mass=tau_mass, r_lo_bp=r_lo_bp, r_hi_bp=r_hi_bp, clamp=clamp)


def check_groups(tag, w, gpu, b, r: O.GroupedResult):
    """Compare GPU outputs of sequence b (per-KV-group selection rows) with the
    reference result r of the per-KV-group variant."""
    ctx = f"{tag} seq {b}"
    np.testing.assert_allclose(gpu["mass_head"][b], r.mass_head, rtol=MASS_RTOL, atol=MASS_ATOL,
                               err_msg=f"{ctx}: mass_head")
    np.testing.assert_allclose(gpu["mass_seq"][b], np.stack([r.M_vis, r.M_vis_max], axis=1), rtol=MASS_RTOL,
                               atol=MASS_ATOL, err_msg=f"{ctx}: group M_vis / M_vis_max")
    nv = r.scores.shape[1]
    np.testing.assert_allclose(gpu["scores"][b, :, :nv], r.scores, rtol=MASS_RTOL, atol=MASS_ATOL,
                               err_msg=f"{ctx}: group scores")
    assert np.array_equal(gpu["k"][b], r.k), f"{ctx}: k {gpu['k'][b]} != {r.k}"
    for g in range(w.Hkv):
        idx = gpu["vis_idx"][b, g]
        k = int(r.k[g])
        assert np.array_equal(idx[:k], r.vis_idx[g]), f"{ctx} group {g}: kept index set differs"
        assert np.all(idx[k:] == -1), f"{ctx} group {g}: padding"
    atol, rtol = OUT_TOL[w.dtype]
    np.testing.assert_allclose(gpu["out"][b], r.out, atol=atol, rtol=rtol, err_msg=f"{ctx}: out")
