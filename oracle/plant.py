"""Make the reference answer unique on a generated workload (test infrastructure).

TEST INFRASTRUCTURE. Used by the test suite and the smoke check only.

Two discrete decisions of the path are taken from real numbers: the budget
K_t = ceil(M_vis,max * N_v) (Eq. (7)) and the Top-K_t cut of the scores
(Eq. (3)). An fp32 GPU path and the fp64 reference agree on them only when the
real numbers are not within rounding distance of the decision boundary. This
module edits the stored keys of a workload, a few rows at a time, until

* budget margin: budget(M (1 - mu)) == budget(M (1 + mu)) with mu = 1e-4, and
* score gap: S_(k) >= (1 + gap) * S_(k+1) with gap = 1e-3 (S sorted descending),

both measured by the fp64 reference. Edits move a key row along the unit
direction q_hat_g of its KV group (the same direction the generator spikes
along) and are re-rounded to the stored precision, so the stored tensor is
exactly what both sides read. Every edit is logged (sequence, position).
"""
from __future__ import annotations

import math

import numpy as np

from . import vp_oracle as O

MU = 1e-4
GAP = 1e-3
BAND = 2.5e-3          # tokens this close (in log S) to the cut are pushed apart
PUSH = 0.05            # step along q_hat_g, in key units


def _round_like(x32: np.ndarray, stored_dtype) -> np.ndarray:
    if stored_dtype == np.uint16:
        u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
        r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
        return r.astype(np.uint16)
    return x32.astype(stored_dtype)


def _to_f32(x):
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return x.astype(np.float32)


def _group_dirs(q_b, Hkv):
    q = O.as_f64(q_b)
    Hq, d = q.shape
    s = q.reshape(Hkv, Hq // Hkv, d).sum(axis=1)
    n = np.linalg.norm(s, axis=1, keepdims=True)
    n[n == 0] = 1.0
    return (s / n).astype(np.float32)


def _push_rows(Kb, dirs, positions, signs, eps):
    """Kb[g, pos] += sign * eps * dirs[g] for every KV head g, re-rounded in place."""
    pos = np.asarray(positions, dtype=np.int64)
    if pos.size == 0:
        return
    step = (np.asarray(signs, dtype=np.float64) * eps).astype(np.float32)       # [n]
    rows = _to_f32(Kb[:, pos, :]) + step[None, :, None] * dirs[:, None, :]       # [Hkv, n, d]
    Kb[:, pos, :] = _round_like(rows, Kb.dtype)


def margin_ok(M_max, n_vis, params: O.OracleParams, mu=MU) -> bool:
    lo = O.budget(M_max * (1 - mu), n_vis, params.r_lo_bp, params.r_hi_bp, params.clamp)
    hi = O.budget(M_max * (1 + mu), n_vis, params.r_lo_bp, params.r_hi_bp, params.clamp)
    return lo == hi


def boundary_gap(S: np.ndarray, vis_pos: np.ndarray, k: int) -> float:
    """Relative gap S_(k)/S_(k+1) - 1 at the cut (inf when there is no cut)."""
    if k <= 0 or k >= len(S):
        return math.inf
    order = np.lexsort((vis_pos, -S))
    a, b = S[order[k - 1]], S[order[k]]
    if b <= 0:
        return math.inf
    return a / b - 1.0


def plant_sequence(q_b, K_b, V_b, seq_len, segments, params: O.OracleParams,
                   max_iter=12, log=None):
    """Edit K_b in place until margin and gap hold; returns the final reference result.

    Raises RuntimeError if the conditions cannot be met within ``max_iter`` passes.
    """
    Hkv = K_b.shape[0]
    dirs = _group_dirs(q_b, Hkv)
    vis_pos = O.visual_positions(seq_len, segments)
    n_vis = len(vis_pos)
    edits = []
    for it in range(max_iter):
        r = O.decode_step_sequence(q_b, K_b, V_b, seq_len, segments, params)
        if not margin_ok(r.M_vis_max, n_vis, params):
            # move the visual token that carries most tempered mass in the
            # head-max head; try growing steps in both directions
            Z = O.decode_step_sequence(q_b, K_b, V_b, seq_len, segments, params,
                                       keep_logits=True).Z
            h = int(np.argmax(r.mass_head))
            A = O.tempered_attention(Z[h], params.tau_mass)
            j = int(vis_pos[np.argmax(A[vis_pos])])
            saved = K_b[:, j, :].copy()
            fixed = False
            for eps in (0.02, -0.02, 0.05, -0.05, 0.1, -0.1, 0.2, -0.2):
                K_b[:, j, :] = saved
                _push_rows(K_b, dirs, [j], [1.0], eps)
                r2 = O.decode_step_sequence(q_b, K_b, V_b, seq_len, segments, params)
                if margin_ok(r2.M_vis_max, n_vis, params):
                    fixed = True
                    break
            if not fixed:
                K_b[:, j, :] = saved
                raise RuntimeError("budget margin could not be planted")
            edits.append(("margin", j))
            continue
        g = boundary_gap(r.scores, vis_pos, r.k)
        if g >= GAP:
            if log is not None:
                log.append({"iterations": it, "edits": edits, "gap": g})
            return r, edits
        order = np.lexsort((vis_pos, -r.scores))
        theta = math.sqrt(r.scores[order[r.k - 1]] * r.scores[order[r.k]])
        lg = np.abs(np.log(np.maximum(r.scores, 1e-300) / theta))
        rank = np.empty(n_vis, dtype=np.int64)
        rank[order] = np.arange(n_vis)
        band = np.nonzero(lg < BAND)[0]
        pos = vis_pos[band]
        sgn = np.where(rank[band] < r.k, 1.0, -1.0)
        _push_rows(K_b, dirs, pos, sgn, PUSH)
        edits.extend(("gap", int(p)) for p in pos)
    raise RuntimeError("score gap could not be planted")


def plant_loop_step(q_b, K_b, Kf_b, V_b, Vf_b, seq_len, segments, params: O.OracleParams,
                    max_iter=12, with_output=True):
    """Planting for one step of a decode loop whose cache carries over from step
    to step (edits made at a step stay in the cache for the later steps).

    K_b / V_b hold the stored rows [Hkv, S, d] (K_b edited in place, re-rounded to
    the stored precision as in plant_sequence); Kf_b / Vf_b are their float64
    copies, which the caller keeps equal to the stored values (this function
    updates Kf_b for the rows it edits). Between edits the Eq. (6) logits are
    updated for the edited rows only, and the masses, the budget and the Eq. (2)
    scores are recomputed from them with the reference's own functions; the
    result returned is a fresh reference evaluation of the planted step.
    A budget margin that does not hold is planted by plant_sequence.

    Returns (edited positions, SequenceResult of the planted step).
    """
    Hkv = K_b.shape[0]
    Hq, d = q_b.shape
    G = Hq // Hkv
    sm = params.sm_scale if params.sm_scale is not None else 1.0 / math.sqrt(d)
    vis_pos = O.visual_positions(seq_len, segments)
    n_vis = len(vis_pos)
    r = O.decode_step_sequence(q_b, Kf_b, Vf_b, seq_len, segments, params, keep_logits=True, with_output=False)
    if not margin_ok(r.M_vis_max, n_vis, params):
        _, edits = plant_sequence(q_b, K_b, V_b, seq_len, segments, params, max_iter=max_iter)
        pos = sorted({p for _, p in edits})
        if pos:
            Kf_b[:, pos] = O.as_f64(K_b[:, pos])
        return pos, O.decode_step_sequence(q_b, Kf_b, Vf_b, seq_len, segments, params, with_output=with_output)
    if boundary_gap(r.scores, vis_pos, r.k) >= GAP:
        if with_output:
            r = O.decode_step_sequence(q_b, Kf_b, Vf_b, seq_len, segments, params)
        return [], r
    dirs = _group_dirs(q_b, Hkv)
    qf = O.as_f64(q_b)
    Z = r.Z
    S, k = r.scores, r.k
    edited = set()
    for _ in range(max_iter):
        order = np.lexsort((vis_pos, -S))
        theta = math.sqrt(S[order[k - 1]] * S[order[k]])
        lg = np.abs(np.log(np.maximum(S, 1e-300) / theta))
        rank = np.empty(n_vis, dtype=np.int64)
        rank[order] = np.arange(n_vis)
        band = np.nonzero(lg < BAND)[0]
        pos = vis_pos[band]
        _push_rows(K_b, dirs, pos, np.where(rank[band] < k, 1.0, -1.0), PUSH)
        Kf_b[:, pos] = O.as_f64(K_b[:, pos])
        edited.update(int(p) for p in pos)
        for g in range(Hkv):
            Z[g * G:(g + 1) * G, pos] = O.logits(qf[g * G:(g + 1) * G], Kf_b[g, pos], sm)
        _, _, M_max = O.visual_mass(Z, vis_pos, params.tau_mass)
        k = O.budget(M_max, n_vis, params.r_lo_bp, params.r_hi_bp, params.clamp)
        S = O.importance_scores(Z, vis_pos, params.tau_score)
        if margin_ok(M_max, n_vis, params) and boundary_gap(S, vis_pos, k) >= GAP:
            r = O.decode_step_sequence(q_b, Kf_b, Vf_b, seq_len, segments, params, with_output=with_output)
            if margin_ok(r.M_vis_max, n_vis, params) and boundary_gap(r.scores, vis_pos, r.k) >= GAP:
                return sorted(edited), r
    raise RuntimeError("score gap could not be planted at this loop step")


def plant(w, params: O.OracleParams, seqs=None):
    """Plant every sequence of workload ``w`` (in place). Returns {b: SequenceResult}, log."""
    res, log = {}, []
    for b in (range(w.B) if seqs is None else seqs):
        lg = []
        r, edits = plant_sequence(w.q[b], w.K[b], w.V[b], int(w.seq_len[b]),
                                  w.segments[b], params, log=lg)
        res[b] = r
        log.append({"seq": b, **(lg[0] if lg else {}), "n_edits": len(edits)})
    return res, log


def plant_kv_groups(w, params: O.OracleParams, seqs=None):
    """plant() for the per-KV-group variant: every KV group of every sequence is
    planted as the one-KV-head sequence it is in that variant (edits stay inside
    the group's own KV head). Returns {b: GroupedResult}, log."""
    res, log = {}, []
    G = w.Hq // w.Hkv
    for b in (range(w.B) if seqs is None else seqs):
        for g in range(w.Hkv):
            lg = []
            _, edits = plant_sequence(w.q[b, g * G:(g + 1) * G], w.K[b, g:g + 1], w.V[b, g:g + 1],
                                      int(w.seq_len[b]), w.segments[b], params, log=lg)
            log.append({"seq": b, "group": g, **(lg[0] if lg else {}), "n_edits": len(edits)})
        res[b] = O.decode_step_sequence_kv_groups(w.q[b], w.K[b], w.V[b], int(w.seq_len[b]),
                                                  w.segments[b], params)
    return res, log


def plant_queries(w, params: O.OracleParams, seqs=None, kv_groups=False, rounds=4):
    """plant() for T queries per sequence (w.q: [B, T, Hq, d]): each query is
    planted as the step it is (its visible prefix, visual segments cut at
    L - T + 1), in rounds until every query of the sequence holds its margin
    and gap at once (an edit for one query moves the others' scores too).
    Returns {b: [T results]}, {b: True when every query holds}."""
    res, ok = {}, {}
    T = w.q.shape[1]
    G = w.Hq // w.Hkv
    for b in (range(w.B) if seqs is None else seqs):
        L = int(w.seq_len[b])
        L0 = L - T + 1
        segs = O.clip_segments(w.segments[b], max(L0, 0))
        vis = O.visual_positions(max(L0, 0), segs)
        good = False
        for _ in range(rounds):
            good = True
            for t in range(T):
                n = max(L0 + t, 0)
                units = ([(w.q[b, t], w.K[b], w.V[b])] if not kv_groups else
                         [(w.q[b, t, g * G:(g + 1) * G], w.K[b, g:g + 1], w.V[b, g:g + 1]) for g in range(w.Hkv)])
                for (qq, KK, VV) in units:
                    r = O.decode_step_sequence(qq, KK, VV, n, segs, params, with_output=False)
                    if margin_ok(r.M_vis_max, len(vis), params) and boundary_gap(r.scores, vis, r.k) >= GAP:
                        continue
                    good = False
                    try:
                        plant_sequence(qq, KK, VV, n, segs, params)
                    except RuntimeError:
                        pass
            if good:
                break
        ok[b] = good
        res[b] = O.decode_step_queries(w.q[b], w.K[b], w.V[b], L, w.segments[b], params, kv_groups=kv_groups)
    return res, ok


def params_of(w) -> O.OracleParams:
    return O.OracleParams(tau_mass=w.tau_mass, tau_score=w.tau_score,
                          r_lo_bp=w.r_lo_bp, r_hi_bp=w.r_hi_bp, clamp=w.clamp)
