"""fp64 reference ("oracle") for the VisionPulse per-decode-step path.

TEST INFRASTRUCTURE. Only the test suite, the smoke check and the CPU-baseline
leg of the benchmark may import this module. The HIP library never calls it and
shares no code with it; the two meet only through the seeded inputs produced by
``paper_2605_31457_amd.workloads`` (which holds none of the method's arithmetic).

Everything here is the plain definition written out in float64, in the paper's
order and notation (VisionPulse, arXiv 2605.31457):

* Eq. (6), Sec. 4.3 -- Z_{t,h}(q_t, j): the pre-softmax logit of head h at the
  anchor layer, and A^{(tau)}_{t,h} = softmax_j(Z / tau) over every cached token j.
* Eq. (5), Sec. 4.3 -- visual attention mass m^{vis}_{t,h} = sum_{i in V} A_{t,h},
  M_vis = mean over heads; the head-max variant M_vis,max (Sec. 4.3, text
  after Eq. (6)) drives the budget.
* Eq. (7), Sec. 4.3 -- budget K_t = M_vis,max * N_v, clamped to the retention
  presets of Sec. 5.2 ((0.01N, 0.05N) for the 5% setting, (0.05N, 0.10N) for 10%).
* Eq. (2), Sec. 4.2 -- importance S_i = (1/H) sum_h A_{t,h}(q_t, v_i).
* Eq. (3), Sec. 4.2 -- X_v^t = the Top-K_t visual tokens by S.
* Sec. 4.1/4.2 -- decoding attends over the pruned context: kept visual tokens
  plus every text token (dropped tokens are simply absent from the softmax).

Readings where the paper is silent:
  A1 the softmax of Eq. (6) runs over all cached tokens of the sequence;
  A2 Z includes the 1/sqrt(d) scale (sm_scale);
  A3 the scores of Eq. (2) use the untempered attention (tau_score = 1);
  A4 H counts query heads; query head h reads KV head h // (Hq/Hkv);
  A5 one k and one index set per sequence, shared by all heads;
  A6 K_t = M*N_v is rounded up;  A7/A8 the clamp is [ceil(r_lo N_v), floor(r_hi N_v)]
     with N = N_v and r in basis points (integer arithmetic);
  A10 ties in Top-K go to the lower position; the index set is returned ascending;
  A12 the pruned softmax is renormalised over the kept context only; an empty
     context yields a zero output;
  A18 the Top-p budget counts visual tokens in the Eq. (3) order until their
     Eq. (2) scores sum to p (all of them if they never do);
  A19 the per-KV-group variant (an extension; the paper keeps one set per
     sequence) runs the whole method on each KV group g as if it were a
     sequence of its own: the G query heads that read KV head g give the head
     mean and head max of Eq. (5)/(7), the head average of Eq. (2) and a budget
     k_g, and those G heads attend over their group's own kept set;
  A20 several queries per sequence (an extension: speculative or multi-token
     decoding): the T queries are the last T positions of the sequence, query t
     sees the positions before L - T + 1 + t (itself included) and is a decode
     step of its own (its own masses, budget, kept set and output); the other
     queries' positions are text, so the visual segments are cut at L - T + 1.

Parity status: every function below is pinned by tests/test_oracle_pins.py
(closed forms, invariants, brute force, library cross-checks and the
hand-derived fixtures under tests/golden/).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "as_f64", "logits", "tempered_attention", "visual_mass", "retention_bounds",
    "budget", "budget_top_p", "importance_scores", "select_top_k", "pruned_attention", "attention",
    "OracleParams", "SequenceResult", "decode_step_sequence", "decode_step",
    "visual_positions", "text_positions", "GroupedResult", "decode_step_sequence_kv_groups",
    "clip_segments", "decode_step_queries",
]


# --------------------------------------------------------------------------
# input decoding (the oracle's own; it never uses the HIP path's converters)
# --------------------------------------------------------------------------
def as_f64(x: np.ndarray) -> np.ndarray:
    """Widen stored values exactly to float64.

    uint16 arrays are bfloat16 bit patterns (the upper half of an IEEE binary32);
    float32 / float64 arrays are taken as they are.
    """
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if x.dtype == np.float64:
        return x
    if x.dtype == np.float32:
        return x.astype(np.float64)
    raise TypeError(f"unsupported stored dtype {x.dtype}")


# --------------------------------------------------------------------------
# token classes of one sequence (Sec. 4.2: X_v = {v_1..v_N}; text = the rest)
# --------------------------------------------------------------------------
def visual_positions(seq_len: int, segments) -> np.ndarray:
    """Absolute positions of the visual tokens, ascending (visual rank order).

    ``segments`` is a list of (start, length) pairs, ascending and disjoint.
    """
    pos = [np.arange(s, s + n, dtype=np.int64) for (s, n) in segments]
    out = np.concatenate(pos) if pos else np.zeros(0, dtype=np.int64)
    assert np.all(out < seq_len), "visual segment beyond the sequence"
    return out


def text_positions(seq_len: int, segments) -> np.ndarray:
    """Every cached position that is not visual (system prompt, text, generated)."""
    mask = np.ones(seq_len, dtype=bool)
    mask[visual_positions(seq_len, segments)] = False
    return np.nonzero(mask)[0].astype(np.int64)


# --------------------------------------------------------------------------
# Eq. (6): logits and tempered attention
# --------------------------------------------------------------------------
def logits(q_h: np.ndarray, K_g: np.ndarray, sm_scale: float) -> np.ndarray:
    """Z_{t,h}(q_t, j) for every row j of K_g: sm_scale * <q_h, k_j> (Eq. (6), reading A2).

    q_h is one head's query [d] (result [rows]) or the queries of several heads
    that read the same KV head, [n, d] (result [n, rows], one row per head).
    """
    return sm_scale * (as_f64(q_h) @ as_f64(K_g).T)


def tempered_attention(Z: np.ndarray, tau: float) -> np.ndarray:
    """A^{(tau)}(j) = exp(Z_j / tau) / sum_j' exp(Z_j' / tau)  (Eq. (6); A1: j over all tokens).

    Z is one head's logits [n], or [H, n] for H heads (one softmax per head, over
    the last axis). The common factor exp(-max Z / tau) is divided out of
    numerator and denominator, which leaves the quotient unchanged and avoids
    overflow.
    """
    x = np.asarray(Z, dtype=np.float64) / tau
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


# --------------------------------------------------------------------------
# Eq. (5) with Eq. (6): visual attention mass and its head-max
# --------------------------------------------------------------------------
def visual_mass(Z_heads: np.ndarray, vis_pos: np.ndarray, tau: float):
    """Per-head m^{vis}_{t,h}, M_vis (mean over heads) and M_vis,max (max over heads).

    Z_heads: [H, n] logits of every query head over every cached token.
    Returns (m_head [H], M_vis, M_vis_max).
    """
    A = tempered_attention(Z_heads, tau)          # [H, n], one softmax per head
    m_head = A[:, vis_pos].sum(axis=1)
    return m_head, float(m_head.mean()), float(m_head.max())


# --------------------------------------------------------------------------
# Eq. (7) and the retention clamp of Sec. 5.2
# --------------------------------------------------------------------------
def retention_bounds(n_vis: int, r_lo_bp: int, r_hi_bp: int):
    """(k_lo, k_hi) = (ceil(r_lo N_v), floor(r_hi N_v)) with r in basis points (A7).

    k_hi is raised to k_lo if rounding would invert the interval.
    """
    k_lo = -((-r_lo_bp * n_vis) // 10000)          # integer ceil
    k_hi = (r_hi_bp * n_vis) // 10000               # integer floor
    return k_lo, max(k_hi, k_lo)


def budget(m_max: float, n_vis: int, r_lo_bp: int = 100, r_hi_bp: int = 500,
           clamp: bool = True) -> int:
    """K_t = M_vis,max * N_v (Eq. (7)), rounded up (A6), clamped (Sec. 5.2), 0 <= K_t <= N_v."""
    if n_vis <= 0:
        return 0
    k = math.ceil(float(m_max) * n_vis)
    if clamp:
        k_lo, k_hi = retention_bounds(n_vis, r_lo_bp, r_hi_bp)
        k = min(max(k, k_lo), k_hi)
    return int(min(max(k, 0), n_vis))


# --------------------------------------------------------------------------
# Eq. (2): importance scores;  Eq. (3): Top-K_t
# --------------------------------------------------------------------------
def importance_scores(Z_heads: np.ndarray, vis_pos: np.ndarray,
                      tau_score: float = 1.0) -> np.ndarray:
    """S_i = (1/H) sum_h A_{t,h}(q_t, v_i), i over visual tokens in rank order (Eq. (2), A3, A4)."""
    H = Z_heads.shape[0]
    A = tempered_attention(Z_heads, tau_score)    # [H, n], one softmax per head
    return A[:, vis_pos].sum(axis=0) / H


def select_top_k(S: np.ndarray, vis_pos: np.ndarray, k: int) -> np.ndarray:
    """Positions of the k visual tokens with the largest S (Eq. (3)).

    Order: descending S, ties to the lower position (A10); the chosen positions
    are returned ascending.
    """
    if k <= 0:
        return np.zeros(0, dtype=np.int64)
    order = np.lexsort((vis_pos, -S))          # primary key -S, secondary position
    return np.sort(vis_pos[order[:k]])


def budget_top_p(S: np.ndarray, vis_pos: np.ndarray, p: float) -> int:
    """The Top-p budget the paper compares against (Sec. 5, budgeting strategies):
    the smallest number of visual tokens, taken in the Eq. (3) order (descending
    S, ties to the lower position), whose scores sum to at least p; every visual
    token when all of them sum to less (reading A18). p <= 0 gives 0.
    """
    if p <= 0 or len(S) == 0:
        return 0
    order = np.lexsort((vis_pos, -S))
    csum = np.cumsum(S[order])
    reach = np.nonzero(csum >= p)[0]
    return int(reach[0] + 1) if len(reach) else len(S)


# --------------------------------------------------------------------------
# pruned decode attention (Sec. 4.1/4.2)
# --------------------------------------------------------------------------
def pruned_attention(q_h: np.ndarray, K_g: np.ndarray, V_g: np.ndarray,
                     J: np.ndarray, sm_scale: float) -> np.ndarray:
    """softmax over J of Z_{t,h}(q_t, j), applied to V rows in J (A11, A12).

    J: positions of the pruned context (kept visual + all text). Empty J -> zeros.
    """
    d = V_g.shape[-1]
    if len(J) == 0:
        return np.zeros(d, dtype=np.float64)
    return attention(q_h, K_g[J], V_g[J], sm_scale)


def attention(q_h: np.ndarray, K_rows: np.ndarray, V_rows: np.ndarray, sm_scale: float) -> np.ndarray:
    """softmax over the given rows of Z_{t,h}(q_t, j), applied to their V rows
    (temperature 1; at least one row). q_h: [d], or [n, d] for n heads that read
    the same rows (one softmax per head)."""
    Z = logits(q_h, K_rows, sm_scale)
    p = np.exp(Z - Z.max(axis=-1, keepdims=True))
    return (p / p.sum(axis=-1, keepdims=True)) @ as_f64(V_rows)


# --------------------------------------------------------------------------
# one decode step over a batch
# --------------------------------------------------------------------------
@dataclass
class OracleParams:
    tau_mass: float = 0.1        # Eq. (6) temperature, 5% preset (App. B.1)
    tau_score: float = 1.0       # reading A3
    sm_scale: float | None = None  # default 1/sqrt(d) (reading A2)
    r_lo_bp: int = 100           # Sec. 5.2, 5% preset: (0.01N, 0.05N)
    r_hi_bp: int = 500
    clamp: bool = True


@dataclass
class SequenceResult:
    mass_head: np.ndarray        # [Hq] m^{vis}_{t,h}
    M_vis: float
    M_vis_max: float
    scores: np.ndarray           # [N_v] S_i, visual rank order
    k: int
    vis_idx: np.ndarray          # [k] positions, ascending
    out: np.ndarray | None       # [Hq, d] (None when not requested)
    Z: np.ndarray | None = field(default=None, repr=False)


def decode_step_sequence(q: np.ndarray, K: np.ndarray, V: np.ndarray,
                         seq_len: int, segments, params: OracleParams,
                         keep_logits: bool = False,
                         k_override: int | None = None,
                         with_output: bool = True) -> SequenceResult:
    """The whole per-step path for one sequence at the anchor layer.

    q: [Hq, d]; K, V: [Hkv, >=seq_len, d] (stored values: uint16 bf16 bits or
    float32; float64 arrays are taken as already widened).
    ``k_override`` replaces the Eq. (7) budget (used to test selection and
    attention on their own). ``with_output=False`` stops after the selection
    (out is None): the attention output is the costly part on long contexts.
    """
    Hq, d = q.shape
    Hkv = K.shape[0]
    assert Hq % Hkv == 0
    G = Hq // Hkv
    sm_scale = params.sm_scale if params.sm_scale is not None else 1.0 / math.sqrt(d)
    vis_pos = visual_positions(seq_len, segments)
    txt_pos = text_positions(seq_len, segments)
    n_vis = len(vis_pos)

    # stored values widened once per KV head (exact: bf16/fp32 -> fp64)
    Kf = [as_f64(K[g, :seq_len]) for g in range(Hkv)]
    Vf = [as_f64(V[g, :seq_len]) for g in range(Hkv)]
    qf = as_f64(q)

    # Eq. (6) logits of every query head over every cached token (A1, A4)
    # (the G query heads of KV head g in one product)
    Z = np.empty((Hq, seq_len), dtype=np.float64)
    for g in range(Hkv):
        Z[g * G:(g + 1) * G] = logits(qf[g * G:(g + 1) * G], Kf[g], sm_scale)

    # Eq. (5)/(6) and the head-max; Eq. (7) with the clamp
    if seq_len > 0:
        m_head, M_vis, M_max = visual_mass(Z, vis_pos, params.tau_mass)
    else:
        m_head, M_vis, M_max = np.zeros(Hq), 0.0, 0.0
    k = budget(M_max, n_vis, params.r_lo_bp, params.r_hi_bp, params.clamp)
    if k_override is not None:
        k = int(k_override)

    # Eq. (2) scores and Eq. (3) selection
    S = importance_scores(Z, vis_pos, params.tau_score) if n_vis else np.zeros(0)
    sel = select_top_k(S, vis_pos, k)

    # attention over the pruned context J = kept visual U text
    out = None
    if with_output:
        J = np.sort(np.concatenate([sel, txt_pos]))
        out = np.zeros((Hq, d), dtype=np.float64)
        if len(J):
            # softmax over J of the same logits Z (temperature 1): the dropped
            # visual tokens are absent, i.e. carry weight exactly zero
            inJ = np.zeros(seq_len, dtype=bool)
            inJ[J] = True
            ZJ = np.where(inJ, Z, -np.inf)
            P = np.exp(ZJ - ZJ.max(axis=1, keepdims=True))
            P /= P.sum(axis=1, keepdims=True)
            for g in range(Hkv):
                out[g * G:(g + 1) * G] = P[g * G:(g + 1) * G] @ Vf[g]

    return SequenceResult(m_head, M_vis, M_max, S, k, sel, out,
                          Z if keep_logits else None)


def decode_step(q, K, V, seq_len, segments, params: OracleParams,
                seqs=None, keep_logits=False):
    """decode_step_sequence for every sequence b (or the subset ``seqs``).

    q: [B, Hq, d]; K, V: [B, Hkv, S_cap, d]; seq_len: [B]; segments: list of
    per-sequence (start, len) lists. Returns {b: SequenceResult}.
    """
    B = q.shape[0]
    seqs = range(B) if seqs is None else seqs
    return {b: decode_step_sequence(q[b], K[b], V[b], int(seq_len[b]), segments[b],
                                    params, keep_logits=keep_logits)
            for b in seqs}


# --------------------------------------------------------------------------
# per-KV-group budgets and kept sets (reading A19)
# --------------------------------------------------------------------------
@dataclass
class GroupedResult:
    mass_head: np.ndarray        # [Hq] m^{vis}_{t,h} (the same as per sequence)
    M_vis: np.ndarray            # [Hkv] mean of m^{vis} over the group's heads
    M_vis_max: np.ndarray        # [Hkv] max over the group's heads
    scores: np.ndarray           # [Hkv, N_v] S_{g,i} = (1/G) sum_{h in g} A_{t,h}(v_i)
    k: np.ndarray                # [Hkv] K_{t,g}
    vis_idx: list                # Hkv arrays of kept positions, ascending
    out: np.ndarray | None       # [Hq, d]; head h attends over its group's kept set + text


def decode_step_sequence_kv_groups(q: np.ndarray, K: np.ndarray, V: np.ndarray,
                                   seq_len: int, segments, params: OracleParams,
                                   with_output: bool = True) -> GroupedResult:
    """The per-step path with one budget and one kept set per KV group (A19).

    KV group g is the sub-problem made of query heads g*G .. (g+1)*G - 1 and KV
    head g alone; each is solved by decode_step_sequence, which is the whole
    definition of the variant.
    """
    Hq, d = q.shape
    Hkv = K.shape[0]
    assert Hq % Hkv == 0
    G = Hq // Hkv
    parts = [decode_step_sequence(q[g * G:(g + 1) * G], K[g:g + 1], V[g:g + 1], seq_len, segments,
                                  params, with_output=with_output) for g in range(Hkv)]
    return GroupedResult(
        mass_head=np.concatenate([r.mass_head for r in parts]),
        M_vis=np.array([r.M_vis for r in parts]),
        M_vis_max=np.array([r.M_vis_max for r in parts]),
        scores=np.stack([r.scores for r in parts]),
        k=np.array([r.k for r in parts], dtype=np.int64),
        vis_idx=[r.vis_idx for r in parts],
        out=np.concatenate([r.out for r in parts]) if with_output else None)


# --------------------------------------------------------------------------
# several queries per sequence (reading A20)
# --------------------------------------------------------------------------
def clip_segments(segments, n: int):
    """The visual segments cut to the first n positions (empty pieces dropped)."""
    out = []
    for (st, ln) in segments:
        ln = min(ln, n - st)
        if ln > 0:
            out.append((st, ln))
    return out


def decode_step_queries(q: np.ndarray, K: np.ndarray, V: np.ndarray, seq_len: int, segments,
                        params: OracleParams, kv_groups: bool = False, with_output: bool = True):
    """T queries of one sequence (q: [T, Hq, d]), each a decode step of its own (A20).

    Query t sees the first L0 + t positions, L0 = seq_len - T + 1; positions from
    L0 on are never visual. Returns a list of T results (SequenceResult, or
    GroupedResult with ``kv_groups``).
    """
    T = q.shape[0]
    L0 = seq_len - T + 1
    segs = clip_segments(segments, max(L0, 0))
    # a sequence shorter than T leaves the first queries without positions
    n = [max(L0 + t, 0) for t in range(T)]
    if kv_groups:
        return [decode_step_sequence_kv_groups(q[t], K, V, n[t], segs, params, with_output=with_output)
                for t in range(T)]
    return [decode_step_sequence(q[t], K, V, n[t], segs, params, with_output=with_output)
            for t in range(T)]
