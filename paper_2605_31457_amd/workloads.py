"""Seeded synthetic inputs shaped like the paper's LMM decode workloads.

This module builds inputs only: layouts, seeded Gaussian draws, key spikes and
bfloat16 rounding. It holds none of the method's arithmetic (no logits, no
softmax, no mass, no budget, no selection) and is shared by the HIP path's
tests/benchmark and by the fp64 reference; neither side's code lives here.

Shapes follow the paper's setting (Sec. 3.1 cost model, Sec. 5.1 / App. B.1
models and decoding setup): a KV cache of one anchor layer holding system text,
one or more images of visual tokens (a 36x36 patch grid is 1296 tokens) and a
long reasoning trace, with 7B-class (28 query / 4 KV heads) and 72B-class
(64 / 8) attention shapes, head_dim 128.

Storage: bfloat16 tensors are numpy ``uint16`` bit patterns (round to nearest
even from float32); the fp32 configuration stores ``float32``. KV caches are
[B, Hkv, S_cap, d] with d contiguous; q is [B, Hq, d].
"""
from __future__ import annotations

import os
from dataclasses import dataclass, field

import numpy as np

__all__ = ["Workload", "CONFIGS", "generate", "bf16_round", "bf16_to_f32",
           "Cfg5Stream", "layout_arrays", "with_queries"]


# --------------------------------------------------------------------------
# bfloat16 storage helpers (pure data conversion)
# --------------------------------------------------------------------------
def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest, ties to even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.size >= (1 << 16):
        import torch  # vectorised, multi-threaded RNE conversion for large tensors
        return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    u = x.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.asarray(b).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# workload container
# --------------------------------------------------------------------------
@dataclass
class Workload:
    name: str
    dtype: str                    # "bf16" | "f32"
    B: int
    Hq: int
    Hkv: int
    d: int
    S_cap: int                    # cache capacity (max_seq_len)
    seq_len: np.ndarray           # [B] int32
    segments: list                # per sequence: list of (start, len) visual segments
    q: np.ndarray                 # [B, Hq, d]
    K: np.ndarray                 # [B, Hkv, S_cap, d]
    V: np.ndarray                 # [B, Hkv, S_cap, d]
    tau_mass: float = 0.1         # 5% preset (App. B.1)
    tau_score: float = 1.0
    r_lo_bp: int = 100            # (0.01N, 0.05N) clamp (Sec. 5.2)
    r_hi_bp: int = 500
    clamp: bool = True
    meta: dict = field(default_factory=dict)

    @property
    def n_vis(self) -> np.ndarray:
        return np.array([sum(n for _, n in segs) for segs in self.segments], dtype=np.int32)

    @property
    def max_vis(self) -> int:
        return int(max(1, self.n_vis.max()))

    @property
    def max_segs(self) -> int:
        return int(max(1, max(len(s) for s in self.segments)))

    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4


def layout_arrays(segments):
    """CSR form of per-sequence segment lists: (seg_off [B+1] int32, seg [nseg, 2] int32)."""
    off = [0]
    flat = []
    for segs in segments:
        flat.extend(segs)
        off.append(len(flat))
    seg = np.array(flat, dtype=np.int32).reshape(-1, 2) if flat else np.zeros((0, 2), np.int32)
    return np.array(off, dtype=np.int32), seg


# --------------------------------------------------------------------------
# seeded streams: one independent stream per (config, sequence, purpose)
# --------------------------------------------------------------------------
_STREAMS = {"q": 0, "K": 1, "V": 2, "spike": 3, "lengths": 4, "offset": 5, "steps": 6, "queries": 7}


def _rng(cfg: int, stream: str, b: int = 0, seed: int | None = None) -> np.random.Generator:
    base = 1000 + cfg if seed is None else seed
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence(entropy=base, spawn_key=(_STREAMS[stream], b))))


def _normal(rng, shape, scale=1.0):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x


def _group_dirs(q_b: np.ndarray, Hkv: int) -> np.ndarray:
    """q_hat_g = sum_{h in g} q_h / ||sum_{h in g} q_h|| per KV group (spike direction)."""
    Hq, d = q_b.shape
    G = Hq // Hkv
    s = q_b.astype(np.float64).reshape(Hkv, G, d).sum(axis=1)
    n = np.linalg.norm(s, axis=1, keepdims=True)
    n[n == 0] = 1.0
    return (s / n).astype(np.float32)


# --------------------------------------------------------------------------
# the five configurations
# --------------------------------------------------------------------------
# cfg3: additive offset on every visual key along q_hat_g, drawn per sequence so
# that the head-max visual mass at tau = 0.1 spans roughly 0.01 .. 0.6
# (the range was found once by sweeping the offset; it is a constant here).
CFG3_OFFSET_RANGE = (-4.2, -2.7)

CONFIGS = {
    1: dict(name="tiny-fp32", dtype="f32", B=1, Hq=4, Hkv=1, d=64),
    2: dict(name="7b-b1", dtype="bf16", B=1, Hq=28, Hkv=4, d=128),
    3: dict(name="7b-b16-ragged", dtype="bf16", B=16, Hq=28, Hkv=4, d=128),
    4: dict(name="7b-b64-multiimage-32k", dtype="bf16", B=64, Hq=28, Hkv=4, d=128),
    5: dict(name="72b-b8-decode-loop", dtype="bf16", B=8, Hq=64, Hkv=8, d=128),
}


def _layout(cfg: int, B: int, seed=None):
    """Per-sequence (seq_len, segments, S_cap)."""
    if cfg == 1:
        return [384] * B, [[(16, 256)] for _ in range(B)], 384
    if cfg == 2:
        return [3358] * B, [[(14, 1296)] for _ in range(B)], 3358
    if cfg == 3:
        rng = _rng(3, "lengths", 0, seed)
        T = rng.integers(1024, 8192, size=B, endpoint=True)
        lens = [4096 + int(t) for t in T]
        return lens, [[(0, 4096)] for _ in range(B)], 4096 + 8192
    if cfg == 4:
        segs, p = [], 16
        for _ in range(4):
            segs.append((p, 4096))
            p += 4096 + 4092
        assert p == 32768
        return [32768] * B, [list(segs) for _ in range(B)], 32768
    if cfg == 5:
        # initial cache 6400 visual + 4096 text; one text token appended per step
        return [6400 + 4096] * B, [[(0, 6400)] for _ in range(B)], 6400 + 4096 + 512
    raise ValueError(cfg)


def _spike_fraction(cfg):
    return {1: 0.04, 2: 0.05, 3: 0.05, 4: 0.03, 5: 0.05}[cfg]


def generate(cfg: int, B: int | None = None, seqs=None, seed: int | None = None,
             S_cap: int | None = None) -> Workload:
    """Build configuration ``cfg`` (1..5).

    ``B`` overrides the batch size (smaller test cases keep the per-sequence
    shape); ``seqs`` restricts generation to a subset of sequence indices of the
    full batch (rows are drawn from per-sequence streams, so a subset is
    byte-identical to the same rows of the full batch). ``seed`` replaces the
    per-config base seed.
    """
    c = CONFIGS[cfg]
    Bfull = c["B"] if B is None else B
    lens_all, segs_all, S_def = _layout(cfg, Bfull, seed)
    idx = list(range(Bfull)) if seqs is None else list(seqs)
    Bn = len(idx)
    Hq, Hkv, d = c["Hq"], c["Hkv"], c["d"]
    S_cap = S_def if S_cap is None else S_cap
    f32 = c["dtype"] == "f32"
    st = np.float32 if f32 else np.uint16
    q = np.zeros((Bn, Hq, d), dtype=st)
    K = np.zeros((Bn, Hkv, S_cap, d), dtype=st)
    V = np.zeros((Bn, Hkv, S_cap, d), dtype=st)
    kv_scale = 1.0 if cfg == 1 else 0.5
    frac = _spike_fraction(cfg)
    offsets = [0.0] * Bn

    def one(i):
        b = idx[i]
        L = lens_all[b]
        segs = segs_all[b]
        qb = _normal(_rng(cfg, "q", b, seed), (Hq, d))
        Kb = _normal(_rng(cfg, "K", b, seed), (Hkv, L, d), kv_scale)
        Vb = _normal(_rng(cfg, "V", b, seed), (Hkv, L, d), kv_scale)
        dirs = _group_dirs(qb, Hkv)                     # [Hkv, d]
        vis = np.concatenate([np.arange(s, s + n) for s, n in segs])
        rs = _rng(cfg, "spike", b, seed)
        n_spike = int(round(frac * len(vis)))
        spiked = np.sort(rs.choice(vis, size=n_spike, replace=False))
        Kb[:, spiked, :] += np.float32(3.0) * dirs[:, None, :]
        if cfg == 3:
            ro = _rng(cfg, "offset", b, seed)
            s_b = float(ro.uniform(*CFG3_OFFSET_RANGE))
            Kb[:, vis, :] += np.float32(s_b) * dirs[:, None, :]
            offsets[i] = s_b
        if f32:
            q[i] = qb
            K[i, :, :L] = Kb
            V[i, :, :L] = Vb
        else:
            q[i] = bf16_round(qb)
            K[i, :, :L] = bf16_round(Kb)
            V[i, :, :L] = bf16_round(Vb)

    if Bn > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=min(Bn, 8, os.cpu_count() or 1)) as ex:
            list(ex.map(one, range(Bn)))
    else:
        one(0)
    w = Workload(name=c["name"], dtype=c["dtype"], B=Bn, Hq=Hq, Hkv=Hkv, d=d, S_cap=S_cap,
                 seq_len=np.array([lens_all[b] for b in idx], dtype=np.int32),
                 segments=[list(segs_all[b]) for b in idx], q=q, K=K, V=V,
                 meta={"cfg": cfg, "seqs": idx, "seed": seed, "cfg3_offsets": offsets})
    return w


# --------------------------------------------------------------------------
# configuration 5: the 512-step decode loop
# --------------------------------------------------------------------------
class Cfg5Stream:
    """Per-step inputs of the 72B-class decode loop.

    Step t (0-based) appends one text token's K/V row at position 10496 + t and
    then runs the path with seq_len = 10497 + t. The query drifts as
    q_t = 0.9 q_{t-1} + 0.1 eps_t (eps ~ N(0, 1)), carried in float32 and rounded
    to bfloat16 for use. Spikes toward q_hat_g(q_0) sit on 5% of the visual keys.
    """

    def __init__(self, B: int | None = None, steps: int = 512, seed: int | None = None):
        self.w = generate(5, B=B, seed=seed)
        self.steps = steps
        self.seed = seed
        self._q = bf16_to_f32(self.w.q).astype(np.float32)
        self.base_len = int(self.w.seq_len[0])

    def step_inputs(self, t: int):
        """(q_t bits [B, Hq, d], new K row bits [B, Hkv, d], new V row bits, position)."""
        w = self.w
        rng = _rng(5, "steps", t, self.seed)
        eps = _normal(rng, (w.B, w.Hq, w.d))
        if t > 0:
            self._q = np.float32(0.9) * self._q + np.float32(0.1) * eps
        kr = _normal(rng, (w.B, w.Hkv, w.d), 0.5)
        vr = _normal(rng, (w.B, w.Hkv, w.d), 0.5)
        return bf16_round(self._q), bf16_round(kr), bf16_round(vr), self.base_len + t


# --------------------------------------------------------------------------
# several queries per sequence (speculative / multi-token decoding)
# --------------------------------------------------------------------------
def with_queries(w: Workload, T: int, seed: int = 0) -> Workload:
    """A copy of ``w`` whose q holds T queries per sequence, [B, T, Hq, d]:
    query 0 is w's query and q_t = 0.9 q_{t-1} + 0.1 eps_t (eps ~ N(0, 1)), the
    drift of the decode loop, carried in float32 and rounded to the stored
    dtype. The queries stand for the last T positions of each sequence (whose
    K/V rows are the text rows the generator already wrote there)."""
    f32 = w.dtype == "f32"
    q = (w.q if f32 else bf16_to_f32(w.q)).astype(np.float32)
    qs = [q]
    cur = q.copy()
    for t in range(1, T):
        eps = _normal(_rng(0, "queries", t, 7000 + seed), q.shape)
        cur = np.float32(0.9) * cur + np.float32(0.1) * eps
        qs.append(cur.copy())
    qt = np.stack(qs, axis=1)
    return Workload(name=f"{w.name}-q{T}", dtype=w.dtype, B=w.B, Hq=w.Hq, Hkv=w.Hkv, d=w.d, S_cap=w.S_cap,
                    seq_len=w.seq_len.copy(), segments=[list(x) for x in w.segments],
                    q=qt if f32 else bf16_round(qt), K=w.K.copy(), V=w.V.copy(), tau_mass=w.tau_mass,
                    tau_score=w.tau_score, r_lo_bp=w.r_lo_bp, r_hi_bp=w.r_hi_bp, clamp=w.clamp,
                    meta=dict(w.meta, queries=T))
