"""Device buffers for one decode step and the four C-ABI calls in order.

Marshalling only: uploads a ``workloads.Workload`` to the GPU (torch
allocations), fills the ABI structs and calls vp_visual_mass -> vp_budget ->
vp_select_topk -> vp_sparse_decode_attn through ``vp``. All arithmetic runs in
libvisionpulse.so.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import vp
from .workloads import Workload, layout_arrays


def _dev(a: np.ndarray, device) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def make_params(w: Workload, sm_scale: float = 0.0) -> vp.vp_params:
    return vp.vp_params(tau_mass=w.tau_mass, tau_score=w.tau_score, sm_scale=sm_scale,
                        r_lo_bp=w.r_lo_bp, r_hi_bp=w.r_hi_bp, clamp=int(w.clamp))


def paged_cache(K: np.ndarray, V: np.ndarray, block_size: int, seed: int = 0):
    """The caches [B][Hkv][S][d] as paged caches [NB][Hkv][block_size][d]:
    block j of sequence b (rows j*block_size ...) goes to physical block
    table[b, j], a seeded permutation of B*nblk + nblk//2 + 1 blocks (the spare
    blocks stay zero). Returns (K_paged, V_paged, table int32 [B][nblk])."""
    B, Hkv, S, d = K.shape
    nblk = -(-S // block_size)
    nb = B * nblk + nblk // 2 + 1
    perm = np.random.default_rng(seed).permutation(nb)[:B * nblk].astype(np.int32)
    table = perm.reshape(B, nblk)
    Kp = np.zeros((nb, Hkv, block_size, d), K.dtype)
    Vp = np.zeros((nb, Hkv, block_size, d), V.dtype)
    for b in range(B):
        for j in range(nblk):
            r0, r1 = j * block_size, min(S, (j + 1) * block_size)
            Kp[table[b, j], :, :r1 - r0] = K[b, :, r0:r1]
            Vp[table[b, j], :, :r1 - r0] = V[b, :, r0:r1]
    return Kp, Vp, np.ascontiguousarray(table)


class DeviceStep:
    """Device-resident inputs, outputs and workspace of one step of workload ``w``.

    ``kv_groups``: one budget and kept set per KV group (VP_SCOPE_KV_GROUP);
    results() then returns mass_seq [B, Hkv, 2], scores [B, Hkv, max_vis],
    k [B, Hkv] and vis_idx [B, Hkv, k_cap]. A workload whose q is
    [B, T, Hq, d] runs T queries per sequence (n_queries = T); results() then
    has a query axis after the batch axis (mass_head [B, T, Hq], out
    [B, T, Hq, d], k [B, T] or [B, T, Hkv], ...).
    """

    def __init__(self, w: Workload, device="cuda:0", k_cap: int | None = None, max_vis: int | None = None,
                 kv=None, block_size: int = 0, block_seed: int = 0, kv_groups: bool = False):
        self.w = w
        self.T = w.q.shape[1] if w.q.ndim == 4 else 1
        self.kv_groups = kv_groups
        self.rows = w.Hkv if kv_groups else 1  # selection rows per query
        self.device = torch.device(device)
        self.q = _dev(w.q, self.device)
        self.block_size = block_size
        self.block_table = None
        if block_size:
            # paged caches: the sequences' blocks of block_size rows dealt to
            # physical blocks in a seeded random order (plus unused spare blocks)
            Kp, Vp, table = paged_cache(w.K, w.V, block_size, block_seed)
            self.K, self.V = _dev(Kp, self.device), _dev(Vp, self.device)
            self.block_table = torch.from_numpy(table).to(self.device)
        elif kv is None:
            self.K = _dev(w.K, self.device)
            self.V = _dev(w.V, self.device)
        else:
            self.K, self.V = kv
        off, seg = layout_arrays(w.segments)
        self.seq_len = torch.from_numpy(w.seq_len.astype(np.int32)).to(self.device)
        self.seg_off = torch.from_numpy(off).to(self.device)
        self.seg = torch.from_numpy(seg.reshape(-1) if seg.size else np.zeros(2, np.int32)).to(self.device)
        B, Hq, d = w.B, w.Hq, w.d
        self.max_vis = max_vis or w.max_vis
        self.params = make_params(w)
        # row capacity of the kept-index output: the largest budget the rule
        # allows for max_vis visual tokens (its value at full visual mass)
        self.k_cap = k_cap or max(1, int(vp.lib().vp_budget_host(1.0, self.max_vis, ctypes.byref(self.params))))
        st = self.K.stride()
        self.shape = vp.vp_shape(batch=B, n_q_heads=Hq, n_kv_heads=w.Hkv, head_dim=d,
                                 dtype=vp.VP_BF16 if w.dtype == "bf16" else vp.VP_F32,
                                 max_seq_len=w.S_cap, max_vis=self.max_vis, max_segs=w.max_segs,
                                 k_cap=self.k_cap, block_size=block_size,
                                 scope=vp.VP_SCOPE_KV_GROUP if kv_groups else vp.VP_SCOPE_SEQUENCE,
                                 n_queries=self.T,
                                 kv_stride_b=st[0], kv_stride_h=st[1], kv_stride_s=st[2])
        self.layout = vp.vp_layout(seq_len=self.seq_len.data_ptr(), vis_seg_off=self.seg_off.data_ptr(),
                                   vis_seg=self.seg.data_ptr(),
                                   block_table=self.block_table.data_ptr() if block_size else None)
        f32 = dict(dtype=torch.float32, device=self.device)
        i32 = dict(dtype=torch.int32, device=self.device)
        T = self.T
        self.mass_head = torch.zeros(B * T, Hq, **f32)
        R = B * T * self.rows  # selection rows
        self.mass_seq = torch.zeros(R, 2, **f32)
        self.scores = torch.zeros(R, self.max_vis, **f32)
        self.k = torch.zeros(R, **i32)
        self.vis_idx = torch.full((R, self.k_cap), -7, **i32)
        self.out = torch.zeros(B * T, Hq, d, dtype=self.q.dtype, device=self.device)
        self.ws_bytes = vp.vp_workspace_size(self.shape)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)

    # the four calls ------------------------------------------------------
    def visual_mass(self, fused=True, stream=None):
        vp.vp_visual_mass(self.shape, self.layout, self.params, self.q, self.K, self.V if fused else None,
                          self.mass_head, self.mass_seq, self.scores, self.ws, self.ws_bytes, stream)

    def budget(self, stream=None):
        vp.vp_budget(self.shape, self.layout, self.params, self.mass_seq, self.k, stream)

    def select_topk(self, stream=None):
        vp.vp_select_topk(self.shape, self.layout, self.scores, self.k, self.vis_idx, stream)

    def sparse_decode_attn(self, fused=True, stream=None):
        vp.vp_sparse_decode_attn(self.shape, self.layout, self.params, self.q, self.K, self.V, self.vis_idx,
                                 self.k, self.out, vp.VP_ATTN_TEXT_FROM_WORKSPACE if fused else 0,
                                 self.ws, self.ws_bytes, stream)

    def decode_step(self, stream=None, events=()):
        vp.vp_decode_step(self.shape, self.layout, self.params, self.q, self.K, self.V, self.mass_head,
                          self.mass_seq, self.scores, self.k, self.vis_idx, self.out, self.ws, self.ws_bytes,
                          stream, events)

    def run(self, fused=True, stream=None):
        self.visual_mass(fused, stream)
        self.budget(stream)
        self.select_topk(stream)
        self.sparse_decode_attn(fused, stream)

    def results(self) -> dict:
        torch.cuda.synchronize(self.device)
        B, T = self.w.B, self.T
        qlead = (B, T) if T > 1 else (B,)
        lead = qlead + ((self.rows,) if self.kv_groups else ())
        rows = lambda t: t.cpu().numpy().reshape(lead + tuple(t.shape[1:]))
        per_query = lambda t: t.cpu().numpy().reshape(qlead + tuple(t.shape[1:]))
        return dict(mass_head=per_query(self.mass_head), mass_seq=rows(self.mass_seq),
                    scores=rows(self.scores), k=rows(self.k), vis_idx=rows(self.vis_idx),
                    out=per_query(self.out.float()))
