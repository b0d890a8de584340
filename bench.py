#!/usr/bin/env python3
"""Throughput of the VisionPulse per-decode-step path on one MI355X.

One step = one vp_decode_step call (the results of vp_visual_mass ->
vp_budget -> vp_select_topk -> vp_sparse_decode_attn, in fewer launches) over
the whole batch on one layer's KV cache (the anchor layer); --calls times the
four separate calls instead. Inputs are seeded synthetic tensors shaped
like the paper's LMM decode workloads (paper_2605_31457_amd.workloads), resident
in HBM before timing. To keep the 256 MB Infinity Cache from serving the cache
reads, the step rotates over R distinct copies of the KV cache (R * KV bytes
>= 1 GiB), as a real model's layers would.

Prints one JSON line: steps/s, the roofline of the kernel that carries most of
the step's bytes (the text pass: every text K and V row; its duration comes from
HIP events attached to that launch in steps run after the timed ones, so the
timed steps record no events), the streaming-read ceiling measured on the same
GPU, and the fp64 reference timed on this host's cores (one thread, and all the
cores this process may use).

The default workload is config 4 (64 sequences of 32k tokens, 3.33 GB of
algorithmic bytes per step), the largest that fits one GPU.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 4]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import re
import sys
import time

PEAK_HBM_GBS = 8000.0   # MI355X HBM3E, 8 TB/s
MALL_DEFEAT_BYTES = 1 << 30

WORKLOAD_NAMES = {
    1: "tiny fp32 check: B=1, 4/1 heads, d=64, 16 text + 256 visual + 112 text",
    2: "7B-class decode layer: B=1, 28/4 heads, d=128, 1296 visual (36x36) at 14 + 2048 text",
    3: "7B-class ragged batch: B=16, 28/4 heads, d=128, 4096 visual + U{1024..8192} text",
    4: "7B-class multi-image 32k: B=64, 28/4 heads, d=128, 4 x 4096 visual + 16384 text",
    5: "72B-class decode loop: B=8, 64/8 heads, d=128, 6400 visual + 4097..4608 text over 512 steps",
}
DEFAULT_STEPS = {1: (200, 20), 2: (400, 40), 3: (200, 10), 4: (100, 5), 5: (512, 16)}


def workload_name(cfg: int, batch=None) -> str:
    """The configuration's name; with --batch, its batch size replaced."""
    name = WORKLOAD_NAMES[cfg]
    if batch is not None:
        name = re.sub(r"B=\d+", f"B={batch}", name, count=1)
    return f"config {cfg}: {name}"


class Hip:
    """hipEvent helpers through the HIP runtime's C API."""

    def __init__(self):
        self.h = ctypes.CDLL("libamdhip64.so")
        self.h.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.h.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.h.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def event(self):
        e = ctypes.c_void_p()
        assert self.h.hipEventCreate(ctypes.byref(e)) == 0
        return e

    def elapsed_ms(self, a, b):
        t = ctypes.c_float()
        assert self.h.hipEventElapsedTime(ctypes.byref(t), a, b) == 0
        return t.value


def algorithmic_bytes(w, ks, lens=None, rows=1, kv_per_row=None):
    """Bytes the method must move at least once per step, by kernel.

    Visual pass: the K rows of visual tokens (their Eq. (6) logits). Text pass:
    the K and V rows of text tokens. Kept pass: K and V rows of the k kept
    visual tokens. q, outputs, scores and indices are < 1% and not counted.
    lens: per-step sequence lengths of a decode loop (same for every sequence);
    the figures are then averages over its steps. rows: selection rows per
    sequence (T queries x (1, or Hkv with per-KV-group budgets)); kv_per_row:
    the KV heads whose kept rows a selection row's list names (Hkv, or 1)."""
    kv_per_row = w.Hkv if kv_per_row is None else kv_per_row
    esz = 2 if w.dtype == "bf16" else 4
    row = w.Hkv * w.d * esz
    vis = text = kept = 0
    for b in range(w.B):
        Ls = [int(w.seq_len[b])] if lens is None else list(lens)
        nv = sum(n for _, n in w.segments[b])
        vis += nv * row
        text += sum(2 * (L - nv) * row for L in Ls) / len(Ls)
        kept += 2 * int(sum(ks[b * rows:(b + 1) * rows])) * w.d * esz * kv_per_row
    return {"visual": vis, "text": text, "kept": kept}


# the sources that set what the context passes (the roofline kernels) read and
# write: their kernels, their launch plan and their arguments
ROOFLINE_SOURCES = ("vp_attend.hip", "vp_common.h", "vp_internal.h", "vp_plan.hip")


def kernel_source_hash(root: str) -> str:
    """sha256 over the roofline kernels' sources with comments and blank space
    removed, so that a comment edit does not mark the stored counter figures stale."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in sorted(ROOFLINE_SOURCES):
        f = os.path.join(root, "paper_2605_31457_amd", "csrc", name)
        with open(f) as src:
            text = src.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(os.path.basename(f).encode())
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def counter_traffic(cfg: int, kernel: str):
    """HBM bytes per launch of the roofline kernel ("text": the text pass;
    "one_launch": both context passes in one launch) from the FETCH_SIZE /
    WRITE_SIZE counter runs summarised in profiles/ (FETCH_SIZE scaled by a
    plain copy's reading), or None when they were taken on other kernel
    sources, another configuration or another kernel."""
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", "text_pass_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    entry = rec.get("configs", {}).get(str(cfg))
    if kernel_source_hash(root) != rec.get("source_sha256") or entry is None or entry.get("kernel") != kernel:
        return None
    return entry["traffic_bytes"]


def stream_ceiling(hip, sp, nbytes=4 << 30, reps=5):
    """Streaming-read ceiling of this GPU (informational): one read of a 4 GiB
    buffer (16x the Infinity Cache) through vector loads and through the LDS
    copies of the decode-step kernels (vp_stream_read), each timed with HIP
    events around single launches; the best of `reps` per path."""
    import numpy as np
    import torch
    from paper_2605_31457_amd import vp
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = {"buffer_bytes": nbytes, "unit": "GB/s"}
    e0, e1 = hip.event(), hip.event()
    for mode, name in ((0, "vector_loads"), (1, "lds_copies")):
        times = []
        for r in range(reps + 1):
            hip.h.hipEventRecord(e0, sp)
            vp.vp_stream_read(buf, nbytes, mode, sink, sp)
            hip.h.hipEventRecord(e1, sp)
            hip.h.hipEventSynchronize(e1)
            if r:
                times.append(hip.elapsed_ms(e0, e1))
        out[name] = nbytes / (min(times) * 1e-3) / 1e9
        out[name + "_median"] = nbytes / (float(np.median(times)) * 1e-3) / 1e9
    out["ceiling"] = max(out["vector_loads"], out["lds_copies"])
    del buf
    torch.cuda.empty_cache()
    return out


def _cores():
    """Cores this process may use for the reference: its CPU affinity, capped by
    OMP_NUM_THREADS when that is set (one machine's share of a larger host)."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, n)


def cpu_baseline(w, budget_s: float, kv_groups: bool = False, gpu=None):
    """fp64 reference on this host, in two legs of about budget_s seconds each:
    one thread (sequences one after another, single-threaded BLAS), then every
    core this process may use (that many sequences at once, one thread each).
    steps/s = sequence-steps done / wall time / B.

    With ``gpu`` (the GPU step's results on the same inputs, one query per
    sequence, budgets per sequence), every sequence the reference finished is
    also compared with them: parity of the measured run's outputs."""
    from concurrent.futures import ThreadPoolExecutor

    import threadpoolctl

    from oracle import vp_oracle as O
    from oracle.plant import params_of
    p = params_of(w)
    done = {}

    def one(b):
        if w.q.ndim == 4:  # several queries per sequence
            return O.decode_step_queries(w.q[b], w.K[b], w.V[b], int(w.seq_len[b]), w.segments[b], p,
                                         kv_groups=kv_groups)
        run = O.decode_step_sequence_kv_groups if kv_groups else O.decode_step_sequence
        return run(w.q[b], w.K[b], w.V[b], int(w.seq_len[b]), w.segments[b], p)

    def leg(workers):
        n = 0
        t0 = time.perf_counter()
        with threadpoolctl.threadpool_limits(1), ThreadPoolExecutor(workers) as ex:
            while True:
                bs = [(n + i) % w.B for i in range(workers)]
                for b, r in zip(bs, ex.map(one, bs)):
                    if w.q.ndim == 3 and b not in done:
                        done[b] = r
                n += workers
                el = time.perf_counter() - t0
                if el >= budget_s:
                    break
        return {"value": n / el / w.B, "unit": "steps/s", "cores": workers, "sequence_steps": n,
                "wall_s": round(el, 2)}

    one_thread = leg(1)
    cores = _cores()
    all_cores = leg(cores) if cores > 1 else dict(one_thread)
    model = ""
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
    except OSError:
        pass
    out = {"value": all_cores["value"], "unit": "steps/s", "cores": all_cores["cores"], "kind": "oracle",
           "host_cpu": model, "one_thread": one_thread, "all_cores": all_cores,
           "sample": f"whole sequence-steps of this workload's batch, sequences 0, 1, ... in turn: "
                     f"{one_thread['sequence_steps']} on one thread in {one_thread['wall_s']} s, then "
                     f"{all_cores['sequence_steps']} on {all_cores['cores']} threads (one sequence each, "
                     f"single-threaded BLAS) in {all_cores['wall_s']} s; steps/s = sequence-steps / s / B={w.B}"}
    if gpu is not None and w.q.ndim == 3 and not kv_groups:
        out["parity_of_measured_run"] = measured_parity(w, gpu, done, p, O)
    return out


def loop_parity(w, gpu, q_t, L_t, seqs=(0, 1)):
    """The decode loop's last timed step (query q_t, length L_t) against the
    reference, on a few of its sequences (the cpu_baseline leg's oracle use)."""
    import dataclasses
    import numpy as np
    from oracle import vp_oracle as O
    from oracle.plant import params_of
    wl = dataclasses.replace(w, q=np.ascontiguousarray(q_t), seq_len=np.full(w.B, L_t, np.int32))
    p = params_of(wl)
    ref = {b: O.decode_step_sequence(wl.q[b], wl.K[b], wl.V[b], L_t, wl.segments[b], p) for b in seqs}
    rep = measured_parity(wl, gpu, ref, p, O)
    rep["step"] = f"loop step with length {L_t}"
    return rep


def measured_parity(w, gpu, ref, p, O):
    """The timed run's outputs against the reference on the same (unplanted)
    inputs: masses and scores to 1e-5 relative; the budget exact unless
    M_vis,max * N_v lies within 2e-5 of a rounding boundary; the kept set exact,
    or differing only in tokens within 2e-5 relative of the cut score; outputs to
    the dtype's tolerance wherever the sets agree."""
    import numpy as np
    band = 2e-5
    atol, rtol = (2e-2, 1e-2) if w.dtype == "bf16" else (1e-5, 1e-5)
    rep = {"sequences": len(ref), "masses_and_scores": True, "budgets_exact": 0, "budgets_in_band": 0,
           "sets_exact": 0, "sets_in_band": 0, "outputs_checked": 0, "outputs_ok": True, "ok": True}
    for b, r in ref.items():
        vis = O.visual_positions(int(w.seq_len[b]), w.segments[b])
        nv = len(vis)
        close = lambda x, y: np.allclose(x, y, rtol=1e-5, atol=1e-30)
        if not (close(gpu["mass_head"][b], r.mass_head) and close(gpu["mass_seq"][b], [r.M_vis, r.M_vis_max])
                and close(gpu["scores"][b, :nv], r.scores)):
            rep["masses_and_scores"] = False
        k = int(gpu["k"][b])
        ks = {O.budget(r.M_vis_max * (1 + s * band), nv, p.r_lo_bp, p.r_hi_bp, p.clamp) for s in (-1, 0, 1)}
        if k == r.k:
            rep["budgets_exact"] += 1
        elif k in ks:
            rep["budgets_in_band"] += 1
        else:
            rep["ok"] = False
        sel = gpu["vis_idx"][b, :k]
        want = O.select_top_k(r.scores, vis, k)
        if np.array_equal(sel, want):
            rep["sets_exact"] += 1
            if k == r.k:
                rep["outputs_checked"] += 1
                if not np.allclose(gpu["out"][b], r.out, atol=atol, rtol=rtol):
                    rep["outputs_ok"] = False
        else:
            order = np.lexsort((vis, -r.scores))
            cut = r.scores[order[k - 1]] if k > 0 else 0.0
            diff = np.searchsorted(vis, np.setxor1d(sel, want))
            if np.all(np.abs(r.scores[diff] - cut) <= band * cut):
                rep["sets_in_band"] += 1
            else:
                rep["ok"] = False
    rep["ok"] = rep["ok"] and rep["masses_and_scores"] and rep["outputs_ok"]
    return rep


def bench_layers(args, w, ds, bufs, loop, steps, warmup, sp, hip):
    """A per-token attention step over L layers, timed as a whole: A =
    --anchor-layer layers of full attention (pruning starts at the anchor layer,
    Sec. 4.1), the anchor layer's vp_decode_step, and L-A-1 calls of
    vp_sparse_decode_attn on the later layers' caches with the anchor's kept set
    (they reuse its selection); with --dense, L layers of full attention
    (vp_sparse_decode_attn on a layout with no visual segments, so every cached
    row goes through the streaming text pass). Layer l of step i reads cache
    copy (i * L + l) mod R."""
    import numpy as np
    import torch
    from paper_2605_31457_amd import vp
    L, R = args.layers, len(bufs)
    A = 0 if args.dense else args.anchor_layer
    out_l = torch.empty_like(ds.out)
    lay_dense = None
    if args.dense or A > 0:
        seg_off0 = torch.zeros(w.B + 1, dtype=torch.int32, device=ds.device)
        seg0 = torch.zeros(2, dtype=torch.int32, device=ds.device)
        k0 = torch.zeros(w.B, dtype=torch.int32, device=ds.device)
        lay_dense = [vp.vp_layout(seq_len=(loop[2][t].seq_len if loop else ds.layout.seq_len),
                                  vis_seg_off=seg_off0.data_ptr(), vis_seg=seg0.data_ptr(),
                                  block_table=ds.layout.block_table)
                     for t in range(loop[0] if loop else 1)]

    def one(i):
        t = i % loop[0] if loop else 0
        q = loop[1][t] if loop else ds.q
        lay = loop[2][t] if loop else ds.layout
        if args.dense:
            for layer in range(L):
                K, V = bufs[(i * L + layer) % R]
                vp.vp_sparse_decode_attn(ds.shape, lay_dense[t], ds.params, q, K, V, ds.vis_idx, k0, out_l, 0,
                                         ds.ws, ds.ws_bytes, sp)
            return
        for layer in range(A):
            K, V = bufs[(i * L + layer) % R]
            vp.vp_sparse_decode_attn(ds.shape, lay_dense[t], ds.params, q, K, V, ds.vis_idx, k0, out_l, 0,
                                     ds.ws, ds.ws_bytes, sp)
        K, V = bufs[(i * L + A) % R]
        vp.vp_decode_step(ds.shape, lay, ds.params, q, K, V, ds.mass_head, ds.mass_seq, ds.scores, ds.k,
                          ds.vis_idx, ds.out, ds.ws, ds.ws_bytes, sp)
        for layer in range(A + 1, L):
            K, V = bufs[(i * L + layer) % R]
            vp.vp_sparse_decode_attn(ds.shape, lay, ds.params, q, K, V, ds.vis_idx, ds.k, out_l, 0,
                                     ds.ws, ds.ws_bytes, sp)

    for i in range(warmup):
        one(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        one(warmup + i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ks = ds.k.cpu().numpy()
    nb = algorithmic_bytes(w, ks, None if loop is None else loop[3], rows=ds.T * ds.rows,
                           kv_per_row=w.Hkv // ds.rows)
    esz = 2 if w.dtype == "bf16" else 4
    row = w.Hkv * w.d * esz
    # a dense layer: every cached K and V row of every sequence
    if loop:
        per_dense = w.B * 2 * row * sum(loop[3]) / len(loop[3])
    else:
        per_dense = sum(2 * int(n) * row for n in w.seq_len)
    if args.dense:
        step_bytes = L * per_dense
    else:
        step_bytes = A * per_dense + nb["visual"] + nb["text"] + nb["kept"] + (L - A - 1) * (nb["text"] + nb["kept"])
    ms = wall * 1e3 / steps
    res = {"metric": "per-token attention steps/s over several layers", "value": steps / wall, "unit": "steps/s",
           "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": ms, "higher_is_better": True,
           "layers": L, "anchor_layer": A,
           "mode": "dense" if args.dense else "dense layers, anchor decode step, sparse layers",
           "step_algorithmic_bytes": step_bytes, "step_achieved_GBps": step_bytes / (ms * 1e-3) / 1e9,
           "dtype": w.dtype, "data": "synthetic", "config": {"workload": workload_name(args.config, args.batch),
                                                             "kv_copies": R}}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--config", type=int, default=4, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--rotate", type=int, default=0, help="KV copies to rotate over (0: >= 1 GiB)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="seconds of reference work per leg (one thread, then all cores)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calls", action="store_true", help="time the four separate calls instead of vp_decode_step")
    ap.add_argument("--layers", type=int, default=1,
                    help="time a per-token step over this many layers, each on its own KV cache: the layers "
                         "before the anchor (--anchor-layer) attend densely, the anchor runs the decode step, the "
                         "later layers attend over the anchor's kept set")
    ap.add_argument("--batch", type=int, default=None, metavar="B",
                    help="configs 3 and 4: B sequences of the configuration's per-sequence shape")
    ap.add_argument("--anchor-layer", type=int, default=0, metavar="A",
                    help="with --layers L: layers 0..A-1 attend densely, layer A is the anchor (0 <= A < L)")
    ap.add_argument("--dense", action="store_true",
                    help="with --layers: every layer attends to all of its cached tokens instead")
    ap.add_argument("--paged", type=int, default=0, metavar="P",
                    help="paged KV caches: blocks of P rows (a power of two) dealt to physical blocks in a "
                         "seeded random order, addressed through a block table")
    ap.add_argument("--queries", type=int, default=1, metavar="T",
                    help="T queries per sequence in one step (speculative / multi-token decoding; configs 1-4): "
                         "the last T positions are the queries, each a step of its own over its prefix")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of a HIP graph holding one step per rotated cache copy")
    ap.add_argument("--kv-groups", action="store_true",
                    help="one budget and kept set per KV group (VP_SCOPE_KV_GROUP) instead of per sequence")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (3 times): the reference "
                         "for scaling the FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the VisionPulse step is measured on a single MI355X "
              "(sequences shard across GPUs with no exchange; see the design notes). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2605_31457_amd import step as S
    from paper_2605_31457_amd import vp
    from paper_2605_31457_amd import workloads as W

    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 3}), flush=True)
        return

    cfg = args.config
    if not 0 <= args.anchor_layer < max(1, args.layers):
        print("bench.py --anchor-layer A: 0 <= A < --layers", file=sys.stderr)
        sys.exit(2)
    if args.graph and (cfg == 5 or args.calls or args.layers > 1 or args.dense):
        print("bench.py --graph: configs 1-4, one-call steps, one layer", file=sys.stderr)
        sys.exit(2)
    if args.batch is not None and (cfg not in (3, 4) or not 1 <= args.batch <= 64):
        print("bench.py --batch B: configs 3 and 4, 1 <= B <= 64 (the per-sequence shape is kept)", file=sys.stderr)
        sys.exit(2)
    if args.paged and cfg == 4 and (args.batch is None or args.batch > 16):
        # one run of this case ended in a host-side segmentation fault before
        # its first kernel launch (while the 2.2 GB paged caches were built and
        # uploaded), with no cause found in this code: held back until there is
        # one; batches of up to 16 sequences (paged caches under 0.6 GB) run
        print("bench.py --paged: configs 1-3 and 5, and config 4 with --batch 16 or fewer (the paged "
              "64 x 32k batch is held back after an unexplained host-side crash during its set-up)",
              file=sys.stderr)
        sys.exit(2)
    if args.queries > 1 and cfg == 5:
        print("bench.py --queries: configs 1-4 (the decode loop of config 5 runs one query per step)",
              file=sys.stderr)
        sys.exit(2)
    steps, warmup = DEFAULT_STEPS[cfg]
    steps = args.steps if args.steps is not None else steps
    warmup = args.warmup if args.warmup is not None else warmup

    vp.lib()  # fail loudly if the HIP library is missing
    print(f"[bench] generating config {cfg}", file=sys.stderr, flush=True)
    loop = None
    if cfg == 5:
        # the decode loop: all 512 appended rows and drifting queries are
        # generated and made resident first; step t runs with q_t and length
        # 10497 + t (rows past a step's length are not part of its cache)
        stream5 = W.Cfg5Stream(steps=512)
        w = stream5.w
        qs = []
        for t in range(stream5.steps):
            q_t, kr, vr, pos = stream5.step_inputs(t)
            w.K[:, :, pos] = kr
            w.V[:, :, pos] = vr
            qs.append(q_t)
        ds = S.DeviceStep(w, block_size=args.paged, kv_groups=args.kv_groups)
        q_all = torch.from_numpy(np.ascontiguousarray(np.stack(qs)).view(np.int16)).view(torch.bfloat16).to(ds.device)
        lens = torch.tensor([[stream5.base_len + t + 1] * w.B for t in range(stream5.steps)], dtype=torch.int32,
                            device=ds.device)
        layouts = [vp.vp_layout(seq_len=lens[t].data_ptr(), vis_seg_off=ds.seg_off.data_ptr(),
                                vis_seg=ds.seg.data_ptr(), block_table=ds.layout.block_table)
                   for t in range(stream5.steps)]
        loop = (stream5.steps, q_all, layouts, [stream5.base_len + t + 1 for t in range(stream5.steps)])
    else:
        w = W.generate(cfg, B=args.batch)
        if args.queries > 1:
            w = W.with_queries(w, args.queries)
        ds = S.DeviceStep(w, block_size=args.paged, kv_groups=args.kv_groups)
    kv_bytes = ds.K.numel() * ds.K.element_size() * 2
    R = args.rotate or max(1, math.ceil(MALL_DEFEAT_BYTES / kv_bytes))
    layered = args.layers > 1 or args.dense
    if layered:
        R = max(R, args.layers)  # every layer of a step reads its own cache copy
    bufs = [(ds.K, ds.V)]
    for _ in range(R - 1):
        bufs.append((ds.K.clone(), ds.V.clone()))
    torch.cuda.synchronize()
    print(f"[bench] {w.name}: KV {kv_bytes / 1e6:.1f} MB x {R} rotated copies; steps={steps} warmup={warmup}",
          file=sys.stderr, flush=True)

    hip = Hip()
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    if layered:
        bench_layers(args, w, ds, bufs, loop, steps, warmup, sp, hip)
        return
    # step events: [0] visual pass [1] text pass [2] tail [3] kept pass [4] merge [5].
    # An event record costs microseconds of queue time, which shows on small
    # steps, so the timed steps record none; the roofline launch's duration and
    # the per-phase split come from further steps run after the timed ones.
    NEV = vp.VP_STEP_EVENTS
    n_phase = 50
    evs_phase = [[hip.event() for _ in range(NEV)] for _ in range(n_phase)]
    # argument arrays built ahead of the runs
    arr_phase = [vp.event_array(e) for e in evs_phase]
    arr_phase3 = [vp.event_array(e[:3]) for e in evs_phase]
    ev_t0, ev_t1 = hip.event(), hip.event()

    def one_step(i, evs=(), arr6=(), arr3=()):
        K, V = bufs[i % R]
        q, lay = ds.q, ds.layout
        if loop is not None:
            q, lay = loop[1][i % loop[0]], loop[2][i % loop[0]]
        if not args.calls:
            vp.vp_decode_step(ds.shape, lay, ds.params, q, K, V, ds.mass_head, ds.mass_seq, ds.scores,
                              ds.k, ds.vis_idx, ds.out, ds.ws, ds.ws_bytes, sp, events=arr6)
            return
        vp.vp_visual_mass_timed(ds.shape, lay, ds.params, q, K, V, ds.mass_head, ds.mass_seq,
                                ds.scores, ds.ws, ds.ws_bytes, sp, events=arr3)
        vp.vp_budget(ds.shape, lay, ds.params, ds.mass_seq, ds.k, sp)
        vp.vp_select_topk(ds.shape, lay, ds.scores, ds.k, ds.vis_idx, sp)
        if evs and evs[3]:
            hip.h.hipEventRecord(evs[3], sp)
        vp.vp_sparse_decode_attn(ds.shape, lay, ds.params, q, K, V, ds.vis_idx, ds.k, ds.out,
                                 vp.VP_ATTN_TEXT_FROM_WORKSPACE, ds.ws, ds.ws_bytes, sp)
        if evs and evs[5]:
            hip.h.hipEventRecord(evs[5], sp)

    gs = None
    if args.graph:
        # capture needs a stream of its own; every step of the run goes there
        gs = torch.cuda.Stream()
        sp = gs.cuda_stream
        torch.cuda.set_stream(gs)
    for i in range(warmup):
        one_step(i)
    torch.cuda.synchronize()
    ks = ds.k.cpu().numpy().copy()

    graph = None
    if args.graph:
        # one step per rotated cache copy in one graph; the timed region replays it
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=gs):
            for i in range(R):
                one_step(warmup + i)
        torch.cuda.synchronize()
        reps = max(1, round(steps / R))
        steps = reps * R
    hip.h.hipEventRecord(ev_t0, sp)
    t0 = time.perf_counter()
    if graph is not None:
        for _ in range(reps):
            graph.replay()
    else:
        for i in range(steps):
            one_step(warmup + i)
    hip.h.hipEventRecord(ev_t1, sp)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = hip.elapsed_ms(ev_t0, ev_t1)
    for i in range(n_phase):
        one_step(warmup + steps + i, evs_phase[i], arr_phase[i], arr_phase3[i])
    torch.cuda.synchronize()

    def phase(i, j):
        return float(np.mean([hip.elapsed_ms(e[i], e[j]) for e in evs_phase]))
    # [1]..[2]: the roofline launch's execution alone (events attached to it)
    vis_ms, text_ms, tail_ms, attn_ms = phase(0, 1), phase(1, 2), phase(2, 3), phase(3, 5)
    ceiling = stream_ceiling(hip, sp)
    if loop is None:
        assert np.array_equal(ds.k.cpu().numpy(), ks), "budget changed between warm-up and timed steps"

    nb = algorithmic_bytes(w, ks, None if loop is None else loop[3], rows=ds.T * ds.rows,
                           kv_per_row=w.Hkv // ds.rows)
    step_bytes = nb["visual"] + nb["text"] + nb["kept"]
    ms_per_step = wall * 1e3 / steps
    plan = vp.vp_step_plan(ds.shape, ds.params)
    one_launch = bool(plan & vp.VP_PLAN_ONE_CONTEXT_LAUNCH)
    # the roofline kernel: the text pass, or (small caches) the one launch that
    # runs the visual and text passes together
    roof_bytes = nb["text"] + (nb["visual"] if one_launch else 0)
    achieved = roof_bytes / (text_ms * 1e-3) / 1e9
    step_gbs = step_bytes / (ms_per_step * 1e-3) / 1e9

    res = {
        "metric": "pruned decode-attention steps/s per layer; achieved HBM GB/s vs peak",
        "value": steps / wall,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded; shapes of the paper's LMM decode workloads)",
        "config": {"workload": workload_name(cfg, args.batch), "batch": w.B, "q_heads": w.Hq,
                   "kv_heads": w.Hkv, "head_dim": w.d, "max_seq_len": w.S_cap, "visual_tokens": int(w.n_vis[0]),
                   "tau_mass": w.tau_mass, "retention_clamp_bp": [w.r_lo_bp, w.r_hi_bp],
                   "kept_k": [int(x) for x in ks[:8]], "kv_rotation": R, "parallelism": "single GPU",
                   "kv_block_size": args.paged or None,
                   "budget_scope": "per KV group" if args.kv_groups else "per sequence",
                   "queries_per_sequence": ds.T},
        "step_algorithmic_bytes": step_bytes,
        "step_achieved_GBps": step_gbs,
        "step_frac_of_peak": step_gbs / PEAK_HBM_GBS,
        "gpu_event_ms_per_step": gpu_ms / steps,
        "roofline": {"kernel": (f"context pass, one launch (attend_dual_kernel<{w.dtype},{w.d}>: visual K and "
                                "text K/V, Eq. (6)/(5)/(2) statistics, logit spill, attention partial)")
                     if one_launch else
                     (f"text pass (attend_kernel<{w.dtype},{w.d},MODE_TEXT_BOTH>: text K/V, "
                      "Eq. (6)/(2) statistics, attention partial)"), "bound": "hbm",
                     "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS,
                     "traffic": counter_traffic(cfg, "one_launch" if one_launch else "text"),
                     "algorithmic_bytes_per_launch": roof_bytes,
                     "avg_launch_ms": text_ms, "share_of_step": text_ms / ms_per_step,
                     "launch_time_source": f"HIP events attached to the launch, mean of {n_phase} steps run "
                                           "after the timed ones",
                     "frac_of_measured_ceiling": achieved / ceiling["ceiling"]},
        "stream_read_ceiling": ceiling,
        "step_frac_of_measured_ceiling": step_gbs / ceiling["ceiling"],
        # separate visual launch: [0]..[1] runs from before it to the text pass's start
        "visual_pass": None if one_launch else {"achieved": nb["visual"] / (vis_ms * 1e-3) / 1e9, "unit": "GB/s",
                                                "algorithmic_bytes_per_launch": nb["visual"],
                                                "avg_phase_ms": vis_ms},
        "phases_ms": {"visual_pass": vis_ms, "text_pass": text_ms,
                      "mass_budget_scores_topk": tail_ms, "kept_pass_and_merge": attn_ms},
        "entry_point": ("four calls" if args.calls else "vp_decode_step") + (" (HIP graph replays)" if args.graph else ""),
        "plan": {"one_context_launch": one_launch, "select_in_one_group": bool(plan & vp.VP_PLAN_FUSED_TAIL)},
    }
    res["query_tokens_per_s"] = res["value"] * w.B * ds.T
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 reference on the host", file=sys.stderr, flush=True)
        # the reference on the timed run's inputs; for a single-step workload its
        # sequences are also compared with the run's own outputs
        gpu = ds.results() if loop is None and ds.T == 1 else None
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, args.kv_groups, gpu)
        if loop is not None and not args.kv_groups:
            t_last = (warmup + steps + n_phase - 1) % loop[0]
            res["cpu_baseline"]["parity_of_measured_run"] = loop_parity(w, ds.results(), qs[t_last], loop[3][t_last])
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
