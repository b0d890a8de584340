"""GPU parity over the 72B-class decode loop (config 5): 512 steps, B = 8,
64/8 heads, 6400 visual + 4096 text tokens, one text row appended per step and
the query drifting as q_t = 0.9 q_{t-1} + 0.1 N(0, 1).

Every step is planted after its append (oracle/plant.py plant_loop_step: key
rows near the Eq. (3) cut are moved apart until the fp64 reference shows a
score gap of at least 1e-3 at the cut and a 1e-4 margin on the Eq. (7)
rounding); the planted rows stay in the cache for the later steps, as the
appended ones do. The step's appended and planted rows, its query and its length
are written to the device, vp_decode_step runs, and every (step, sequence) is
held to the bar of every other configuration: masses and scores within 1e-5
relative, the budget exactly, the kept index set bit-exact, and the attention
output within bf16 atol 2e-2 / rtol 1e-2 of the reference's own pruned
attention (over the reference's own kept set).
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import threadpoolctl
import torch

from _parity import check_sequence
from oracle import plant as P
from oracle import vp_oracle as O
from paper_2605_31457_amd import step as S
from paper_2605_31457_amd import workloads as W

pytestmark = pytest.mark.gpu

STEPS = 512


def _bf16_dev(bits, device):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def test_config5_decode_loop_planted_every_step():
    stream = W.Cfg5Stream(B=8, steps=STEPS)
    w = stream.w
    p = P.params_of(w)
    ds = S.DeviceStep(w)
    B = w.B
    # the reference's float64 copies of the caches, kept equal to the stored rows
    Kf = [O.as_f64(w.K[b]) for b in range(B)]
    Vf = [O.as_f64(w.V[b]) for b in range(B)]
    log = dict(edited_rows=0, k_exact=0, set_exact=0, outputs=0)
    # one reference thread per sequence, each with a single-threaded BLAS
    with ThreadPoolExecutor(B) as ex, threadpoolctl.threadpool_limits(1):
        for t in range(STEPS):
            q, kr, vr, pos = stream.step_inputs(t)
            w.K[:, :, pos] = kr
            w.V[:, :, pos] = vr
            for b in range(B):
                Kf[b][:, pos] = O.as_f64(kr[b])
                Vf[b][:, pos] = O.as_f64(vr[b])
            L = pos + 1
            planted = list(ex.map(lambda b: P.plant_loop_step(q[b], w.K[b], Kf[b], w.V[b], Vf[b], L,
                                                               w.segments[b], p), range(B)))
            # step t's inputs on the device: appended row, planted rows, query, length
            ds.K[:, :, pos] = _bf16_dev(kr, ds.device)
            ds.V[:, :, pos] = _bf16_dev(vr, ds.device)
            for b, (edits, _) in enumerate(planted):
                if edits:
                    idx = torch.tensor(edits, dtype=torch.long, device=ds.device)
                    ds.K[b][:, idx] = _bf16_dev(w.K[b][:, edits], ds.device)
                    log["edited_rows"] += len(edits)
            ds.q.copy_(_bf16_dev(q, ds.device))
            ds.seq_len.fill_(L)
            ds.decode_step()
            g = ds.results()
            for b, (_, r) in enumerate(planted):
                check_sequence(f"config 5 step {t}", w, g, b, r)
                log["k_exact"] += 1
                log["set_exact"] += 1
                log["outputs"] += 1
            if t % 64 == 0 or t == STEPS - 1:
                print(f"step {t}: k={list(g['k'])} {log}", flush=True)
    total = STEPS * B
    print(f"config 5 loop: {total} sequence-steps; budgets exact {log['k_exact']}, kept sets bit-exact "
          f"{log['set_exact']}, outputs within tolerance {log['outputs']}; {log['edited_rows']} rows planted",
          flush=True)
    assert log["set_exact"] == log["k_exact"] == log["outputs"] == total
