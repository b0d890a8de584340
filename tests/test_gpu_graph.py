"""vp_decode_step captured in a HIP graph (the library enqueues kernels only:
no allocation, no memset, no synchronisation), replayed several times with
eager work and synchronisation between replays; every replay must reproduce
the eager step bit for bit."""
import numpy as np
import pytest
import torch

from paper_2605_31457_amd import step as S
from paper_2605_31457_amd import workloads as W

pytestmark = pytest.mark.gpu

KEYS = ("mass_head", "mass_seq", "scores", "k", "vis_idx", "out")


@pytest.mark.parametrize("cfg,kw", [(2, {}), (3, {}), (5, dict(kv_groups=True)), (2, dict(block_size=32))])
def test_decode_step_graph_replays(cfg, kw):
    w = W.generate(cfg, seqs=[0, 1] if cfg == 5 else None)
    ds = S.DeviceStep(w, **kw)
    ds.decode_step()
    want = ds.results()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        ds.decode_step()  # warm-up on the capture stream
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        ds.decode_step()
    for rep in range(4):
        # scribble over the outputs eagerly, then replay
        for t in (ds.mass_head, ds.mass_seq, ds.scores, ds.out):
            t.fill_(7)
        ds.k.fill_(-3)
        ds.vis_idx.fill_(-9)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = ds.results()
        for key in KEYS:
            assert np.array_equal(got[key], want[key]), f"replay {rep}: {key}"
