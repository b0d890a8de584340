"""vp_validate_layout: the debug check of a device-resident layout (host copies
only; no kernel runs on a malformed layout here)."""
import numpy as np
import pytest
import torch

from _parity import small_workload
from paper_2605_31457_amd import step as S
from paper_2605_31457_amd import vp

pytestmark = pytest.mark.gpu


def _ds(**kw):
    w = small_workload(seed=51, B=3, Hq=4, Hkv=1, d=64, lens=[300, 200, 120],
                       segs=[[(10, 100), (150, 50)], [(0, 64)], []])
    return S.DeviceStep(w, **kw)


def _bad(ds, match, layout=None):
    with pytest.raises(vp.VPError, match="VP_ERR_SHAPE") as e:
        vp.vp_validate_layout(ds.shape, layout or ds.layout)
    assert match in str(e.value), str(e.value)


def test_valid_layouts_pass():
    vp.vp_validate_layout(_ds().shape, _ds().layout)
    ds = _ds(block_size=32, block_seed=2)
    vp.vp_validate_layout(ds.shape, ds.layout)


def test_each_violation_is_named():
    ds = _ds()
    seq_len, seg = ds.seq_len.clone(), ds.seg.clone()
    ds.seq_len[1] = ds.w.S_cap + 1
    _bad(ds, "seq_len")
    ds.seq_len.copy_(seq_len)
    ds.seg[2] = 90          # second segment of sequence 0 starts inside the first
    _bad(ds, "before the previous end")
    ds.seg.copy_(seg)
    ds.seg[3] = 500         # ends past seq_len
    _bad(ds, "ends past seq_len")
    ds.seg.copy_(seg)
    ds.seg[1] = 0           # empty segment
    _bad(ds, "length 0")
    ds.seg.copy_(seg)
    ds.shape.max_vis = 100  # sequence 0 holds 150 visual tokens
    _bad(ds, "max_vis")
    ds.shape.max_vis = ds.max_vis
    ds.shape.max_segs = 1   # sequence 0 has two segments
    _bad(ds, "max_segs")
    ds.shape.max_segs = ds.w.max_segs
    vp.vp_validate_layout(ds.shape, ds.layout)


def test_negative_block_id_is_named():
    ds = _ds(block_size=32, block_seed=3)
    ds.block_table[2, 1] = -5
    _bad(ds, "block_table")


def test_offsets_may_start_inside_a_larger_segment_array():
    """vis_seg_off[0] > 0: the sequences' segments sit after unrelated entries."""
    ds = _ds()
    pad = torch.tensor([999999, -5], dtype=torch.int32, device=ds.device)  # never read
    seg = torch.cat([pad, ds.seg])
    off = ds.seg_off + 1
    lay = vp.vp_layout(seq_len=ds.seq_len.data_ptr(), vis_seg_off=off.data_ptr(), vis_seg=seg.data_ptr())
    vp.vp_validate_layout(ds.shape, lay)
    seg[2 + 2] = 90  # the second segment of sequence 0 now overlaps the first
    _bad(ds, "before the previous end", layout=lay)
