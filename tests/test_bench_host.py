"""Host logic of bench.py (no GPU): the algorithmic bytes every roofline figure
divides by, the source hash that decides whether stored counter traffic is
reported, and the runs it refuses."""
import os
import shutil
import subprocess
import sys
import types

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2605_31457_amd import workloads as W  # noqa: E402


def _layout_only(cfg, B, Hkv, d, dtype):
    """A workload stand-in with the fields algorithmic_bytes reads (no KV draws)."""
    lens, segs, _ = W._layout(cfg, B)
    return types.SimpleNamespace(B=B, Hkv=Hkv, d=d, dtype=dtype, seq_len=np.asarray(lens, np.int32),
                                 segments=[list(s) for s in segs])


def test_algorithmic_bytes_single_image_step():
    # 1296 visual + 2062 text rows, 4 KV heads of 128 bf16, 64 kept rows:
    # visual K 1296 x 1024 B, text K+V 2 x 2062 x 1024 B, kept K+V 2 x 64 x 1024 B
    w = _layout_only(2, 1, 4, 128, "bf16")
    nb = bench.algorithmic_bytes(w, [64])
    assert nb == {"visual": 1296 * 1024, "text": 2 * 2062 * 1024, "kept": 2 * 64 * 1024}
    assert sum(nb.values()) == 5_681_152


def test_algorithmic_bytes_multi_image_batch():
    # 64 sequences of 32768 rows (16384 visual in four images), k = 819 each
    w = _layout_only(4, 64, 4, 128, "bf16")
    nb = bench.algorithmic_bytes(w, [819] * 64)
    assert nb["visual"] == 64 * 16384 * 1024
    assert nb["text"] == 64 * 2 * 16384 * 1024
    assert sum(nb.values()) == 3_328_573_440


def test_algorithmic_bytes_decode_loop_average():
    # 8 sequences, 8 KV heads of 128 bf16, 6400 visual rows; lengths 10497 .. 11008
    # over the 512 steps (text rows averaged), k = 320 each
    lens, segs, _ = W._layout(5, 8)
    w = types.SimpleNamespace(B=8, Hkv=8, d=128, dtype="bf16", seq_len=np.asarray(lens, np.int32),
                              segments=[list(s) for s in segs])
    nb = bench.algorithmic_bytes(w, [320] * 8, lens=[10497 + t for t in range(512)])
    assert sum(nb.values()) == 257_966_080


def test_algorithmic_bytes_per_group_rows():
    # per-KV-group budgets: each selection row names the kept rows of one KV head
    w = _layout_only(2, 1, 4, 128, "bf16")
    nb = bench.algorithmic_bytes(w, [10, 20, 30, 40], rows=4, kv_per_row=1)
    assert nb["kept"] == 2 * (10 + 20 + 30 + 40) * 128 * 2


def _copy_sources(dst):
    src = os.path.join(ROOT, "paper_2605_31457_amd", "csrc")
    os.makedirs(os.path.join(dst, "paper_2605_31457_amd", "csrc"))
    for name in bench.ROOFLINE_SOURCES:
        shutil.copy(os.path.join(src, name), os.path.join(dst, "paper_2605_31457_amd", "csrc", name))
    return os.path.join(dst, "paper_2605_31457_amd", "csrc", "vp_plan.hip")


def test_source_hash_ignores_comments_not_code(tmp_path):
    base = bench.kernel_source_hash(ROOT)
    plan = _copy_sources(str(tmp_path))
    assert bench.kernel_source_hash(str(tmp_path)) == base
    text = open(plan).read()
    open(plan, "w").write(text + "\n// a comment\n/* another\n   one */\n\n")
    assert bench.kernel_source_hash(str(tmp_path)) == base
    open(plan, "w").write(text.replace("#define VP_MIN_TILES 2", "#define VP_MIN_TILES 3"))
    assert bench.kernel_source_hash(str(tmp_path)) != base


def test_counter_traffic_only_for_the_measured_kernel():
    # the stored figures name one kernel per configuration; asking for the
    # other one (or a configuration never measured) gives None
    import json
    rec = json.load(open(os.path.join(ROOT, "profiles", "text_pass_traffic.json")))
    for cfg, e in rec["configs"].items():
        other = "text" if e["kernel"] == "one_launch" else "one_launch"
        assert bench.counter_traffic(int(cfg), other) is None
    assert bench.counter_traffic(99, "text") is None


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=300, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_held_back_cases_are_refused():
    r = _run("--config", "4", "--paged", "32")
    assert r.returncode == 2 and "held back" in r.stderr
    r = _run("--config", "4", "--paged", "32", "--batch", "32")
    assert r.returncode == 2 and "held back" in r.stderr
    r = _run("--config", "5", "--queries", "2")
    assert r.returncode == 2
    r = _run("--config", "2", "--batch", "4")
    assert r.returncode == 2 and "--batch" in r.stderr


def test_anchor_layer_must_precede_the_last_layer():
    for args in (("--layers", "4", "--anchor-layer", "4"), ("--anchor-layer", "-1")):
        r = _run("--config", "2", *args)
        assert r.returncode == 2 and "--anchor-layer" in r.stderr
