"""bench.py's contract points that need no GPU: more than one GPU is refused
with a message, and the algorithmic byte model counts what a step must move."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and res.stdout == ""


def test_step_bytes_llama_layer():
    """The Llama-3.1-8B layer after its first append: 16 x 32769 tokens of
    8 KV heads x 128 dims x 2 B for K and V (the footprint formula of the
    scaling policy with L = 1), plus q, page ids, route rows and partials."""
    sys.path.insert(0, ROOT)
    import bench
    from kf_workloads import make_instance, workload
    wl = workload("llama8b_32k", num_seqs=2, ctx=1000, part_tokens=300)
    inst = make_instance(wl, seed=1, steps=3)
    b = bench.step_bytes(inst, 0)
    tokens = 2 * 1001
    assert b["tokens"] == tokens
    assert b["kv"] == 2 * tokens * 8 * 128 * 2
    R = len(inst.routes)
    pages = sum(-(-(int(r[3] - r[2]) + (1 if i in set(inst.tail_route.tolist()) else 0)) // 16)
                for i, r in enumerate(inst.routes))
    assert b["partial"] == b["kv"] + 2 * 32 * 128 * 2 + pages * 4 + R * 24 + R * 32 * 129 * 4
    assert b["merge"] == R * 32 * 129 * 4 + 3 * 4 + 2 * 32 * 129 * 4
    assert bench.step_bytes(inst, 2)["tokens"] == tokens + 4
    assert np.isclose(b["kv"] / tokens, 4096)
