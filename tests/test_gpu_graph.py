"""kf_decode_step captured in a HIP graph (through torch's CUDAGraph) and
replayed once per decode step: every replay, with eager work and
synchronisations between replays, must leave exactly the state that the
same steps run eagerly leave (the graph records kernel launches only; the
library records no memset and allocates nothing)."""
import numpy as np
import pytest

from kf_testlib import host
from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]

KEYS = ("o_part", "lse_part", "out", "lse", "k_pool", "v_pool", "routes", "k_scale", "v_scale",
        "flags")


@pytest.mark.parametrize("name,over,lens", [
    ("llama8b_32k", dict(num_seqs=3, num_q_heads=8, num_kv_heads=2, part_tokens=1000),
     [2100, 999, 1500]),
    ("wide_gqa_fp8", dict(num_seqs=2, num_q_heads=16, num_kv_heads=2, part_tokens=1024, appends=1),
     [2048, 1500]),
])
def test_decode_step_graph_replays_match_eager(gpu, name, over, lens):
    import torch
    from paper_2606_29207_amd.step import DecodeState
    steps = 6
    inst = make_instance(workload(name, **over), seed=2, steps=steps, seq_lens=lens)
    eager = DecodeState.from_instance(inst)
    graphed = DecodeState.from_instance(inst)
    kbuf, vbuf = graphed.upload_new_tokens(*inst.new_tokens(0))     # the graph's inputs
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side), torch.cuda.graph(graph, stream=side):
        graphed.step_fused(kbuf, vbuf)                               # recorded, not run
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    scratch = torch.zeros(1 << 20, device="cuda")
    for s in range(steps):
        kn, vn = eager.upload_new_tokens(*inst.new_tokens(s))
        kbuf.copy_(kn)
        vbuf.copy_(vn)
        graph.replay()
        scratch.add_(1.0)                                            # eager work between replays
        eager.step_fused(kn, vn)
        torch.cuda.synchronize()
        a, b = host(graphed), host(eager)
        for k in KEYS:
            x, y = a[k], b[k]
            if x is None or y is None:
                assert x is None and y is None, k
                continue
            assert np.array_equal(np.asarray(x), np.asarray(y), equal_nan=True), (s, k)
    assert host(graphed)["flags"] == 0
