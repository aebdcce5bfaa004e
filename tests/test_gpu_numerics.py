"""Degenerate score patterns on the GPU, against closed forms and the fp64
oracle: a zero query (uniform weights: out = mean of V, lse = ln n), one
dominant key (out = its value), and a wide score range (|s| up to ~50, where
the online softmax rescales by large factors between tiles)."""
import numpy as np
import pytest

import oracle
from kf_testlib import compare_all, host, run_oracle
from kf_workloads import bf16_bits_to_f32, f32_to_bf16_bits, make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]


def gpu_with_q(inst, q_bits):
    import torch
    from paper_2606_29207_amd.step import DecodeState
    st = DecodeState(q=q_bits, k_pool=inst.k_pool, v_pool=inst.v_pool, routes=inst.routes,
                     page_ids=inst.page_ids, seq_route_begin=inst.seq_route_begin,
                     tail_route=inst.tail_route, scale=inst.scale,
                     max_pages_per_route=inst.max_pages_per_route, k_scale=inst.k_scale,
                     v_scale=inst.v_scale)
    st.step()
    torch.cuda.synchronize()
    return host(st)


def base(name="llama8b_32k", **over):
    """A static context (no append), as gpu_with_q runs the step without one."""
    kw = dict(num_seqs=2, num_q_heads=8, num_kv_heads=2, part_tokens=1000, appends=0)
    kw.update(over)
    return make_instance(workload(name, **kw), seed=11, seq_lens=[2500, 777])


@pytest.mark.parametrize("name", ["llama8b_32k", "wide_gqa_fp8"])
def test_zero_query_gives_mean_of_values(gpu, name):
    inst = base(name, part_tokens=1024) if name == "wide_gqa_fp8" else base()
    q0 = np.zeros_like(inst.q)
    g = gpu_with_q(inst, q0)
    G = inst.wl.group
    for b, n in enumerate(inst.seq_lens):
        for gk in range(inst.wl.num_kv_heads):
            vals = []
            for r in range(inst.seq_route_begin[b], inst.seq_route_begin[b + 1]):
                _, V = oracle.gather_kv(inst.routes[r], inst.page_ids, inst.k_pool, inst.v_pool, gk,
                                        inst.k_scale, inst.v_scale)
                vals.append(V)
            mean = np.concatenate(vals).mean(axis=0)
            for h in range(gk * G, (gk + 1) * G):
                assert np.abs(g["out"][b, h] - mean).max() <= 2e-3
                assert abs(g["lse"][b, h] - np.log(n)) <= 1e-4


def test_one_dominant_key(gpu):
    """Key t* of sequence 0 set along the group's mean query with norm 120:
    its score exceeds 30 for every head of the group while the others stay
    near N(0, 1), so out = v_{t*} to fp32 precision."""
    inst = base()
    q = bf16_bits_to_f32(inst.q)
    G, D = inst.wl.group, inst.wl.head_dim
    r, j = 1, 333                                   # route 1 of seq 0, local token 333
    pid = inst.page_ids[inst.routes[r, 4] + j // 16]
    for gk in range(inst.wl.num_kv_heads):
        u = q[0, gk * G:(gk + 1) * G].mean(axis=0)
        k = u / np.linalg.norm(u) * 120.0
        inst.k_pool[pid, gk, j % 16, :] = f32_to_bf16_bits(k.astype(np.float32))
    o = run_oracle(inst, 1)
    g = gpu_with_q(inst, inst.q)
    compare_all(g, o, pools=False)
    for gk in range(inst.wl.num_kv_heads):
        v = oracle.bf16_to_f64(inst.v_pool[pid, gk, :, j % 16])
        for h in range(gk * G, (gk + 1) * G):
            s = oracle.bf16_to_f64(inst.q[0, h]) @ oracle.bf16_to_f64(inst.k_pool[pid, gk, j % 16]) * inst.scale
            assert s > 30, s                            # dominant for every head
            assert np.abs(g["out"][0, h] - v).max() <= 2e-3


def test_wide_score_range(gpu):
    """q scaled by 8 (scores up to ~50): the running max jumps by large steps
    between tiles and the rescaling factors underflow to 0."""
    inst = base()
    q8 = f32_to_bf16_bits(bf16_bits_to_f32(inst.q) * np.float32(8.0))
    inst.q = q8
    o = run_oracle(inst, 1)
    g = gpu_with_q(inst, q8)
    compare_all(g, o, pools=False)
    assert np.abs(o["lse"]).max() > 20
