"""Unsplit bf16 launches that run two (route, KV head) units per 512-thread
workgroup (units u and u + ceil(U/2) share one).  Every shape here is
planned that way, which each test checks through kf_partial_attn_plan; an
odd route count leaves the last workgroup half idle.
The halves see every mix of states: a tail taking the step's token beside a
route that does not, empty and broken routes beside working ones.  Checked
against the oracle and, for the fused step, bit for bit against the three
separate calls."""
import numpy as np
import pytest

import oracle
from kf_testlib import compare_all, host, run_gpu, run_oracle
from kf_workloads import make_instance, workload
from test_gpu_fused import same_bits

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]


def _instance(seed, steps):
    rng = np.random.default_rng(seed)
    lens = [int(x) for x in rng.integers(0, 400, 170)]
    lens[3] = lens[50] = 0                       # requests without tokens: empty tail routes
    wl = workload("llama8b_32k", num_seqs=len(lens), num_q_heads=8, num_kv_heads=2,
                  part_tokens=128, appends=1)
    inst = make_instance(wl, seed=seed, steps=steps, seq_lens=lens)
    if len(inst.routes) % 2 == 0:                 # make the route count odd
        lens[0] += 128 if lens[0] else 200        # one more route for sequence 0
        inst = make_instance(wl, seed=seed, steps=steps, seq_lens=lens)
    assert len(inst.routes) % 2 == 1
    assert len(inst.routes) * 2 >= 512 and inst.max_pages_per_route <= 16
    return inst


def _assert_two_units(st, route_list=False):
    from paper_2606_29207_amd import kf
    plan = kf.partial_attn_plan(st.shape, st.routes.shape[0], st.max_pages_per_route, route_list)
    assert plan[1:] == ((1, 1) if route_list else (1, 2)), plan


def test_two_units_per_workgroup_match_oracle_and_separate_calls(gpu):
    from paper_2606_29207_amd.step import DecodeState
    inst = _instance(seed=21, steps=3)
    _assert_two_units(DecodeState.from_instance(inst))
    o = run_oracle(inst, 3)
    f = host(run_gpu(inst, 3, fused=True))
    compare_all(f, o)
    same_bits(f, host(run_gpu(inst, 3)))


def test_two_units_per_workgroup_with_broken_rows(gpu):
    """A broken row, a page outside the pool and a bad tail index in one half
    of a workgroup, next to working units in the other half."""
    import torch
    from paper_2606_29207_amd.step import DecodeState
    inst = _instance(seed=22, steps=2)
    R = len(inst.routes)
    half = (R + 1) // 2
    routes = inst.routes.copy()
    page_ids = inst.page_ids.copy()
    tail = inst.tail_route.copy()
    routes[1, 3] = routes[1, 2] - 3                  # tok_end < tok_begin (partner: route 1 + half)
    r = 2 if routes[2, 3] > routes[2, 2] else 4      # a route with pages: one id outside the pool
    page_ids[routes[r, 4]] = inst.num_pages + 7
    tail[5] = tail[6]                                # sequence 5's tail names another sequence's route
    assert routes[1 + half, 3] >= routes[1 + half, 2]
    outs = []
    for fused in (False, True):
        st = DecodeState(q=inst.q, k_pool=inst.k_pool, v_pool=inst.v_pool, routes=routes,
                         page_ids=page_ids, seq_route_begin=inst.seq_route_begin,
                         tail_route=tail, scale=inst.scale,
                         max_pages_per_route=inst.max_pages_per_route)
        _assert_two_units(st)
        for s in range(2):
            kn, vn = st.upload_new_tokens(*inst.new_tokens(s))
            (st.step_fused if fused else st.step)(kn, vn)
        torch.cuda.synchronize()
        outs.append(host(st))
    same_bits(outs[1], outs[0])
    assert outs[1]["flags"] == oracle.EFLAG_BAD_ROUTE | oracle.EFLAG_BAD_PAGE
    kp, vp, rt = inst.k_pool, inst.v_pool, routes.copy()
    flags = 0
    for s in range(2):
        kn, vn = inst.new_tokens(s)
        kp, vp, rt, f = oracle.kv_append(kp, vp, rt, page_ids, tail, kn, vn)
        flags |= f
    o_part, lse_part, f1 = oracle.partial_attn(inst.q, kp, vp, rt, page_ids, num_kv_heads=2,
                                               scale=inst.scale,
                                               max_pages_per_route=inst.max_pages_per_route)
    out, lse, f2 = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    compare_all(outs[1], dict(k_pool=kp, v_pool=vp, k_scale=None, v_scale=None, routes=rt,
                              o_part=o_part, lse_part=lse_part, out=out, lse=lse,
                              flags=flags | f1 | f2))
    # the broken unit's partner in the other half of its workgroup is untouched
    assert np.isfinite(outs[1]["o_part"][1 + half]).all()


@pytest.mark.parametrize("shape", ["odd_routes", "full_round"])
def test_two_units_per_workgroup_bitwise_equal_to_one(gpu, shape):
    """Two units per workgroup keep each unit's four waves, tile order and
    LDS combine, so the partials equal the one-unit kernel's bit for bit.
    kf_partial_attn_subset over the identity list has the same plan at one
    unit per workgroup."""
    import torch
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    if shape == "odd_routes":
        inst = _instance(seed=23, steps=1)
    else:   # 64 routes x 8 KV heads: one unsplit unit per slot, 129 pages each
        wl = workload("llama8b_32k", num_seqs=16, part_tokens=2048)
        inst = make_instance(wl, seed=24, steps=1, seq_lens=[8192] * 16)
        assert len(inst.routes) * wl.num_kv_heads == 512
    st = DecodeState.from_instance(inst)
    _assert_two_units(st)
    _assert_two_units(st, route_list=True)
    st.partial()
    torch.cuda.synchronize()
    o2, l2 = st.o_part.clone(), st.lse_part.clone()
    st.o_part.fill_(float("nan"))
    st.lse_part.fill_(float("nan"))
    ident = torch.arange(len(inst.routes), dtype=torch.int32, device=st.device)
    kf.partial_attn(st.shape, st.q, st.k_pool, st.v_pool, st.routes, st.max_pages_per_route,
                    st.page_ids, st.o_part, st.lse_part, st.workspace, st.err_flags,
                    route_list=ident)
    torch.cuda.synchronize()
    assert st.flags() == 0
    assert torch.equal(o2.view(torch.int32), st.o_part.view(torch.int32))
    assert torch.equal(l2.view(torch.int32), st.lse_part.view(torch.int32))
