"""Split launches of several rounds run their work items in a computed order
(largest page ranges first, written by a one-workgroup kernel into the
workspace).  Which workgroup computes an item never changes a result: these
tests run such launches against the fp64 oracle, with empty and bad routes
(one item each, for their outputs), fused appends over several steps and a
route-list launch, and check that repeated runs are bit-identical although
the order within a size class varies from run to run."""
import numpy as np
import pytest

import oracle
from kf_testlib import (assert_close_lse, assert_close_o, compare_all, host, run_gpu,
                        run_oracle)
from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]

MAX_ORDER_ITEMS = 1 << 20


def _ordered(st, num_launch, route_list=False):
    """Whether a launch of num_launch routes runs in a computed order on this
    GPU: split, with at least two work items per resident slot (two per CU)."""
    import torch
    from paper_2606_29207_amd import kf
    cp, mc, up = kf.partial_attn_plan(st.shape, num_launch, st.max_pages_per_route,
                                      route_list=route_list)
    slots = 2 * torch.cuda.get_device_properties(0).multi_processor_count
    items = mc * st.shape.num_kv_heads * num_launch
    return mc > 1 and 2 * slots <= items <= MAX_ORDER_ITEMS, (cp, mc, up, items)


def _ragged_instance(appends):
    lens = [0, 37, 16, 900, 4096, 9000, 23000, 511, 3000, 12000, 7777, 40000,
            64, 2048, 15000, 1025, 6000, 300, 18000, 8191]
    return make_instance(workload("agentic_mix", num_seqs=len(lens), part_tokens=4096,
                                  appends=appends), seed=21, steps=4, seq_lens=lens)


@pytest.mark.parametrize("fused", [False, True])
def test_ordered_split_launch_matches_oracle(gpu, fused):
    from paper_2606_29207_amd.step import DecodeState
    inst = _ragged_instance(appends=1)
    ok, plan = _ordered(DecodeState.from_instance(inst), len(inst.routes))
    assert ok, f"the launch should run in a computed order: plan {plan}"
    print(f"[order] {len(inst.routes)} routes, plan (chunk pages, ranges, units/wg, items) {plan}",
          flush=True)
    compare_all(host(run_gpu(inst, 3, fused=fused)), run_oracle(inst, 3))


def test_ordered_launch_with_bad_routes(gpu):
    """A bad route row and a bad page id in an ordered launch: NaN in their
    units only, the flags raised, every other unit to the oracle's bar."""
    inst = _ragged_instance(appends=0)
    routes = inst.routes.copy()
    routes[5, 3] = routes[5, 2] + 16 * (routes[5, 5] + 1)   # more pages than page_cap
    inst.routes[:] = routes
    inst.page_ids[int(inst.routes[9, 4]) + 3] = inst.num_pages + 5   # a page outside the pool
    g, o = host(run_gpu(inst, 1)), run_oracle(inst, 1)
    assert g["flags"] == o["flags"] == (oracle.EFLAG_BAD_ROUTE | oracle.EFLAG_BAD_PAGE)
    compare_all(g, o)


def test_ordered_launch_is_bitwise_repeatable(gpu):
    inst = _ragged_instance(appends=0)
    runs = [host(run_gpu(inst, 1)) for _ in range(3)]
    for k in ("o_part", "lse_part", "out", "lse"):
        for r in runs[1:]:
            assert np.array_equal(runs[0][k], r[k], equal_nan=True), k


def test_ordered_route_list_launch(gpu):
    """kf_partial_attn_subset over a list long enough for a computed order,
    with a list entry naming no route: listed rows to the oracle's bar, the
    rest untouched, the bad entry flagged."""
    import torch
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    lens = [(i * 997) % 9000 + 100 for i in range(80)]
    inst = make_instance(workload("agentic_mix", num_seqs=len(lens), part_tokens=8192, appends=0),
                         seed=22, steps=1, seq_lens=lens)
    st = DecodeState.from_instance(inst)
    R = len(inst.routes)
    listed = [r for r in range(R) if r % 5 != 2]
    lst = torch.tensor(listed + [R + 7], dtype=torch.int32, device="cuda")
    ok, plan = _ordered(st, len(lst), route_list=True)
    assert ok, f"the list launch should run in a computed order: plan {plan}"
    st.o_part.fill_(7.0)
    st.lse_part.fill_(7.0)
    ws = kf.alloc_workspace(st.shape, R + 1, inst.max_pages_per_route)
    kf.partial_attn(st.shape, st.q, st.k_pool, st.v_pool, st.routes, inst.max_pages_per_route,
                    st.page_ids, st.o_part, st.lse_part, ws, st.err_flags, route_list=lst)
    torch.cuda.synchronize()
    assert st.flags() == oracle.EFLAG_BAD_ROUTE
    o = st.o_part.cpu().double().numpy()
    lse = st.lse_part.cpu().double().numpy()
    ref_o, ref_l, _ = oracle.partial_attn(inst.q, inst.k_pool, inst.v_pool, inst.routes,
                                          inst.page_ids, num_kv_heads=inst.wl.num_kv_heads,
                                          scale=inst.scale,
                                          max_pages_per_route=inst.max_pages_per_route)
    others = [r for r in range(R) if r not in listed]
    assert_close_o(o[listed], ref_o[listed], "o_part listed")
    assert_close_lse(lse[listed], ref_l[listed], "lse_part listed")
    assert np.all(o[others] == 7.0) and np.all(lse[others] == 7.0)
