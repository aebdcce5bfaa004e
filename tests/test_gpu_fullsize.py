"""Parity at the workloads' full sizes, over whole tensors, in the launch
configuration bench.py times: the same route table (the bench's tail-page
reservation) and the same schedule -- kf_decode_step per step when the
workload appends, kf_partial_attn then kf_merge_partials when it does not.

For every workload and seeds 1 and 2, after the first step and (appending
workloads) after the 17th -- by then every Llama-3.1-8B tail has filled the
page its first append opened and opened the next (Section 3.2 step 3: the
tail appends, then attends):
* every (route, KV head) partial and every merged (sequence, query head)
  output against the fp64 oracle, one unit at a time over a thread pool:
  max|d| and rel-L2 over each whole tensor (o_part, out), max|d| for
  lse_part and lse (the merge equals attention over the whole range,
  Section 5.1);
* appending workloads: the K/V pools, fp8 scales and route rows bit-exact,
  whole, against the oracle's appends;
* no error flags and no NaN anywhere.
Host generation of the largest instance (million-token contexts, 17 GB of
bf16 KV) takes seconds on the GPU host.
"""
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from kf_testlib import assert_close_lse, assert_close_o
from kf_workloads import make_instance, workload

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402  (the reservation and thread count the benchmark uses)

pytestmark = [pytest.mark.gpu, pytest.mark.slow,
              pytest.mark.filterwarnings("ignore::RuntimeWarning")]

WORKLOADS = ["tiny", "llama8b_32k", "agentic_mix", "million_ctx", "wide_gqa_fp8",
             "wide_gqa_fp8_decode"]
CHECK_AFTER = (1, 17)          # steps after which appending workloads are compared


def _oracle_partials(inst, kp, vp, ks, vs, routes):
    """o_part [R, Hq, d], lse_part [R, Hq] of every (route, KV head) unit."""
    wl = inst.wl
    R, H, G = len(routes), wl.num_kv_heads, wl.group
    units = [(r, g) for r in range(R) for g in range(H)]

    def f(u):
        return oracle.route_partial(inst.q, kp, vp, routes[u[0]], inst.page_ids, u[1],
                                    num_kv_heads=H, scale=inst.scale,
                                    max_pages_per_route=inst.max_pages_per_route,
                                    k_scale=ks, v_scale=vs)
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1), \
            ThreadPoolExecutor(bench.cpu_threads(bench.visible_cores())) as ex:
        res = list(ex.map(f, units))
    o_part = np.zeros((R, wl.num_q_heads, wl.head_dim))
    lse_part = np.zeros((R, wl.num_q_heads))
    flags = 0
    for (r, g), (o, lse, fl) in zip(units, res):
        o_part[r, g * G:(g + 1) * G] = o
        lse_part[r, g * G:(g + 1) * G] = lse
        flags |= fl
    return o_part, lse_part, flags


def _pool_bits(t):
    import torch
    t = t.cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if t.element_size() == 2 else \
        t.view(torch.uint8).numpy()


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("name", WORKLOADS)
def test_fullsize_whole_tensors(gpu, name, seed):
    import torch
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    wl = workload(name)
    t0 = time.perf_counter()
    inst = make_instance(wl, seed=seed, steps=bench.RESERVE_APPENDS)
    st = DecodeState.from_instance(inst)
    plan = kf.partial_attn_plan(st.shape, st.routes.shape[0], st.max_pages_per_route)
    print(f"[fullsize] {name} seed {seed}: {len(inst.routes)} routes, {inst.num_pages} pages, "
          f"plan (chunk pages, max chunks, units/workgroup) {plan}, "
          f"set up in {time.perf_counter() - t0:.1f}s", flush=True)
    # the oracle's state: the instance's own arrays, appended to in place
    kp, vp, ks, vs, routes = inst.k_pool, inst.v_pool, inst.k_scale, inst.v_scale, inst.routes
    steps = max(CHECK_AFTER) if wl.appends else 1
    for s in range(steps):
        for t in (st.o_part, st.lse_part, st.out, st.lse):
            t.fill_(float("nan"))
        if wl.appends:
            kn, vn = inst.new_tokens(s)
            st.step_fused(*st.upload_new_tokens(kn, vn))
            res = oracle.kv_append(kp, vp, routes, inst.page_ids, inst.tail_route, kn, vn,
                                   ks, vs, inplace=True)
            assert res[-1] == 0
        else:
            st.step()
        if (s + 1) not in CHECK_AFTER and s + 1 != steps:
            continue
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        assert st.flags() == 0
        got = {k: getattr(st, k).cpu().double().numpy() for k in ("o_part", "lse_part", "out", "lse")}
        for k, a in got.items():
            assert not np.isnan(a).any(), f"{name}: {k} has NaN (unwritten or wrong)"
        if wl.appends:
            assert np.array_equal(st.routes.cpu().numpy(), routes), "route rows differ"
            assert np.array_equal(_pool_bits(st.k_pool), kp), "K pool differs"
            assert np.array_equal(_pool_bits(st.v_pool), vp), "V pool differs"
            if ks is not None:
                assert np.array_equal(st.k_scale.cpu().numpy(), ks), "K scales differ"
                assert np.array_equal(st.v_scale.cpu().numpy(), vs), "V scales differ"
        o_part, lse_part, f1 = _oracle_partials(inst, kp, vp, ks, vs, routes)
        out, lse, f2 = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
        assert f1 == f2 == 0
        e_op = assert_close_o(got["o_part"], o_part, f"{name} o_part after step {s + 1}")
        e_lp = assert_close_lse(got["lse_part"], lse_part, f"{name} lse_part after step {s + 1}")
        e_o = assert_close_o(got["out"], out, f"{name} out after step {s + 1}")
        e_l = assert_close_lse(got["lse"], lse, f"{name} lse after step {s + 1}")
        print(f"[fullsize] {name} seed {seed} after step {s + 1}: "
              f"o_part max|d| {e_op[0]:.2e} rel-L2 {e_op[1]:.2e} ({o_part.size} elements), "
              f"lse_part max|d| {e_lp:.2e}, out max|d| {e_o[0]:.2e} rel-L2 {e_o[1]:.2e}, "
              f"lse max|d| {e_l:.2e}"
              + (", pools/scales/routes bit-exact" if wl.appends else "")
              + f" ({time.perf_counter() - t1:.1f}s)", flush=True)
