"""Parity at the workloads' full sizes, in the launch configuration bench.py
times (one decode step of its default schedule: kf_decode_step when the
workload appends, partial attention and merge when it does not), on outputs
the oracle can compute one unit at a time.

Per workload:
* sampled (route, KV head) partials and sampled merged (sequence, KV group)
  outputs against the fp64 oracle, same tolerances as the reduced tests;
* the route rows bit-exact, and the K/V pages the append wrote bit-exact
  (every tail page in full, untouched pages compared by sampling);
* properties over every output: no NaN, no error flags, and the GPU's
  merged output equal to the oracle's merge of the GPU's own partials.
Host generation of the largest instance (million-token contexts, 17 GB of
bf16 KV) takes tens of seconds on the GPU host.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from kf_testlib import assert_close_lse, assert_close_o, host
from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.slow,
              pytest.mark.filterwarnings("ignore::RuntimeWarning")]

SAMPLE_UNITS = 12       # (route, KV head) partials checked per workload
SAMPLE_GROUPS = 3       # (sequence, KV head) merged outputs checked per workload


def _threads():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return 4


def _oracle_units(inst, kp, vp, routes, units):
    wl = inst.wl
    f = lambda u: oracle.route_partial(  # noqa: E731
        inst.q, kp, vp, routes[u[0]], inst.page_ids, u[1], num_kv_heads=wl.num_kv_heads,
        scale=inst.scale, max_pages_per_route=inst.max_pages_per_route,
        k_scale=inst.k_scale, v_scale=inst.v_scale)
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1), ThreadPoolExecutor(_threads()) as ex:
        return list(ex.map(f, units))


@pytest.mark.parametrize("name", ["tiny", "llama8b_32k", "agentic_mix", "million_ctx",
                                  "wide_gqa_fp8"])
def test_fullsize_sampled(gpu, name):
    import torch
    from paper_2606_29207_amd.step import DecodeState
    wl = workload(name)
    inst = make_instance(wl, seed=1, steps=1)
    print(f"[fullsize] {name}: {len(inst.routes)} routes, {inst.num_pages} pages", flush=True)
    st = DecodeState.from_instance(inst)
    for t in (st.o_part, st.lse_part, st.out, st.lse):
        t.fill_(float("nan"))
    if wl.appends:
        kn, vn = inst.new_tokens(0)
        st.step_fused(*st.upload_new_tokens(kn, vn))
    else:
        st.step()
    torch.cuda.synchronize()
    o_part = st.o_part.cpu().double().numpy()
    lse_part = st.lse_part.cpu().double().numpy()
    out = st.out.cpu().double().numpy()
    lse = st.lse.cpu().double().numpy()
    assert st.flags() == 0
    for a, n in ((o_part, "o_part"), (lse_part, "lse_part"), (out, "out"), (lse, "lse")):
        assert not np.isnan(a).any(), f"{n} has NaN (unwritten or wrong)"

    # ---- append: routes and pages bit-exact
    kp, vp, routes = inst.k_pool, inst.v_pool, inst.routes
    if wl.appends:
        kp, vp, routes, f0 = oracle.kv_append(inst.k_pool, inst.v_pool, inst.routes,
                                              inst.page_ids, inst.tail_route, kn, vn)
        assert f0 == 0
        g = host(st)
        assert np.array_equal(g["routes"], routes)
        tails = routes[inst.tail_route]
        tail_pages = np.concatenate([inst.page_ids[r[4]:r[4] + r[5]] for r in tails])
        rng = np.random.default_rng(0)
        other = rng.choice(inst.num_pages, size=min(2048, inst.num_pages), replace=False)
        for pages in (tail_pages, other):
            assert np.array_equal(g["k_pool"][pages], kp[pages])
            assert np.array_equal(g["v_pool"][pages], vp[pages])
        del g

    # ---- sampled partials
    rng = np.random.default_rng(1)
    R, H, G = len(routes), wl.num_kv_heads, wl.group
    units = [(int(rng.integers(R)), int(rng.integers(H))) for _ in range(SAMPLE_UNITS)]
    units += [(int(t), int(rng.integers(H))) for t in inst.tail_route[:2] if t >= 0]
    ref = _oracle_units(inst, kp, vp, routes, units)
    got_o = np.stack([o_part[r, g * G:(g + 1) * G] for r, g in units])
    got_l = np.stack([lse_part[r, g * G:(g + 1) * G] for r, g in units])
    mx, rel = assert_close_o(got_o, np.stack([x[0] for x in ref]), f"{name} o_part (sampled)")
    ml_err = assert_close_lse(got_l, np.stack([x[1] for x in ref]), f"{name} lse_part (sampled)") or 0.0
    print(f"[fullsize] {name}: {len(units)} sampled units, o_part max|d| {mx:.2e} rel-L2 {rel:.2e}, "
          f"lse_part max|d| {ml_err:.2e}", flush=True)

    # ---- sampled merged outputs: all routes of a sequence, one KV group
    srb = inst.seq_route_begin
    groups = [(int(rng.integers(wl.num_seqs)), int(rng.integers(H))) for _ in range(SAMPLE_GROUPS)]
    worst = (0.0, 0.0, 0.0)
    for b, g in groups:
        rows = list(range(int(srb[b]), int(srb[b + 1])))
        parts = _oracle_units(inst, kp, vp, routes, [(r, g) for r in rows])
        mo, ml = oracle.merge([p[0] for p in parts], [p[1] for p in parts])
        e_o = assert_close_o(out[b, g * G:(g + 1) * G], mo, f"{name} out[{b}, group {g}]")
        e_l = assert_close_lse(lse[b, g * G:(g + 1) * G], ml, f"{name} lse[{b}, group {g}]") or 0.0
        worst = (max(worst[0], e_o[0]), max(worst[1], e_o[1]), max(worst[2], e_l))
    print(f"[fullsize] {name}: {len(groups)} sampled (sequence, group) merges, out max|d| "
          f"{worst[0]:.2e} rel-L2 {worst[1]:.2e}, lse max|d| {worst[2]:.2e}", flush=True)

    # ---- every sequence: GPU merge == oracle merge of the GPU partials
    mo, ml, mf = oracle.merge_partials(o_part, lse_part, srb)
    assert mf == 0
    assert_close_o(out, mo, f"{name} out vs merge(GPU partials)")
    assert_close_lse(lse, ml, f"{name} lse vs merge(GPU partials)")
