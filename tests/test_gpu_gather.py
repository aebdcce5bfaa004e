"""Route snapshot + page lookup, bit-exact (GPU): kf_debug_gather copies a
route's tokens out through the same route checks and page lookup as the
attention kernels; every element must equal the oracle's gather through the
routing table (Section 4.1), independent of any floating-point arithmetic."""
import numpy as np
import pytest

import oracle
from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]

SENTINEL16 = 0x7E01      # a bf16 NaN pattern no pool holds
SENTINEL8 = 0x7F


def gather_all(inst, routes=None, page_ids=None, max_tokens=None, max_pages=None, sel=None):
    """Gather the routes ``sel`` (default: all) on the GPU; returns
    ({route: (out_k, out_v)}, flags)."""
    import torch
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    routes = inst.routes if routes is None else routes
    page_ids = inst.page_ids if page_ids is None else page_ids
    st = DecodeState(q=inst.q, k_pool=inst.k_pool, v_pool=inst.v_pool, routes=routes,
                     page_ids=page_ids, seq_route_begin=inst.seq_route_begin,
                     tail_route=inst.tail_route, scale=inst.scale,
                     max_pages_per_route=max_pages or inst.max_pages_per_route,
                     k_scale=inst.k_scale, v_scale=inst.v_scale)
    H = inst.wl.num_kv_heads
    fp8 = inst.wl.kv_dtype == "fp8"
    dt, sent = (torch.uint8, SENTINEL8) if fp8 else (torch.int16, SENTINEL16)
    outs = []
    sel = range(len(routes)) if sel is None else sel
    for r in sel:
        n = max(int(routes[r, 3]) - int(routes[r, 2]), 0)
        m = n + 5 if max_tokens is None else max_tokens
        ok = torch.full((m, H, 128), sent, dtype=dt, device="cuda")
        ov = torch.full((m, H, 128), sent, dtype=dt, device="cuda")
        if not fp8:
            ok, ov = ok.view(torch.bfloat16), ov.view(torch.bfloat16)
        kf.debug_gather(st.shape, st.k_pool, st.v_pool, st.routes, r, st.max_pages_per_route,
                        st.page_ids, m, ok, ov, st.err_flags)
        outs.append((r, ok, ov))
    torch.cuda.synchronize()
    res = {}
    for r, ok, ov in outs:
        if fp8:
            res[r] = (ok.cpu().numpy(), ov.cpu().numpy())
        else:
            res[r] = (ok.view(torch.int16).cpu().numpy().view(np.uint16),
                      ov.view(torch.int16).cpu().numpy().view(np.uint16))
    return res, st.flags()


def decode(x, fp8):
    return oracle.e4m3_to_f64(x) if fp8 else oracle.bf16_to_f64(x)


def check_routes(inst, got, routes=None, page_ids=None, clamp=None):
    routes = inst.routes if routes is None else routes
    page_ids = inst.page_ids if page_ids is None else page_ids
    fp8 = inst.wl.kv_dtype == "fp8"
    ones = None if not fp8 else np.ones_like(inst.k_scale)
    sent = SENTINEL8 if fp8 else SENTINEL16
    for r, (ok, ov) in got.items():
        n = int(routes[r, 3] - routes[r, 2])
        n_out = n if clamp is None else min(n, clamp)
        for g in range(inst.wl.num_kv_heads):
            K, V = oracle.gather_kv(routes[r], page_ids, inst.k_pool, inst.v_pool, g, ones, ones)
            assert np.array_equal(decode(ok[:n_out, g], fp8), K[:n_out]), (r, g)
            assert np.array_equal(decode(ov[:n_out, g], fp8), V[:n_out]), (r, g)
        assert np.all(ok[n_out:] == sent) and np.all(ov[n_out:] == sent), r


@pytest.mark.parametrize("name,over,lens", [
    ("llama8b_32k", dict(num_seqs=3, part_tokens=1000), [3001, 1700, 4103]),   # unaligned route starts
    ("agentic_mix", dict(num_seqs=5, ctx_range=(100, 6000), part_tokens=2048), None),  # permuted pool
    ("wide_gqa_fp8", dict(num_seqs=2, part_tokens=1024), [3000, 1111]),       # E4M3 codes
    ("llama8b_32k", dict(num_seqs=2, num_q_heads=8, num_kv_heads=2, part_tokens=512), [1024, 7]),
])
def test_gather_every_route_bit_exact(gpu, name, over, lens):
    inst = make_instance(workload(name, **over), seed=1, seq_lens=lens, empty_tail=True)
    got, flags = gather_all(inst)
    assert flags == 0
    check_routes(inst, got)


def test_gather_clamps_to_max_tokens(gpu):
    inst = make_instance(workload("llama8b_32k", num_seqs=2, part_tokens=700), seed=2,
                         seq_lens=[1500, 900])
    got, flags = gather_all(inst, max_tokens=37)
    assert flags == 0
    check_routes(inst, got, clamp=37)


def test_gather_bad_rows_and_pages(gpu):
    inst = make_instance(workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2,
                                  part_tokens=512), seed=3, seq_lens=[1300, 900])
    routes = inst.routes.copy()
    routes[1, 3] = routes[1, 2] - 1                  # bad row: nothing written
    page_ids = inst.page_ids.copy()
    page_ids[routes[2, 4] + 1] = inst.num_pages     # second page of route 2 outside the pool
    got, flags = gather_all(inst, routes=routes, page_ids=page_ids)
    assert flags == oracle.EFLAG_BAD_ROUTE | oracle.EFLAG_BAD_PAGE
    ok1, ov1 = got[1]
    assert np.all(ok1 == SENTINEL16) and np.all(ov1 == SENTINEL16)
    ok2, ov2 = got[2]
    assert np.all(ok2[16:32] == SENTINEL16) and np.all(ov2[16:32] == SENTINEL16)  # the bad page
    check_routes(inst, {r: got[r] for r in (0, 3)}, routes=routes, page_ids=page_ids)
    for g in range(2):                                 # route 2's other pages are intact
        K, V = oracle.gather_kv(inst.routes[2], inst.page_ids, inst.k_pool, inst.v_pool, g)
        for lo, hi in ((0, 16), (32, len(K))):
            assert np.array_equal(oracle.bf16_to_f64(ok2[lo:hi, g]), K[lo:hi])
            assert np.array_equal(oracle.bf16_to_f64(ov2[lo:hi, g]), V[lo:hi])


def test_gather_fullsize_llama_sampled_routes(gpu):
    """The benchmark's Llama-3.1-8B layer: four routes, including a tail."""
    inst = make_instance(workload("llama8b_32k"), seed=1)
    got, flags = gather_all(inst, sel=[0, 17, 38, 63])
    assert flags == 0
    check_routes(inst, got)
