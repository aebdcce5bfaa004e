"""kf_decode_step (append fused into partial attention) on the
GPU: against the oracle at the usual bars, and bit for bit against the
three separate calls on the same inputs, including every error path of the
append."""
import numpy as np
import pytest

import oracle
from kf_testlib import compare_all, host, run_gpu, run_oracle
from kf_workloads import make_instance, workload
from test_gpu_parity import CASES

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]

KEYS = ("o_part", "lse_part", "out", "lse", "k_pool", "v_pool", "routes", "k_scale", "v_scale",
        "flags")


def same_bits(a, b):
    for k in KEYS:
        x, y = a[k], b[k]
        if x is None or y is None:
            assert x is None and y is None, k
            continue
        assert np.array_equal(np.asarray(x), np.asarray(y), equal_nan=True), k


@pytest.mark.parametrize("case", list(CASES))
def test_fused_step_matches_oracle_and_separate_calls(gpu, case):
    """Every parity shape, with one append per step (whatever the workload's
    default): the fused step equals the oracle and the three calls."""
    name, over, lens, steps = CASES[case]
    wl = workload(name, **dict(over, appends=1))
    steps = max(steps, 3)
    inst = make_instance(wl, seed=1, steps=steps, seq_lens=lens)
    o = run_oracle(inst, steps)
    f = host(run_gpu(inst, steps, fused=True))
    compare_all(f, o)
    same_bits(f, host(run_gpu(inst, steps)))


def test_fused_tail_full(gpu):
    wl = workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2, part_tokens=256)
    inst = make_instance(wl, seed=4, steps=2, seq_lens=[270, 300])   # tails run out of pages
    o = run_oracle(inst, 5)
    assert o["flags"] == oracle.EFLAG_TAIL_FULL
    f = host(run_gpu(inst, 5, fused=True))
    compare_all(f, o)
    same_bits(f, host(run_gpu(inst, 5)))


def test_fused_inactive_and_bad_tail_index(gpu):
    wl = workload("llama8b_32k", num_seqs=3, num_q_heads=8, num_kv_heads=2, part_tokens=256)
    inst = make_instance(wl, seed=5, steps=1, seq_lens=[300, 400, 500])
    tail = inst.tail_route.copy()
    tail[0] = -1
    tail[1] = inst.tail_route[2]          # another sequence's route
    o = run_oracle(inst, 1, tail_route=tail)
    assert o["flags"] == oracle.EFLAG_BAD_ROUTE
    f = host(run_gpu(inst, 1, tail_route=tail, fused=True))
    compare_all(f, o)
    same_bits(f, host(run_gpu(inst, 1, tail_route=tail)))
    tail2 = inst.tail_route.copy()
    tail2[2] = len(inst.routes) + 4       # outside the table
    f = host(run_gpu(inst, 1, tail_route=tail2, fused=True))
    same_bits(f, host(run_gpu(inst, 1, tail_route=tail2)))
    assert f["flags"] == oracle.EFLAG_BAD_ROUTE


def test_fused_empty_tail_route(gpu):
    """A route published at a token boundary takes its first token in the
    fused step: a one-token route."""
    wl = workload("llama8b_32k", num_seqs=3, num_q_heads=8, num_kv_heads=2, part_tokens=512)
    inst = make_instance(wl, seed=3, steps=3, empty_tail=True, seq_lens=[1024, 700, 512])
    o = run_oracle(inst, 3)
    f = host(run_gpu(inst, 3, fused=True))
    compare_all(f, o)
    same_bits(f, host(run_gpu(inst, 3)))


def test_fused_bad_rows_and_page_ids(gpu):
    """Broken route rows and page ids on tails and historical routes: the
    same flags, NaNs, pools and routes as the three calls."""
    import torch
    from paper_2606_29207_amd.step import DecodeState
    wl = workload("llama8b_32k", num_seqs=4, num_q_heads=8, num_kv_heads=2, part_tokens=512,
                  appends=1)
    inst = make_instance(wl, seed=6, steps=2, seq_lens=[1300, 900, 700, 1030])
    routes = inst.routes.copy()
    tails = inst.tail_route
    routes[0, 3] = routes[0, 2] - 5                   # historical: tok_end < tok_begin
    routes[tails[1], 0] = 9                            # tail whose seq is out of range
    page_ids = inst.page_ids.copy()
    t2 = routes[tails[2]]
    j = int(t2[3] - t2[2])
    page_ids[t2[4] + j // 16] = inst.num_pages + 3    # the page the tail's token goes to
    t3 = routes[tails[3]]
    page_ids[t3[4]] = -2                               # a page the tail only reads
    outs = []
    for fused in (False, True):
        st = DecodeState(q=inst.q, k_pool=inst.k_pool, v_pool=inst.v_pool, routes=routes,
                         page_ids=page_ids, seq_route_begin=inst.seq_route_begin,
                         tail_route=inst.tail_route, scale=inst.scale,
                         max_pages_per_route=inst.max_pages_per_route)
        for s in range(2):
            kn, vn = st.upload_new_tokens(*inst.new_tokens(s))
            (st.step_fused if fused else st.step)(kn, vn)
        torch.cuda.synchronize()
        outs.append(host(st))
    same_bits(outs[1], outs[0])
    assert outs[1]["flags"] == oracle.EFLAG_BAD_ROUTE | oracle.EFLAG_BAD_PAGE
    # the oracle on the same tables agrees
    kp, vp, rt = inst.k_pool, inst.v_pool, routes.copy()
    flags = 0
    for s in range(2):
        kn, vn = inst.new_tokens(s)
        kp, vp, rt, f = oracle.kv_append(kp, vp, rt, page_ids, inst.tail_route, kn, vn)
        flags |= f
    o_part, lse_part, f1 = oracle.partial_attn(inst.q, kp, vp, rt, page_ids, num_kv_heads=2,
                                               scale=inst.scale,
                                               max_pages_per_route=inst.max_pages_per_route)
    out, lse, f2 = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    compare_all(outs[1], dict(k_pool=kp, v_pool=vp, k_scale=None, v_scale=None, routes=rt,
                              o_part=o_part, lse_part=lse_part, out=out, lse=lse,
                              flags=flags | f1 | f2))


def test_fused_fullsize_llama_sampled(gpu):
    """The benchmark's Llama-3.1-8B layer, one fused step against the three
    calls, bit for bit."""
    inst = make_instance(workload("llama8b_32k"), seed=1, steps=2)
    same_bits(host(run_gpu(inst, 2, fused=True, nan_fill=False)),
              host(run_gpu(inst, 2, nan_fill=False)))


def test_fused_tail_crossing_max_pages(gpu):
    """A tail full to its last page takes a token on a new page beyond
    max_pages_per_route: the token is stored, the route's partial is NaN with
    KF_EFLAG_BAD_ROUTE, exactly as with the three calls."""
    import torch
    from paper_2606_29207_amd.step import DecodeState
    wl = workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2, part_tokens=256,
                  appends=1)
    inst = make_instance(wl, seed=8, steps=1, seq_lens=[512, 320])   # seq 0's tail: 16 full pages
    assert inst.max_pages_per_route == 17
    outs = []
    for fused in (False, True):
        st = DecodeState(q=inst.q, k_pool=inst.k_pool, v_pool=inst.v_pool, routes=inst.routes,
                         page_ids=inst.page_ids, seq_route_begin=inst.seq_route_begin,
                         tail_route=inst.tail_route, scale=inst.scale, max_pages_per_route=16)
        kn, vn = st.upload_new_tokens(*inst.new_tokens(0))
        (st.step_fused if fused else st.step)(kn, vn)
        torch.cuda.synchronize()
        outs.append(host(st))
    same_bits(outs[1], outs[0])
    kp, vp, rt, f0 = oracle.kv_append(inst.k_pool, inst.v_pool, inst.routes.copy(), inst.page_ids,
                                      inst.tail_route, *inst.new_tokens(0))
    o_part, lse_part, f1 = oracle.partial_attn(inst.q, kp, vp, rt, inst.page_ids, num_kv_heads=2,
                                               scale=inst.scale, max_pages_per_route=16)
    out, lse, f2 = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    assert f0 == 0 and f1 | f2 == oracle.EFLAG_BAD_ROUTE
    compare_all(outs[1], dict(k_pool=kp, v_pool=vp, k_scale=None, v_scale=None, routes=rt,
                              o_part=o_part, lse_part=lse_part, out=out, lse=lse, flags=f1 | f2))


def test_fused_fp8_reencode_of_pages_begun_by_appends(gpu):
    """E4M3 pools through kf_decode_step with one step's tokens 100x larger:
    the tail workgroups re-encode their pages and attend with the new scales
    (passed through LDS), bit for bit as the three calls."""
    from kf_workloads import bf16_bits_to_f32, f32_to_bf16_bits
    wl = workload("wide_gqa_fp8", num_seqs=3, part_tokens=1024, appends=1)
    inst = make_instance(wl, seed=5, steps=24, seq_lens=[3000, 2048, 1111])

    def tokens(s):
        kn, vn = inst.new_tokens(s)
        if s != 12:
            return kn, vn
        up = lambda t: f32_to_bf16_bits(bf16_bits_to_f32(t) * np.float32(100.0))  # noqa: E731
        return up(kn), up(vn)

    f = host(run_gpu(inst, 24, new_tokens=tokens, fused=True))
    same_bits(f, host(run_gpu(inst, 24, new_tokens=tokens)))
    o = run_oracle(inst, 24, new_tokens=tokens)
    for key in ("routes", "k_pool", "v_pool", "k_scale", "v_scale"):
        assert np.array_equal(f[key], o[key]), key


@pytest.mark.parametrize("page", [1, 2, 5, 9, 30])
def test_bad_page_in_any_wave_raises_the_flag(gpu, page):
    """A page id outside the pool, at local pages that fall to different
    waves (each wave takes every fourth 2-page tile, from a per-route
    rotation), and a broken route row: NaN for the unit and its sequence,
    BAD_PAGE and BAD_ROUTE raised whichever wave loads the bad page, the rest
    as the oracle has it; the fused step equals the three calls."""
    wl = workload("llama8b_32k", num_seqs=3, num_q_heads=8, num_kv_heads=2, part_tokens=600,
                  appends=1)
    inst = make_instance(wl, seed=9, steps=2, seq_lens=[1300, 700, 1000])
    inst.routes[1, 3] = inst.routes[1, 2] - 5          # tok_end < tok_begin
    inst.page_ids[int(inst.routes[3, 4]) + page] = inst.num_pages + 7
    o = run_oracle(inst, 2)
    assert o["flags"] == oracle.EFLAG_BAD_ROUTE | oracle.EFLAG_BAD_PAGE
    f = host(run_gpu(inst, 2, fused=True))
    compare_all(f, o)
    same_bits(f, host(run_gpu(inst, 2)))
