"""Seeded random shapes through the whole step, against the oracle: KV dtype,
KV heads, group size, sequence count and lengths (empty and page-edge ones
included), route length, pool placement, appends and step count are all
drawn from one generator per case.  Every fourth case draws many short
routes, so that launches with at least 512 unsplit units (two units per
workgroup for bf16) are among them; the others mostly split their units.
The plan each case takes is checked to be a valid one.  A second set draws
equal-length batches of 32 to 1100 units, for the planner's equal-unit rules."""
import numpy as np
import pytest

from kf_testlib import compare_all, host, run_gpu, run_oracle
from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]

EDGE_LENS = (0, 1, 15, 16, 17, 31, 32, 33)


def draw(case):
    rng = np.random.default_rng([2606, 29207, case])
    fp8 = bool(rng.random() < 0.35)
    hkv = int(rng.choice([1, 2, 4, 8]))
    group = int(rng.integers(1, 17))
    many = case % 4 == 0
    if many:        # many routes of at most 15 pages, tails included
        B = int(rng.integers(20, 41))
        part = 16 * int(rng.integers(1, 14))
        lens = rng.integers(100, 1500, B)
    else:
        B = int(rng.integers(1, 13))
        part = 16 * int(rng.integers(1, 160))
        lens = rng.integers(0, 4000, B)
    for i in range(B):
        if rng.random() < 0.2:
            lens[i] = EDGE_LENS[int(rng.integers(len(EDGE_LENS)))]
    appends = int(rng.random() < 0.7)
    steps = int(rng.integers(1, 4)) if appends else 1
    over = dict(num_seqs=B, num_q_heads=group * hkv, num_kv_heads=hkv, part_tokens=part,
                appends=appends, permuted=bool(rng.random() < 0.5))
    wl = workload("wide_gqa_fp8" if fp8 else "llama8b_32k", **over)
    return make_instance(wl, seed=1000 + case, steps=steps, seq_lens=[int(x) for x in lens]), steps


@pytest.mark.parametrize("case", range(48))
def test_random_shape(gpu, case):
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    inst, steps = draw(case)
    st = DecodeState.from_instance(inst)
    chunk_pages, max_chunks, units = kf.partial_attn_plan(st.shape, st.routes.shape[0],
                                                          st.max_pages_per_route)
    assert chunk_pages * max_chunks >= inst.max_pages_per_route and units in (1, 2)
    assert units == 1 or (inst.wl.kv_dtype == "bf16" and max_chunks == 1)
    del st
    o = run_oracle(inst, steps)
    g = host(run_gpu(inst, steps, fused=bool(inst.wl.appends)))
    compare_all(g, o)


@pytest.mark.parametrize("ragged", [True, False])
def test_full_round_of_units_ragged_or_equal(gpu, ragged):
    """512 units (64 single-route sequences x 8 KV heads) fill whole rounds of
    the resident slots.  Equal routes stay whole, two units per workgroup;
    ragged ones (a page table well under routes x max pages; routes of
    up to ~560 pages here, longer than the 256-page range floor) are cut
    into page ranges.  Both match the oracle over fused steps."""
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    rng = np.random.default_rng(606)
    lens = [int(x) for x in rng.integers(16, 9000, 64)] if ragged else [700] * 64
    wl = workload("llama8b_32k", num_seqs=64, part_tokens=1 << 20, appends=1)
    inst = make_instance(wl, seed=31, steps=2, seq_lens=lens)
    assert len(inst.routes) * wl.num_kv_heads == 512
    st = DecodeState.from_instance(inst)
    _, max_chunks, units = kf.partial_attn_plan(st.shape, st.routes.shape[0], st.max_pages_per_route)
    assert (max_chunks > 1 and units == 1) if ragged else (max_chunks == 1 and units == 2)
    del st
    o = run_oracle(inst, 2)
    compare_all(host(run_gpu(inst, 2, fused=True)), o)


@pytest.mark.parametrize("num_seqs,tokens,plan_tail", [(56, 700, (1, 1)), (96, 700, (1, 1)),
                                                      (120, 700, (1, 2)), (40, 1400, (3, 1))])
def test_equal_units_spread_over_the_cus(gpu, num_seqs, tokens, plan_tail):
    """Equal routes whose (route, KV head) units do not fill whole rounds of
    the resident slots but spread evenly over the compute units (448, 768
    and 960 units on 256 CUs) stay whole: one unit per workgroup, or two
    where pairs leave every CU an even count (960).  320 units take the
    fewest ranges whose work items spread evenly (3: 960 items).  They match
    the oracle over fused steps."""
    import torch
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    wl = workload("llama8b_32k", num_seqs=num_seqs, part_tokens=1 << 20, appends=1)
    inst = make_instance(wl, seed=37, steps=2, seq_lens=[tokens] * num_seqs)
    st = DecodeState.from_instance(inst)
    plan = kf.partial_attn_plan(st.shape, st.routes.shape[0], st.max_pages_per_route)
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:
        assert plan[1:] == plan_tail, plan
    del st
    o = run_oracle(inst, 2)
    compare_all(host(run_gpu(inst, 2, fused=True)), o)


def draw_equal(case):
    """An equal-length batch: every sequence holds the same number of tokens,
    split into routes of one drawn length, with 32 to 1100 (route, KV head)
    units, so that the planner's rules for equal units (whole units spread
    evenly over the CUs, the fewest evenly spread ranges, pairs per
    workgroup) are all taken across the cases."""
    rng = np.random.default_rng([7, 7, case])
    fp8 = bool(rng.random() < 0.35)
    hkv = int(rng.choice([1, 2, 4, 8]))
    group = int(rng.integers(1, 9))
    L = int(rng.integers(200, 2500))
    part = 16 * int(rng.integers(max(1, L // 16 // 4), L // 16 + 2))
    units_target = int(rng.integers(32, 1100))
    B = max(1, units_target // (-(-L // part) * hkv))
    appends = int(rng.random() < 0.6)
    over = dict(num_seqs=B, num_q_heads=group * hkv, num_kv_heads=hkv, part_tokens=part,
                appends=appends, permuted=bool(rng.random() < 0.3))
    wl = workload("wide_gqa_fp8" if fp8 else "llama8b_32k", **over)
    steps = 2 if appends else 1
    return make_instance(wl, seed=5000 + case, steps=steps, seq_lens=[L] * B), steps


@pytest.mark.parametrize("case", range(24))
def test_random_equal_shape(gpu, case):
    inst, steps = draw_equal(case)
    o = run_oracle(inst, steps)
    compare_all(host(run_gpu(inst, steps, fused=bool(inst.wl.appends))), o)
