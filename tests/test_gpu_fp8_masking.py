"""fp8 pools: pages past a range's end are loaded only to be masked, so no
value of a page the routes do not reference may reach an output.

Each case prepends one poisoned page to the pool -- every code the E4M3 NaN
(0x7F) and the page's K/V scales +Inf and NaN -- and shifts the page table
by one, so the routes reference exactly the pages they did before and the
oracle, which reads only referenced pages, gives the unpoisoned results.
Route lengths leave 1, 2 and 3 pages past a multiple of the 4-page fp8 tile,
in whole units, in chunked units and in the tails of an appending layer
(Section 3.2, step 3: local attention over the tokens a route holds).
"""
import dataclasses

import numpy as np
import pytest

from kf_testlib import compare_all, host, run_gpu, run_oracle
from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]


def _poison_page_zero(inst):
    fp8 = inst.k_pool.dtype == np.uint8
    assert fp8
    H = inst.k_pool.shape[1]
    bad_k = np.full((1,) + inst.k_pool.shape[1:], 0x7F, np.uint8)
    bad_v = np.full((1,) + inst.v_pool.shape[1:], 0x7F, np.uint8)
    ks = np.concatenate([np.full((1, H), np.inf, np.float32), inst.k_scale])
    vs = np.concatenate([np.full((1, H), np.nan, np.float32), inst.v_scale])
    return dataclasses.replace(
        inst, k_pool=np.concatenate([bad_k, inst.k_pool]),
        v_pool=np.concatenate([bad_v, inst.v_pool]), k_scale=ks, v_scale=vs,
        page_ids=(inst.page_ids + 1).astype(np.int32))


CASES = {
    # whole units: 1, 3, 3, 6 and 10 pages (1, 3, 3, 2, 2 past a multiple of 4)
    "whole": (dict(num_seqs=5, num_q_heads=16, num_kv_heads=2, part_tokens=1024),
              [16, 37, 48, 95, 151], 1),
    # chunked units: ranges of 12 and 13 pages inside 38- and 51-page routes
    "chunked": (dict(num_seqs=2, num_q_heads=16, num_kv_heads=2, part_tokens=2048),
                [16 * 37 + 5, 16 * 50 + 9], 1),
    # appending tails (E4M3 append rule) over three steps
    "append": (dict(num_seqs=3, num_q_heads=16, num_kv_heads=2, part_tokens=512, appends=1),
               [16 * 9 + 14, 530, 33], 3),
}


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("fused", [False, True])
def test_unreferenced_nonfinite_page_never_reaches_outputs(gpu, case, fused):
    over, lens, steps = CASES[case]
    if fused and not over.get("appends"):
        pytest.skip("the fused step applies to appending layers")
    inst = _poison_page_zero(make_instance(workload("wide_gqa_fp8", **over), seed=7,
                                           steps=steps, seq_lens=lens))
    o = run_oracle(inst, steps)
    g = host(run_gpu(inst, steps, fused=fused))
    for key in ("o_part", "lse_part", "out", "lse"):
        assert not np.isnan(g[key]).any(), f"{key}: NaN from the unreferenced page"
    compare_all(g, o)
    assert np.isinf(g["k_scale"][0]).all() and np.isnan(g["v_scale"][0]).all()
