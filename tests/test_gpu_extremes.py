"""Degenerate and extreme shapes on the GPU against the oracle: a sequence
cut into thousands of 1-17 token routes (merge fan-in in the thousands),
beside a sequence with a few long routes and one with no tokens; and the
largest route count one launch takes."""
import numpy as np
import pytest

import oracle
from kf_testlib import compare_all, host, run_gpu, run_oracle
from kf_workloads import bf16_bits_to_f32, make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]


def tiny_route_table(lens_per_route, other_lens):
    """Routes of sequence 0 with the given lengths, then one route per
    length in other_lens (one sequence each); consecutive pages."""
    rows, srb, base = [], [0], 0
    tok = 0
    for k, n in enumerate(lens_per_route):
        cap = -(-n // 16)
        rows.append([0, k, tok, tok + n, base, cap])
        tok += n
        base += cap
    srb.append(len(rows))
    for b, n in enumerate(other_lens, start=1):
        cap = max(-(-n // 16), 1)
        rows.append([b, 0, 0, n, base, cap])
        base += cap
        srb.append(len(rows))
    tails = [-1] * (1 + len(other_lens))
    return np.array(rows, np.int32), np.arange(base, dtype=np.int32), np.array(srb, np.int32), \
        np.array(tails, np.int32), tok


def test_thousands_of_tiny_routes(gpu):
    rng = np.random.default_rng(4)
    lens = [int(x) for x in rng.integers(1, 18, 9000)]
    routes, page_ids, srb, tails, n0 = tiny_route_table(lens, [5000, 0])
    wl = workload("llama8b_32k", num_seqs=3, num_q_heads=4, num_kv_heads=1, part_tokens=1 << 20)
    inst = make_instance(wl, seed=9, seq_lens=[n0, 5000, 0], routing=(routes, page_ids, srb, tails))
    o = run_oracle(inst, 1)
    g = host(run_gpu(inst, 1))
    compare_all(g, o)
    # the merge over 9000 partials equals attention over the whole sequence
    q = bf16_bits_to_f32(inst.q).astype(np.float64)
    K, V = inst.logical_kv(0, 0, n0)
    ref_o, ref_l = oracle.attend(q[0], oracle.bf16_to_f64(K[:, 0]), oracle.bf16_to_f64(V[:, 0]),
                                 inst.scale)
    assert np.abs(g["out"][0] - ref_o).max() <= 2e-3
    assert np.abs(g["lse"][0] - ref_l).max() <= 1e-4
    assert np.all(g["out"][2] == 0) and np.all(np.isneginf(g["lse"][2]))   # no tokens


def test_route_count_limit(gpu):
    """65535 routes, the most one launch takes (its grid's z extent): one
    sequence cut into 65534 routes of 1-4 tokens (merge fan-in 65534) beside
    a one-route sequence; 65536 routes are refused on the host."""
    rng = np.random.default_rng(5)
    lens = [int(x) for x in rng.integers(1, 5, 65534)]
    routes, page_ids, srb, tails, n0 = tiny_route_table(lens, [37])
    wl = workload("llama8b_32k", num_seqs=2, num_q_heads=4, num_kv_heads=1, part_tokens=1 << 20)
    inst = make_instance(wl, seed=11, seq_lens=[n0, 37], routing=(routes, page_ids, srb, tails))
    assert len(inst.routes) == 65535
    o = run_oracle(inst, 1)
    g = host(run_gpu(inst, 1))
    compare_all(g, o)
    q = bf16_bits_to_f32(inst.q).astype(np.float64)
    K, V = inst.logical_kv(0, 0, n0)
    ref_o, ref_l = oracle.attend(q[0], oracle.bf16_to_f64(K[:, 0]), oracle.bf16_to_f64(V[:, 0]),
                                 inst.scale)
    assert np.abs(g["out"][0] - ref_o).max() <= 2e-3
    assert np.abs(g["lse"][0] - ref_l).max() <= 1e-4
