"""The seeded input generator (kf_workloads), which serves both the oracle
and the GPU path: rounding bit-equal to torch, determinism, independence
from how a sequence is cut into routes, a permuted page table that is a
bijection, NaN in every unused slot."""
import numpy as np
import torch

import oracle
from kf_workloads import bf16_bits_to_f32, f32_to_bf16_bits, make_instance, workload
from kf_workloads.synth import BF16_NAN, E4M3_NAN


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10 ** rng.uniform(-30, 30, 100000).astype(np.float32),
                        np.array([0.0, -0.0, 1e-40, -1e-40, 3.4e38, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8],
                                 np.float32)]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(x), ref)
    assert np.array_equal(bf16_bits_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(
        torch.bfloat16).float().numpy())


def test_same_seed_same_instance_other_seed_differs():
    wl = workload("agentic_mix", num_seqs=3, ctx_range=(100, 3000), part_tokens=1024)
    a, b = make_instance(wl, seed=4), make_instance(wl, seed=4)
    c = make_instance(wl, seed=5)
    for k in ("q", "k_pool", "v_pool", "routes", "page_ids", "seq_route_begin", "tail_route"):
        assert np.array_equal(getattr(a, k), getattr(b, k)), k
    assert not np.array_equal(a.q, c.q)
    kn1, vn1 = a.new_tokens(3)
    kn2, vn2 = b.new_tokens(3)
    assert np.array_equal(kn1, kn2) and np.array_equal(vn1, vn2)
    assert not np.array_equal(a.new_tokens(4)[0], kn1)


def _tokens(inst, b):
    """Logical K, V of sequence b gathered through its routes (fp64)."""
    ks, vs = [], []
    for r in range(inst.seq_route_begin[b], inst.seq_route_begin[b + 1]):
        K, V = oracle.gather_kv(inst.routes[r], inst.page_ids, inst.k_pool, inst.v_pool, 0)
        ks.append(K)
        vs.append(V)
    return np.concatenate(ks), np.concatenate(vs)


def test_tokens_do_not_depend_on_route_cut_or_permutation():
    lens = [3100, 777]
    base = make_instance(workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2,
                                  part_tokens=4096), seed=2, seq_lens=lens)
    for over in (dict(part_tokens=1000), dict(part_tokens=333), dict(part_tokens=512, permuted=True)):
        other = make_instance(workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2,
                                       **over), seed=2, seq_lens=lens)
        for b in range(2):
            K0, V0 = _tokens(base, b)
            K1, V1 = _tokens(other, b)
            assert np.array_equal(K0, K1) and np.array_equal(V0, V1), (over, b)
            Kl, Vl = other.logical_kv(b, 0, lens[b])
            assert np.array_equal(oracle.bf16_to_f64(Kl[:, 0]), K0)


def test_permuted_page_table_is_a_bijection():
    inst = make_instance(workload("agentic_mix", num_seqs=5, ctx_range=(100, 4000),
                                  part_tokens=1024), seed=3)
    assert np.array_equal(np.sort(inst.page_ids), np.arange(inst.num_pages))
    assert not np.array_equal(inst.page_ids, np.arange(inst.num_pages))


def test_unused_slots_hold_nan():
    for name, nan in (("llama8b_32k", BF16_NAN), ("wide_gqa_fp8", E4M3_NAN)):
        inst = make_instance(workload(name, num_seqs=2, num_q_heads=16, num_kv_heads=2,
                                      part_tokens=1024, appends=1), seed=1, steps=40,
                             seq_lens=[1500, 100])
        used = np.zeros((inst.num_pages, 16), bool)
        for r in inst.routes:
            n = int(r[3] - r[2])
            for j in range(n):
                used[inst.page_ids[r[4] + j // 16], j % 16] = True
        free = ~used
        assert free.any()
        assert np.all(inst.k_pool.transpose(0, 2, 1, 3)[free] == nan)
        assert np.all(inst.v_pool.transpose(0, 3, 1, 2)[free] == nan)
        assert not np.any(inst.k_pool.transpose(0, 2, 1, 3)[used] == nan)


def test_contiguous_pool_hands_out_pages_in_pairs():
    """Every route of a contiguous pool starts on an even page id, its pages
    are consecutive, no page is shared, and capacities are as requested
    (odd reservations leave one unused page behind them)."""
    for steps in (1, 2, 65):
        inst = make_instance(workload("llama8b_32k", num_seqs=3, part_tokens=1000), seed=2,
                             steps=steps, seq_lens=[2100, 999, 3001])
        seen = []
        for r in inst.routes:
            base, cap = int(r[4]), int(r[5])
            ids = inst.page_ids[base:base + cap]
            assert ids[0] % 2 == 0
            assert np.array_equal(ids, ids[0] + np.arange(cap))
            assert cap == -(-(int(r[3] - r[2]) + (steps if r[1] == inst.routes[
                inst.seq_route_begin[r[0] + 1] - 1, 1] else 0)) // 16)
            seen.append(ids)
        seen = np.concatenate(seen)
        assert len(np.unique(seen)) == len(seen) and seen.max() < inst.num_pages
