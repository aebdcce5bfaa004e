"""Pins of the fp64 oracle against facts fixed outside it.

Each test checks the oracle against something other than itself: a
hand-worked example (tests/golden), closed forms, library routines
(torch's scaled_dot_product_attention with GQA, torch.logsumexp, scipy's
logsumexp/softmax, torch's bf16 and float8_e4m3fn decoders), brute force with
Python loops, and invariants the paper states (the merge of partials over any
split equals attention over the whole range, Section 5.1; the tail attends
after its append, Section 3.2).  The mutation tests at the end plant plausible
mistakes in copies of oracle functions and check that a pin catches each.
"""
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle import kf_oracle
from kf_workloads import make_instance, workload, f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _read_golden(name):
    rows = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            rows.setdefault(key, []).append([float(v) for v in vals])
    return {k: np.array(v) for k, v in rows.items()}


# ------------------------------------------------------------------ decoding
def test_bf16_decode_matches_torch():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 1 << 16, 20000, dtype=np.uint32).astype(np.uint16)
    exp = (bits >> 7) & 0xFF
    bits = bits[exp != 0xFF]                       # drop inf/NaN patterns
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(oracle.bf16_to_f64(bits), ref)


def test_e4m3_table_matches_torch_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    got = oracle.e4m3_to_f64(codes)
    np.testing.assert_array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(got[ok], ref[ok])
    assert set(np.flatnonzero(np.isnan(got))) == {0x7F, 0xFF}


def test_e4m3_landmarks():
    t = oracle.e4m3_table()
    assert t[0x7E] == 448.0 and t[0xFE] == -448.0      # largest finite
    assert t[0x01] == 2.0 ** -9                          # smallest subnormal
    assert t[0x08] == 2.0 ** -6                          # smallest normal
    assert t[0x38] == 1.0 and t[0x80] == 0.0


# ----------------------------------------------------------------- attention
def _brute_attend(q_rows, K, V, scale):
    """Python loops with math.exp of raw scores (no max shift)."""
    G, d = len(q_rows), len(q_rows[0])
    o = np.zeros((G, d))
    lse = np.zeros(G)
    for h in range(G):
        w = [math.exp(scale * sum(q_rows[h][i] * K[t][i] for i in range(d)))
             for t in range(len(K))]
        z = math.fsum(w)
        for i in range(d):
            o[h, i] = math.fsum(w[t] * V[t][i] for t in range(len(K))) / z
        lse[h] = math.log(z)
    return o, lse


@pytest.mark.parametrize("n,d,G", [(1, 4, 1), (3, 5, 2), (6, 8, 3), (9, 3, 4)])
def test_attend_brute_force(n, d, G):
    rng = np.random.default_rng(n * 100 + d)
    q, K, V = rng.normal(size=(G, d)), rng.normal(size=(n, d)), rng.normal(size=(n, d))
    o, lse = oracle.attend(q, K, V, 0.7)
    bo, blse = _brute_attend(q.tolist(), K.tolist(), V.tolist(), 0.7)
    np.testing.assert_allclose(o, bo, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse, blse, rtol=1e-13, atol=1e-14)


def test_attend_matches_torch_sdpa_fp64():
    rng = np.random.default_rng(3)
    G, n, d = 4, 300, 128
    q, K, V = rng.normal(size=(G, d)), rng.normal(size=(n, d)), rng.normal(size=(n, d))
    scale = 1 / math.sqrt(d)
    o, lse = oracle.attend(q, K, V, scale)
    tq = torch.from_numpy(q)[None, :, None, :]              # [1, G, 1, d]
    tk = torch.from_numpy(K)[None, None].expand(1, G, n, d)
    tv = torch.from_numpy(V)[None, None].expand(1, G, n, d)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale)
    np.testing.assert_allclose(o, ref[0, :, 0].numpy(), rtol=1e-12, atol=1e-13)
    ref_lse = torch.logsumexp(torch.from_numpy(scale * (q @ K.T)), dim=1).numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-13, atol=1e-13)


def test_attend_huge_scores_stay_finite():
    rng = np.random.default_rng(4)
    q, K, V = rng.normal(size=(2, 16)) * 40, rng.normal(size=(50, 16)) * 40, rng.normal(size=(50, 16))
    o, lse = oracle.attend(q, K, V, 1.0)
    s = q @ K.T
    np.testing.assert_allclose(lse, scipy.special.logsumexp(s, axis=1), rtol=1e-13)
    np.testing.assert_allclose(o, scipy.special.softmax(s, axis=1) @ V, rtol=1e-10, atol=1e-12)


def test_attend_single_key_returns_its_value():
    rng = np.random.default_rng(5)
    q, K, V = rng.normal(size=(3, 128)), rng.normal(size=(1, 128)), rng.normal(size=(1, 128))
    o, lse = oracle.attend(q, K, V, 0.125)
    np.testing.assert_array_equal(o, np.repeat(V, 3, axis=0))
    np.testing.assert_allclose(lse, 0.125 * (q @ K[0]), rtol=1e-15)


def test_attend_equal_scores_return_mean():
    rng = np.random.default_rng(6)
    n = 37
    K, V = rng.normal(size=(n, 128)), rng.normal(size=(n, 128))
    o, lse = oracle.attend(np.zeros((2, 128)), K, V, 0.1)
    np.testing.assert_allclose(o, np.repeat(V.mean(axis=0)[None], 2, axis=0), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(lse, math.log(n), rtol=1e-15)


def test_attend_empty_range():
    o, lse = oracle.attend(np.ones((2, 8)), np.zeros((0, 8)), np.zeros((0, 8)), 1.0)
    assert np.all(o == 0) and np.all(np.isneginf(lse))


def test_golden_three_keys():
    g = _read_golden("three_keys.txt")
    o, lse = oracle.attend(g["q"], g["k"], g["v"], 1.0)
    np.testing.assert_allclose(o[0], g["o"][0], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(lse[0], g["lse"][0, 0], rtol=1e-15)
    oA, lA = oracle.attend(g["q"], g["k"][:1], g["v"][:1], 1.0)
    oB, lB = oracle.attend(g["q"], g["k"][1:], g["v"][1:], 1.0)
    np.testing.assert_allclose(oA[0], g["oA"][0], atol=1e-14)
    np.testing.assert_allclose(lA[0], g["lseA"][0, 0], atol=1e-15)
    np.testing.assert_allclose(oB[0], g["oB"][0], rtol=1e-14)
    np.testing.assert_allclose(lB[0], g["lseB"][0, 0], rtol=1e-15)
    om, lm = oracle.merge([oA, oB], [lA, lB])
    np.testing.assert_allclose(om[0], g["o"][0], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(lm[0], g["lse"][0, 0], rtol=1e-15)


# --------------------------------------------------------------------- merge
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_merge_of_any_split_equals_unsplit(seed):
    """Section 5.1: merging the partials equals attention over the full range.
    Splits include empty and one-token ranges and non-page-aligned cuts."""
    rng = np.random.default_rng(seed)
    n, G, d = 211, 4, 128
    q, K, V = rng.normal(size=(G, d)), rng.normal(size=(n, d)), rng.normal(size=(n, d))
    o_full, l_full = oracle.attend(q, K, V, 1 / math.sqrt(d))
    cuts = np.sort(np.r_[0, rng.integers(0, n + 1, 6), 5, 5, 6, n])
    parts = [oracle.attend(q, K[a:b], V[a:b], 1 / math.sqrt(d)) for a, b in zip(cuts[:-1], cuts[1:])]
    om, lm = oracle.merge([p[0] for p in parts], [p[1] for p in parts])
    np.testing.assert_allclose(om, o_full, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lm, l_full, rtol=1e-13, atol=1e-13)
    # one-token ranges throughout
    singles = [oracle.attend(q, K[t:t + 1], V[t:t + 1], 1 / math.sqrt(d)) for t in range(n)]
    om, lm = oracle.merge([p[0] for p in singles], [p[1] for p in singles])
    np.testing.assert_allclose(om, o_full, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lm, l_full, rtol=1e-13)


def test_merge_order_and_empty_identity():
    rng = np.random.default_rng(9)
    o = rng.normal(size=(5, 3, 16))
    lse = rng.normal(size=(5, 3)) * 3
    om, lm = oracle.merge(o, lse)
    perm = rng.permutation(5)
    om2, lm2 = oracle.merge(o[perm], lse[perm])
    np.testing.assert_allclose(om2, om, rtol=1e-13)
    np.testing.assert_allclose(lm2, lm, rtol=1e-14)
    o3 = np.concatenate([o, np.zeros((1, 3, 16))])
    l3 = np.concatenate([lse, np.full((1, 3), -np.inf)])
    om3, lm3 = oracle.merge(o3, l3)
    np.testing.assert_array_equal(om3, om)
    np.testing.assert_array_equal(lm3, lm)


def test_merge_all_empty_and_no_partials():
    om, lm = oracle.merge(np.zeros((3, 2, 8)), np.full((3, 2), -np.inf))
    assert np.all(om == 0) and np.all(np.isneginf(lm))
    om, lm = oracle.merge(np.zeros((0, 2, 8)), np.zeros((0, 2)))
    assert np.all(om == 0) and np.all(np.isneginf(lm))


# ---------------------------------------------- whole pipeline vs dense GQA
def _dense_reference(inst, tail_extra=None):
    """torch SDPA (fp64, enable_gqa: query head h reads KV head h // G) over the
    logical tokens of each sequence, drawn afresh from the generator streams."""
    wl = inst.wl
    outs, lses = [], []
    for b in range(wl.num_seqs):
        n = int(inst.seq_lens[b])
        K, V = inst.logical_kv(b, 0, n)
        if tail_extra is not None:
            K = np.concatenate([K, tail_extra[0][b][None]])
            V = np.concatenate([V, tail_extra[1][b][None]])
        Kf = oracle.bf16_to_f64(K).transpose(1, 0, 2)[None]       # [1, Hkv, n, d]
        Vf = oracle.bf16_to_f64(V).transpose(1, 0, 2)[None]
        qf = oracle.bf16_to_f64(inst.q[b])[None, :, None, :]       # [1, Hq, 1, d]
        o = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(qf), torch.from_numpy(Kf), torch.from_numpy(Vf),
            scale=inst.scale, enable_gqa=True)
        outs.append(o[0, :, 0].numpy())
        kk = np.repeat(Kf[0], wl.group, axis=0)                    # [Hq, n, d]
        s = inst.scale * np.einsum("hd,hnd->hn", qf[0, :, 0], kk)
        lses.append(scipy.special.logsumexp(s, axis=1))
    return np.stack(outs), np.stack(lses)


def _oracle_pipeline(inst, routes=None):
    wl = inst.wl
    routes = inst.routes if routes is None else routes
    o_part, lse_part, f1 = oracle.partial_attn(
        inst.q, inst.k_pool, inst.v_pool, routes, inst.page_ids,
        num_kv_heads=wl.num_kv_heads, scale=inst.scale,
        max_pages_per_route=inst.max_pages_per_route)
    out, lse, f2 = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    assert f1 == 0 and f2 == 0
    return out, lse


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("agentic_mix", dict(num_seqs=3, ctx_range=(100, 1500), part_tokens=256)),
    ("llama8b_32k", dict(num_seqs=2, num_q_heads=8, num_kv_heads=2, ctx=700, part_tokens=160)),
])
def test_pipeline_matches_dense_gqa_attention(name, over):
    inst = make_instance(workload(name, **over), seed=2)
    out, lse = _oracle_pipeline(inst)
    ref_o, ref_l = _dense_reference(inst)
    np.testing.assert_allclose(out, ref_o, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse, ref_l, rtol=1e-12, atol=1e-12)


def test_score_offset_keys_gain_four():
    """The agentic workload shifts 5% of keys so that their score rises by
    +4.0 for every query head of the group (up to bf16 rounding of K)."""
    inst = make_instance(workload("agentic_mix", num_seqs=2, ctx_range=(3000, 3001)), seed=1)
    from kf_workloads.synth import _rng, _T_BIAS, _T_K
    b, g, G = 0, 1, inst.wl.group
    mask = _rng(1, inst.wl.wid, _T_BIAS, b, 0).random((2048, 8)) < 0.05
    raw = _rng(1, inst.wl.wid, _T_K, b, 0).standard_normal((2048, 8, 128), dtype=np.float32)
    K, _ = inst.logical_kv(b, 0, 2048)
    q = oracle.bf16_to_f64(inst.q[b, g * G:(g + 1) * G])
    ds = inst.scale * (oracle.bf16_to_f64(K[:, g]) - raw[:, g].astype(np.float64)) @ q.T
    assert 0.03 < mask[:, g].mean() < 0.07
    np.testing.assert_allclose(ds[mask[:, g]], 4.0, atol=0.05)
    np.testing.assert_allclose(ds[~mask[:, g]], 0.0, atol=0.02)


# -------------------------------------------------------------------- gather
@pytest.mark.parametrize("permuted", [False, True])
def test_gather_reads_logical_tokens(permuted):
    wl = workload("llama8b_32k", num_seqs=3, ctx=1000, part_tokens=176, permuted=permuted)
    inst = make_instance(wl, seed=3)
    for r, row in enumerate(inst.routes):
        b, _, tb, te = (int(x) for x in row[:4])
        Kl, Vl = inst.logical_kv(b, tb, te)
        for g in (0, 5):
            K, V = oracle.gather_kv(row, inst.page_ids, inst.k_pool, inst.v_pool, g)
            np.testing.assert_array_equal(K, oracle.bf16_to_f64(Kl[:, g]))
            np.testing.assert_array_equal(V, oracle.bf16_to_f64(Vl[:, g]))


def test_gather_fp8_dequantises_with_page_scale():
    wl = workload("wide_gqa_fp8", num_seqs=1, ctx=100, part_tokens=64)
    inst = make_instance(wl, seed=1)
    row = inst.routes[1]
    K, V = oracle.gather_kv(row, inst.page_ids, inst.k_pool, inst.v_pool, 3,
                            inst.k_scale, inst.v_scale)
    pid = inst.page_ids[int(row[4]) + 1]                     # second page, token 16+5
    code = inst.k_pool[pid, 3, 5, 7]
    ref = torch.tensor([code], dtype=torch.uint8).view(torch.float8_e4m3fn).double().item()
    assert K[21, 7] == ref * np.float64(inst.k_scale[pid, 3])
    code = inst.v_pool[pid, 3, 9, 5]
    ref = torch.tensor([code], dtype=torch.uint8).view(torch.float8_e4m3fn).double().item()
    assert V[21, 9] == ref * np.float64(inst.v_scale[pid, 3])
    assert np.all(np.isfinite(K)) and np.all(np.isfinite(V))


# -------------------------------------------------------------------- append
def test_append_list_model_across_pages():
    """Appending one token per step behaves like appending to a list,
    across page boundaries, until the reserved pages run out."""
    wl = workload("llama8b_32k", num_seqs=2, num_q_heads=4, num_kv_heads=2,
                  ctx=45, part_tokens=32, permuted=True)
    inst = make_instance(wl, seed=4, steps=10)
    kp, vp, routes = inst.k_pool, inst.v_pool, inst.routes.copy()
    lists = {}
    for b in range(2):
        K, V = inst.logical_kv(b, 0, 45)
        lists[b] = ([k for k in K], [v for v in V])
    for step in range(24):
        kn, vn = inst.new_tokens(step)
        kp, vp, routes, flags = oracle.kv_append(kp, vp, routes, inst.page_ids,
                                                 inst.tail_route, kn, vn)
        tail_len = 13 + step + 1                      # 45 = 32 + 13 resident in the tail
        cap_tokens = int(inst.routes[inst.tail_route[0], 5]) * 16
        if tail_len <= cap_tokens:
            assert flags == 0
            for b in range(2):
                lists[b][0].append(kn[b])
                lists[b][1].append(vn[b])
        else:
            assert flags == oracle.EFLAG_TAIL_FULL
        for b in range(2):
            Kl, Vl = np.stack(lists[b][0]), np.stack(lists[b][1])
            rows = routes[inst.seq_route_begin[b]:inst.seq_route_begin[b + 1]]
            for g in range(2):
                K = np.concatenate([oracle.gather_kv(r, inst.page_ids, kp, vp, g)[0] for r in rows])
                V = np.concatenate([oracle.gather_kv(r, inst.page_ids, kp, vp, g)[1] for r in rows])
                np.testing.assert_array_equal(K, oracle.bf16_to_f64(Kl[:, g]))
                np.testing.assert_array_equal(V, oracle.bf16_to_f64(Vl[:, g]))
    # non-tail routes never change
    np.testing.assert_array_equal(routes[[0, 2]], inst.routes[[0, 2]])


def test_append_then_attend_includes_new_token():
    """Section 3.2 step 3: the tail appends the new K/V, then attends over the
    updated range, so the step's query sees its own token."""
    wl = workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2,
                  ctx=300, part_tokens=128)
    inst = make_instance(wl, seed=5, steps=1)
    kn, vn = inst.new_tokens(0)
    kp, vp, routes, flags = oracle.kv_append(inst.k_pool, inst.v_pool, inst.routes,
                                             inst.page_ids, inst.tail_route, kn, vn)
    assert flags == 0
    o_part, lse_part, _ = oracle.partial_attn(inst.q, kp, vp, routes, inst.page_ids,
                                              num_kv_heads=2, scale=inst.scale,
                                              max_pages_per_route=inst.max_pages_per_route)
    out, lse, _ = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    ref_o, ref_l = _dense_reference(inst, tail_extra=(kn, vn))
    np.testing.assert_allclose(out, ref_o, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse, ref_l, rtol=1e-12)


def test_append_skips_inactive_and_flags_bad_routes():
    wl = workload("tiny", num_seqs=3, ctx=40, part_tokens=32, appends=1)
    inst = make_instance(wl, seed=6, steps=2)
    kn, vn = inst.new_tokens(0)
    tail = inst.tail_route.copy()
    tail[1] = -1                                 # inactive sequence
    tail[2] = inst.tail_route[0]                 # names a route of another sequence
    kp, vp, routes, flags = oracle.kv_append(inst.k_pool, inst.v_pool, inst.routes,
                                             inst.page_ids, tail, kn, vn)
    assert flags == oracle.EFLAG_BAD_ROUTE
    changed = np.flatnonzero(np.any(routes != inst.routes, axis=1))
    assert list(changed) == [inst.tail_route[0]]
    assert routes[inst.tail_route[0], 3] == 41
    bad = inst.routes.copy()
    bad[inst.tail_route[0], 3] = 5               # tok_end < tok_begin
    _, _, r2, f2 = oracle.kv_append(inst.k_pool, inst.v_pool, bad, inst.page_ids,
                                    inst.tail_route, kn, vn)
    assert f2 & oracle.EFLAG_BAD_ROUTE


def test_new_empty_tail_route_receives_append():
    """A route published at a token boundary (Section 4.2) starts empty,
    contributes nothing (lse = -inf) until its first append, then holds it."""
    wl = workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2,
                  ctx=256, part_tokens=128)
    inst = make_instance(wl, seed=7, steps=3, empty_tail=True)
    tail = inst.tail_route
    assert np.all(inst.routes[tail, 2] == inst.routes[tail, 3])
    o_part, lse_part, _ = oracle.partial_attn(inst.q, inst.k_pool, inst.v_pool, inst.routes,
                                              inst.page_ids, num_kv_heads=2, scale=inst.scale,
                                              max_pages_per_route=inst.max_pages_per_route)
    assert np.all(np.isneginf(lse_part[tail])) and np.all(o_part[tail] == 0)
    kn, vn = inst.new_tokens(0)
    kp, vp, routes, flags = oracle.kv_append(inst.k_pool, inst.v_pool, inst.routes,
                                             inst.page_ids, tail, kn, vn)
    assert flags == 0 and np.all(routes[tail, 3] == 257)
    o_part, lse_part, _ = oracle.partial_attn(inst.q, kp, vp, routes, inst.page_ids,
                                              num_kv_heads=2, scale=inst.scale,
                                              max_pages_per_route=inst.max_pages_per_route)
    out, lse, _ = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    ref_o, ref_l = _dense_reference(inst, tail_extra=(kn, vn))
    np.testing.assert_allclose(out, ref_o, rtol=1e-11, atol=1e-12)


def test_bad_route_and_bad_page_give_nan_and_flags():
    wl = workload("tiny", num_seqs=1, ctx=64, part_tokens=32)
    inst = make_instance(wl, seed=8)
    args = dict(num_kv_heads=2, scale=inst.scale, max_pages_per_route=inst.max_pages_per_route)
    bad = inst.routes.copy()
    bad[0, 3] = -1
    o, l, f = oracle.partial_attn(inst.q, inst.k_pool, inst.v_pool, bad, inst.page_ids, **args)
    assert f == oracle.EFLAG_BAD_ROUTE and np.all(np.isnan(o[0])) and np.all(np.isfinite(o[1]))
    pids = inst.page_ids.copy()
    pids[3] = inst.num_pages
    o, l, f = oracle.partial_attn(inst.q, inst.k_pool, inst.v_pool, inst.routes, pids, **args)
    assert f == oracle.EFLAG_BAD_PAGE and np.all(np.isnan(l[1])) and np.all(np.isfinite(l[0]))
    o, l, f = oracle.merge_partials(np.zeros((2, 8, 128)), np.zeros((2, 8)), np.array([0, 3]))
    assert f == oracle.EFLAG_BAD_ROUTE and np.all(np.isnan(o))


# --------------------------------------------------------------------- bytes
def test_kv_footprint_formula():
    """Section 4.2: C_total = sum_i 2 s_i H_kv d_h L * 2 B.  One Llama-3.1-8B
    layer, 16 sequences of 32768 + 1 tokens: 2,147,549,184 bytes."""
    assert oracle.kv_footprint_bytes([32769] * 16, 8, 128) == 2_147_549_184
    assert oracle.kv_footprint_bytes([1], 8, 128, num_layers=32) == 2 * 8 * 128 * 32 * 2
    assert oracle.kv_footprint_bytes([10, 20], 8, 128, elem_bytes=1) == 2 * 30 * 8 * 128


# ---------------------------------------------------------- planted mistakes
def _pipeline_error(attend_fn=None, gather_fn=None, merge_fn=None):
    """Max deviation of the oracle pipeline from the dense GQA reference,
    optionally with one oracle function swapped for a mutant."""
    inst = make_instance(workload("llama8b_32k", num_seqs=2, num_q_heads=8, num_kv_heads=2,
                                  ctx=300, part_tokens=96), seed=11)
    saved = (kf_oracle.attend, kf_oracle.gather_kv, kf_oracle.merge)
    try:
        if attend_fn:
            kf_oracle.attend = attend_fn
        if gather_fn:
            kf_oracle.gather_kv = gather_fn
        if merge_fn:
            kf_oracle.merge = merge_fn
        out, lse = _oracle_pipeline(inst)
    finally:
        kf_oracle.attend, kf_oracle.gather_kv, kf_oracle.merge = saved
    ref_o, ref_l = _dense_reference(inst)
    return max(np.nanmax(np.abs(out - ref_o)), np.nanmax(np.abs(lse - ref_l)),
               float(np.isnan(out).any()))


def _mut_no_scale(q, K, V, scale):
    return saved_attend(q, K, V, 1.0)


def _mut_log2(q, K, V, scale):
    o, lse = saved_attend(q, K, V, scale)
    return o, lse / math.log(2.0)


def _mut_unnormalised(q, K, V, scale):
    o, lse = saved_attend(q, K, V, scale)
    return o * K.shape[0], lse


def _mut_gather_v_transposed(route, page_ids, k_pool, v_pool, kv_head, ks=None, vs=None):
    K, V = saved_gather(route, page_ids, k_pool, v_pool, kv_head, ks, vs)
    return K, V[::-1]


def _mut_gather_off_by_one(route, page_ids, k_pool, v_pool, kv_head, ks=None, vs=None):
    r = np.array(route)
    r[3] = max(r[2], r[3] - 1)
    return saved_gather(r, page_ids, k_pool, v_pool, kv_head, ks, vs)


def _mut_gather_wrong_head(route, page_ids, k_pool, v_pool, kv_head, ks=None, vs=None):
    return saved_gather(route, page_ids, k_pool, v_pool, (kv_head + 1) % k_pool.shape[1], ks, vs)


def _mut_merge_plain_mean(o_list, lse_list):
    o = np.asarray(o_list)
    return o.mean(axis=0), np.asarray(lse_list).max(axis=0)


def _mut_merge_sign(o_list, lse_list):
    lse = np.asarray(lse_list)
    return saved_merge(o_list, -lse)


saved_attend, saved_gather, saved_merge = kf_oracle.attend, kf_oracle.gather_kv, kf_oracle.merge


def test_unmutated_pipeline_is_exact():
    assert _pipeline_error() < 1e-11


@pytest.mark.parametrize("kw", [
    dict(attend_fn=_mut_no_scale), dict(attend_fn=_mut_log2), dict(attend_fn=_mut_unnormalised),
    dict(gather_fn=_mut_gather_v_transposed), dict(gather_fn=_mut_gather_off_by_one),
    dict(gather_fn=_mut_gather_wrong_head),
    dict(merge_fn=_mut_merge_plain_mean), dict(merge_fn=_mut_merge_sign),
], ids=lambda kw: next(iter(kw.values())).__name__)
def test_planted_mistake_is_caught(kw):
    assert _pipeline_error(**kw) > 1e-3


# ------------------------------------------------------------- fp8 append
def test_e4m3_encode_matches_torch_cast():
    """Nearest-even encoding onto the E4M3FN grid equals torch's float8_e4m3fn
    cast (on values clamped to +-448), including ties, subnormals and -0."""
    rng = np.random.default_rng(21)
    x = np.concatenate([rng.normal(size=5000).astype(np.float32) * s
                        for s in (1e-3, 0.05, 1, 30, 200, 1000)])
    grid = oracle.e4m3_table()[:0x7F]
    mids = ((grid[:-1] + grid[1:]) / 2).astype(np.float32)
    x = np.concatenate([x, mids, -mids, np.float32([0.0, -0.0, 448, -448, 464, 1e6, 2.0 ** -12])])
    ref = torch.from_numpy(np.clip(x, -448, 448)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(oracle.e4m3_encode_rne(x), ref)


def _fp8_append_run(steps, kv_append=None, big=None):
    """Appends into an E4M3 pool; ``big`` = (step, factor) scales one step's
    new tokens up so that their pages must be re-encoded."""
    wl = workload("wide_gqa_fp8", num_seqs=2, num_q_heads=16, num_kv_heads=2, part_tokens=64,
                  appends=1)
    inst = make_instance(wl, seed=22, steps=steps, seq_lens=[70, 45])
    kv_append = kv_append or oracle.kv_append
    kp, vp, ks, vs, routes = inst.k_pool, inst.v_pool, inst.k_scale, inst.v_scale, inst.routes
    written = []               # (step, b, local index j, k bits, v bits, k scales, v scales)
    for s in range(steps):
        if big is not None and s == big[0]:
            inst.before_big = tuple(a.copy() for a in (kp, vp, ks, vs, routes))
        kn, vn = inst.new_tokens(s)
        if big is not None and s == big[0]:
            kn = f32_to_bf16_bits(oracle.bf16_to_f64(kn).astype(np.float32) * big[1])
            vn = f32_to_bf16_bits(oracle.bf16_to_f64(vn).astype(np.float32) * big[1])
        for b in range(2):
            r = inst.tail_route[b]
            written.append((s, b, int(routes[r, 3] - routes[r, 2]), kn[b], vn[b]))
        kp, vp, ks, vs, routes, f = kv_append(kp, vp, routes, inst.page_ids, inst.tail_route,
                                              kn, vn, ks, vs)
        assert f == 0
        for i in range(len(written) - 2, len(written)):       # page scales right after the write
            s_, b, j, kb, vb = written[i][:5]
            pid = inst.page_ids[int(routes[inst.tail_route[b], 4]) + j // 16]
            written[i] = (s_, b, j, kb, vb, ks[pid].copy(), vs[pid].copy())
    return inst, kp, vp, ks, vs, routes, written


def _stored(inst, routes, pool, b, j, g, kmajor):
    r = inst.tail_route[b]
    pid = inst.page_ids[int(routes[r, 4]) + j // 16]
    return pid, (pool[pid, g][j % 16, :] if kmajor else pool[pid, g][:, j % 16])


def _torch_e4m3(x):
    return torch.from_numpy(np.clip(np.asarray(x, np.float32), -448, 448)).to(
        torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_fp8_append_first_token_scale_and_codes():
    """E4M3 append rule on N(0,1) tokens: a page begun by an append has
    scale = amax(first token)/28 in float32 and is never re-encoded; every
    token whose page scale has not changed since it was written equals
    torch's float8_e4m3fn cast of x/scale, so it lies within half an E4M3 step
    of its bf16 value."""
    inst, kp, vp, ks, vs, routes, written = _fp8_append_run(40)
    checked = 0
    for s_, b, j, kb, vb, ks_then, vs_then in written:
        for pool, scl, then, bits, kmajor in ((kp, ks, ks_then, kb, True), (vp, vs, vs_then, vb, False)):
            for g in range(2):
                pid, codes = _stored(inst, routes, pool, b, j, g, kmajor)
                x = oracle.bf16_to_f64(bits[g]).astype(np.float32)
                first = [w for w in written if w[1] == b and w[2] == j - j % 16]
                if first:                                  # page begun by an append
                    fx = oracle.bf16_to_f64((first[0][3] if kmajor else first[0][4])[g])
                    assert scl[pid, g] == np.float32(np.float32(np.abs(fx).max()) / np.float32(28.0))
                if then[g] != scl[pid, g]:                 # re-encoded later (prefilled page)
                    continue
                checked += 1
                s32 = np.float32(scl[pid, g])
                np.testing.assert_array_equal(codes, _torch_e4m3((x / s32).astype(np.float32)))
                deq = oracle.e4m3_to_f64(codes) * np.float64(s32)
                assert np.all(np.abs(deq - x) <= 2.0 ** -4 * np.abs(x) + np.float64(s32) * 2.0 ** -10)
    assert checked >= 0.9 * 4 * len(written)


def test_fp8_append_reencodes_page_for_large_token():
    """A token 100x larger than its page's first token: the page's earlier
    slots are re-encoded to scale' = amax/28 (torch's cast of
    decode(code)*scale/scale'), and every value stays within two E4M3
    roundings of its bf16 value."""
    steps, at = 12, 5                  # tail of b=1 starts a page at j=48 (step 3)
    inst, kp, vp, ks, vs, routes, written = _fp8_append_run(steps, big=(at, 100.0))
    kp0, vp0, ks0, vs0, routes0 = inst.before_big
    b = 1
    j_big = [w[2] for w in written if w[0] == at and w[1] == b][0]
    assert j_big % 16 > 0
    for pool0, sc0, pool, sc, kmajor, idx in ((kp0, ks0, kp, ks, True, 3), (vp0, vs0, vp, vs, False, 4)):
        for g in range(2):
            pid, _ = _stored(inst, routes, pool, b, j_big, g, kmajor)
            big = oracle.bf16_to_f64(written[[i for i, w in enumerate(written)
                                              if w[0] == at and w[1] == b][0]][idx][g])
            new_scale = np.float32(np.float32(np.abs(big).max()) / np.float32(28.0))
            assert sc[pid, g] == new_scale
            for jj in range(j_big - j_big % 16, j_big):
                _, old_codes = _stored(inst, routes0, pool0, b, jj, g, kmajor)
                vals = (oracle.e4m3_to_f64(old_codes).astype(np.float32) * np.float32(sc0[pid, g]))
                expect = _torch_e4m3((vals.astype(np.float32) / new_scale).astype(np.float32))
                _, codes = _stored(inst, routes, pool, b, jj, g, kmajor)
                np.testing.assert_array_equal(codes, expect)
    for s_, b_, j, kb, vb, _, _ in written:
        for pool, scl, bits, kmajor in ((kp, ks, kb, True), (vp, vs, vb, False)):
            for g in range(2):
                pid, codes = _stored(inst, routes, pool, b_, j, g, kmajor)
                x = oracle.bf16_to_f64(bits[g])
                deq = oracle.e4m3_to_f64(codes) * np.float64(scl[pid, g])
                bound = (2.0 ** -3 + 2.0 ** -8) * np.abs(x) + np.float64(scl[pid, g]) * 2.0 ** -9
                assert np.all(np.abs(deq - x) <= bound)


def test_fp8_append_without_reencode_is_caught():
    """Planted mistake: never re-encode a page when a larger token arrives
    (that token then saturates at 448*scale); the re-encode pin must fail."""
    saved = kf_oracle._append_e4m3

    def no_reencode(page, scales, pid, g, slot, x_bits, kmajor):
        if slot == 0:
            return saved(page, scales, pid, g, slot, x_bits, kmajor)
        x = (np.asarray(x_bits, np.uint16).astype(np.uint32) << 16).view(np.float32)
        codes = oracle.e4m3_encode_rne((x / np.float32(scales[pid, g])).astype(np.float32))
        if kmajor:
            page[slot, :] = codes
        else:
            page[:, slot] = codes
    kf_oracle._append_e4m3 = no_reencode
    try:
        with pytest.raises(AssertionError):
            test_fp8_append_reencodes_page_for_large_token()
    finally:
        kf_oracle._append_e4m3 = saved


def test_append_in_place_equals_append_on_copies():
    """kv_append(..., inplace=True) -- for pools too large to copy every step --
    writes exactly what the copying form returns, for bf16 and E4M3 pools over
    steps that cross pages and re-encode one (and leaves its inputs as the
    copying form would have returned them)."""
    for name, over, lens in (("llama8b_32k", dict(num_seqs=2, num_q_heads=8, num_kv_heads=2,
                                                  part_tokens=64, appends=1), [70, 45]),
                             ("wide_gqa_fp8", dict(num_seqs=2, num_q_heads=16, num_kv_heads=2,
                                                   part_tokens=64, appends=1), [70, 45])):
        inst = make_instance(workload(name, **over), seed=4, steps=20, seq_lens=lens)
        fp8 = inst.k_scale is not None
        ref = [inst.k_pool, inst.v_pool, inst.routes] + ([inst.k_scale, inst.v_scale] if fp8 else [])
        mut = [a.copy() for a in ref]
        for s in range(20):
            kn, vn = inst.new_tokens(s)
            if s == 7:
                kn = f32_to_bf16_bits(oracle.bf16_to_f64(kn).astype(np.float32) * 60)
            if fp8:
                kp, vp, ks, vs, rt, f = oracle.kv_append(ref[0], ref[1], ref[2], inst.page_ids,
                                                         inst.tail_route, kn, vn, ref[3], ref[4])
                ref = [kp, vp, rt, ks, vs]
                out = oracle.kv_append(mut[0], mut[1], mut[2], inst.page_ids, inst.tail_route,
                                       kn, vn, mut[3], mut[4], inplace=True)
                assert out[0] is mut[0] and out[2] is mut[3] and out[4] is mut[2]
            else:
                kp, vp, rt, f = oracle.kv_append(ref[0], ref[1], ref[2], inst.page_ids,
                                                 inst.tail_route, kn, vn)
                ref = [kp, vp, rt]
                out = oracle.kv_append(mut[0], mut[1], mut[2], inst.page_ids, inst.tail_route,
                                       kn, vn, inplace=True)
                assert out[0] is mut[0] and out[2] is mut[2]
            assert f == out[-1] == 0
            for a, b in zip(ref, mut):
                assert np.array_equal(a, b)
        assert not np.array_equal(inst.routes, mut[2])    # the instance's own arrays untouched
