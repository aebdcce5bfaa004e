"""The scaling policy's routing table drives the decode kernels.

A Llama-3.1-8B-shaped layer (32/8 heads) whose six requests are placed on
three attention nodes by the policy (Section 4.2, Algorithm 1) and decode 40
steps while the monitor moves tails to newly published nodes.  The table the
kernels get is the oracle policy's; the library's policy must produce the
same table.  The GPU runs the appends with each step's tails, then partial
attention over the policy's ranges and the merge, and is compared with
(a) the oracle's appends and partials on the same table (pools and routes
bit-exact, floats within the usual bars) and (b) plain attention of each
request's query over its whole token sequence, which does not depend on how
the policy cut it.
"""
import numpy as np
import pytest

import oracle
from oracle import kf_policy as O
from kf_testlib import assert_close_lse, assert_close_o, compare_all
from kf_workloads import bf16_bits_to_f32, make_instance, workload

pytestmark = [pytest.mark.filterwarnings("ignore::RuntimeWarning")]

LENS = [1500, 2900, 640, 2222, 1800, 1037]
GENS = [40, 40, 25, 40, 10, 40]
STEPS = 40


def plan():
    T = sum(LENS)
    p = dict(num_kv_heads=8, head_dim=128, num_layers=1, elem_bytes=2, beta_mem=1.0,
             beta_slo=1.0, gamma=0.9, t_a_max=1.0, bw_hbm=1e15,
             c_kv_cap=T * 4096 / 3 * 1.01, t_step=1.0, t_prewarm=5.0)
    sim = O.simulate(p, LENS, GENS, STEPS)
    routes, srb, r2r, pages = O.build_routes(sim["ranges"], len(LENS), LENS)
    row_of = {(seq, node): r2r[k] for k, (seq, node, b, e) in enumerate(sim["ranges"])}
    tails = [[row_of[(i, n)] if n >= 0 else -1 for i, n in enumerate(row)]
             for row in sim["tails_per_step"]]
    return p, sim, np.array(routes, np.int32), np.array(srb, np.int32), r2r, pages, tails


def test_policy_table_matches_library_and_has_scale_ups():
    from paper_2606_29207_amd import policy as L
    p, sim, routes, srb, r2r, pages, tails = plan()
    assert sim["init"]["num_nodes"] == 3
    assert sum(e[1] == O.PUBLISH for e in sim["events"]) >= 2
    lp = L.params(**p)
    ls = L.simulate(lp, LENS, GENS, STEPS)
    rt = L.build_routes(ls.state.live_ranges(), len(LENS), LENS)
    assert rt.routes.tolist() == routes.tolist() and rt.seq_route_begin.tolist() == srb.tolist()
    assert rt.page_ids.tolist() == list(range(pages))


def build(with_gpu_state=False):
    p, sim, routes, srb, r2r, pages, tails = plan()
    wl = workload("llama8b_32k", num_seqs=len(LENS), appends=1)
    inst = make_instance(wl, seed=31, seq_lens=LENS,
                         routing=(routes, np.arange(pages, dtype=np.int32), srb, tails[0]))
    # oracle appends with each step's tails, then partials on the final table
    kp, vp, rt = inst.k_pool, inst.v_pool, routes.copy()
    for t in range(STEPS):
        kn, vn = inst.new_tokens(t)
        kp, vp, rt, f = oracle.kv_append(kp, vp, rt, inst.page_ids, np.array(tails[t], np.int32),
                                         kn, vn)
        assert f == 0
    o_part, lse_part, f1 = oracle.partial_attn(inst.q, kp, vp, rt, inst.page_ids,
                                               num_kv_heads=wl.num_kv_heads, scale=inst.scale,
                                               max_pages_per_route=inst.max_pages_per_route)
    out, lse, f2 = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    ref = dict(k_pool=kp, v_pool=vp, k_scale=None, v_scale=None, routes=rt, o_part=o_part,
               lse_part=lse_part, out=out, lse=lse, flags=f1 | f2)
    return wl, inst, sim, r2r, tails, ref


def whole_sequence_check(wl, inst, sim, tails, out, lse):
    """Attention of each request's query over its whole token sequence (the
    resident tokens, then the appended ones in step order)."""
    G = wl.group
    q = bf16_bits_to_f32(inst.q).astype(np.float64)
    for i, n0 in enumerate(LENS):
        K, V = inst.logical_kv(i, 0, n0)
        extra = [inst.new_tokens(t) for t in range(STEPS) if tails[t][i] >= 0]
        K = np.concatenate([K] + [kn[i][None] for kn, _ in extra])
        V = np.concatenate([V] + [vn[i][None] for _, vn in extra])
        assert len(K) == sim["seq_len"][i]
        for gk in range(wl.num_kv_heads):
            hs = slice(gk * G, (gk + 1) * G)
            o_ref, lse_ref = oracle.attend(q[i, hs], oracle.bf16_to_f64(K[:, gk]),
                                           oracle.bf16_to_f64(V[:, gk]), inst.scale)
            assert_close_o(out[i, hs], o_ref, f"out seq {i} head {gk}")
            assert_close_lse(lse[i, hs], lse_ref, f"lse seq {i} head {gk}")


def test_oracle_on_policy_table_equals_whole_sequence_attention():
    """CPU: the policy's cut of each request, appended to and merged by the
    oracle, gives plain attention over the whole request (Section 5.1: the
    merge of partials equals attention over the full range)."""
    wl, inst, sim, r2r, tails, ref = build()
    assert [int(ref["routes"][r2r[k], 3]) for k in range(len(r2r))] == [r[3] for r in sim["ranges"]]
    whole_sequence_check(wl, inst, sim, tails, ref["out"], ref["lse"])


@pytest.mark.gpu
def test_decode_on_policy_routes():
    import torch
    from kf_testlib import host
    from paper_2606_29207_amd.step import DecodeState
    wl, inst, sim, r2r, tails, ref = build()
    st = DecodeState.from_instance(inst)
    for t in range(STEPS):
        st.tail_route.copy_(torch.from_numpy(np.array(tails[t], np.int32)))
        kn, vn = st.upload_new_tokens(*inst.new_tokens(t))
        st.append(kn, vn)
    st.partial()
    st.merge()
    torch.cuda.synchronize()
    g = host(st)
    compare_all(g, ref)
    whole_sequence_check(wl, inst, sim, tails, g["out"], g["lse"])
