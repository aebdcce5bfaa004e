"""Parity of the library's scaling policy (include/kf_policy.h, host code)
with the oracle (oracle/kf_policy.py), on the hand-worked example and on
seeded random batches: every integer, index and event bit-exact, and every
double bit-exact too (both sides evaluate the same expressions in the same
order).  Host-only: runs without a GPU."""
import math

import numpy as np
import pytest

from oracle import kf_policy as O
from paper_2606_29207_amd import kf, policy as L

from test_policy_pins import example_params, golden

FIELDS = ("num_kv_heads", "head_dim", "num_layers", "elem_bytes", "beta_mem", "beta_slo", "gamma",
          "t_a_max", "bw_hbm", "c_kv_cap", "t_step", "t_prewarm")


def both(p):
    return p, L.params(**{k: p[k] for k in FIELDS})


def ranges_list(st):
    return [[int(r["seq"]), int(r["node"]), int(r["tok_begin"]), int(r["tok_end"])]
            for r in st.live_ranges()]


def same_float(a, b):
    return (math.isnan(a) and math.isnan(b)) or a == b


def compare_sim(po, pl, lens, gens, steps):
    o = O.simulate(po, lens, gens, steps)
    s = L.simulate(pl, lens, gens, steps)
    st = s.state
    assert st.num_nodes == len(o["nodes"])
    assert [tuple(int(x) for x in e) for e in st.events[:st.num_events]] == o["events"]
    assert ranges_list(st) == o["ranges"]
    assert st.tail.tolist() == o["tail"]
    nodes = st.nodes[:st.num_nodes]
    assert nodes["bytes"].tolist() == [nd["bytes"] for nd in o["nodes"]]
    assert nodes["live"].tolist() == [nd["live"] for nd in o["nodes"]]
    assert nodes["prewarm"].tolist() == [nd["prewarm"] for nd in o["nodes"]]
    assert nodes["prewarm_ready"].tolist() == [nd["ready"] for nd in o["nodes"]]
    assert all(same_float(float(a), b["tau"]) for a, b in zip(nodes["tau_fill"], o["nodes"]))
    assert s.tails_per_step.tolist() == (o["tails_per_step"] if steps else [])
    assert s.seq_len.tolist() == o["seq_len"]
    assert s.max_node_bytes == o["max_node_bytes"]
    return o, s


def test_golden_example_through_the_library():
    g = golden()
    po, pl = both(example_params())
    assert L.token_bytes(pl) == 8
    assert L.threshold(pl) == (30.0, 100.0, 30.0)
    st = L.init(pl, [5, 3, 2])
    assert (st.c_total, st.num_nodes) == (80, 3)
    assert ranges_list(st) == g["init_ranges"]
    o, s = compare_sim(po, pl, [5, 3, 2], [4, 10, 1], 6)
    assert [list(int(x) for x in e) for e in s.state.events[:s.state.num_events]] == g["events"]
    rt = L.build_routes(s.state.live_ranges(), 3, [5, 3, 2])
    assert rt.routes.tolist() == g["routes"]
    assert rt.seq_route_begin.tolist() == [int(x) for x in g["seq_route_begin"]]
    assert rt.range_to_route.tolist() == [int(x) for x in g["range_to_route"]]
    assert rt.page_ids.tolist() == list(range(int(g["pages"][0])))


def random_params(rng, tb_scale=1):
    return example_params(
        num_kv_heads=int(rng.integers(1, 4)), head_dim=int(rng.integers(1, 5)),
        num_layers=int(rng.integers(1, 4)), elem_bytes=int(rng.choice([1, 2])),
        beta_mem=float(rng.uniform(0.3, 1.0)), beta_slo=float(rng.uniform(0.3, 1.0)),
        gamma=float(rng.choice([0.5, 0.75, 0.9, 1.0, rng.uniform(0.1, 1.0)])),
        t_a_max=float(rng.uniform(0.5, 4.0)), bw_hbm=float(rng.uniform(10, 400)),
        c_kv_cap=float(rng.uniform(50, 5000)), t_step=float(rng.uniform(0.2, 2.0)),
        t_prewarm=float(rng.choice([0.0, rng.uniform(0.0, 8.0)])))


@pytest.mark.parametrize("seed", range(40))
def test_random_batches_match_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    po, pl = both(random_params(rng))
    B = int(rng.integers(0, 12))
    lens = [int(x) for x in rng.integers(0, 300, B)]
    if B and rng.random() < 0.2:
        lens[int(rng.integers(0, B))] = 0
    gens = [int(x) for x in rng.integers(0, 80, B)]
    steps = int(rng.integers(0, 90))
    assert L.threshold(pl) == O.threshold(po)
    st = L.init(pl, lens)
    oi = O.init(po, lens)
    assert (st.c_total, st.num_nodes) == (oi["c_total"], oi["num_nodes"])
    assert ranges_list(st) == oi["ranges"] and st.tail.tolist() == oi["tail"]
    assert st.nodes[:st.num_nodes]["bytes"].tolist() == oi["node_bytes"]
    o, s = compare_sim(po, pl, lens, gens, steps)
    now = [int(x) for x in rng.integers(0, 400, B)]
    rt = L.build_routes(s.state.live_ranges(), B, now)
    routes, srb, r2r, pages = O.build_routes(o["ranges"], B, now)
    assert rt.routes.tolist() == routes and rt.seq_route_begin.tolist() == srb
    assert rt.range_to_route.tolist() == r2r and len(rt.page_ids) == pages


def test_monitor_step_by_step_matches_oracle():
    """Drive the monitor entry point directly (caller-owned state, the
    caller flips readiness) and compare each pass."""
    rng = np.random.default_rng(7)
    for trial in range(15):
        po, pl = both(random_params(rng))
        B = int(rng.integers(1, 9))
        lens = [int(x) for x in rng.integers(0, 200, B)]
        oi = O.init(po, lens)
        room = B * 40                               # per pass: <= one node, range per request
        st = L.init(pl, lens, max_nodes=oi["num_nodes"] + room,
                    max_ranges=len(oi["ranges"]) + room, max_events=2 * room)
        onodes = O.new_nodes(oi["num_nodes"])
        for k, b in enumerate(oi["node_bytes"]):
            onodes[k]["bytes"] = b
        oranges, otail, oevents = [list(r) for r in oi["ranges"]], list(oi["tail"]), []
        seq_len = list(lens)
        tb = O.token_bytes(po)
        for t in range(40):
            active = [bool(rng.random() < 0.8) for _ in range(B)]
            for k in range(st.num_nodes):          # the caller decides readiness
                if st.nodes[k]["prewarm"] >= 0 and rng.random() < 0.3:
                    st.nodes[k]["prewarm_ready"] = 1
                    onodes[k]["ready"] = 1
            L.monitor(pl, t, st, np.array(active, np.uint8), np.array(seq_len, np.int64))
            O.monitor(po, t, onodes, oranges, otail, active, seq_len, oevents)
            assert st.num_nodes == len(onodes) and ranges_list(st) == oranges
            assert st.tail.tolist() == otail
            assert [tuple(int(x) for x in e) for e in st.events[:st.num_events]] == oevents
            for a, b in zip(st.nodes[:st.num_nodes], onodes):
                assert same_float(float(a["tau_fill"]), b["tau"])
                assert (int(a["prewarm"]), int(a["prewarm_ready"]), int(a["live"])) == \
                    (b["prewarm"], b["ready"], b["live"])
            for i in range(B):                     # append one token to active tails
                if active[i]:
                    r = int(st.tail[i])
                    st.ranges[r]["tok_end"] += 1
                    st.nodes[int(st.ranges[r]["node"])]["bytes"] += tb
                    oranges[otail[i]][3] += 1
                    onodes[oranges[otail[i]][1]]["bytes"] += tb
                    seq_len[i] += 1


def test_llama_scale_agentic_batch():
    """Llama-3.1-8B constants (128 KiB per token), a 64-request batch with
    contexts log-uniform in 2K..128K, MI355X-sized budgets: parity over 3000
    steps with several scale-ups."""
    rng = np.random.default_rng(5)
    lens = [int(x) for x in np.exp(rng.uniform(np.log(2048), np.log(131072), 64))]
    gens = [int(x) for x in rng.integers(100, 3000, 64)]
    # capacity such that three nodes start 0.3% below the memory budget
    cap = sum(lens) * 131072 / 3 / 0.9 * 1.003
    po, pl = both(dict(num_kv_heads=8, head_dim=128, num_layers=32, elem_bytes=2, beta_mem=0.9,
                       beta_slo=0.8, gamma=0.9, t_a_max=1.0e-3, bw_hbm=6.7e12, c_kv_cap=cap,
                       t_step=0.035, t_prewarm=2.0))
    o, s = compare_sim(po, pl, lens, gens, 3000)
    assert o["init"]["num_nodes"] == 3 and s.state.num_nodes >= 5
    assert sum(e[1] == O.PUBLISH for e in o["events"]) >= 2


def test_many_empty_nodes_and_empty_batches():
    po, pl = both(example_params(c_kv_cap=8.0, beta_mem=1.0, beta_slo=1.0, t_a_max=1e9))
    for lens in ([], [0, 0], [3, 0, 2], [1], [0, 7, 0]):
        st = L.init(pl, lens)
        oi = O.init(po, lens)
        assert st.num_nodes == oi["num_nodes"] and ranges_list(st) == oi["ranges"]
        assert st.tail.tolist() == oi["tail"]
        compare_sim(po, pl, lens, [2] * len(lens), 5)


def test_budget_and_pipeline_match_oracle():
    rng = np.random.default_rng(9)
    for _ in range(200):
        a = [float(x) for x in rng.uniform(0, 0.1, 3)]
        L_ = int(rng.integers(1, 128))
        assert L.layer_budget(a[0], a[1], L_, a[2] / 64) == O.layer_budget(a[0], a[1], L_, a[2] / 64)
        assert L.pipeline(*a) == O.pipeline(*a)


def test_free_page_list_is_used_in_route_order():
    po, pl = both(example_params())
    s = L.simulate(pl, [5, 3, 2], [4, 10, 1], 6)
    free = np.array([40, 7, 33, 2, 19, 5, 11, 23], np.int32)
    rt = L.build_routes(s.state.live_ranges(), 3, [5, 3, 2], free_pages=free)
    assert rt.page_ids.tolist() == free[:7].tolist()
    with pytest.raises(kf.KFError):
        L.build_routes(s.state.live_ranges(), 3, [5, 3, 2], free_pages=free[:6])


def test_capacity_and_argument_errors_leave_state_unchanged():
    po, pl = both(example_params())
    with pytest.raises(kf.KFError):
        L.init(pl, [5, 3, 2], max_nodes=2, max_ranges=10)
    with pytest.raises(kf.KFError):
        L.init(pl, [5, -1, 2])
    st = L.init(pl, [5, 3, 2], max_nodes=3, max_ranges=5, max_events=4)
    before = (st.nodes.copy(), st.ranges.copy(), st.tail.copy(), st.num_nodes, st.num_ranges)
    with pytest.raises(kf.KFError):       # two spawns need two more node slots
        L.monitor(pl, 0, st, np.ones(3, np.uint8), np.array([5, 3, 2], np.int64))
    assert st.nodes.tobytes() == before[0].tobytes() and np.array_equal(st.ranges, before[1])
    assert np.array_equal(st.tail, before[2]) and (st.num_nodes, st.num_ranges) == before[3:]
    for bad in (dict(gamma=0.0), dict(gamma=1.5), dict(beta_mem=0.0), dict(elem_bytes=3),
                dict(t_step=0.0), dict(t_prewarm=-1.0), dict(bw_hbm=float("nan")),
                dict(num_layers=0)):
        p = L.params(**{k: v for k, v in dict(example_params(), **bad).items()})
        with pytest.raises(kf.KFError):
            L.threshold(p)
    assert L.layer_budget(0.05, 0.06, 32, 0.0) is None
