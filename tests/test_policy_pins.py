"""Pins of the scaling-policy oracle (Section 4.2: Algorithm 1, Eqs. (1), (2);
Section 5.2 pipeline model) against things other than itself: a hand-worked
example, closed forms, brute force over all contiguous partitions, step-by-
step recounts of the monitor's timing, and conservation laws.  Planted
mistakes (source mutations of the oracle) must each fail a pin."""
import inspect
import math
import types
from itertools import combinations
from pathlib import Path

import numpy as np
import pytest

from oracle import kf_policy

GOLDEN = Path(__file__).parent / "golden" / "policy_example.txt"


def golden():
    out = {}
    for line in GOLDEN.read_text().splitlines():
        if not line.strip() or line.startswith("#"):
            continue
        k, v = line.split(":", 1)
        items = v.split()
        out[k] = [[int(x) for x in it.split(",")] if "," in it else it for it in items]
    return out


def example_params(**kw):
    p = dict(num_kv_heads=1, head_dim=2, num_layers=1, elem_bytes=2, beta_mem=0.5,
             beta_slo=0.5, gamma=0.9, t_a_max=2.0, bw_hbm=30.0, c_kv_cap=200.0,
             t_step=1.0, t_prewarm=3.0)
    p.update(kw)
    return p


def _ints(xs):
    return [int(x) for x in xs]


# ------------------------------------------------------------- the pins
def pin_golden(P):
    g = golden()
    p = example_params()
    assert P.token_bytes(p) == int(g["token_bytes"][0])
    c, c_mem, c_slo = P.threshold(p)
    assert (c, c_mem, c_slo) == (30.0, 100.0, 30.0)
    st = P.init(p, [5, 3, 2])
    assert st["c_total"] == 80 and st["num_nodes"] == 3
    assert st["ranges"] == g["init_ranges"]
    assert [st["ranges"][t][1] for t in st["tail"]] == _ints(g["init_tail_nodes"])
    assert st["node_bytes"] == _ints(g["init_node_bytes"])
    # tau at the first boundary
    nodes = P.new_nodes(3)
    for k, b in enumerate(st["node_bytes"]):
        nodes[k]["bytes"] = b
    ev = []
    P.monitor(p, 0, nodes, [list(r) for r in st["ranges"]], list(st["tail"]),
              [True] * 3, [5, 3, 2], ev)
    taus = [nd["tau"] for nd in nodes[:3]]
    assert math.isnan(taus[0]) and taus[1] == 0.75 and taus[2] == -0.125
    sim = P.simulate(p, [5, 3, 2], [4, 10, 1], 6)
    assert [list(e) for e in sim["events"]] == g["events"]
    assert sim["tails_per_step"] == g["tails_per_step"]
    assert sim["ranges"] == g["final_ranges"]
    assert [nd["bytes"] for nd in sim["nodes"]] == _ints(g["final_node_bytes"])
    assert [nd["live"] for nd in sim["nodes"]] == _ints(g["final_live"])
    assert sim["seq_len"] == _ints(g["final_seq_len"])
    assert sim["max_node_bytes"] == int(g["max_node_bytes"][0])
    routes, srb, r2r, pages = P.build_routes(sim["ranges"], 3, [5, 3, 2])
    assert routes == g["routes"]
    assert srb == _ints(g["seq_route_begin"]) and r2r == _ints(g["range_to_route"])
    assert pages == int(g["pages"][0])


def pin_threshold_branches(P):
    """Eq. (1): the tighter of the two budgets binds; the SLO term is
    beta_slo * T_A^max * BW * L (whole-node bytes), linear in each factor."""
    base = dict(num_kv_heads=8, head_dim=128, num_layers=32, elem_bytes=2, beta_mem=0.9,
                beta_slo=0.8, gamma=0.9, t_a_max=1e-4, bw_hbm=6e12, c_kv_cap=280e9,
                t_step=0.05, t_prewarm=2.0)
    c, c_mem, c_slo = P.threshold(base)
    assert c_mem == 0.9 * 280e9
    assert c_slo == pytest.approx(0.8 * 1e-4 * 6e12 * 32, rel=1e-15)
    assert c == min(c_mem, c_slo) == c_slo                 # SLO binds here
    c2 = P.threshold(dict(base, t_a_max=1.0))[0]
    assert c2 == c_mem                                       # memory binds
    # doubling L doubles the footprint and the SLO budget: same node count
    lens = [30000, 70000, 123457]
    n1 = P.init(base, lens)["num_nodes"]
    n2 = P.init(dict(base, num_layers=64), lens)["num_nodes"]
    assert n1 == n2 >= 2


def pin_token_bytes(P):
    """Llama-3.1-8B: 2 * 8 * 128 * 32 * 2 B = 128 KiB per token (K and V)."""
    assert P.bytes_per_token(8, 128, 32, 2) == 131072
    assert P.bytes_per_token(8, 128, 80, 1) == 163840


def pin_min_nodes_and_balance(P):
    """N_A is the least node count whose thresholds hold C_total, and the
    initial ranges tile every request exactly once with node loads within one
    token of each other."""
    rng = np.random.default_rng(3)
    for trial in range(60):
        B = int(rng.integers(1, 9))
        lens = [int(x) for x in rng.integers(0, 400, B)]
        p = example_params(c_kv_cap=float(rng.integers(50, 4000)), beta_mem=1.0,
                           beta_slo=1.0, t_a_max=1e9)
        st = P.init(p, lens)
        tb = P.token_bytes(p)
        n, c = st["num_nodes"], P.threshold(p)[0]
        assert st["c_total"] == sum(lens) * tb
        assert n >= 1 and n * c >= st["c_total"]
        if st["c_total"] > 0:
            assert (n - 1) * c < st["c_total"]
        per_seq = {}
        for seq, node, b, e in st["ranges"]:
            per_seq.setdefault(seq, []).append((b, e, node))
        for i, s in enumerate(lens):
            rs = per_seq[i]
            assert rs[0][0] == 0 and rs[-1][1] == s
            assert all(rs[k][1] == rs[k + 1][0] for k in range(len(rs) - 1))
            assert all(rs[k][2] < rs[k + 1][2] for k in range(len(rs) - 1))
            assert st["ranges"][st["tail"][i]][1] == rs[-1][2]
        loads = st["node_bytes"]
        assert sum(loads) == st["c_total"]
        assert max(loads) - min(loads) <= tb


def pin_minimax_bruteforce(P):
    """Brute force: over every way to cut the batch's token sequence into N_A
    contiguous pieces, none has a smaller largest piece than the policy's."""
    for lens in ([3, 1, 4], [5, 0, 2, 2], [1, 1, 1, 1, 1, 6], [7, 2]):
        T = sum(lens)
        for cap in (8.0, 16.0, 24.0, 40.0):
            p = example_params(c_kv_cap=cap, beta_mem=1.0, beta_slo=1.0, t_a_max=1e9)
            st = P.init(p, lens)
            n = st["num_nodes"]
            if n > T:
                continue
            best = min(max(b - a for a, b in zip((0,) + cuts, cuts + (T,)))
                       for cuts in combinations(range(1, T), n - 1))
            assert max(st["node_bytes"]) == best * P.token_bytes(p)


def pin_spawn_and_publish_timing(P):
    """One request on one node growing by one token per step: recount by hand
    when Eq. (2) first predicts a fill sooner than the prewarm, and when the
    watermark and readiness both hold."""
    for b0, prewarm, gamma in ((3, 4.0, 0.9), (0, 2.0, 0.5), (4, 6.0, 1.0), (1, 1.0, 0.25)):
        p = example_params(c_kv_cap=40.0, beta_mem=1.0, beta_slo=1.0, t_a_max=1e9,
                           t_prewarm=prewarm, t_step=1.0, gamma=gamma)
        c = P.threshold(p)[0]                     # 40 B = 5 tokens of 8 B
        steps = 12
        # a second request with no tokens and none to generate shares the
        # node: it is not active, so n_i = 1
        sim = P.simulate(p, [b0, 0], [steps, 0], steps)
        assert sim["init"]["num_nodes"] == 1
        bytes_at = [8 * (b0 + t) for t in range(steps)]       # b_i at boundary t
        spawn = next(t for t in range(steps) if (c - bytes_at[t]) / 8 * 1.0 < prewarm)
        ready = next(t for t in range(spawn + 1, steps + 1) if (t - spawn) * 1.0 >= prewarm)
        pub = next((t for t in range(ready, steps) if bytes_at[t] >= gamma * c), None)
        evs = [e for e in sim["events"] if e[2] == 0]
        assert evs[0] == (spawn, kf_policy.SPAWN, 0, 1, 0)
        if pub is None:
            assert len(evs) == 1
        else:
            assert evs[1] == (pub, kf_policy.PUBLISH, 0, 1, 1)
            assert sim["tails_per_step"][pub][0] == 1 and sim["tails_per_step"][pub - 1][0] == 0


def pin_publish_waits_for_watermark(P):
    """Four requests on one node, three of which stop after one step: the
    steep first-step growth triggers a prewarm, which is ready before the
    node reaches gamma * C_thresh, so the route is published only once the
    watermark is reached (recounted by hand)."""
    p = example_params(c_kv_cap=80.0, beta_mem=1.0, beta_slo=1.0, t_a_max=1e9,
                       t_prewarm=3.0, t_step=1.0, gamma=1.0)
    sim = P.simulate(p, [0, 0, 0, 0], [1, 1, 1, 12], 12)
    # boundary 0: n = 4, tau = 80 / 32 = 2.5 < 3 -> spawn; b = 32 after step 0,
    # then +8 per step: b at boundary t >= 1 is 32 + 8 (t - 1); ready at t = 3;
    # b >= 80 first at t = 7
    assert sim["events"] == [(0, kf_policy.SPAWN, 0, 1, 0), (7, kf_policy.PUBLISH, 0, 1, 1)]


def pin_conservation(P):
    """Every active request appends exactly one token per step to its tail
    node: node bytes sum to the batch's final footprint and every request's
    ranges still tile [0, final length)."""
    rng = np.random.default_rng(11)
    for trial in range(20):
        B = int(rng.integers(1, 7))
        lens = [int(x) for x in rng.integers(0, 60, B)]
        gens = [int(x) for x in rng.integers(0, 40, B)]
        p = example_params(c_kv_cap=float(rng.integers(40, 600)), beta_mem=1.0, beta_slo=1.0,
                           t_a_max=1e9, t_prewarm=float(rng.integers(0, 6)),
                           gamma=float(rng.choice([0.5, 0.8, 1.0])))
        steps = 30
        sim = P.simulate(p, lens, gens, steps)
        tb = P.token_bytes(p)
        final = [s + min(g, steps) for s, g in zip(lens, gens)]
        assert sim["seq_len"] == final
        assert sum(nd["bytes"] for nd in sim["nodes"]) == sum(final) * tb
        for i in range(B):
            rs = sorted((b, e) for seq, node, b, e in sim["ranges"] if seq == i)
            assert rs[0][0] == 0 and rs[-1][1] == final[i]
            assert all(rs[k][1] == rs[k + 1][0] for k in range(len(rs) - 1))
        for t, row in enumerate(sim["tails_per_step"]):
            assert [x >= 0 for x in row] == [t < g for g in gens]
        per_node = {}
        for seq, node, b, e in sim["ranges"]:
            per_node[node] = per_node.get(node, 0) + (e - b) * tb
        assert all(per_node.get(k, 0) == nd["bytes"] for k, nd in enumerate(sim["nodes"]))


def pin_pipeline_and_budget(P):
    """Section 5.2: exposed time is the slower stage; the pipelined/serial
    ratio is 2 for equal stages and tends to 1 when one stage vanishes.
    Section 4.2: T_A^max = (T_slo - overhead) / L, infeasible when the W-side
    stage alone exceeds it."""
    assert P.pipeline(1.0, 2.0, 3.0) == (3.0, 2.0)
    assert P.pipeline(0.5, 0.5, 0.25) == (1.0, 1.25)
    assert P.pipeline(1.0, 0.0, 1e-12)[1] == pytest.approx(1.0)
    assert P.layer_budget(0.050, 0.002, 32, 0.001) == pytest.approx(0.0015)
    assert P.layer_budget(0.050, 0.002, 32, 0.002) is None
    assert P.layer_budget(0.001, 0.002, 32, 0.0) is None


PINS = [pin_golden, pin_threshold_branches, pin_token_bytes, pin_min_nodes_and_balance,
        pin_minimax_bruteforce, pin_spawn_and_publish_timing, pin_publish_waits_for_watermark,
        pin_conservation,
        pin_pipeline_and_budget]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_policy_oracle_pin(pin):
    pin(kf_policy)


# ------------------------------------------------------- planted mistakes
MUTANTS = {
    "max_not_min": ("return min(c_mem, c_slo), c_mem, c_slo", "return max(c_mem, c_slo), c_mem, c_slo"),
    "no_kv_factor": ("return 2 * num_kv_heads * head_dim", "return num_kv_heads * head_dim"),
    "floor_nodes": ("n = max(1, math.ceil(c_total / c_thresh))", "n = max(1, int(c_total // c_thresh))"),
    "slo_without_L": ('* p["bw_hbm"] * p["num_layers"]', '* p["bw_hbm"]'),
    "tail_first_range": ("tail.append(len(ranges) - 1)", "tail.append(len(ranges) - len(mine))"),
    "uneven_cuts": ("cut = [k * total_tokens // n for k in range(n + 1)]",
                    "cut = [min(total_tokens, k * (-(-total_tokens // n))) for k in range(n + 1)]"),
    "tau_watermark": ("tau = (c_thresh - b_i) / g_i", 'tau = (p["gamma"] * c_thresh - b_i) / g_i'),
    "double_spawn": ('p["t_prewarm"] and nd["prewarm"] < 0', 'p["t_prewarm"]'),
    "publish_ignores_watermark": ('if b_i >= p["gamma"] * c_thresh and nd["prewarm"] >= 0',
                                  'if nd["prewarm"] >= 0'),
    "publish_before_ready": ('and nd["ready"]:', ':'),
    "ready_one_early": ('(t - spawned_at[j]) * p["t_step"] >= p["t_prewarm"]',
                        '(t + 1 - spawned_at[j]) * p["t_step"] >= p["t_prewarm"]'),
    "inactive_counted": ("if active[r] and ranges[tail[r]][1] == i)", "if ranges[tail[r]][1] == i)"),
    "append_to_first_range": ("rg = ranges[tail[i]]", "rg = ranges[[k for k, r in enumerate(ranges) if r[0] == i][0]]"),
    "routes_full_cap_end": ("now = max(b, min(e, int(seq_len_now[seq])))", "now = e"),
}


def mutant(name):
    src = inspect.getsource(kf_policy)
    old, new = MUTANTS[name]
    assert src.count(old) == 1, name
    mod = types.ModuleType(f"kf_policy_{name}")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_policy_mutant_is_caught(name):
    mod = mutant(name)
    failed = []
    for pin in PINS:
        try:
            pin(mod)
        except (AssertionError, StopIteration, IndexError, KeyError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
