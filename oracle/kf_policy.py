"""Oracle of the attention-node scaling policy (KernelFlume, arXiv 2606.29207,
Section 4.2 "Elastic Scaling Policy": Algorithm 1, Eqs. (1) and (2); Section
5.2 for the two-stage pipeline model).

TEST INFRASTRUCTURE ONLY: imported by tests/ and nothing in the product.
Plain Python integers for bytes and token counts, Python floats (IEEE
double) for times and budgets, loops in the paper's order.

Readings taken where the paper leaves a choice (the same in the library):

* Bytes per token of one request: 2 (K and V) * H_kv * d_h * L * elem_bytes,
  with elem_bytes = 2 in the paper (16-bit KV); 1 is accepted for 8-bit KV.
* Eq. (1) compares a whole-node KV budget (all L layers, the memory term)
  with the bytes one layer may scan in T_A^max (the SLO term).  Every layer
  scans the node's per-layer share C/L in C/(L * BW_HBM), so the SLO term in
  whole-node bytes is beta_slo * T_A^max * BW_HBM * L.  With L = 1 this is
  the printed formula.
* Per-layer budget: T_A^max = (T_slo - T_overhead) / L; infeasible when the
  W-side stage T_p + T_f alone exceeds it.
* N_A = max(1, ceil(C_total / C_thresh)).
* Byte-balanced initial ranges: the batch's tokens, request after request,
  form one sequence of T tokens; node k owns positions
  [floor(k T / N_A), floor((k+1) T / N_A)).  Every request then has one range
  per node it overlaps (node loads differ by at most one token).  A request's
  tail is the node of its highest range; a request with no tokens gets an
  empty range on the node that owns its start position (the last node when
  it starts at T).
* The monitor runs at every token boundary over the nodes that are the tail
  of at least one active request, in increasing node id.  A prewarm spawned
  for node i reserves the next node id.  Publishing moves every active tail
  on i to the prewarmed node, opening an empty range there at the request's
  current length; node i then holds no active tail.
* In simulation a prewarm spawned at boundary t0 is ready at boundary t once
  (t - t0) * T_step >= T_prewarm.  At boundary t the readiness update comes
  first, then the monitor, then step t appends one token to every active
  request's tail; a request with g tokens to generate is active for steps
  0 .. g-1.
"""
from __future__ import annotations

import math

SPAWN = 1
PUBLISH = 2


def bytes_per_token(num_kv_heads, head_dim, num_layers, elem_bytes=2):
    """KV bytes one request adds per decode token (Section 4.2, the growth term
    of Eq. (2)): K and V, every KV head, every layer."""
    return 2 * num_kv_heads * head_dim * num_layers * elem_bytes


def layer_budget(t_slo, t_overhead, num_layers, t_w_stage):
    """T_A^max from the TPOT target (Section 4.2, per-node budget): the time left
    after per-token overheads, split evenly over the layers.  None when the
    W-side stage T_p + T_f already exceeds that per-layer budget."""
    bud = (t_slo - t_overhead) / num_layers
    if bud <= 0 or t_w_stage > bud:
        return None
    return bud


def threshold(p):
    """Eq. (1): C_thresh = min(C_mem, C_slo), C_mem = beta_mem * C_kv_cap,
    C_slo = beta_slo * T_A^max * BW_HBM * L (whole-node bytes, see above).
    Returns (C_thresh, C_mem, C_slo)."""
    c_mem = p["beta_mem"] * p["c_kv_cap"]
    c_slo = p["beta_slo"] * p["t_a_max"] * p["bw_hbm"] * p["num_layers"]
    return min(c_mem, c_slo), c_mem, c_slo


def token_bytes(p):
    return bytes_per_token(p["num_kv_heads"], p["head_dim"], p["num_layers"], p["elem_bytes"])


def pipeline(t_p, t_f, t_a):
    """Section 5.2 two-stage model: exposed per-layer time max(T_p + T_f, T_A)
    and pipelined-to-serial throughput ratio (T_p + T_A + T_f) / that."""
    exposed = max(t_p + t_f, t_a)
    return exposed, (t_p + t_a + t_f) / exposed


def init(p, seq_lens):
    """Post-prefill initialisation (Algorithm 1, first block; Section 4.2).

    Returns dict(c_total, c_thresh, num_nodes, ranges, tail, node_bytes) where
    ranges is a list of [seq, node, tok_begin, tok_end] ordered by (seq,
    tok_begin) and tail[i] is the index in ranges of request i's tail range.
    """
    tb = token_bytes(p)
    c_thresh = threshold(p)[0]
    lens = [int(s) for s in seq_lens]
    total_tokens = sum(lens)
    c_total = total_tokens * tb
    n = max(1, math.ceil(c_total / c_thresh))
    cut = [k * total_tokens // n for k in range(n + 1)]   # node k: [cut[k], cut[k+1])

    def node_of(g):
        for k in range(n):
            if cut[k] <= g < cut[k + 1]:
                return k
        return n - 1

    ranges, tail = [], []
    start = 0
    for i, s in enumerate(lens):
        mine = []
        for k in range(n):
            lo = max(cut[k], start)
            hi = min(cut[k + 1], start + s)
            if lo < hi:
                mine.append([i, k, lo - start, hi - start])
        if not mine:
            mine.append([i, node_of(start), 0, 0])
        ranges.extend(mine)
        tail.append(len(ranges) - 1)
        start += s
    node_bytes = [0] * n
    for seq, k, b, e in ranges:
        node_bytes[k] += (e - b) * tb
    return dict(c_total=c_total, c_thresh=c_thresh, num_nodes=n, ranges=ranges,
                tail=tail, node_bytes=node_bytes)


def new_nodes(num_nodes):
    """Per-node monitor state: bytes, live, prewarm node id (-1: none),
    prewarm ready flag, last fill horizon."""
    return [dict(bytes=0, live=1, prewarm=-1, ready=0, tau=math.nan) for _ in range(num_nodes)]


def monitor(p, step, nodes, ranges, tail, active, seq_len, events):
    """One pass of Algorithm 1's per-step loop at a token boundary (Eq. (2)).

    nodes: list of node dicts (mutated; spawned prewarms are appended as
    reserved, not-yet-live nodes); ranges/tail as from init (publishing
    appends empty ranges and repoints tail); active[i], seq_len[i] per request.
    Appends (step, kind, node, new_node, count) tuples to events.
    """
    tb = token_bytes(p)
    c_thresh = threshold(p)[0]
    for nd in nodes:
        nd["tau"] = math.nan
    holders = sorted({ranges[tail[i]][1] for i in range(len(tail)) if active[i]})
    for i in holders:
        nd = nodes[i]
        n_i = sum(1 for r in range(len(tail)) if active[r] and ranges[tail[r]][1] == i)
        g_i = n_i * tb
        b_i = nd["bytes"]
        if g_i > 0:
            tau = (c_thresh - b_i) / g_i
            nd["tau"] = tau
            if tau * p["t_step"] < p["t_prewarm"] and nd["prewarm"] < 0:
                nodes.append(dict(bytes=0, live=0, prewarm=-1, ready=0, tau=math.nan))
                nd["prewarm"] = len(nodes) - 1
                nd["ready"] = 0
                events.append((step, SPAWN, i, nd["prewarm"], 0))
        if b_i >= p["gamma"] * c_thresh and nd["prewarm"] >= 0 and nd["ready"]:
            j = nd["prewarm"]
            moved = 0
            for r in range(len(tail)):
                if active[r] and ranges[tail[r]][1] == i:
                    ranges.append([r, j, seq_len[r], seq_len[r]])
                    tail[r] = len(ranges) - 1
                    moved += 1
            nodes[j]["live"] = 1
            nd["prewarm"] = -1
            nd["ready"] = 0
            events.append((step, PUBLISH, i, j, moved))


def simulate(p, seq_lens, gen_lens, steps):
    """Post-prefill init, then `steps` decode steps each preceded by a monitor
    pass at its token boundary (readings above).

    Returns dict(init=..., nodes, ranges, tail, events, tails_per_step
    [steps][B] (tail node used by each step's append, -1 when inactive),
    max_node_bytes (largest b_i seen at any boundary or after any step)).
    """
    st = init(p, seq_lens)
    tb = token_bytes(p)
    ranges = [list(r) for r in st["ranges"]]
    tail = list(st["tail"])
    nodes = new_nodes(st["num_nodes"])
    for k, b in enumerate(st["node_bytes"]):
        nodes[k]["bytes"] = b
    seq_len = [int(s) for s in seq_lens]
    left = [int(g) for g in gen_lens]
    active = [g > 0 for g in left]
    spawned_at = {}
    events, tails_per_step = [], []
    peak = max(nd["bytes"] for nd in nodes)
    for t in range(steps):
        for i, nd in enumerate(nodes):
            j = nd["prewarm"]
            if j >= 0 and not nd["ready"] and (t - spawned_at[j]) * p["t_step"] >= p["t_prewarm"]:
                nd["ready"] = 1
        before = len(events)
        monitor(p, t, nodes, ranges, tail, active, seq_len, events)
        for ev in events[before:]:
            if ev[1] == SPAWN:
                spawned_at[ev[3]] = t
        tails_per_step.append([ranges[tail[i]][1] if active[i] else -1 for i in range(len(tail))])
        for i in range(len(tail)):
            if not active[i]:
                continue
            rg = ranges[tail[i]]
            rg[3] += 1
            nodes[rg[1]]["bytes"] += tb
            seq_len[i] += 1
            left[i] -= 1
            if left[i] == 0:
                active[i] = False
        peak = max(peak, max(nd["bytes"] for nd in nodes))
    return dict(init=st, nodes=nodes, ranges=ranges, tail=tail, events=events,
                tails_per_step=tails_per_step, max_node_bytes=peak, seq_len=seq_len)


def build_routes(ranges, num_seqs, seq_len_now, page_size=16):
    """Routing table for the kernels from policy ranges (Section 4.1 single-GPU
    form): one route per range, grouped by request and ordered by tok_begin;
    capacity = the range's final length in pages; pages numbered in route
    order; tok_end = the request's length now, clamped to the range.
    Returns (routes [R,6] rows (seq, part, tok_begin, tok_end, page_base,
    page_cap), seq_route_begin [B+1], range_to_route [len(ranges)], page count).
    """
    order = sorted(range(len(ranges)), key=lambda k: (ranges[k][0], ranges[k][2], k))
    routes, srb, r2r = [], [0] * (num_seqs + 1), [0] * len(ranges)
    base = 0
    for k in order:
        seq, node, b, e = ranges[k]
        cap = -(-(e - b) // page_size)
        now = max(b, min(e, int(seq_len_now[seq])))
        r2r[k] = len(routes)
        routes.append([seq, node, b, now, base, cap])
        base += cap
        srb[seq + 1] += 1
    for i in range(num_seqs):
        srb[i + 1] += srb[i]
    return routes, srb, r2r, base
