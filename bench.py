"""Benchmark of one decode step of the weightless attention node on one GPU.

A step is the whole hot path over one synthetic batch: tail append of the
step's K/V token, partial attention of every token-range route, and the
log-sum-exp merge per sequence, all through the C ABI on one stream.
Default workload: one Llama-3.1-8B attention layer (16 sequences x 32768
tokens, 32 query / 8 KV heads, head_dim 128, 4 routes of 8192 tokens per
sequence, bf16 KV in 16-token pages, one appended token per step).

Prints ONE JSON line: achieved GB/s over the step's algorithmic bytes
(``value``), microseconds per step, the per-call breakdown, a roofline entry
for the partial-attention kernel and the fp64 oracle timed on host cores.

Flags: --gpus N (only 1 is supported: the path runs on one GPU)
       --steps K --warmup W --workload NAME --seed S --no-cpu-baseline
       --calibrate-copy MiB (time a plain device copy instead; for counter
       calibration under rocprofv3)
       --schedule fused|serial|query_first (default fused: kf_decode_step)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "achieved HBM GB/s + µs/step for partial decode attn+merge (Llama-3.1-8B layer)"
# Tail pages reserved for at least this many appends (more if warmup + 3 x
# steps needs it), so the route table, and with it the launch plan, is the
# same for every short run; tests take the same reservation.
RESERVE_APPENDS = 192
# Host threads of the oracle baseline: the host share of a one-GPU job
# (KF_CPU_THREADS overrides); the visible core count is reported beside it.
CPU_THREADS_DEFAULT = 16
HBM_PEAK_GBPS = 8000.0            # MI355X HBM3E, vendor figure
KERNEL_SRC = os.path.join(ROOT, "paper_2606_29207_amd", "csrc", "kf_kernels.hip")
COUNTERS = os.path.join(ROOT, "profiles", "partial_kernel_{workload}_counters.md")


# ---------------------------------------------------------------- bytes model
def step_bytes(inst, step: int, rows=None) -> dict:
    """Algorithmic HBM bytes of decode step ``step`` (0-based), per call;
    ``rows`` restricts the partial-attention bytes to a list of routes (one
    launch of the query-first schedule).

    KV bytes follow the footprint formula of the paper's scaling policy
    (2 * tokens * H_kv * d_h * element bytes per layer); the rest is what each
    call must read or write at least once."""
    wl = inst.wl
    B, Hq, H, D = wl.num_seqs, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    esz = 1 if wl.kv_dtype == "fp8" else 2
    R = len(inst.routes)
    lens = inst.routes[:, 3].astype(np.int64) - inst.routes[:, 2]
    if wl.appends:
        lens = lens.copy()
        tails = inst.tail_route[inst.tail_route >= 0]
        lens[tails] += step + 1
    if rows is not None:
        lens = lens[np.asarray(rows, np.int64)]
    Rl = len(lens)
    tokens = int(lens.sum())
    pages = int((-(-lens // 16)).sum())
    kv = 2 * tokens * H * D * esz + (2 * pages * H * 4 if esz == 1 else 0)
    partial = kv + B * Hq * D * 2 + pages * 4 + Rl * 24 + Rl * Hq * (D + 1) * 4
    merge = R * Hq * (D + 1) * 4 + (B + 1) * 4 + B * Hq * (D + 1) * 4
    n_app = int((inst.tail_route >= 0).sum()) if wl.appends else 0
    # read the new K/V token, write it into the pool (and, for fp8, read and
    # write the page's K and V scales), read and write the route row
    append = n_app * (2 * H * D * 2 + 2 * H * D * esz + (2 * H * 4 * 2 if esz == 1 else 0) + 2 * 24)
    return dict(append=append, partial=partial, merge=merge, kv=kv, tokens=tokens)


# --------------------------------------------------------------- cpu baseline
def visible_cores() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_threads(host_cores: int) -> int:
    """Threads the oracle baseline uses: KF_CPU_THREADS if set, else the
    visible cores up to CPU_THREADS_DEFAULT."""
    env = os.environ.get("KF_CPU_THREADS")
    if env:
        return max(1, int(env))
    return max(1, min(CPU_THREADS_DEFAULT, host_cores))


def cpu_baseline(inst, min_s=10.0, max_s=30.0) -> dict:
    """The fp64 oracle on the host: partials of (route, KV head) units of the
    same instance, spread over a thread pool with one BLAS thread each, then
    the merge of the sequences completed; repeated until ``min_s`` elapses."""
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    import oracle
    wl = inst.wl
    host_cores = visible_cores()
    cores = cpu_threads(host_cores)
    G = wl.group

    def unit(args):
        r, g = args
        return oracle.route_partial(inst.q, inst.k_pool, inst.v_pool, inst.routes[r],
                                    inst.page_ids, g, num_kv_heads=wl.num_kv_heads,
                                    scale=inst.scale, max_pages_per_route=inst.max_pages_per_route,
                                    k_scale=inst.k_scale, v_scale=inst.v_scale)

    esz = 1 if wl.kv_dtype == "fp8" else 2
    done_bytes, done_seqs = 0, 0
    t0 = time.perf_counter()
    with threadpool_limits(limits=1), ThreadPoolExecutor(cores) as ex:
        b = 0
        while True:
            rows = range(int(inst.seq_route_begin[b]), int(inst.seq_route_begin[b + 1]))
            res = list(ex.map(unit, [(r, g) for r in rows for g in range(wl.num_kv_heads)]))
            o = np.zeros((len(rows), wl.num_q_heads, wl.head_dim))
            lse = np.zeros((len(rows), wl.num_q_heads))
            for i, (oo, ll, _) in enumerate(res):
                r, g = divmod(i, wl.num_kv_heads)
                o[r, g * G:(g + 1) * G], lse[r, g * G:(g + 1) * G] = oo, ll
            oracle.merge(o, lse)
            toks = int((inst.routes[list(rows), 3] - inst.routes[list(rows), 2]).sum())
            done_bytes += 2 * toks * wl.num_kv_heads * wl.head_dim * esz
            done_seqs += 1
            b = (b + 1) % wl.num_seqs
            el = time.perf_counter() - t0
            if el >= min_s or el >= max_s:
                break
    el = time.perf_counter() - t0
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), None)
    except OSError:
        pass
    return {"value": round(done_bytes / el / 1e9, 4), "unit": "GB/s", "cores": cores,
            "host_cores_visible": host_cores, "cpu_model": model,
            "kind": "oracle",
            "sample": f"{done_seqs} sequence(s) of the same instance (all routes x KV heads, "
                      f"fp64 partials + merge, append not timed), {el:.1f} s on {cores} threads, "
                      f"KV bytes {done_bytes}"}


# ------------------------------------------------------------------- counters
def kernel_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def counter_traffic(workload_name: str, seed: int):
    """Per-launch HBM bytes of the partial kernel from the committed rocprofv3
    counter summary of this workload (seed 1), or None when there is none or
    the kernel has changed since it was taken."""
    path = COUNTERS.format(workload=workload_name)
    if seed != 1 or not os.path.exists(path):
        return None
    txt = open(path).read()
    m = re.search(r"kernel_sha256_16:\s*([0-9a-f]+)", txt)
    t = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not m or not t or m.group(1) != kernel_hash():
        return None
    return float(t.group(1))


# ------------------------------------------------------------------------ main
def calibrate_copy(mib: int):
    import torch
    n = mib * (1 << 20)
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    dst.copy_(src)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    print(json.dumps({"copy_bytes_each_way": n, "seconds": dt, "GBps_rw": 2 * n / dt / 1e9}),
          flush=True)


def policy_report(inst, wl, bw_gbps: float, attn_us: float, hbm_bytes: int) -> dict:
    """Scaling-policy calculator (Section 4.2: Algorithm 1, Eqs. (1), (2)) fed
    with this run's measured partial-attention bandwidth, for this batch at
    the full model's depth, through the library's host entry points."""
    from paper_2606_29207_amd import policy as pol
    layers = 80 if wl.num_q_heads == 64 else 32          # 70B-like wide GQA, else Llama-3.1-8B
    t_slo = 0.080 if layers == 80 else 0.050              # the paper's TPOT targets for 70B / 8B
    t_a_max = pol.layer_budget(t_slo, 0.0, layers, 0.0)
    p = pol.params(num_kv_heads=wl.num_kv_heads, head_dim=wl.head_dim, num_layers=layers,
                   elem_bytes=2 if wl.kv_dtype == "bf16" else 1, beta_mem=0.9, beta_slo=0.8,
                   gamma=0.9, t_a_max=t_a_max, bw_hbm=bw_gbps * 1e9, c_kv_cap=float(hbm_bytes),
                   t_step=layers * attn_us * 1e-6, t_prewarm=1.0)
    c, c_mem, c_slo = pol.threshold(p)
    lens = np.asarray(inst.seq_lens, np.int64)
    B = len(lens)
    st = pol.init(p, lens, max_events=4 * B + 8)
    st.nodes = np.concatenate([st.nodes, np.zeros(B + 1, pol.NODE_DT)])
    st.ranges = np.concatenate([st.ranges, np.zeros(B + 1, pol.RANGE_DT)])
    act = np.ones(B, np.uint8)
    pol.monitor(p, 0, st, act, lens)
    taus = st.nodes["tau_fill"][:st.num_nodes]
    tau = float(np.nanmin(taus)) if np.isfinite(taus).any() else None
    pol.monitor(p, 1, st, act, lens)          # a first pass may spawn; the next ones do not
    mon_us = pol.time_monitor(p, st, act, lens) * 1e6
    return {"model_layers": layers, "t_slo_ms": t_slo * 1e3, "t_a_max_us": round(t_a_max * 1e6, 2),
            "bw_hbm_GBps": round(bw_gbps, 2), "c_kv_cap_GB": round(hbm_bytes / 1e9, 2),
            "c_mem_GB": round(c_mem / 1e9, 2), "c_slo_GB": round(c_slo / 1e9, 2),
            "c_thresh_GB": round(c / 1e9, 2), "binding": "slo" if c_slo < c_mem else "mem",
            "c_total_GB": round(st.c_total / 1e9, 2), "n_a": st.num_nodes,
            "node_GB_max": round(float(st.nodes["bytes"][:st.num_nodes].max()) / 1e9, 2),
            "tau_fill_steps_min": None if tau is None else round(tau, 1),
            "t_step_ms": round(layers * attn_us * 1e-3, 3),
            "monitor_us_per_call": round(mon_us, 3),
            "assumptions": "beta_mem 0.9, beta_slo 0.8, gamma 0.9, no per-token overhead, "
                           "T_step = layers x measured attention+merge, T_prewarm 1 s"}


ORDER_MAX_ITEMS = 1 << 20   # largest split launch given a dispatch order


def kernel_label(st, wl, route_list=None) -> str:
    """The partial-attention launch the timed step makes (route_list: a launch
    over those routes), from the library's own plan: its kernel, units per
    workgroup and any combine launch."""
    from paper_2606_29207_amd import kf
    n = st.routes.shape[0] if route_list is None else len(route_list)
    chunk_pages, max_chunks, units = kf.partial_attn_plan(st.shape, n, st.max_pages_per_route,
                                                          route_list=route_list is not None)
    name = f"partial_kernel<{wl.kv_dtype}" + (", 2 units/workgroup>" if units == 2 else ">")
    if route_list is not None:
        name += f" over {n} listed routes"
    if max_chunks > 1:
        name += f" + combine_kernel ({chunk_pages}-page chunks, up to {max_chunks} per unit)"
        # split launches of at least two rounds of resident workgroups (two per CU) run
        # largest ranges first, in an order the one-workgroup order_kernel writes
        import torch
        slots = 2 * torch.cuda.get_device_properties(0).multi_processor_count
        items = max_chunks * st.shape.num_kv_heads * n
        if 2 * slots <= items <= ORDER_MAX_ITEMS:
            name = "order_kernel + " + name
    return name


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="llama8b_32k")
    ap.add_argument("--kv-layout", choices=("page", "head"), default="page",
                    help="pool layout: page-major [P][Hkv][...] (default) or head-major [Hkv][P][...]")
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MiB")
    ap.add_argument("--schedule", choices=("fused", "serial", "query_first"), default="fused",
                    help="fused: kf_decode_step (append fused into the partial-attention "
                         "launch, then the merge); serial: append -> partial -> "
                         "merge as three calls on one stream; query_first: historical partials "
                         "from q alone on one stream, append + tail partials on a second, merge "
                         "after both")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this path runs on exactly one GPU (the decode kernels of one "
              "attention node); --gpus above 1 is not supported", file=sys.stderr)
        return 2
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return 0

    from kf_workloads import make_instance, workload
    wl = workload(args.workload)
    K, W = args.steps, args.warmup
    t = time.perf_counter()
    inst = make_instance(wl, seed=args.seed, steps=max(W + 3 * K, RESERVE_APPENDS))
    print(f"[bench] generated {wl.name} in {time.perf_counter() - t:.1f}s", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:   # host-only work, before the GPU is touched
        cpu = cpu_baseline(inst)
        print(f"[bench] cpu baseline {cpu['value']} GB/s on {cpu['cores']} threads",
              file=sys.stderr, flush=True)

    import torch
    from paper_2606_29207_amd.step import DecodeState
    torch.cuda.set_device(0)
    from paper_2606_29207_amd import kf as _kf
    st = DecodeState.from_instance(
        inst, kv_layout=_kf.KV_HEAD_MAJOR if args.kv_layout == "head" else _kf.KV_PAGE_MAJOR)
    news = [st.upload_new_tokens(*inst.new_tokens(s)) if wl.appends else (None, None)
            for s in range(W + 3 * K)]
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    print(f"[bench] uploaded; warmup {W} steps", file=sys.stderr, flush=True)

    qf = args.schedule == "query_first"
    if qf:
        if not wl.appends:
            print("bench.py: --schedule query_first needs a workload that appends", file=sys.stderr)
            return 2
        st.setup_query_first()
    fused = args.schedule == "fused" and wl.appends > 0

    def one_step(kv):
        if qf:
            st.step_query_first(*kv)
        elif fused:
            st.step_fused(*kv)
        else:
            st.step(*kv)

    for s in range(W):
        one_step(news[s])
    torch.cuda.synchronize()

    # timed region: K whole steps, nothing recorded between the kernels (an
    # event marker between two launches lengthens the gap between them)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        one_step(news[W + i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # breakdown pass: the next K steps as three calls with HIP events around
    # each, on the stream the kernels are launched on (the fused schedule
    # runs the same partial kernel; its launch cannot be bracketed alone)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        e = ev[i]
        e[0].record(stream)
        if qf:
            st.step_query_first(*news[W + K + i], hist_events=(e[1], e[2]))
            e[3].record(stream)
            continue
        if wl.appends:
            st.append(*news[W + K + i])
        e[1].record(stream)
        st.partial()
        e[2].record(stream)
        st.merge()
        e[3].record(stream)
    torch.cuda.synchronize()

    # flushed pass: the next K steps as three calls, each after a 512 MiB
    # scrub write that evicts the 256 MB Infinity Cache (outside the events)
    flushed = None
    if not qf:
        scrub = torch.empty(512 << 20, dtype=torch.uint8, device=st.device)
        evf = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
        for i in range(K):
            scrub.fill_(i & 0xFF)
            e = evf[i]
            e[0].record(stream)
            if wl.appends:
                st.append(*news[W + 2 * K + i])
            e[1].record(stream)
            st.partial()
            e[2].record(stream)
            st.merge()
            e[3].record(stream)
        torch.cuda.synchronize()
        del scrub
        med = lambda a, b: round(float(np.median([e[a].elapsed_time(e[b]) for e in evf])) * 1e3, 2)  # noqa: E731
        flushed = {"scrub_MiB": 512, "append_us_median": med(0, 1) if wl.appends else None,
                   "partial_attn_us_median": med(1, 2), "merge_us_median": med(2, 3),
                   "step_us_median": med(0, 3)}
    flags = st.flags()
    if flags:
        print(f"[bench] device error flags {flags}", file=sys.stderr, flush=True)
        return 1

    t_app = np.array([e[0].elapsed_time(e[1]) for e in ev]) * 1e3      # us
    t_par = np.array([e[1].elapsed_time(e[2]) for e in ev]) * 1e3
    t_mrg = np.array([e[2].elapsed_time(e[3]) for e in ev]) * 1e3
    by = [step_bytes(inst, W + i) for i in range(K)]
    step_b = np.mean([b["append"] + b["partial"] + b["merge"] for b in by])
    by2 = [step_bytes(inst, W + K + i) for i in range(K)]
    if qf:   # the events bracket the launch over the historical routes only
        par_b = np.mean([step_bytes(inst, W + K + i, rows=st.hist_rows)["partial"]
                         for i in range(K)])
    else:
        par_b = np.mean([b["partial"] for b in by2])
    am_b = np.mean([b["partial"] + b["merge"] for b in by2])
    us_step = wall / K * 1e6
    achieved = par_b / (t_par.mean() * 1e-6) / 1e9
    t_step = np.array([e[0].elapsed_time(e[3]) for e in ev]) * 1e3
    # attention + merge: the two calls, or (query-first) the whole overlapped step
    t_am = t_step if qf else t_par + t_mrg
    # the committed counter profiles were taken on page-major pools, for the
    # partial call over the whole route table (not the query-first launch)
    traffic = counter_traffic(wl.name, args.seed) if args.kv_layout == "page" and not qf else None
    out = {
        "metric": METRIC,
        "value": round(step_b / (us_step * 1e-6) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(us_step / 1e3, 4),
        "us_per_step": round(us_step, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.kv_dtype == "bf16" else "fp8_e4m3/bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.num_seqs, "q_heads": wl.num_q_heads,
                   "kv_heads": wl.num_kv_heads, "head_dim": wl.head_dim,
                   "context": int(inst.seq_lens.max()), "route_tokens": wl.part_tokens,
                   "routes": int(len(inst.routes)), "page_tokens": 16,
                   "appends_per_step": wl.appends, "kv_dtype": wl.kv_dtype,
                   "kv_layout": args.kv_layout},
        "schedule": "query_first" if qf else "fused" if fused else "serial",
        "breakdown_pass": ("a second run of K query-first steps with HIP events on the first "
                           "stream around the launch over the historical routes and around the "
                           "whole step" if qf else
                           "a second run of K steps as three calls with HIP events around each"),
        "breakdown_us": ({"historical_partial_attn": round(float(t_par.mean()), 2),
                          "historical_partial_attn_median": round(float(np.median(t_par)), 2),
                          "historical_routes": int(len(st.hist_rows)),
                          "tail_routes": int(len(st.tail_rows)),
                          "step": round(float(t_step.mean()), 2)} if qf else
                         {"append": round(float(t_app.mean()), 2) if wl.appends else None,
                          "partial_attn": round(float(t_par.mean()), 2),
                          "partial_attn_median": round(float(np.median(t_par)), 2),
                          "partial_attn_p10_p90": [round(float(np.percentile(t_par, 10)), 2),
                                                   round(float(np.percentile(t_par, 90)), 2)],
                          "merge": round(float(t_mrg.mean()), 2)}),
        "flushed": flushed,
        "attn_merge_us": round(float(t_am.mean()), 2),
        "attn_merge_GBps": round(am_b / (t_am.mean() * 1e-6) / 1e9, 2),
        "bytes_per_step": int(step_b),
        "roofline": {"bound": "hbm",
                     "kernel": kernel_label(st, wl, st.hist_rows if qf else None),
                     "achieved": round(achieved, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic, "algorithmic_bytes_per_launch": int(par_b)},
        "cpu_baseline": cpu,
        "policy": policy_report(inst, wl, achieved, float(t_am.mean()),
                                torch.cuda.mem_get_info()[1]),
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
