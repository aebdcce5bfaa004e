"""C-ABI checks that need no GPU: libkf.so loads, exports every function
include/kf.h declares, and rejects bad arguments on the host before it
launches anything (each call below carries at least one error)."""
import ctypes
import os
import re

import pytest

from paper_2606_29207_amd import kf, policy

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kf.h")
POLICY_HEADER = os.path.join(ROOT, "include", "kf_policy.h")

FAKE = 0x10000      # non-null, 256-byte aligned stand-in; never dereferenced here


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(kf._LIB_PATH):
        from paper_2606_29207_amd import build
        build.build()
    return kf.load()


def _declared_functions(header=HEADER):
    src = open(header).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kf_[a-z0-9_]+)\s*\(", src)))


def test_header_and_binding_agree():
    assert _declared_functions() == sorted(kf.EXPORTS)
    assert _declared_functions(POLICY_HEADER) == sorted(policy.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in _declared_functions() + _declared_functions(POLICY_HEADER):
        assert hasattr(lib, name), name
    assert kf.version().startswith("kf ")


def test_struct_layouts_match_header():
    assert ctypes.sizeof(kf.Route) == 24
    assert ctypes.sizeof(kf.Shape) == 40
    assert ctypes.sizeof(policy.Params) == 80
    assert policy.RANGE_DT.itemsize == 24 and policy.NODE_DT.itemsize == 32
    assert policy.EVENT_DT.itemsize == 24 and policy.ROUTE_DT.itemsize == 24


def test_status_strings(lib):
    for code, text in ((0, "ok"), (-1, "invalid argument"), (-2, "unsupported"),
                       (-3, "workspace"), (-4, "HIP"), (-5, "too small"), (-6, "infeasible"),
                       (-7, "host memory"), (-8, "scratch")):
        assert text in kf.status_str(code)
    assert kf.status_str(12345) == "unknown status"


def _shape(**kw):
    d = dict(num_seqs=2, num_q_heads=8, num_kv_heads=2, kv_dtype=kf.KV_BF16, num_pages=10,
             num_page_ids=10, scale=0.088)
    d.update(kw)
    s = kf.make_shape(d["num_seqs"], d["num_q_heads"], d["num_kv_heads"], d["kv_dtype"],
                      d["num_pages"], d["num_page_ids"], d["scale"])
    for k in ("head_dim", "page_size", "kv_layout"):
        if k in kw:
            setattr(s, k, kw[k])
    return s


def _partial(lib, shape, **kw):
    p = dict(q=FAKE, k=FAKE, v=FAKE, ks=None, vs=None, routes=FAKE, R=4, maxp=8, pids=FAKE,
             o=FAKE, lse=FAKE, ws=FAKE, wsb=1 << 30, flags=FAKE)
    p.update(kw)
    v = lambda x: None if x is None else ctypes.c_void_p(x)  # noqa: E731
    return lib.kf_partial_attn(ctypes.byref(shape), v(p["q"]), v(p["k"]), v(p["v"]), v(p["ks"]),
                               v(p["vs"]), v(p["routes"]), p["R"], p["maxp"], v(p["pids"]),
                               v(p["o"]), v(p["lse"]), v(p["ws"]), p["wsb"], v(p["flags"]), None)


@pytest.mark.parametrize("shape_kw,call_kw,status", [
    ({}, dict(q=None), -1),
    ({}, dict(o=None), -1),
    ({}, dict(q=FAKE + 2), -1),                       # misaligned
    ({}, dict(ws=None), -3),
    ({}, dict(wsb=16), -3),
    ({}, dict(ws=FAKE + 64), -3),                    # workspace not 256-byte aligned
    ({"head_dim": 64}, {}, -2),
    ({"page_size": 32}, {}, -2),
    ({"num_q_heads": 7}, {}, -1),                    # not a multiple of Hkv
    ({"num_q_heads": 34, "num_kv_heads": 2}, {}, -2),  # group 17 > 16
    ({"kv_dtype": 1}, {}, -1),                       # fp8 without scales
    ({"kv_dtype": 5}, {}, -2),
    ({"kv_layout": 2}, {}, -2),                      # unknown pool layout
    ({"kv_layout": -1}, {}, -2),
    ({"num_pages": 0}, {}, -1),
    ({"scale": float("nan")}, {}, -1),
    ({}, dict(R=-1), -1),
    ({}, dict(R=65536), -2),                         # launch grid: at most 65535 routes
    ({}, dict(R=70000), -2),
])
def test_partial_attn_host_checks(lib, shape_kw, call_kw, status):
    assert _partial(lib, _shape(**shape_kw), **call_kw) == status


def test_partial_attn_subset_host_checks(lib):
    v = lambda x: None if x is None else ctypes.c_void_p(x)  # noqa: E731
    s = _shape()
    base = [v(FAKE)] * 5 + [v(FAKE), 4]
    tail = [8, v(FAKE), v(FAKE), v(FAKE), v(FAKE), 1 << 30, v(FAKE), None]
    assert lib.kf_partial_attn_subset(ctypes.byref(s), *base[:3], None, None, v(FAKE), 4,
                                      None, 3, *tail) == -1          # list missing
    assert lib.kf_partial_attn_subset(ctypes.byref(s), *base[:3], None, None, v(FAKE), 4,
                                      v(FAKE + 2), 3, *tail) == -1   # list misaligned
    assert lib.kf_partial_attn_subset(ctypes.byref(s), *base[:3], None, None, v(FAKE), 4,
                                      None, 0, *tail) == 0           # empty list: no-op


def test_partial_attn_zero_routes_is_a_no_op(lib):
    assert _partial(lib, _shape(), R=0) == 0


def test_append_host_checks(lib):
    v = ctypes.c_void_p
    rest = [v(FAKE), v(FAKE), v(FAKE), 4, v(FAKE), v(FAKE), v(FAKE), None]   # k_new .. stream
    s = _shape(kv_dtype=kf.KV_FP8_E4M3)
    assert lib.kf_kv_append(ctypes.byref(s), v(FAKE), v(FAKE), None, None, *rest) == -1   # fp8 w/o scales
    s = _shape()
    assert lib.kf_kv_append(ctypes.byref(s), v(FAKE), None, None, None, *rest) == -1       # null v_pool
    bad = [v(FAKE), v(FAKE), v(FAKE), 4, v(FAKE + 1), v(FAKE), v(FAKE), None]
    assert lib.kf_kv_append(ctypes.byref(s), v(FAKE), v(FAKE), None, None, *bad) == -1    # misaligned tail
    s0 = _shape(num_seqs=0)
    assert lib.kf_kv_append(ctypes.byref(s0), *([None] * 6), None, 0, None, None, None, None) == 0


def _step(lib, shape, **kw):
    p = dict(q=FAKE, k=FAKE, v=FAKE, ks=None, vs=None, kn=FAKE, vn=FAKE, routes=FAKE, R=4,
             tail=FAKE, maxp=8, pids=FAKE, srb=FAKE, o=FAKE, lse=FAKE, out=FAKE, lse_out=FAKE,
             ws=FAKE, wsb=1 << 30, flags=FAKE)
    p.update(kw)
    v = lambda x: None if x is None else ctypes.c_void_p(x)  # noqa: E731
    return lib.kf_decode_step(ctypes.byref(shape), v(p["q"]), v(p["k"]), v(p["v"]), v(p["ks"]),
                              v(p["vs"]), v(p["kn"]), v(p["vn"]), v(p["routes"]), p["R"],
                              v(p["tail"]), p["maxp"], v(p["pids"]), v(p["srb"]), v(p["o"]),
                              v(p["lse"]), v(p["out"]), v(p["lse_out"]), v(p["ws"]), p["wsb"],
                              v(p["flags"]), None)


@pytest.mark.parametrize("shape_kw,call_kw,status", [
    ({}, dict(kn=None), -1),                  # append arguments
    ({}, dict(tail=FAKE + 2), -1),
    ({"kv_dtype": 1}, {}, -1),                # fp8 without scales
    ({}, dict(q=None), -1),                   # partial arguments
    ({}, dict(wsb=16), -3),
    ({}, dict(R=70000), -2),
    ({}, dict(srb=None), -1),                 # merge arguments
    ({}, dict(out=FAKE + 4), -1),
    ({"head_dim": 64}, {}, -2),
])
def test_decode_step_host_checks(lib, shape_kw, call_kw, status):
    """Every check of the three calls runs before anything is launched (with
    these fake pointers a launch would fault)."""
    assert _step(lib, _shape(**shape_kw), **call_kw) == status


def test_decode_step_no_sequences_is_a_no_op(lib):
    assert _step(lib, _shape(num_seqs=0), R=0) == 0


def test_merge_host_checks(lib):
    v = ctypes.c_void_p
    ok = [v(FAKE)] * 7
    assert lib.kf_merge_partials(2, 4, 8, 64, *ok, None) == -2       # head_dim
    assert lib.kf_merge_partials(-1, 4, 8, 128, *ok, None) == -1
    assert lib.kf_merge_partials(2, 4, 8, 128, v(FAKE + 4), *ok[1:], None) == -1  # o_part 8B align
    assert lib.kf_merge_partials(2, 4, 8, 128, *ok[:2], None, *ok[3:], None) == -1  # null CSR
    assert lib.kf_merge_partials(0, 4, 8, 128, *([None] * 7), None) == 0


def _workspace_need(units_routes, H, G, maxp, ragged, slots=512, fp8=False, listed=False):
    """Bytes one launch of `units_routes` routes needs, by the planner's rule:
    units that fill whole rounds of the resident slots stay whole (no
    records) unless the routes are ragged (a page table under 90% of routes
    x max pages), and so do equal units spread evenly over the compute units
    (units mod CUs is 0 or at least 3/4 of the CUs, with at least 3/4 of a
    unit per CU); other equal units take the fewest ranges per unit (2 to
    16, of at least 16 pages) that give at least two work items per CU
    spread evenly so (not for route-list launches); otherwise chunks of about 12 per slot (more units than
    slots, never under 256 pages; 6 for fp8 pools) or about one per slot
    (fewer; four when ragged), never under 16 pages, an odd chunk count for the longest unit except for one per slot;
    records of (max, sum) and o per query head, and, for a split launch of
    at least two rounds (up to 2^20 work items), a dispatch-order table of
    two words per item after a two-word header, each array rounded up to 256
    bytes."""
    rup = lambda x: -(-x // 256) * 256  # noqa: E731
    units = units_routes * H
    if units == 0 or maxp <= 16 or (units >= slots and units % slots == 0 and not ragged):
        return 256
    cus = slots // 2
    even = lambda n: n % cus == 0 or n % cus * 4 >= cus * 3  # noqa: E731
    if not ragged and not listed and units * 4 >= cus * 3 and even(units):
        return 256
    m = 0
    if not ragged and not listed and units < (6 if fp8 else 12) * slots:
        for mm in range(2, 17):            # the fewest ranges whose items spread evenly
            c = -(-maxp // mm)
            if c < 16:
                break
            if -(-maxp // c) == mm and units * mm >= slots and even(units * mm):
                m = mm
                break
    if m:
        recs, items = units * m * G, units * m
        ordered = 2 * slots <= items <= 1 << 20
        return rup(recs * 2 * 4) + rup(recs * 128 * 4) + (rup((2 + 2 * items) * 4) if ordered else 0)
    target = ((6 if fp8 else 12) if units >= slots else 4 if ragged else 1) * slots
    c = max(-(-units * maxp // target), 16)
    if units >= slots and not fp8:
        c = max(c, 256)                     # at least a round of bf16 units: ranges of >= 256 pages
    if c >= maxp:
        return 256
    m = -(-maxp // c)
    if (units >= slots or ragged) and m % 2 == 0:
        c = max(-(-maxp // (m + 1)), 16)
        m = -(-maxp // c)
        cc, tries = c - 1, 0
        while m % 2 == 0 and cc >= 16 and tries < 64:   # a bounded search
            if -(-maxp // cc) % 2 == 1:
                c, m = cc, -(-maxp // cc)
            cc -= 1
            tries += 1
    recs = units * m * G
    items = units * m                       # (route, KV head, range) work items of the launch
    ordered = m > 1 and 2 * slots <= items <= 1 << 20
    return rup(recs * 2 * 4) + rup(recs * 128 * 4) + (rup((2 + 2 * items) * 4) if ordered else 0)


def test_workspace_bytes(lib):
    """The size covers every launch of at most num_routes routes (a subset
    launch of a table that fills the GPU may split its units)."""
    s = _shape(num_seqs=16, num_q_heads=32, num_kv_heads=8, num_pages=40000, num_page_ids=40000)
    sizes = [kf.partial_attn_workspace_bytes(s, m, 513) for m in range(0, 80)]
    assert all(a <= b for a, b in zip(sizes, sizes[1:]))            # non-decreasing
    need = lambda k, maxp: max(_workspace_need(k, 8, 4, maxp, rg, listed=ls)  # noqa: E731
                               for rg in (False, True) for ls in (False, True))
    for m in range(0, 80):
        assert sizes[m] == max(need(k, 513) for k in range(0, m + 1))
    assert _workspace_need(64, 8, 4, 513, False) == 256           # 512 equal units: unsplit
    assert _workspace_need(64, 8, 4, 513, True) > 256             # ... ragged ones are cut
    assert _workspace_need(63, 8, 4, 513, False) == 256           # 504 equal units: unsplit
    assert _workspace_need(63, 8, 4, 513, True) > 256             # ... ragged ones are cut
    assert _workspace_need(40, 8, 4, 513, False) > 256            # 320 equal units are cut
    # 1 sequence, 2 routes of 128 pages, 2 KV heads: 8 splits of 16 pages
    s = _shape(num_seqs=1, num_q_heads=8, num_kv_heads=2, num_pages=256, num_page_ids=256)
    recs = 2 * 2 * 8 * 4
    assert kf.partial_attn_workspace_bytes(s, 2, 128) == 1024 + recs * 128 * 4
    # 142 routes x 8 KV heads of up to 1025 pages
    s = _shape(num_seqs=64, num_q_heads=32, num_kv_heads=8, num_pages=10, num_page_ids=10)
    assert kf.partial_attn_workspace_bytes(s, 142, 1025) == max(need(k, 1025) for k in range(143))
    # the size does not depend on the page table's size
    for pids in (10, 36000, 10 ** 9):
        s = _shape(num_seqs=24, num_q_heads=32, num_kv_heads=8, num_pages=10, num_page_ids=pids)
        assert kf.partial_attn_workspace_bytes(s, 48, 1024) == max(need(k, 1024) for k in range(49))
    assert kf.partial_attn_workspace_bytes(s, -1, 5) == 0
    assert kf.partial_attn_workspace_bytes(_shape(head_dim=64), 4, 5) == 0


def test_workspace_query_is_bounded(lib):
    """The query refuses what no launch accepts (above 65535 routes or KV
    heads) and stays fast for any argument: only route counts whose units can
    be split are visited."""
    for H in (1, 2, 8, 65535, 65536):
        for dt in (kf.KV_BF16, kf.KV_FP8_E4M3):
            for R in (1, 6144, 65535, 65536, 2 ** 31 - 1):
                for maxp in (0, 17, 1000, 2 ** 31 - 1):
                    s = _shape(num_seqs=4, num_q_heads=H, num_kv_heads=H, kv_dtype=dt)
                    best = min(_timed(lambda: kf.partial_attn_workspace_bytes(s, R, maxp))
                               for _ in range(3))
                    n = kf.partial_attn_workspace_bytes(s, R, maxp)
                    assert (n == 0) == (R > 65535 or H > 65535), (H, dt, R, maxp, n)
                    assert best < 1e-3, (H, dt, R, maxp, best)


def _timed(fn):
    import time
    t = time.perf_counter()
    fn()
    return time.perf_counter() - t


def test_partial_attn_plan(lib):
    """Launch plans without a GPU (256 compute units assumed: 512 resident
    workgroups).  Whole-table bf16 launches of at least 512 unsplit units of
    at most 2048 pages run two units per workgroup; fp8, route-list and
    chunked launches one."""
    s = _shape(num_seqs=16, num_q_heads=32, num_kv_heads=8, num_pages=40000, num_page_ids=40000)
    big = _shape(num_seqs=16, num_q_heads=32, num_kv_heads=8, num_pages=200000,
                 num_page_ids=200000)
    plan = kf.partial_attn_plan
    assert plan(s, 64, 516) == (516, 1, 2)                  # Llama layer: 512 units, unsplit
    assert plan(s, 64, 516, route_list=True) == (516, 1, 1)
    assert plan(big, 64, 2048) == (2048, 1, 2)
    assert plan(big, 64, 2049) == (2049, 1, 1)              # longer units: one per workgroup
    assert plan(big, 128, 1024) == (1024, 1, 2)             # two rounds of units
    # the same 128 routes in a page table of 40000 (31%): ragged, so ranges
    c, m, u = plan(s, 128, 1024)
    assert m > 1 and m % 2 == 1 and u == 1 and c * m >= 1024
    assert plan(s, 63, 516) == (516, 1, 1)                  # 504 units: all but 8 CUs hold two
    c, m, u = plan(s, 63, 516, route_list=True)             # ... a list's routes may be ragged:
    assert m == 2 and u == 1 and c * m >= 516               # about one range per slot
    c, m, u = plan(s, 40, 516)                              # 320 units: a quarter of the CUs
    assert m > 1 and u == 1 and c * m >= 516 and c * (m - 1) < 516   # would hold two: split
    assert plan(big, 96, 516) == (516, 1, 1)                # 768 units, three per CU: pairs
    assert plan(big, 120, 516) == (516, 1, 2)               # would leave a CU four; 960 units
    assert plan(big, 88, 516) == (516, 1, 1)                # 704 units: three on 3/4 of the CUs
    fp8 = _shape(num_seqs=32, num_q_heads=64, num_kv_heads=8, kv_dtype=kf.KV_FP8_E4M3,
                 num_pages=131072, num_page_ids=131072)
    assert plan(fp8, 128, 1024) == (1024, 1, 1)
    fp8t = _shape(num_seqs=20, num_q_heads=64, num_kv_heads=8, kv_dtype=kf.KV_FP8_E4M3,
                  num_pages=81920, num_page_ids=60000)
    bf16t = _shape(num_seqs=20, num_q_heads=64, num_kv_heads=8, num_pages=81920,
                   num_page_ids=60000)
    assert plan(fp8t, 80, 1024) == (214, 5, 1)               # 640 ragged units: ~6 ranges per slot
    assert plan(bf16t, 80, 1024) == (205, 5, 1)             # ... and ~12 for bf16, but ranges
    #                                                         of >= 256 pages (then an odd count)
    fp8e = _shape(num_seqs=20, num_q_heads=64, num_kv_heads=8, kv_dtype=kf.KV_FP8_E4M3,
                  num_pages=81920, num_page_ids=81920)
    assert plan(fp8e, 80, 1024) == (512, 2, 1)               # 640 equal units: 2 ranges, 5 per CU
    assert plan(fp8e, 40, 1024) == (342, 3, 1)               # 320 equal units: 3 ranges, 3.75 per CU
    for pids in (100, 81920):
        sh = _shape(num_seqs=20, num_q_heads=64, num_kv_heads=8, kv_dtype=kf.KV_FP8_E4M3,
                    num_pages=10, num_page_ids=pids)
        assert kf.partial_attn_workspace_bytes(sh, 80, 1024) == max(
            _workspace_need(k, 8, 8, 1024, rg, fp8=True, listed=ls) for k in range(81)
            for rg in (False, True) for ls in (False, True))
    ragged = _shape(num_seqs=24, num_q_heads=32, num_kv_heads=8, num_pages=36000,
                    num_page_ids=36000)
    assert plan(ragged, 48, 1024) == (147, 7, 1)            # 384 units, table at 73%: ~4 per slot
    equal = _shape(num_seqs=24, num_q_heads=32, num_kv_heads=8, num_pages=49152,
                   num_page_ids=49152)
    assert plan(equal, 48, 1024) == (512, 2, 1)             # full table: 384 units, 2 ranges (3 per CU)
    tiny = _shape(num_seqs=1, num_q_heads=8, num_kv_heads=2, num_pages=256, num_page_ids=256)
    assert plan(tiny, 2, 128) == (16, 8, 1)                 # 4 units: 8 splits of 16 pages
    assert plan(tiny, 2, 16) == (16, 1, 1)                  # too short to split
    assert plan(tiny, 0, 16) == (16, 1, 1)
    # errors: null outputs are allowed, bad sizes and shapes are not
    i32 = ctypes.c_int32
    assert lib.kf_partial_attn_plan(ctypes.byref(s), 64, 516, 0, None, None, None) == 0
    out = [i32(-7) for _ in range(3)]
    refs = [ctypes.byref(o) for o in out]
    for args, status in (((-1, 5, 0), kf.ERR_INVALID_ARG), ((4, -1, 0), kf.ERR_INVALID_ARG),
                         ((4, 5, 2), kf.ERR_INVALID_ARG), ((65536, 5, 0), kf.ERR_UNSUPPORTED)):
        assert lib.kf_partial_attn_plan(ctypes.byref(s), *args, *refs) == status
    assert lib.kf_partial_attn_plan(None, 4, 5, 0, *refs) == kf.ERR_INVALID_ARG
    assert lib.kf_partial_attn_plan(ctypes.byref(_shape(head_dim=64)), 4, 5, 0,
                                    *refs) == kf.ERR_UNSUPPORTED
    assert [o.value for o in out] == [-7, -7, -7]           # nothing written on error


def test_debug_gather_host_checks(lib):
    v = lambda x: None if x is None else ctypes.c_void_p(x)  # noqa: E731
    s = _shape()

    def call(route=0, R=4, maxp=8, max_tokens=16, out=FAKE):
        return lib.kf_debug_gather(ctypes.byref(s), v(FAKE), v(FAKE), v(FAKE), R, route, maxp,
                                   v(FAKE), max_tokens, v(out), v(out), v(FAKE), None)
    assert call(route=4) == -1           # route outside [0, num_routes)
    assert call(route=-1) == -1
    assert call(max_tokens=-3) == -1
    assert call(out=None) == -1          # outputs needed when max_tokens > 0
    assert call(out=FAKE + 2) == -1      # misaligned
    assert call(max_tokens=0, out=None) == 0   # nothing to gather: no launch


def test_binding_refuses_host_tensors_and_bad_shapes(lib):
    """The binding fails loudly before any call: host (CPU) tensors where the
    library needs device memory, and mismatched shapes."""
    import torch
    s = _shape(num_seqs=1, num_q_heads=8, num_kv_heads=2, num_pages=4, num_page_ids=4)
    q = torch.zeros(1, 8, 128, dtype=torch.bfloat16)
    pool = torch.zeros(4, 2, 16, 128, dtype=torch.bfloat16)
    routes = torch.zeros(1, 6, dtype=torch.int32)
    pids = torch.zeros(4, dtype=torch.int32)
    o = torch.zeros(1, 8, 128)
    lse = torch.zeros(1, 8)
    ws = torch.zeros(256, dtype=torch.uint8)
    flags = torch.zeros(1, dtype=torch.int32)
    with pytest.raises(kf.KFError, match="device tensor"):
        kf.partial_attn(s, q, pool, pool, routes, 1, pids, o, lse, ws, flags)
    with pytest.raises(kf.KFError, match="device tensor"):
        kf.kv_append(s, pool, pool, q[:, :2], q[:, :2], routes, flags, pids, flags)
    with pytest.raises(kf.KFError, match="device tensor"):
        kf.merge_partials(1, o, lse, torch.zeros(2, dtype=torch.int32), o, lse, flags)
    with pytest.raises(kf.KFError, match="device tensor"):
        kf.decode_step(s, q, pool, pool, q[:, :2], q[:, :2], routes, flags, 1, pids,
                       torch.zeros(2, dtype=torch.int32), o, lse, o, lse, ws, flags)


def test_plan_invariants_over_random_shapes(lib):
    """Planner invariants for 3000 seeded random launches (256 compute units
    assumed): the ranges cover the longest unit, no range is under 16 pages
    unless the unit stays whole, the range count is odd when units outnumber
    slots or the routes are ragged (unless ranges hit the 16-page floor, or
    equal units take the fewest ranges that spread evenly over the CUs), two
    units per workgroup only for unsplit bf16 launches over the whole table,
    and the workspace sized for the table covers the launch under any page
    table size."""
    import numpy as np
    rng = np.random.default_rng(2606)
    for _ in range(3000):
        hkv = int(rng.choice([1, 2, 4, 8, 16]))
        group = int(rng.integers(1, 17))
        dtype = kf.KV_FP8_E4M3 if rng.random() < 0.3 else kf.KV_BF16
        routes = int(rng.integers(1, 3000))
        maxp = int(rng.integers(1, 5000))
        pids = int(rng.integers(1, routes * maxp + 1))
        s = _shape(num_seqs=4, num_q_heads=group * hkv, num_kv_heads=hkv, kv_dtype=dtype,
                   num_pages=10, num_page_ids=pids)
        launch = int(rng.integers(1, routes + 1))
        listed = bool(rng.random() < 0.3)
        c, m, u = kf.partial_attn_plan(s, launch, maxp, listed)
        assert c * m >= maxp and (m == 1 or c * (m - 1) < maxp)
        assert m == 1 or c >= 16
        units = launch * hkv
        ragged = pids * 10 < launch * maxp * 9
        spread = lambda n: n % 256 == 0 or n % 256 >= 192  # noqa: E731
        if m > 1 and (units >= 512 or ragged) and c > 16:
            assert m % 2 == 1 or (not ragged and not listed and spread(units * m)), \
                (units, maxp, pids, c, m)
        if m > 1 and not ragged and not listed:   # equal units: the fewest evenly spread ranges
            fits = [k for k in range(2, 17) if -(-maxp // k) >= 16 and
                    -(-maxp // -(-maxp // k)) == k and units * k >= 512 and spread(units * k)]
            assert (fits and m == fits[0]) or not fits, (units, maxp, pids, c, m)
        if u == 2:
            assert m == 1 and dtype == kf.KV_BF16 and not listed and units >= 512 and maxp <= 2048
            assert maxp <= 16 or -(-units // 256) % 2 == 0
        if not ragged and not listed and maxp > 16 and units * 4 >= 768 and \
                (units % 256 == 0 or units % 256 >= 192):
            assert m == 1, (units, maxp, pids, c, m)
        need = 256 if m == 1 else -(-units * m * group * 2 * 4 // 256) * 256 + \
            -(-units * m * group * 128 * 4 // 256) * 256
        if routes <= 200:   # the sizing loop is linear in the table's routes
            assert kf.partial_attn_workspace_bytes(s, routes, maxp) >= need


def test_no_alloc_step_refuses_launches_beyond_its_scratch(lib):
    """kf_decode_step_no_alloc checks every argument first, then refuses a
    launch whose split units need more than KF_SCRATCH_BYTES of scratch,
    before anything is launched: 200 routes x 8 KV heads x a group of 16, up
    to 1000 pages, split into 3 ranges, need 40.0 MB."""
    from paper_2606_29207_amd import kf as k
    assert k.SCRATCH_BYTES == 32 << 20
    s = _shape(num_seqs=16, num_q_heads=128, num_kv_heads=8, num_pages=10 ** 6,
               num_page_ids=200 * 1000)
    assert k.partial_attn_plan(s, 200, 1000)[1] == 3
    v = lambda x: ctypes.c_void_p(x)  # noqa: E731
    args = [ctypes.byref(s), v(FAKE), v(FAKE), v(FAKE), None, None, v(FAKE), v(FAKE), v(FAKE), 200,
            v(FAKE), 1000, v(FAKE), v(FAKE), v(FAKE), v(FAKE), v(FAKE), v(FAKE), v(FAKE), None]
    assert lib.kf_decode_step_no_alloc(*args) == k.ERR_SCRATCH_LIMIT
    assert "KF_SCRATCH_BYTES" in k.status_str(k.ERR_SCRATCH_LIMIT)
    bad = list(args)
    bad[16] = None                                      # null out: an argument error comes first
    assert lib.kf_decode_step_no_alloc(*bad) == k.ERR_INVALID_ARG
