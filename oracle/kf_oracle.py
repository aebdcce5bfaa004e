"""Plain fp64 oracle for the weightless attention node's decode step.

TEST INFRASTRUCTURE ONLY (see the package docstring): imported by tests, the
smoke check and the CPU-baseline leg of the benchmark, never by the product.

Source: KernelFlume (arXiv 2606.29207).
* Section 3.2 (Workflow of Elastic Decoding), step 3: an attention node that
  owns a request's live tail range first appends the step's new K/V token,
  then every node computes local core attention over the token range(s) it
  stores; step 4: each node returns a partial (o_i, m_i, l_i) and the weight
  node combines the partials with the log-sum-exp (online-softmax) reduction.
* Section 4.1 (Elastic Communication): a routing table maps the logical token
  ranges of a request to the nodes that store their KV; one of them owns the
  live tail.
* Section 5.1 (Query-First Attention): the merge of the partials equals
  attention over the full KV range.
* Section 4.2 (Elastic Scaling Policy), post-prefill initialisation and
  Algorithm 1: KV footprint C_total = sum_i 2 s_i H_kv d_h L * 2 B.

Readings where the paper is silent (the kernels take the same ones): a
partial is exported as (normalised o, lse = m + ln l) instead of
(unnormalised o, m, l); the softmax scale is 1/sqrt(d) applied to the fp64
score; query head h reads KV head h // (H_q / H_kv); the tail attends to the
token it has just appended; an empty range gives (o = 0, lse = -inf).

Storage formats read here (the boundary's, see include/kf.h): 16-token pages;
K page ``[kv_head][slot][d]``; V page ``[kv_head][d][slot]``; bf16 elements as
uint16 bits, fp8 elements as OCP E4M3FN codes with one float32 scale per
(page, kv head).
"""
from __future__ import annotations

import math

import numpy as np

PAGE = 16

EFLAG_TAIL_FULL = 1   # the tail route has no reserved page for the new token
EFLAG_BAD_ROUTE = 2   # a route row, tail index or CSR row is inconsistent
EFLAG_BAD_PAGE = 4    # a page id lies outside the pool


# ------------------------------------------------------------------ decoding
def bf16_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns -> float64 (exact: bf16 is the top half of fp32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def e4m3_table() -> np.ndarray:
    """Value of each of the 256 OCP E4M3FN codes, from the format's definition:
    1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits; exponent field 0
    holds subnormals m/8 * 2^-6; S.1111.111 is NaN; there is no infinity."""
    out = np.empty(256, dtype=np.float64)
    for code in range(256):
        s = -1.0 if code & 0x80 else 1.0
        e = (code >> 3) & 0xF
        m = code & 0x7
        if e == 0xF and m == 0x7:
            out[code] = math.nan
        elif e == 0:
            out[code] = s * (m / 8.0) * 2.0 ** (1 - 7)
        else:
            out[code] = s * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return out


_E4M3 = e4m3_table()


def e4m3_to_f64(codes) -> np.ndarray:
    return _E4M3[np.asarray(codes, dtype=np.uint8)]


_E4M3_POS = _E4M3[:0x7F]          # codes 0x00..0x7E: 0 .. 448, increasing


def e4m3_encode_rne(x) -> np.ndarray:
    """Nearest E4M3FN code to each value (ties to the even code), after
    clamping to [-448, 448]: the format's definition of round-to-nearest-even
    applied to the 127 non-negative grid values; the sign bit is the value's
    (a negative value that rounds to zero gives -0, code 0x80)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), 448.0)
    hi = np.searchsorted(_E4M3_POS, a, side="left")          # first grid value >= a
    hi = np.minimum(hi, 0x7E)
    lo = np.maximum(hi - 1, 0)
    dlo, dhi = a - _E4M3_POS[lo], _E4M3_POS[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    code = np.where(a == _E4M3_POS[hi], hi, np.where(pick_hi, hi, lo)).astype(np.uint8)
    return (code | (np.signbit(x).astype(np.uint8) << 7)).astype(np.uint8)


# -------------------------------------------------------------------- gather
def gather_kv(route, page_ids, k_pool, v_pool, kv_head, k_scale=None, v_scale=None):
    """Logical K, V [n, d] (fp64) of one route and KV head.

    Token t of the route's range [tok_begin, tok_end) is local index
    j = t - tok_begin, stored in page page_ids[page_base + j // 16], slot j % 16
    (the single-GPU form of the routing table of Section 4.1: one route names
    one token range and the pages that hold it)."""
    _, _, tb, te, base, _ = (int(x) for x in route)
    j = np.arange(te - tb)
    pid = np.asarray(page_ids)[base + j // PAGE].astype(np.int64)
    slot = j % PAGE
    kc = k_pool[pid, kv_head, slot, :]          # [n, d]
    vc = v_pool[pid, kv_head, :, slot]          # [n, d]
    if k_pool.dtype == np.uint8:
        K = e4m3_to_f64(kc) * np.asarray(k_scale, np.float64)[pid, kv_head][:, None]
        V = e4m3_to_f64(vc) * np.asarray(v_scale, np.float64)[pid, kv_head][:, None]
    else:
        K, V = bf16_to_f64(kc), bf16_to_f64(vc)
    return K, V


# ----------------------------------------------------------------- attention
def attend(q_rows, K, V, scale):
    """Softmax attention of query rows [G, d] over keys/values [n, d], fp64.

    Local core attention of Section 3.2, step 3:
      s_t = scale * (q . k_t),  o = sum_t softmax(s)_t v_t,  lse = ln sum_t e^{s_t}.
    Returns (o [G, d], lse [G]); an empty range gives (0, -inf)."""
    q_rows = np.asarray(q_rows, np.float64)
    G, d = q_rows.shape
    if K.shape[0] == 0:
        return np.zeros((G, d)), np.full(G, -np.inf)
    s = scale * (K @ q_rows.T)                   # [n, G]
    m = s.max(axis=0)
    e = np.exp(s - m)
    ell = e.sum(axis=0)
    o = (e.T @ V) / ell[:, None]
    return o, m + np.log(ell)


def _route_ok(route, B, num_page_ids, max_pages):
    seq, _, tb, te, base, cap = (int(x) for x in route)
    n = te - tb
    npg = -(-n // PAGE) if n > 0 else 0
    return (0 <= seq < B and n >= 0 and base >= 0 and npg <= cap
            and npg <= max_pages and base + npg <= num_page_ids)


def route_partial(q, k_pool, v_pool, route, page_ids, kv_head, *, num_kv_heads,
                  scale, max_pages_per_route, k_scale=None, v_scale=None):
    """Partial of one (route, KV head): o [G, d], lse [G], error flags.

    q is bf16 bits [B, Hq, d].  A route that fails the consistency checks, or
    that names a page outside the pool, yields NaN with a flag set."""
    B, Hq, d = q.shape
    G = Hq // num_kv_heads
    flags = 0
    if not _route_ok(route, B, len(page_ids), max_pages_per_route):
        return np.full((G, d), np.nan), np.full(G, np.nan), EFLAG_BAD_ROUTE
    seq, _, tb, te, base, _ = (int(x) for x in route)
    n = te - tb
    npg = -(-n // PAGE) if n > 0 else 0
    pids = np.asarray(page_ids[base:base + npg])
    if np.any((pids < 0) | (pids >= k_pool.shape[0])):
        return np.full((G, d), np.nan), np.full(G, np.nan), EFLAG_BAD_PAGE
    K, V = gather_kv(route, page_ids, k_pool, v_pool, kv_head, k_scale, v_scale)
    qg = bf16_to_f64(q[seq, kv_head * G:(kv_head + 1) * G, :])
    o, lse = attend(qg, K, V, scale)
    return o, lse, flags


def partial_attn(q, k_pool, v_pool, routes, page_ids, *, num_kv_heads, scale,
                 max_pages_per_route, k_scale=None, v_scale=None):
    """Partials of every route: o_part [R, Hq, d], lse_part [R, Hq], flags."""
    B, Hq, d = q.shape
    G = Hq // num_kv_heads
    R = len(routes)
    o_part = np.zeros((R, Hq, d))
    lse_part = np.zeros((R, Hq))
    flags = 0
    for r in range(R):
        for g in range(num_kv_heads):
            o, lse, f = route_partial(q, k_pool, v_pool, routes[r], page_ids, g,
                                      num_kv_heads=num_kv_heads, scale=scale,
                                      max_pages_per_route=max_pages_per_route,
                                      k_scale=k_scale, v_scale=v_scale)
            o_part[r, g * G:(g + 1) * G] = o
            lse_part[r, g * G:(g + 1) * G] = lse
            flags |= f
    return o_part, lse_part, flags


# --------------------------------------------------------------------- merge
def merge(o_list, lse_list):
    """Log-sum-exp combination of partials (Section 3.2, step 4):
      M = max_r lse_r,  w_r = e^{lse_r - M},
      o = sum_r w_r o_r / sum_r w_r,  lse = M + ln sum_r w_r.
    o_list [R, ..., d], lse_list [R, ...]; no partials or all lse = -inf
    gives (0, -inf)."""
    o = np.asarray(o_list, np.float64)
    lse = np.asarray(lse_list, np.float64)
    if o.shape[0] == 0:
        return np.zeros(o.shape[1:]), np.full(lse.shape[1:], -np.inf)
    with np.errstate(invalid="ignore"):
        M = lse.max(axis=0)
        Ms = np.where(np.isneginf(M), 0.0, M)
        w = np.exp(lse - Ms)
        wsum = w.sum(axis=0)
        out = (w[..., None] * o).sum(axis=0) / np.where(wsum > 0, wsum, 1.0)[..., None]
        out = np.where((wsum > 0)[..., None] | np.isnan(wsum)[..., None], out, 0.0)
        lse_out = Ms + np.log(wsum)
    return out, lse_out


def merge_partials(o_part, lse_part, seq_route_begin):
    """Merged output per sequence: out [B, Hq, d], lse [B, Hq], flags.
    Routes of sequence b are rows seq_route_begin[b] .. seq_route_begin[b+1]-1;
    a malformed CSR row yields NaN with EFLAG_BAD_ROUTE."""
    srb = np.asarray(seq_route_begin, np.int64)
    B = len(srb) - 1
    R, Hq, d = o_part.shape
    out = np.zeros((B, Hq, d))
    lse = np.zeros((B, Hq))
    flags = 0
    for b in range(B):
        a, e = int(srb[b]), int(srb[b + 1])
        if not (0 <= a <= e <= R):
            out[b], lse[b] = np.nan, np.nan
            flags |= EFLAG_BAD_ROUTE
            continue
        out[b], lse[b] = merge(o_part[a:e], lse_part[a:e])
    return out, lse, flags


# -------------------------------------------------------------------- append
def kv_append(k_pool, v_pool, routes, page_ids, tail_route, k_new, v_new,
              k_scale=None, v_scale=None, inplace=False):
    """Tail append (Section 3.2, step 3; Section 5.1): each sequence b with a
    tail route r = tail_route[b] >= 0 stores its new K/V token (bf16 bits
    [B, Hkv, d]) at local index j = tok_end - tok_begin of route r and then
    extends the route by one token.  Works on copies (inplace=True: on the
    arrays given, which must then be writable numpy arrays of the storage
    dtypes -- for pools of many gigabytes); returns
    (k_pool, v_pool, routes, flags) for bf16 pools and
    (k_pool, v_pool, k_scale, v_scale, routes, flags) for E4M3 pools.  A full
    tail (no reserved page for j) or an inconsistent route leaves that
    sequence unchanged and sets a flag.

    E4M3 pools (no fp8 KV in the paper; the rule the kernels share), per page and KV
    head, separately for K and V, in float32 arithmetic:
      * the first token of a page sets scale = amax/28 (1 if amax = 0): its
        largest element lands at 28 = 448/16, leaving 16x headroom, which
        costs no precision (E4M3 keeps 3 mantissa bits in every normal binade);
      * a later token whose amax exceeds 448*scale first re-encodes the
        page's earlier slots to scale' = amax/28 (value = decode(code)*scale,
        code' = RNE(value/scale')), then the scale becomes scale';
      * the token is stored as RNE(x/scale), clamped to +-448."""
    fp8 = k_pool.dtype == np.uint8
    if inplace:
        for a in (k_pool, v_pool, routes) + ((k_scale, v_scale) if fp8 else ()):
            assert isinstance(a, np.ndarray) and a.flags.writeable
        assert routes.dtype == np.int32 and (not fp8 or k_scale.dtype == v_scale.dtype == np.float32)
    else:
        k_pool = k_pool.copy()
        v_pool = v_pool.copy()
        if fp8:
            k_scale = np.array(k_scale, dtype=np.float32, copy=True)
            v_scale = np.array(v_scale, dtype=np.float32, copy=True)
        routes = np.array(routes, dtype=np.int32, copy=True)
    R = len(routes)
    P = k_pool.shape[0]
    flags = 0
    for b, r in enumerate(np.asarray(tail_route)):
        r = int(r)
        if r < 0:
            continue
        if r >= R or int(routes[r, 0]) != b or routes[r, 3] < routes[r, 2]:
            flags |= EFLAG_BAD_ROUTE
            continue
        _, _, tb, te, base, cap = (int(x) for x in routes[r])
        j = te - tb
        if j // PAGE >= cap:
            flags |= EFLAG_TAIL_FULL
            continue
        if base < 0 or base + j // PAGE >= len(page_ids):
            flags |= EFLAG_BAD_ROUTE
            continue
        pid = int(page_ids[base + j // PAGE])
        if not 0 <= pid < P:
            flags |= EFLAG_BAD_PAGE
            continue
        slot = j % PAGE
        if fp8:
            for g in range(k_pool.shape[1]):
                _append_e4m3(k_pool[pid, g], k_scale, pid, g, slot, k_new[b, g], kmajor=True)
                _append_e4m3(v_pool[pid, g], v_scale, pid, g, slot, v_new[b, g], kmajor=False)
        else:
            k_pool[pid, :, slot, :] = k_new[b]
            v_pool[pid, :, :, slot] = v_new[b]
        routes[r, 3] = te + 1
    if fp8:
        return k_pool, v_pool, k_scale, v_scale, routes, flags
    return k_pool, v_pool, routes, flags


def _append_e4m3(page, scales, pid, g, slot, x_bits, kmajor):
    """One (page, KV head) of an E4M3 pool: page is [16, d] (K) or [d, 16] (V)."""
    f32 = np.float32
    x = (np.asarray(x_bits, np.uint16).astype(np.uint32) << 16).view(np.float32)
    amax = f32(np.max(np.abs(x)))
    if slot == 0:
        scale = f32(amax / f32(28.0)) if amax > 0 else f32(1.0)
    else:
        scale = f32(scales[pid, g])
        if amax > f32(f32(448.0) * scale):
            new = f32(amax / f32(28.0))
            old = page[:slot, :] if kmajor else page[:, :slot]
            vals = (e4m3_to_f64(old).astype(np.float32) * scale).astype(np.float32)
            recoded = e4m3_encode_rne((vals / new).astype(np.float32))
            if kmajor:
                page[:slot, :] = recoded
            else:
                page[:, :slot] = recoded
            scale = new
    scales[pid, g] = scale
    codes = e4m3_encode_rne((x / scale).astype(np.float32))
    if kmajor:
        page[slot, :] = codes
    else:
        page[:, slot] = codes


# --------------------------------------------------------------------- bytes
def kv_footprint_bytes(seq_lens, num_kv_heads, head_dim, num_layers=1, elem_bytes=2):
    """KV footprint of a batch (Section 4.2, post-prefill initialisation):
    C_total = sum_i 2 * s_i * H_kv * d_h * L * elem_bytes."""
    return int(sum(2 * int(s) * num_kv_heads * head_dim * num_layers * elem_bytes
                   for s in seq_lens))
