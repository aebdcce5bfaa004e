"""Seeded synthetic inputs for decode attention over token-range KV partitions.

Shapes follow the head configurations the paper evaluates (Q32:KV8 and
Q64:KV8, Section 6.3) at head dimension 128.  Every tensor is drawn from its
own numpy PCG64 stream keyed by ``(seed, workload id, tensor id, sequence,
block)`` so that any part of any instance can be regenerated on its own and
the result does not depend on thread scheduling or on how a sequence is cut
into routes.

Layouts written here are the boundary's storage formats (16-token pages,
head_dim 128):

* K pool  ``[page][kv_head][slot 0..15][d 0..127]``
* V pool  ``[page][kv_head][d 0..127][slot 0..15]``  (dimension-major page)
* fp8 scales ``[page][kv_head]`` float32, real value = decode(code) * scale
* route row ``(seq, part, tok_begin, tok_end, page_base, page_cap)`` int32;
  token ``t`` of a route sits in page ``page_ids[page_base + (t-tok_begin)//16]``
  at slot ``(t-tok_begin) % 16``.

Unused slots of every page are filled with NaN bit patterns so that a reader
that touches them shows it.  A contiguous pool hands out pages in pairs (each
route starts on an even page id); a permuted pool is one random permutation.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

PAGE = 16
HEAD_DIM = 128
BLOCK_TOKENS = 2048          # tokens per independent random stream

BF16_NAN = 0x7FC0
E4M3_NAN = 0x7F

# tensor ids of the random streams
_T_Q, _T_K, _T_V, _T_KNEW, _T_VNEW, _T_BIAS, _T_LENS, _T_PERM = range(1, 9)


@dataclass(frozen=True)
class Workload:
    """A synthetic decode batch for one attention layer."""
    name: str
    wid: int                      # workload id, part of every stream key
    num_seqs: int
    num_q_heads: int
    num_kv_heads: int
    part_tokens: int              # tokens per route when the routes are laid out
    ctx: int | None = None        # resident tokens per sequence (fixed) ...
    ctx_range: tuple | None = None  # ... or log-uniform in [lo, hi]
    kv_dtype: str = "bf16"        # "bf16" or "fp8" (OCP E4M3FN + per-page scales)
    permuted: bool = False        # page table randomly permuted over one pool
    appends: int = 0              # new K/V tokens per sequence per step
    bias_frac: float = 0.0        # fraction of keys given a score offset
    bias: float = 0.0             # the score offset
    head_dim: int = HEAD_DIM
    page_size: int = PAGE

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # 1 sequence, 8 query / 2 KV heads, 4096 tokens in 2 routes of 2048
    "tiny": Workload("tiny", 1, num_seqs=1, num_q_heads=8, num_kv_heads=2,
                     part_tokens=2048, ctx=4096),
    # Llama-3.1-8B layer: 16 x 32768 tokens, 4 routes of 8192, 1 append per step
    "llama8b_32k": Workload("llama8b_32k", 2, num_seqs=16, num_q_heads=32,
                            num_kv_heads=8, part_tokens=8192, ctx=32768,
                            appends=1),
    # agentic mix: 64 sequences, log-uniform 2K..128K, routes of 16384,
    # permuted shared pool, 5% of keys with a +4.0 score offset, 1 append
    "agentic_mix": Workload("agentic_mix", 3, num_seqs=64, num_q_heads=32,
                            num_kv_heads=8, part_tokens=16384,
                            ctx_range=(2048, 131072), permuted=True, appends=1,
                            bias_frac=0.05, bias=4.0),
    # million-token context: 4 x 1048576 tokens, 16 routes of 65536
    "million_ctx": Workload("million_ctx", 4, num_seqs=4, num_q_heads=32,
                            num_kv_heads=8, part_tokens=65536, ctx=1048576),
    # 70B-like wide GQA (64/8) with fp8 E4M3 KV: 32 x 65536, routes of 16384
    "wide_gqa_fp8": Workload("wide_gqa_fp8", 5, num_seqs=32, num_q_heads=64,
                             num_kv_heads=8, part_tokens=16384, ctx=65536,
                             kv_dtype="fp8"),
    # the same layer run as decode steps: 1 appended token per sequence per
    # step into the fp8 tails (same streams, so the same resident tokens)
    "wide_gqa_fp8_decode": Workload("wide_gqa_fp8_decode", 5, num_seqs=32, num_q_heads=64,
                                    num_kv_heads=8, part_tokens=16384, ctx=65536,
                                    kv_dtype="fp8", appends=1),
}


def workload(name: str, **overrides) -> Workload:
    wl = WORKLOADS[name]
    return wl.replace(**overrides) if overrides else wl


# ----------------------------------------------------------------- encodings
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 bits, nearest-even (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = b >> 16
    t &= 1
    t += b
    t += 0x7FFF
    t >>= 16
    return t.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """float32 -> OCP E4M3FN codes, nearest-even (|x| <= 448 expected)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()


def _rng(*key) -> np.random.Generator:
    return np.random.default_rng([int(k) for k in key])


# ------------------------------------------------------------------ instance
@dataclass
class Instance:
    wl: Workload
    seed: int
    seq_lens: np.ndarray          # int64 [B] resident tokens before step 0
    q: np.ndarray                 # uint16 [B, Hq, D] bf16 bits
    k_pool: np.ndarray            # uint16|uint8 [P, Hkv, 16, D]
    v_pool: np.ndarray            # uint16|uint8 [P, Hkv, D, 16]
    k_scale: np.ndarray | None    # float32 [P, Hkv] (fp8 only)
    v_scale: np.ndarray | None
    routes: np.ndarray            # int32 [R, 6]
    page_ids: np.ndarray          # int32 [NP]
    seq_route_begin: np.ndarray   # int32 [B+1]
    tail_route: np.ndarray        # int32 [B]  (-1: no append target)
    scale: float                  # softmax scale 1/sqrt(d)
    bias_dirs: dict               # (seq, kv_head) -> float64 [D] key shift (if any)

    @property
    def num_pages(self) -> int:
        return int(self.k_pool.shape[0])

    @property
    def max_pages_per_route(self) -> int:
        return int(self.routes[:, 5].max()) if len(self.routes) else 0

    def new_tokens(self, step: int):
        """bf16 bits of the K/V token each sequence appends at ``step``."""
        wl = self.wl
        shp = (wl.num_seqs, wl.num_kv_heads, wl.head_dim)
        k = _rng(self.seed, wl.wid, _T_KNEW, step).standard_normal(shp, dtype=np.float32)
        v = _rng(self.seed, wl.wid, _T_VNEW, step).standard_normal(shp, dtype=np.float32)
        return f32_to_bf16_bits(k), f32_to_bf16_bits(v)

    def logical_kv(self, seq: int, t0: int, t1: int):
        """bf16 bits of resident tokens [t0, t1) of ``seq``: (K, V) [n, Hkv, D].

        Drawn from the same streams that filled the pools (bf16 workloads)."""
        assert self.wl.kv_dtype == "bf16"
        ks, vs = [], []
        for blk in range(t0 // BLOCK_TOKENS, (t1 - 1) // BLOCK_TOKENS + 1):
            kb, vb = _draw_block(self, seq, blk)
            b0 = blk * BLOCK_TOKENS
            lo, hi = max(t0, b0) - b0, min(t1, b0 + len(kb)) - b0
            ks.append(f32_to_bf16_bits(kb[lo:hi]))
            vs.append(f32_to_bf16_bits(vb[lo:hi]))
        return np.concatenate(ks), np.concatenate(vs)


def _seq_lens(wl: Workload, seed: int) -> np.ndarray:
    if wl.ctx is not None:
        return np.full(wl.num_seqs, wl.ctx, dtype=np.int64)
    lo, hi = wl.ctx_range
    u = _rng(seed, wl.wid, _T_LENS).uniform(math.log(lo), math.log(hi), wl.num_seqs)
    return np.minimum(np.floor(np.exp(u)).astype(np.int64), hi)


def _draw_block(inst: Instance, seq: int, blk: int):
    """float32 K, V of tokens [blk*2048, ...) of ``seq`` (score offset applied)."""
    wl = inst.wl
    n = int(min(BLOCK_TOKENS, inst.seq_lens[seq] - blk * BLOCK_TOKENS))
    shp = (n, wl.num_kv_heads, wl.head_dim)
    k = _rng(inst.seed, wl.wid, _T_K, seq, blk).standard_normal(shp, dtype=np.float32)
    v = _rng(inst.seed, wl.wid, _T_V, seq, blk).standard_normal(shp, dtype=np.float32)
    if wl.bias_frac > 0:
        mask = _rng(inst.seed, wl.wid, _T_BIAS, seq, blk).random((n, wl.num_kv_heads)) < wl.bias_frac
        for g in range(wl.num_kv_heads):
            sel = np.nonzero(mask[:, g])[0]
            if len(sel):
                k[sel, g, :] = (k[sel, g, :].astype(np.float64)
                                + inst.bias_dirs[(seq, g)]).astype(np.float32)
    return k, v


def _bias_dirs(wl: Workload, q_bits: np.ndarray, scale: float) -> dict:
    """Minimum-norm key shift u_g with q_h . u_g = bias/scale for every query
    head h of KV group g, so that a shifted key's score rises by ``bias``."""
    if wl.bias_frac <= 0:
        return {}
    q = bf16_bits_to_f32(q_bits).astype(np.float64)
    G = wl.group
    out = {}
    for b in range(wl.num_seqs):
        for g in range(wl.num_kv_heads):
            Qg = q[b, g * G:(g + 1) * G, :]
            rhs = np.full(G, wl.bias / scale)
            out[(b, g)] = Qg.T @ np.linalg.solve(Qg @ Qg.T, rhs)
    return out


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def make_instance(wl: Workload, seed: int = 1, *, steps: int = 1,
                  seq_lens=None, empty_tail: bool = False, routing=None) -> Instance:
    """Build one seeded instance of ``wl``.

    ``steps``      appends the tail routes must hold room for (if wl.appends).
    ``seq_lens``   override of the resident lengths (int array [B]).
    ``empty_tail`` additionally open a fresh, empty tail route per sequence
                   (a route published at a token boundary, before its first
                   append).
    ``routing``    an explicit routing table (routes [R, 6], page_ids,
                   seq_route_begin [B+1], tail_route [B]) used verbatim
                   instead of routes of part_tokens; its resident ranges
                   must tile each sequence's [0, seq_lens[b]).
    """
    B, Hq, Hkv, D = wl.num_seqs, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    assert Hq % Hkv == 0 and wl.page_size == PAGE and D == HEAD_DIM
    scale = 1.0 / math.sqrt(D)
    lens = _seq_lens(wl, seed) if seq_lens is None else np.asarray(seq_lens, dtype=np.int64)
    q = f32_to_bf16_bits(
        np.stack([_rng(seed, wl.wid, _T_Q, b).standard_normal((Hq, D), dtype=np.float32)
                  for b in range(B)]))

    if routing is not None:
        routes = np.array(routing[0], dtype=np.int32).reshape(-1, 6)
        page_ids = np.array(routing[1], dtype=np.int32)
        srb = [int(x) for x in routing[2]]
        tails = [int(x) for x in routing[3]]
        P = max(int(page_ids.max()) + 1 if len(page_ids) else 1, 1)
    else:
        # ---- routes: contiguous token ranges of part_tokens; the last is the tail
        grow = steps * wl.appends
        rows, srb, tails = [], [0], []
        for b in range(B):
            n = int(lens[b])
            starts = list(range(0, n, wl.part_tokens)) or [0]
            ends = [min(s + wl.part_tokens, n) for s in starts]
            if empty_tail:
                starts.append(n)
                ends.append(n)
            for k, (s, e) in enumerate(zip(starts, ends)):
                last = k == len(starts) - 1
                cap = -(-((e - s) + (grow if last else 0)) // PAGE)
                rows.append([b, k, s, e, 0, cap])
            tails.append(len(rows) - 1 if wl.appends or empty_tail else -1)
            srb.append(len(rows))
        routes = np.array(rows, dtype=np.int32).reshape(-1, 6)
        caps = routes[:, 5].astype(np.int64)
        total = int(caps.sum())
        routes[:, 4] = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int32)
        if wl.permuted:
            page_ids = _rng(seed, wl.wid, _T_PERM).permutation(total).astype(np.int32)
            P = max(total, 1)
        else:
            # contiguous pool, pages handed out in pairs (64 KiB of bf16 K per
            # pair at 8 KV heads): each route's pages start on an even page id,
            # a route reserving an odd count leaves one unused page behind it
            even = caps + (caps & 1)
            first = np.concatenate([[0], np.cumsum(even)[:-1]])
            page_ids = np.concatenate(
                [first[r] + np.arange(caps[r]) for r in range(len(caps))]
            ).astype(np.int32) if len(caps) else np.zeros(0, np.int32)
            P = max(int(even.sum()), 1)

    fp8 = wl.kv_dtype == "fp8"
    edt = np.uint8 if fp8 else np.uint16
    nan = E4M3_NAN if fp8 else BF16_NAN
    k_pool = np.full((P, Hkv, PAGE, D), nan, dtype=edt)
    v_pool = np.full((P, Hkv, D, PAGE), nan, dtype=edt)
    k_scale = np.ones((P, Hkv), np.float32) if fp8 else None
    v_scale = np.ones((P, Hkv), np.float32) if fp8 else None

    inst = Instance(wl, seed, lens, q, k_pool, v_pool, k_scale, v_scale, routes,
                    page_ids, np.array(srb, np.int32), np.array(tails, np.int32),
                    scale, _bias_dirs(wl, q, scale))

    # ---- token -> (page id, slot) for each sequence, from its routes
    jobs = []
    for b in range(B):
        n = int(lens[b])
        if n == 0:
            continue
        pid = np.empty(n, np.int64)
        slot = np.empty(n, np.int64)
        for r in range(srb[b], srb[b + 1]):
            _, _, s, e, base, _ = (int(x) for x in routes[r])
            j = np.arange(e - s)
            pid[s:e] = page_ids[base + j // PAGE]
            slot[s:e] = j % PAGE
        for blk in range(-(-n // BLOCK_TOKENS)):
            jobs.append((b, blk, pid, slot))

    def fill(job):
        b, blk, pid, slot = job
        kf, vf = _draw_block(inst, b, blk)
        t0 = blk * BLOCK_TOKENS
        p = pid[t0:t0 + len(kf)]
        s = slot[t0:t0 + len(kf)]
        if np.array_equal(s, np.arange(len(s)) % PAGE):
            _fill_pages(inst, p[::PAGE], kf, vf)
        else:
            assert not fp8, "fp8 pools need 16-aligned route starts"
            k_pool[p, :, s, :] = f32_to_bf16_bits(kf)
            v_pool[p, :, :, s] = f32_to_bf16_bits(vf)

    if len(jobs) > 1:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(fill, jobs))
    else:
        for j in jobs:
            fill(j)
    return inst


def _fill_pages(inst: Instance, pages, kf, vf):
    """Write whole pages: tokens arrive in page order, 16 per page, the last
    page possibly partial.  fp8 pools get one scale per (page, kv head): the
    page's absolute maximum over its resident tokens maps to 448."""
    n = len(kf)
    npg = len(pages)
    pad = npg * PAGE - n
    fp8 = inst.wl.kv_dtype == "fp8"
    for src, pool, sc, kmaj in ((kf, inst.k_pool, inst.k_scale, True),
                                (vf, inst.v_pool, inst.v_scale, False)):
        x = src
        if pad:
            x = np.concatenate([x, np.zeros((pad,) + x.shape[1:], np.float32)])
        x = x.reshape(npg, PAGE, x.shape[1], x.shape[2])          # [pg, slot, Hkv, D]
        if fp8:
            amax = np.abs(x).max(axis=(1, 3))                        # [pg, Hkv]
            scl = np.where(amax > 0, amax / np.float32(448.0),
                           np.float32(1.0)).astype(np.float32)
            codes = e4m3_encode(x / scl[:, None, :, None])
            sc[pages] = scl
            fill_val = E4M3_NAN
        else:
            codes = f32_to_bf16_bits(x)
            fill_val = BF16_NAN
        if pad:
            codes[-1, PAGE - pad:] = fill_val
        if kmaj:
            pool[pages] = codes.transpose(0, 2, 1, 3)
        else:
            pool[pages] = codes.transpose(0, 2, 3, 1)
