"""Device-resident decode state of one attention layer on one GPU.

Holds the query batch, the paged K/V pools, the routing table (token-range
routes and page ids) and the output buffers as torch device tensors, and runs
one decode step as the paper orders it (Section 3.2, steps 3-4; Section 5.1):
the tail routes append the step's K/V token, every route computes its partial,
and the partials of each sequence are merged.  Marshalling only: the three
calls are the library's HIP kernels, enqueued on the current stream.  Their
arguments are checked and marshalled once, when the state is built.
"""
from __future__ import annotations

import numpy as np
import torch

from . import kf


def _to_dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(a)
    return t.to(device, non_blocking=False)


class DecodeState:
    """Buffers for one layer's decode step.

    Arrays follow include/kf.h: q uint16 (bf16 bits) [B, Hq, 128]; pools
    uint16 or uint8 (E4M3 codes) [P, Hkv, 16, 128] / [P, Hkv, 128, 16];
    scales float32 [P, Hkv] or None; routes int32 [R, 6]; page_ids int32;
    seq_route_begin int32 [B+1]; tail_route int32 [B].  kv_layout =
    kf.KV_HEAD_MAJOR stores the (page-major) pools given here head-major on
    the device: [Hkv, P, ...].

    The calls are bound to the device tensors built here (kf.BoundCall):
    write into them between steps; replacing one raises AttributeError.
    """

    _BOUND = frozenset(("q", "k_pool", "v_pool", "k_scale", "v_scale", "routes", "page_ids",
                        "seq_route_begin", "tail_route", "workspace", "o_part", "lse_part", "out",
                        "lse", "err_flags", "shape", "max_pages_per_route"))

    def __init__(self, *, q, k_pool, v_pool, routes, page_ids, seq_route_begin, tail_route,
                 scale, max_pages_per_route, k_scale=None, v_scale=None, device="cuda",
                 kv_layout=None):
        self.device = torch.device(device)
        self.kv_layout = kf.KV_PAGE_MAJOR if kv_layout is None else kv_layout
        relayout = ((lambda x: np.ascontiguousarray(np.swapaxes(x, 0, 1)))
                    if self.kv_layout == kf.KV_HEAD_MAJOR else (lambda x: x))
        self.q = _to_dev(q, device)
        self.k_pool = _to_dev(relayout(k_pool), device)
        self.v_pool = _to_dev(relayout(v_pool), device)
        self.k_scale = None if k_scale is None else _to_dev(np.asarray(k_scale, np.float32), device)
        self.v_scale = None if v_scale is None else _to_dev(np.asarray(v_scale, np.float32), device)
        self.routes = _to_dev(np.asarray(routes, np.int32).reshape(-1, 6), device)
        self.page_ids = _to_dev(np.asarray(page_ids, np.int32), device)
        self.seq_route_begin = _to_dev(np.asarray(seq_route_begin, np.int32), device)
        self.tail_route = _to_dev(np.asarray(tail_route, np.int32), device)
        self.max_pages_per_route = int(max_pages_per_route)
        B, Hq, D = self.q.shape
        R = self.routes.shape[0]
        self.num_seqs = B
        self.shape = kf.shape_of(self.q, self.k_pool, self.page_ids, scale, self.kv_layout)
        # sized for any launch over at most R routes (the query-first schedule
        # launches over subsets, which may split their units), so it can be
        # larger than a launch over the whole table needs
        self.workspace = kf.alloc_workspace(self.shape, R, self.max_pages_per_route, device)
        self.o_part = torch.empty((R, Hq, D), dtype=torch.float32, device=device)
        self.lse_part = torch.empty((R, Hq), dtype=torch.float32, device=device)
        self.out = torch.empty((B, Hq, D), dtype=torch.float32, device=device)
        self.lse = torch.empty((B, Hq), dtype=torch.float32, device=device)
        self.err_flags = torch.zeros(1, dtype=torch.int32, device=device)
        self._append = kf.bind_kv_append(self.shape, self.k_pool, self.v_pool, self.routes,
                                         self.tail_route, self.page_ids, self.err_flags,
                                         self.k_scale, self.v_scale)
        self._partial = kf.bind_partial_attn(self.shape, self.q, self.k_pool, self.v_pool,
                                             self.routes, self.max_pages_per_route,
                                             self.page_ids, self.o_part, self.lse_part,
                                             self.workspace, self.err_flags, self.k_scale,
                                             self.v_scale)
        self._merge = kf.bind_merge_partials(self.num_seqs, self.o_part, self.lse_part,
                                             self.seq_route_begin, self.out, self.lse,
                                             self.err_flags)
        self._fused = self._bind_fused(self.workspace)
        self._no_alloc = None
        self._frozen = True

    def __setattr__(self, name, value):
        if name in self._BOUND and self.__dict__.get("_frozen"):
            raise AttributeError(f"DecodeState.{name} is bound into the marshalled calls: "
                                 "write into the tensor instead of replacing it")
        object.__setattr__(self, name, value)

    def _bind_fused(self, workspace):
        return kf.bind_decode_step(self.shape, self.q, self.k_pool, self.v_pool, self.routes,
                                   self.tail_route, self.max_pages_per_route, self.page_ids,
                                   self.seq_route_begin, self.o_part, self.lse_part, self.out,
                                   self.lse, workspace, self.err_flags, self.k_scale,
                                   self.v_scale)

    @classmethod
    def from_instance(cls, inst, device="cuda", kv_layout=None):
        """Upload a kf_workloads.Instance (duck-typed)."""
        return cls(q=inst.q, k_pool=inst.k_pool, v_pool=inst.v_pool, routes=inst.routes,
                   page_ids=inst.page_ids, seq_route_begin=inst.seq_route_begin,
                   tail_route=inst.tail_route, scale=inst.scale,
                   max_pages_per_route=inst.max_pages_per_route,
                   k_scale=inst.k_scale, v_scale=inst.v_scale, device=device,
                   kv_layout=kv_layout)

    def upload_new_tokens(self, k_new: np.ndarray, v_new: np.ndarray):
        return _to_dev(k_new, self.device), _to_dev(v_new, self.device)

    # ---------------------------------------------------------------- calls
    def append(self, k_new: torch.Tensor, v_new: torch.Tensor, stream=None):
        self._append(k_new, v_new, stream)

    def partial(self, stream=None):
        self._partial(stream)

    def merge(self, stream=None):
        self._merge(stream)

    def step(self, k_new: torch.Tensor | None = None, v_new: torch.Tensor | None = None,
             stream=None):
        """One decode step: append (if new tokens are given) -> partial -> merge."""
        if k_new is not None:
            self.append(k_new, v_new, stream)
        self.partial(stream)
        self.merge(stream)

    def step_fused(self, k_new: torch.Tensor, v_new: torch.Tensor, stream=None):
        """One decode step through kf_decode_step: same results as step(),
        with the append fused into the partial-attention launch."""
        self._fused(k_new, v_new, stream)

    def step_no_alloc(self, k_new: torch.Tensor, v_new: torch.Tensor, stream=None):
        """step_fused through kf_decode_step_no_alloc: the library's
        per-device scratch array instead of this state's workspace."""
        if self._no_alloc is None:
            self._no_alloc = self._bind_fused(None)
        self._no_alloc(k_new, v_new, stream)

    # ----------------------------------------------------- query-first step
    def setup_query_first(self):
        """Split the routes into historical ones and the tails (read from the
        device tail table; call again after editing it) for step_query_first."""
        tails = self.tail_route.cpu().numpy()
        tails = np.unique(tails[tails >= 0]).astype(np.int32)
        R = self.routes.shape[0]
        hist = np.setdiff1d(np.arange(R, dtype=np.int32), tails).astype(np.int32)
        self.hist_rows, self.tail_rows = hist, tails
        self.hist_list = _to_dev(hist, self.device)
        self.tail_list = _to_dev(tails, self.device)
        self.ws_hist = kf.alloc_workspace(self.shape, R, self.max_pages_per_route, self.device)
        self.ws_tail = kf.alloc_workspace(self.shape, R, self.max_pages_per_route, self.device)
        self.stream_b = torch.cuda.Stream(device=self.device)   # default priority
        self._qf_hist, self._qf_tail = (
            kf.bind_partial_attn(self.shape, self.q, self.k_pool, self.v_pool, self.routes,
                                 self.max_pages_per_route, self.page_ids, self.o_part,
                                 self.lse_part, ws, self.err_flags, self.k_scale, self.v_scale,
                                 route_list=lst)
            for ws, lst in ((self.ws_hist, self.hist_list), (self.ws_tail, self.tail_list)))
        self._qf_ready = torch.cuda.Event()
        self._qf_tail_done = torch.cuda.Event()

    def step_query_first(self, k_new: torch.Tensor, v_new: torch.Tensor, hist_events=None):
        """One decode step scheduled query-first (Section 5.1): partials of the
        historical routes start on the current stream from q alone; on a second
        stream the tails append the new K/V token and then attend; the merge
        waits for both.  Same kernels as step(), other order.  hist_events:
        two timing events recorded on the current stream around the launch
        over the historical routes."""
        cur = torch.cuda.current_stream(self.device)
        self._qf_ready.record(cur)
        self.stream_b.wait_event(self._qf_ready)
        if hist_events is not None:
            hist_events[0].record(cur)
        if self.hist_list.numel():
            self._qf_hist(cur)
        if hist_events is not None:
            hist_events[1].record(cur)
        self.append(k_new, v_new, self.stream_b)
        if self.tail_list.numel():
            self._qf_tail(self.stream_b)
        self._qf_tail_done.record(self.stream_b)
        cur.wait_event(self._qf_tail_done)
        self.merge(cur)

    def flags(self) -> int:
        return int(self.err_flags.item())
