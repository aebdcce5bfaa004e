"""Thin ctypes binding of libkf.so (include/kf.h) for torch device tensors.

Argument marshalling only: every step runs in the library's HIP kernels on
the current torch stream.  Importing works without a GPU; calling an entry
point without the built library raises ``KFError``.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkf.so")

PAGE_SIZE = 16
HEAD_DIM = 128
MAX_GROUP = 16

KV_BF16 = 0
KV_FP8_E4M3 = 1

ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_WORKSPACE = -3
ERR_HIP = -4
ERR_CAPACITY = -5
ERR_INFEASIBLE = -6
ERR_HOST_MEMORY = -7
ERR_SCRATCH_LIMIT = -8
SCRATCH_BYTES = 32 << 20   # KF_SCRATCH_BYTES

EFLAG_TAIL_FULL = 1
EFLAG_BAD_ROUTE = 2
EFLAG_BAD_PAGE = 4
KV_PAGE_MAJOR = 0
KV_HEAD_MAJOR = 1

# every symbol include/kf.h declares
EXPORTS = ("kf_kv_append", "kf_partial_attn_workspace_bytes", "kf_partial_attn_plan",
           "kf_partial_attn", "kf_partial_attn_subset", "kf_merge_partials", "kf_decode_step",
           "kf_decode_step_no_alloc", "kf_debug_gather", "kf_status_str", "kf_version")


class KFError(RuntimeError):
    pass


class Route(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("seq", "part", "tok_begin", "tok_end", "page_base", "page_cap")]


class Shape(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("kv_dtype", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("num_page_ids", ctypes.c_int32),
                ("scale", ctypes.c_float), ("kv_layout", ctypes.c_int32)]


_lib = None


def load(path: str | None = None) -> ctypes.CDLL:
    """Load libkf.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or _LIB_PATH
    if not os.path.exists(path):
        raise KFError(f"{path} is missing: build it with `python -m paper_2606_29207_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sp = ctypes.POINTER(Shape)
    lib.kf_kv_append.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp]
    lib.kf_kv_append.restype = ctypes.c_int
    lib.kf_partial_attn_workspace_bytes.argtypes = [sp, i32, i32]
    lib.kf_partial_attn_workspace_bytes.restype = sz
    lib.kf_partial_attn_plan.argtypes = [sp, i32, i32, i32, vp, vp, vp]
    lib.kf_partial_attn_plan.restype = ctypes.c_int
    lib.kf_partial_attn.argtypes = [sp, vp, vp, vp, vp, vp, vp, i32, i32, vp, vp, vp, vp, sz, vp, vp]
    lib.kf_partial_attn.restype = ctypes.c_int
    lib.kf_partial_attn_subset.argtypes = [sp, vp, vp, vp, vp, vp, vp, i32, vp, i32, i32, vp, vp, vp,
                                           vp, sz, vp, vp]
    lib.kf_partial_attn_subset.restype = ctypes.c_int
    lib.kf_merge_partials.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.kf_merge_partials.restype = ctypes.c_int
    lib.kf_decode_step.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp, i32, vp, vp, vp, vp,
                                   vp, vp, vp, sz, vp, vp]
    lib.kf_decode_step.restype = ctypes.c_int
    lib.kf_decode_step_no_alloc.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp, i32, vp,
                                            vp, vp, vp, vp, vp, vp, vp]
    lib.kf_decode_step_no_alloc.restype = ctypes.c_int
    lib.kf_debug_gather.argtypes = [sp, vp, vp, vp, i32, i32, i32, vp, i32, vp, vp, vp, vp]
    lib.kf_debug_gather.restype = ctypes.c_int
    lib.kf_status_str.argtypes = [ctypes.c_int]
    lib.kf_status_str.restype = ctypes.c_char_p
    lib.kf_version.argtypes = []
    lib.kf_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().kf_status_str(status).decode()


def version() -> str:
    return load().kf_version().decode()


def _check(status: int, what: str):
    if status != 0:
        raise KFError(f"{what}: {status_str(status)} ({status})")


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


# the current stream's raw handle without building a torch.cuda.Stream object
# (a few microseconds per call through the public API)
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_cur_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(stream):
    """hipStream_t of `stream` (a torch stream), or of the current torch
    stream when None, as an integer for a c_void_p argument."""
    if stream is not None:
        return stream.cuda_stream
    if _raw_stream is not None and _cur_device is not None:
        return _raw_stream(_cur_device())
    return torch.cuda.current_stream().cuda_stream


def _dev(t: torch.Tensor, name: str, dtype=None):
    if not t.is_cuda:
        raise KFError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise KFError(f"{name} must be contiguous")
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise KFError(f"{name} has dtype {t.dtype}, expected {dtype}")
    return t


def _need(cond, msg):
    if not cond:
        raise KFError(msg)


def _check_tables(shape: Shape, k_pool, v_pool, routes, page_ids):
    """Sizes the C ABI cannot see: pools, route rows and page ids."""
    P, H = shape.num_pages, shape.num_kv_heads
    esz = 1 if shape.kv_dtype == KV_FP8_E4M3 else 2
    for t, n in ((k_pool, "k_pool"), (v_pool, "v_pool")):
        _need(t.element_size() == esz and t.numel() == P * H * PAGE_SIZE * HEAD_DIM,
              f"{n} must hold [num_pages, num_kv_heads, 16, 128] elements of the pool dtype")
    _need(routes.dtype == torch.int32 and routes.dim() == 2 and routes.shape[1] == 6,
          "routes must be int32 [R, 6]")
    _need(page_ids.dtype == torch.int32 and page_ids.numel() == shape.num_page_ids,
          "page_ids must be int32 [num_page_ids]")
    _need(shape.num_seqs >= 0, "bad shape")


def make_shape(num_seqs, num_q_heads, num_kv_heads, kv_dtype, num_pages, num_page_ids,
               scale, kv_layout=None) -> Shape:
    return Shape(num_seqs, num_q_heads, num_kv_heads, HEAD_DIM, PAGE_SIZE, kv_dtype,
                 num_pages, num_page_ids, float(scale),
                 KV_PAGE_MAJOR if kv_layout is None else kv_layout)


def _pool_dtype(k_pool: torch.Tensor) -> int:
    return KV_FP8_E4M3 if k_pool.element_size() == 1 else KV_BF16


def shape_of(q, k_pool, page_ids, scale, kv_layout=None) -> Shape:
    """kf_shape from q [B, Hq, 128], the K pool ([P, Hkv, 16, 128] page-major,
    [Hkv, P, 16, 128] head-major) and page_ids."""
    head_major = kv_layout == KV_HEAD_MAJOR
    P, H = (k_pool.shape[1], k_pool.shape[0]) if head_major else (k_pool.shape[0], k_pool.shape[1])
    return make_shape(q.shape[0], q.shape[1], H, _pool_dtype(k_pool), P, page_ids.numel(), scale,
                      kv_layout)


class BoundCall:
    """An entry point with its arguments checked and marshalled once.

    Calling it issues the C call again with the same device pointers, on
    ``stream`` (the current torch stream when None).  It holds a reference
    to every tensor it was bound to, so those pointers stay valid while the
    object lives: writes into the tensors between calls are seen; a tensor
    replaced elsewhere (or resized in place) is not.  The current device
    must stay the tensors' device, and a given stream must belong to it.  A
    per-step decode loop pays the argument checks once instead of on every
    step (tens of microseconds of host time against a few microseconds of
    kernel time for small batches)."""

    __slots__ = ("_fn", "_what", "_args", "_keep", "_dev")

    def __init__(self, fn, what: str, args, keep, device: int | None = None):
        self._fn, self._what, self._args, self._keep = fn, what, tuple(args), tuple(keep)
        self._dev = device

    def _handle(self, stream):
        if self._dev is not None:
            cur = _cur_device() if _cur_device is not None else torch.cuda.current_device()
            if cur != self._dev or (stream is not None and stream.device_index != self._dev):
                raise KFError(f"{self._what}: bound to cuda:{self._dev}, called with the current "
                              f"device cuda:{cur}" + ("" if stream is None else
                                                      f" and a stream of cuda:{stream.device_index}"))
            if stream is None and _raw_stream is not None:
                return _raw_stream(cur)
        return _stream(stream)

    def __call__(self, stream=None):
        st = self._fn(*self._args, self._handle(stream))
        if st != 0:
            _check(st, self._what)


class BoundTokenCall(BoundCall):
    """A BoundCall whose entry point also takes the step's new token: k_new
    and v_new (bf16 device tensors [num_seqs, num_kv_heads, 128]) are given
    per call and checked against the bound shape."""

    __slots__ = ("_tok_at", "_tok_shape")

    def __init__(self, fn, what: str, args, keep, tok_at: int, tok_shape, device=None):
        super().__init__(fn, what, args, keep, device)
        self._tok_at, self._tok_shape = tok_at, torch.Size(tok_shape)

    def __call__(self, k_new, v_new, stream=None):
        for t, n in ((k_new, "k_new"), (v_new, "v_new")):
            if not (isinstance(t, torch.Tensor) and t.is_cuda and t.shape == self._tok_shape
                    and t.element_size() == 2 and t.is_contiguous()):
                raise KFError(f"{n} must be a contiguous bf16 device tensor "
                              f"{list(self._tok_shape)}")
        i, a = self._tok_at, self._args
        st = self._fn(*a[:i], k_new.data_ptr(), v_new.data_ptr(), *a[i:], self._handle(stream))
        if st != 0:
            _check(st, self._what)


def _copy_shape(shape: Shape) -> Shape:
    return Shape.from_buffer_copy(shape)


def _check_scales(shape: Shape, k_scale, v_scale):
    if shape.kv_dtype == KV_FP8_E4M3:
        for t, n in ((k_scale, "k_scale"), (v_scale, "v_scale")):
            _need(t is not None, f"{n} is required for fp8 pools")
            _dev(t, n)
            _need(t.dtype == torch.float32 and t.numel() >= shape.num_pages * shape.num_kv_heads,
                  f"{n} must be float32 [num_pages, num_kv_heads]")


def _check_tokens(shape: Shape, k_new, v_new):
    _dev(k_new, "k_new")
    _dev(v_new, "v_new")
    B, H = shape.num_seqs, shape.num_kv_heads
    _need(tuple(k_new.shape) == (B, H, HEAD_DIM) and tuple(v_new.shape) == (B, H, HEAD_DIM),
          "k_new/v_new must be [num_seqs, num_kv_heads, 128]")
    _need(k_new.element_size() == 2 and v_new.element_size() == 2, "k_new/v_new must be bf16")


def bind_kv_append(shape: Shape, k_pool, v_pool, routes, tail_route, page_ids, err_flags,
                   k_scale=None, v_scale=None) -> BoundTokenCall:
    """kf_kv_append bound to its tables; call it as (k_new, v_new, stream)."""
    lib = load()
    for t, n in ((k_pool, "k_pool"), (v_pool, "v_pool"), (routes, "routes"),
                 (tail_route, "tail_route"), (page_ids, "page_ids"), (err_flags, "err_flags")):
        _dev(t, n)
    B, H = shape.num_seqs, shape.num_kv_heads
    _need(tail_route.numel() >= B and tail_route.dtype == torch.int32, "tail_route: int32 [num_seqs]")
    _check_tables(shape, k_pool, v_pool, routes, page_ids)
    _check_scales(shape, k_scale, v_scale)
    sh = _copy_shape(shape)
    args = (ctypes.byref(sh), _ptr(k_pool), _ptr(v_pool), _ptr(k_scale), _ptr(v_scale),
            _ptr(routes), routes.shape[0], _ptr(tail_route), _ptr(page_ids), _ptr(err_flags))
    return BoundTokenCall(lib.kf_kv_append, "kf_kv_append", args,
                          (sh, k_pool, v_pool, k_scale, v_scale, routes, tail_route, page_ids,
                           err_flags), 5, (B, H, HEAD_DIM), k_pool.device.index)


def kv_append(shape: Shape, k_pool, v_pool, k_new, v_new, routes, tail_route, page_ids,
              err_flags, stream=None, k_scale=None, v_scale=None):
    """kf_kv_append.  routes: int32 [R, 6] (updated in place); fp8 pools also
    take (and update) k_scale/v_scale float32 [P, Hkv]."""
    _check_tokens(shape, k_new, v_new)
    bind_kv_append(shape, k_pool, v_pool, routes, tail_route, page_ids, err_flags,
                   k_scale, v_scale)(k_new, v_new, stream)


def partial_attn_workspace_bytes(shape: Shape, num_routes: int, max_pages_per_route: int) -> int:
    return int(load().kf_partial_attn_workspace_bytes(ctypes.byref(shape), num_routes,
                                                       max_pages_per_route))


def partial_attn_plan(shape: Shape, num_launch: int, max_pages_per_route: int,
                      route_list: bool = False) -> tuple[int, int, int]:
    """kf_partial_attn_plan: (chunk_pages, max_chunks, units_per_wg) of a
    launch of num_launch routes (route_list: a kf_partial_attn_subset launch)."""
    out = [ctypes.c_int32(0) for _ in range(3)]
    st = load().kf_partial_attn_plan(ctypes.byref(shape), int(num_launch), int(max_pages_per_route),
                                     1 if route_list else 0, *[ctypes.byref(o) for o in out])
    _check(st, "kf_partial_attn_plan")
    return tuple(int(o.value) for o in out)


def alloc_workspace(shape: Shape, num_routes: int, max_pages_per_route: int, device="cuda"):
    n = partial_attn_workspace_bytes(shape, num_routes, max_pages_per_route)
    if n == 0:
        raise KFError("invalid workspace request")
    return torch.zeros(n, dtype=torch.uint8, device=device)


def bind_partial_attn(shape: Shape, q, k_pool, v_pool, routes, max_pages_per_route, page_ids,
                      o_part, lse_part, workspace, err_flags, k_scale=None, v_scale=None,
                      route_list=None) -> BoundCall:
    """kf_partial_attn (all routes) or, with ``route_list`` (int32 device
    tensor of route indices), kf_partial_attn_subset, bound to its buffers;
    call it as (stream).  o_part float32 [R, Hq, 128], lse_part float32 [R, Hq]."""
    lib = load()
    for t, n in ((q, "q"), (k_pool, "k_pool"), (v_pool, "v_pool"), (routes, "routes"),
                 (page_ids, "page_ids"), (o_part, "o_part"), (lse_part, "lse_part"),
                 (workspace, "workspace"), (err_flags, "err_flags")):
        _dev(t, n)
    if o_part.dtype != torch.float32 or lse_part.dtype != torch.float32:
        raise KFError("o_part and lse_part must be float32")
    R = routes.shape[0]
    _need(tuple(q.shape) == (shape.num_seqs, shape.num_q_heads, HEAD_DIM) and q.element_size() == 2,
          "q must be bf16 [num_seqs, num_q_heads, 128]")
    _need(tuple(o_part.shape) == (R, shape.num_q_heads, HEAD_DIM), "o_part must be [R, Hq, 128]")
    _need(tuple(lse_part.shape) == (R, shape.num_q_heads), "lse_part must be [R, Hq]")
    _check_tables(shape, k_pool, v_pool, routes, page_ids)
    _check_scales(shape, k_scale, v_scale)
    sh = _copy_shape(shape)
    ws_bytes = workspace.numel() * workspace.element_size()
    head = (ctypes.byref(sh), _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(k_scale), _ptr(v_scale),
            _ptr(routes), R)
    tail = (int(max_pages_per_route), _ptr(page_ids), _ptr(o_part), _ptr(lse_part),
            _ptr(workspace), ws_bytes, _ptr(err_flags))
    keep = (sh, q, k_pool, v_pool, k_scale, v_scale, routes, page_ids, o_part, lse_part,
            workspace, err_flags)
    if route_list is None:
        return BoundCall(lib.kf_partial_attn, "kf_partial_attn", head + tail, keep, q.device.index)
    _dev(route_list, "route_list")
    _need(route_list.dtype == torch.int32 and route_list.dim() == 1, "route_list must be int32 [n]")
    return BoundCall(lib.kf_partial_attn_subset, "kf_partial_attn_subset",
                     head + (_ptr(route_list), route_list.numel()) + tail, keep + (route_list,),
                     q.device.index)


def partial_attn(shape: Shape, q, k_pool, v_pool, routes, max_pages_per_route, page_ids,
                 o_part, lse_part, workspace, err_flags, k_scale=None, v_scale=None,
                 stream=None, route_list=None):
    """kf_partial_attn (all routes) or, with ``route_list`` (int32 device
    tensor of route indices), kf_partial_attn_subset.
    o_part float32 [R, Hq, 128], lse_part float32 [R, Hq]."""
    bind_partial_attn(shape, q, k_pool, v_pool, routes, max_pages_per_route, page_ids, o_part,
                      lse_part, workspace, err_flags, k_scale, v_scale, route_list)(stream)


def bind_merge_partials(num_seqs, o_part, lse_part, seq_route_begin, out, lse_out,
                        err_flags) -> BoundCall:
    """kf_merge_partials bound to its buffers; call it as (stream).
    out float32 [B, Hq, 128], lse_out float32 [B, Hq]."""
    lib = load()
    for t, n in ((o_part, "o_part"), (lse_part, "lse_part"), (seq_route_begin, "seq_route_begin"),
                 (out, "out"), (lse_out, "lse_out"), (err_flags, "err_flags")):
        _dev(t, n)
    R, Hq, D = o_part.shape
    _need(o_part.dtype == torch.float32 and lse_part.dtype == torch.float32, "partials must be float32")
    _need(tuple(lse_part.shape) == (R, Hq), "lse_part must be [R, Hq]")
    _need(seq_route_begin.dtype == torch.int32 and seq_route_begin.numel() >= num_seqs + 1,
          "seq_route_begin must be int32 [num_seqs + 1]")
    _need(tuple(out.shape) == (num_seqs, Hq, D) and out.dtype == torch.float32, "out must be float32 [B, Hq, D]")
    _need(tuple(lse_out.shape) == (num_seqs, Hq) and lse_out.dtype == torch.float32, "lse_out must be float32 [B, Hq]")
    args = (int(num_seqs), R, Hq, D, _ptr(o_part), _ptr(lse_part), _ptr(seq_route_begin),
            _ptr(out), _ptr(lse_out), _ptr(err_flags))
    return BoundCall(lib.kf_merge_partials, "kf_merge_partials", args,
                     (o_part, lse_part, seq_route_begin, out, lse_out, err_flags),
                     o_part.device.index)


def merge_partials(num_seqs, o_part, lse_part, seq_route_begin, out, lse_out, err_flags,
                   stream=None):
    """kf_merge_partials.  out float32 [B, Hq, 128], lse_out float32 [B, Hq]."""
    bind_merge_partials(num_seqs, o_part, lse_part, seq_route_begin, out, lse_out,
                        err_flags)(stream)


def bind_decode_step(shape: Shape, q, k_pool, v_pool, routes, tail_route, max_pages_per_route,
                     page_ids, seq_route_begin, o_part, lse_part, out, lse_out, workspace,
                     err_flags, k_scale=None, v_scale=None) -> BoundTokenCall:
    """kf_decode_step bound to its buffers; call it as (k_new, v_new, stream).
    workspace=None binds kf_decode_step_no_alloc, which uses the library's
    per-device scratch array instead."""
    lib = load()
    for t, n in ((q, "q"), (k_pool, "k_pool"), (v_pool, "v_pool"), (routes, "routes"),
                 (tail_route, "tail_route"), (page_ids, "page_ids"),
                 (seq_route_begin, "seq_route_begin"), (o_part, "o_part"),
                 (lse_part, "lse_part"), (out, "out"), (lse_out, "lse_out"),
                 (err_flags, "err_flags")) + (() if workspace is None else ((workspace, "workspace"),)):
        _dev(t, n)
    B, Hq, H, R = shape.num_seqs, shape.num_q_heads, shape.num_kv_heads, routes.shape[0]
    _need(tuple(q.shape) == (B, Hq, HEAD_DIM) and q.element_size() == 2,
          "q must be bf16 [num_seqs, num_q_heads, 128]")
    _need(tail_route.numel() >= B and tail_route.dtype == torch.int32, "tail_route: int32 [num_seqs]")
    _need(seq_route_begin.dtype == torch.int32 and seq_route_begin.numel() >= B + 1,
          "seq_route_begin must be int32 [num_seqs + 1]")
    for t, shp, n in ((o_part, (R, Hq, HEAD_DIM), "o_part"), (lse_part, (R, Hq), "lse_part"),
                      (out, (B, Hq, HEAD_DIM), "out"), (lse_out, (B, Hq), "lse_out")):
        _need(tuple(t.shape) == shp and t.dtype == torch.float32, f"{n} must be float32 {list(shp)}")
    _check_tables(shape, k_pool, v_pool, routes, page_ids)
    _check_scales(shape, k_scale, v_scale)
    sh = _copy_shape(shape)
    args = (ctypes.byref(sh), _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(k_scale), _ptr(v_scale),
            _ptr(routes), R, _ptr(tail_route), int(max_pages_per_route), _ptr(page_ids),
            _ptr(seq_route_begin), _ptr(o_part), _ptr(lse_part), _ptr(out), _ptr(lse_out))
    keep = (sh, q, k_pool, v_pool, k_scale, v_scale, routes, tail_route, page_ids,
            seq_route_begin, o_part, lse_part, out, lse_out, err_flags)
    if workspace is None:
        return BoundTokenCall(lib.kf_decode_step_no_alloc, "kf_decode_step_no_alloc",
                              args + (_ptr(err_flags),), keep, 6, (B, H, HEAD_DIM), q.device.index)
    return BoundTokenCall(lib.kf_decode_step, "kf_decode_step",
                          args + (_ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _ptr(err_flags)), keep + (workspace,), 6, (B, H, HEAD_DIM),
                          q.device.index)


def decode_step(shape: Shape, q, k_pool, v_pool, k_new, v_new, routes, tail_route,
                max_pages_per_route, page_ids, seq_route_begin, o_part, lse_part, out, lse_out,
                workspace, err_flags, k_scale=None, v_scale=None, stream=None):
    """kf_decode_step: append -> partial attention -> merge in one call (two
    launches).  Arguments as for kv_append, partial_attn and merge_partials.
    workspace=None calls kf_decode_step_no_alloc, which uses the library's
    per-device scratch array instead."""
    _check_tokens(shape, k_new, v_new)
    bind_decode_step(shape, q, k_pool, v_pool, routes, tail_route, max_pages_per_route, page_ids,
                     seq_route_begin, o_part, lse_part, out, lse_out, workspace, err_flags,
                     k_scale, v_scale)(k_new, v_new, stream)


def debug_gather(shape: Shape, k_pool, v_pool, routes, route, max_pages_per_route, page_ids,
                 max_tokens, out_k, out_v, err_flags, stream=None):
    """kf_debug_gather (test export): route ``route``'s tokens through the page
    table into out_k/out_v [max_tokens, num_kv_heads, 128] (pool element type)."""
    lib = load()
    for t, n in ((k_pool, "k_pool"), (v_pool, "v_pool"), (routes, "routes"), (page_ids, "page_ids"),
                 (out_k, "out_k"), (out_v, "out_v"), (err_flags, "err_flags")):
        _dev(t, n)
    _check_tables(shape, k_pool, v_pool, routes, page_ids)
    shp = (int(max_tokens), shape.num_kv_heads, HEAD_DIM)
    for t, n in ((out_k, "out_k"), (out_v, "out_v")):
        _need(tuple(t.shape) == shp and t.element_size() == k_pool.element_size(),
              f"{n} must be [max_tokens, num_kv_heads, 128] of the pool element type")
    st = lib.kf_debug_gather(ctypes.byref(shape), _ptr(k_pool), _ptr(v_pool), _ptr(routes),
                             routes.shape[0], int(route), int(max_pages_per_route), _ptr(page_ids),
                             int(max_tokens), _ptr(out_k), _ptr(out_v), _ptr(err_flags),
                             _stream(stream))
    _check(st, "kf_debug_gather")
