"""Shared helpers of the GPU parity tests: run a decode step on the HIP path
and on the oracle from the same seeded instance, and compare."""
from __future__ import annotations

import numpy as np

import oracle

# tolerances of the path (float32 kernels vs fp64 oracle)
O_MAX_ABS = 2e-3
O_REL_L2 = 1e-3
LSE_MAX_ABS = 1e-4


def run_oracle(inst, steps=1, tail_route=None, new_tokens=None):
    """Oracle decode: per step append (if the workload appends), then
    partials of every route, then the merge.  Returns the final state.
    ``new_tokens(step)`` replaces the instance's token stream."""
    wl = inst.wl
    new_tokens = new_tokens or inst.new_tokens
    kp, vp, routes = inst.k_pool, inst.v_pool, inst.routes.copy()
    ks, vs = inst.k_scale, inst.v_scale
    tail = inst.tail_route if tail_route is None else tail_route
    flags = 0
    for s in range(steps):
        if wl.appends:
            kn, vn = new_tokens(s)
            if ks is None:
                kp, vp, routes, f = oracle.kv_append(kp, vp, routes, inst.page_ids, tail, kn, vn)
            else:
                kp, vp, ks, vs, routes, f = oracle.kv_append(kp, vp, routes, inst.page_ids, tail,
                                                             kn, vn, ks, vs)
            flags |= f
    o_part, lse_part, f1 = oracle.partial_attn(
        inst.q, kp, vp, routes, inst.page_ids, num_kv_heads=wl.num_kv_heads, scale=inst.scale,
        max_pages_per_route=inst.max_pages_per_route, k_scale=ks, v_scale=vs)
    out, lse, f2 = oracle.merge_partials(o_part, lse_part, inst.seq_route_begin)
    return dict(k_pool=kp, v_pool=vp, k_scale=ks, v_scale=vs, routes=routes, o_part=o_part,
                lse_part=lse_part, out=out, lse=lse, flags=flags | f1 | f2)


def run_gpu(inst, steps=1, tail_route=None, nan_fill=True, new_tokens=None, fused=False):
    """HIP path: the same sequence of calls through the C ABI (fused: one
    kf_decode_step per step)."""
    import torch
    new_tokens = new_tokens or inst.new_tokens
    from paper_2606_29207_amd.step import DecodeState
    st = DecodeState.from_instance(inst)
    if tail_route is not None:
        st.tail_route.copy_(torch.from_numpy(np.asarray(tail_route, np.int32)))
    for s in range(steps):
        if nan_fill:
            for t in (st.o_part, st.lse_part, st.out, st.lse):
                t.fill_(float("nan"))
        if inst.wl.appends:
            kn, vn = st.upload_new_tokens(*new_tokens(s))
            if fused:
                st.step_fused(kn, vn)
            else:
                st.step(kn, vn)
        else:
            st.step()
    torch.cuda.synchronize()
    return st


def host(st):
    """Copy the state back: numpy arrays in the oracle's dtypes."""
    import torch
    kp, vp = st.k_pool.cpu(), st.v_pool.cpu()
    if kp.element_size() == 2:
        kp = kp.view(torch.int16).numpy().view(np.uint16)
        vp = vp.view(torch.int16).numpy().view(np.uint16)
    else:
        kp, vp = kp.view(torch.uint8).numpy(), vp.view(torch.uint8).numpy()
    ks = None if st.k_scale is None else st.k_scale.cpu().numpy()
    vs = None if st.v_scale is None else st.v_scale.cpu().numpy()
    return dict(k_pool=kp, v_pool=vp, k_scale=ks, v_scale=vs, routes=st.routes.cpu().numpy(),
                o_part=st.o_part.cpu().numpy().astype(np.float64),
                lse_part=st.lse_part.cpu().numpy().astype(np.float64),
                out=st.out.cpu().numpy().astype(np.float64),
                lse=st.lse.cpu().numpy().astype(np.float64), flags=st.flags())


def assert_close_o(got, ref, what):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, what
    nan_r, nan_g = np.isnan(ref), np.isnan(got)
    assert np.array_equal(nan_r, nan_g), f"{what}: NaN positions differ ({nan_g.sum()} vs {nan_r.sum()})"
    g, r = got[~nan_r], ref[~nan_r]
    if g.size == 0:
        return
    err = np.abs(g - r)
    mx = float(err.max())
    rel = float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))
    assert mx <= O_MAX_ABS, f"{what}: max|d| {mx:.3e} > {O_MAX_ABS}"
    assert rel <= O_REL_L2, f"{what}: rel-L2 {rel:.3e} > {O_REL_L2}"
    return mx, rel


def assert_close_lse(got, ref, what):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, what
    assert np.array_equal(np.isnan(got), np.isnan(ref)), f"{what}: NaN positions differ"
    assert np.array_equal(np.isneginf(got), np.isneginf(ref)), f"{what}: -inf positions differ"
    fin = np.isfinite(ref)
    assert np.all(np.isfinite(got[fin])), f"{what}: non-finite where the oracle is finite"
    if fin.any():
        mx = float(np.abs(got[fin] - ref[fin]).max())
        assert mx <= LSE_MAX_ABS, f"{what}: max|d| {mx:.3e} > {LSE_MAX_ABS}"
        return mx


def _bits(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


def compare_all(g, o, pools=True):
    """Bit-exact pools and routes, toleranced floats, equal flags."""
    if pools:
        assert np.array_equal(g["routes"], o["routes"]), "routes differ"
        assert np.array_equal(g["k_pool"], o["k_pool"]), "K pool differs"
        assert np.array_equal(g["v_pool"], o["v_pool"]), "V pool differs"
        if o.get("k_scale") is not None:   # bit for bit (a NaN scale equals itself)
            assert np.array_equal(_bits(g["k_scale"]), _bits(o["k_scale"])), "K scales differ"
            assert np.array_equal(_bits(g["v_scale"]), _bits(o["v_scale"])), "V scales differ"
    assert g["flags"] == o["flags"], f"flags {g['flags']} != {o['flags']}"
    assert_close_o(g["o_part"], o["o_part"], "o_part")
    assert_close_lse(g["lse_part"], o["lse_part"], "lse_part")
    assert_close_o(g["out"], o["out"], "out")
    assert_close_lse(g["lse"], o["lse"], "lse")
