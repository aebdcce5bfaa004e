"""Head-major pools (kf_shape.kv_layout = KF_KV_HEAD_MAJOR, [Hkv][P][...])
against page-major ones ([P][Hkv][...]) holding the same tokens: every step
(fused and as three calls), every plan mode, bf16 and fp8, gives the same
partials, outputs, flags, routes and scales bit for bit, and the same pools
once swapped back; one case is also checked against the oracle."""
import numpy as np
import pytest

from kf_testlib import compare_all, host, run_oracle
from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]

CASES = {
    # name: (workload, overrides, seq_lens, steps)
    "hkv2_two_units": ("llama8b_32k", dict(num_seqs=64, num_q_heads=8, num_kv_heads=2, part_tokens=256),
                       [1000 + 13 * i for i in range(64)], 2),
    "hkv8_unsplit": ("llama8b_32k", dict(num_seqs=16, part_tokens=1024), [4096] * 16, 2),
    "hkv4_chunked": ("llama8b_32k", dict(num_seqs=5, num_q_heads=16, num_kv_heads=4, part_tokens=2048),
                     [3000, 17, 0, 4100, 999], 3),
    "hkv16_g2": ("llama8b_32k", dict(num_seqs=3, num_q_heads=32, num_kv_heads=16, part_tokens=1024),
                 [2100, 1500, 33], 2),
    "hkv1": ("llama8b_32k", dict(num_seqs=4, num_q_heads=8, num_kv_heads=1, part_tokens=512),
             [900, 1, 1700, 512], 2),
    "fp8_append": ("wide_gqa_fp8", dict(num_seqs=3, part_tokens=1024, appends=1), [3000, 2048, 1111], 3),
    "fp8_hkv2": ("wide_gqa_fp8", dict(num_seqs=4, num_q_heads=16, num_kv_heads=2, part_tokens=768, appends=1),
                 [1600, 1025, 16, 800], 2),
}
KEYS = ("o_part", "lse_part", "out", "lse", "routes", "k_scale", "v_scale", "flags")


def _run(inst, steps, layout, fused):
    import torch
    from paper_2606_29207_amd.step import DecodeState
    st = DecodeState.from_instance(inst, kv_layout=layout)
    for s in range(steps):
        kn, vn = st.upload_new_tokens(*inst.new_tokens(s))
        (st.step_fused if fused else st.step)(kn, vn)
    torch.cuda.synchronize()
    h = host(st)
    if layout:
        h["k_pool"], h["v_pool"] = np.swapaxes(h["k_pool"], 0, 1), np.swapaxes(h["v_pool"], 0, 1)
    return st, h


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("fused", [True, False])
def test_head_major_equals_page_major(gpu, case, fused):
    from paper_2606_29207_amd import kf
    name, over, lens, steps = CASES[case]
    wl = workload(name, **dict(over, appends=1))
    inst = make_instance(wl, seed=41, steps=steps, seq_lens=lens)
    _, a = _run(inst, steps, kf.KV_PAGE_MAJOR, fused)
    st, b = _run(inst, steps, kf.KV_HEAD_MAJOR, fused)
    assert st.shape.kv_layout == kf.KV_HEAD_MAJOR and st.k_pool.shape[0] == wl.num_kv_heads
    for k in KEYS + ("k_pool", "v_pool"):
        x, y = a[k], b[k]
        if x is None:
            assert y is None, k
            continue
        assert np.array_equal(np.asarray(x), np.asarray(y), equal_nan=True), k


def test_head_major_matches_oracle_and_gather(gpu):
    import torch
    from paper_2606_29207_amd import kf
    name, over, lens, steps = CASES["hkv4_chunked"]
    inst = make_instance(workload(name, **dict(over, appends=1)), seed=42, steps=steps, seq_lens=lens)
    st, h = _run(inst, steps, kf.KV_HEAD_MAJOR, True)
    compare_all(h, run_oracle(inst, steps))
    pm, _ = _run(inst, steps, kf.KV_PAGE_MAJOR, True)
    H = inst.wl.num_kv_heads
    routes = st.routes.cpu().numpy()
    for r in range(len(routes)):            # the gather export reads either layout alike
        m = max(int(routes[r, 3]) - int(routes[r, 2]), 0) + 3
        got = []
        for s_ in (pm, st):
            ok = torch.full((m, H, 128), -1, dtype=torch.int16, device="cuda").view(torch.bfloat16)
            ov = torch.full((m, H, 128), -1, dtype=torch.int16, device="cuda").view(torch.bfloat16)
            kf.debug_gather(s_.shape, s_.k_pool, s_.v_pool, s_.routes, r, s_.max_pages_per_route,
                            s_.page_ids, m, ok, ov, s_.err_flags)
            got.append((ok.view(torch.int16), ov.view(torch.int16)))
        torch.cuda.synchronize()
        assert torch.equal(got[0][0], got[1][0]) and torch.equal(got[0][1], got[1][1]), r
    assert pm.flags() == 0 and st.flags() == 0
