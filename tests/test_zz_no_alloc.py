"""kf_decode_step_no_alloc (the decode step for callers that cannot
allocate: its chunk partials use the library's per-device scratch array)
against kf_decode_step with a workspace, through the C ABI.

Two calls in a row on one device, each on its own copy of the same state as
the reference call: first a larger batch whose launch splits its units (so
the chunk partials go through the scratch array), then a smaller one, which
runs over what the first left in the array.  Outputs, pools, scales, route
rows and flags must be bit-identical to kf_decode_step's: both run the same
kernels on the same plan."""
import numpy as np
import pytest

from kf_workloads import make_instance, workload

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]


def _bits(t):
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy()
    return t.view(torch.uint8).numpy() if t.element_size() == 1 else t.view(torch.int16).numpy()


def _step_pair(inst):
    import torch
    from paper_2606_29207_amd import kf
    from paper_2606_29207_amd.step import DecodeState
    ref, got = DecodeState.from_instance(inst), DecodeState.from_instance(inst)
    plan = kf.partial_attn_plan(ref.shape, ref.routes.shape[0], ref.max_pages_per_route)
    assert plan[1] > 1, f"the launch should split its units: plan {plan}"
    for st in (ref, got):
        for t in (st.o_part, st.lse_part, st.out, st.lse):
            t.fill_(float("nan"))
    kn, vn = ref.upload_new_tokens(*inst.new_tokens(0))
    ref.step_fused(kn, vn)
    got.step_no_alloc(kn, vn)
    torch.cuda.synchronize()
    assert ref.flags() == got.flags() == 0
    names = ["o_part", "lse_part", "out", "lse", "k_pool", "v_pool", "routes"]
    if ref.k_scale is not None:
        names += ["k_scale", "v_scale"]
    for n in names:
        assert np.array_equal(_bits(getattr(ref, n)), _bits(getattr(got, n))), f"{n} differs"
    assert not np.isnan(got.out.cpu().numpy()).any()
    return plan


def test_no_alloc_step_equals_decode_step_twice(gpu):
    big = make_instance(workload("agentic_mix", num_seqs=12, ctx_range=(1000, 40000),
                                 part_tokens=8192), seed=3, steps=2)
    small = make_instance(workload("wide_gqa_fp8_decode", num_seqs=2, num_q_heads=16,
                                   num_kv_heads=2, part_tokens=1024), seed=4, steps=2,
                          seq_lens=[2500, 700])
    import torch
    p1 = _step_pair(big)
    # the first launch runs in a computed dispatch order (a table in the scratch array)
    slots = 2 * torch.cuda.get_device_properties(0).multi_processor_count
    items = p1[1] * big.wl.num_kv_heads * len(big.routes)
    assert 2 * slots <= items <= 1 << 20, f"plan {p1}: {items} work items"
    p2 = _step_pair(small)
    print(f"[no_alloc] plans {p1} then {p2}", flush=True)
