"""kf.BoundCall / kf.BoundTokenCall plumbing on the CPU: the bound argument
tuple is passed unchanged with the stream handle appended, the step's token
pointers are inserted at the entry point's position, and host tensors or
wrong token shapes are refused before any call."""
import ctypes

import pytest

torch = pytest.importorskip("torch")
from paper_2606_29207_amd import kf  # noqa: E402


class _Stream:
    cuda_stream = 0xABC
    device_index = 0


def test_bound_call_appends_the_stream():
    seen = []
    call = kf.BoundCall(lambda *a: seen.append(a) or 0, "kf_x", (1, 2, 3), ())
    call(_Stream())
    call(_Stream())
    assert len(seen) == 2
    assert seen[0][:3] == (1, 2, 3) and seen[0][3] == 0xABC


def test_bound_call_refuses_another_device(monkeypatch):
    """A call bound to cuda:1 refuses to run while cuda:0 is current, or on
    a stream of another device, before calling the library."""
    seen = []
    monkeypatch.setattr(kf, "_cur_device", lambda: 0)
    call = kf.BoundCall(lambda *a: seen.append(a) or 0, "kf_x", (1,), (), 1)
    with pytest.raises(kf.KFError, match="bound to cuda:1"):
        call(_Stream())
    monkeypatch.setattr(kf, "_cur_device", lambda: 1)
    with pytest.raises(kf.KFError, match="a stream of cuda:0"):
        call(_Stream())
    s1 = _Stream()
    s1.device_index = 1
    call(s1)
    assert len(seen) == 1


def test_bound_call_raises_on_a_status():
    call = kf.BoundCall(lambda *a: kf.ERR_INVALID_ARG, "kf_x", (), ())
    with pytest.raises(kf.KFError, match="kf_x"):
        call(_Stream())


def test_bound_token_call_refuses_host_tensors_and_bad_shapes():
    called = []
    call = kf.BoundTokenCall(lambda *a: called.append(a) or 0, "kf_y", ("a", "b", "c"), (), 2,
                             (1, 2, 128))
    t = torch.zeros(1, 2, 128, dtype=torch.bfloat16)
    with pytest.raises(kf.KFError, match="k_new must be a contiguous bf16 device tensor"):
        call(t, t, _Stream())
    assert not called
    assert isinstance(call._tok_shape, torch.Size) and call._tok_at == 2
    assert ctypes.sizeof(kf.Shape) == 40
