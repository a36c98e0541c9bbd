"""The Python binding validates every tensor (dtype, exact shape, contiguity,
device) before anything reaches the C library, whose kernels index each
buffer by the shapes taken from q and k.  Runs on the CPU: a mismatched
tensor must raise ValueError naming it, and the library must not be called."""

import pytest

torch = pytest.importorskip("torch")
cowa = pytest.importorskip("paper_2609_32704_amd")


@pytest.fixture
def no_library(monkeypatch):
    def boom():
        raise AssertionError("the library was called")
    monkeypatch.setattr(cowa._abi, "lib", boom)
    import inspect
    for name in dir(cowa._abi):
        if name.startswith("cowa_") and inspect.isfunction(getattr(cowa._abi, name)):
            monkeypatch.setattr(cowa._abi, name, lambda *a, **k: boom())


B, HQ, HK, N, NK, D = 2, 4, 2, 64, 96, 64


def bf(*shape, dtype=torch.bfloat16):
    return torch.zeros(shape, dtype=dtype)


def fwd_args():
    return dict(q=bf(B, HQ, N, D), k=bf(B, HK, NK, D), v=bf(B, HK, NK, D))


@pytest.mark.parametrize("name,bad", [
    ("v", bf(B, HK, NK + 1, D)), ("v", bf(B, HK + 1, NK, D)), ("k", bf(B + 1, HK, NK, D)),
    ("k", bf(B, HK, NK, D + 8)), ("out", bf(B, HQ, N + 1, D)), ("lse", bf(B, HQ, N, dtype=torch.float32)[:, :, :-1]),
    ("lse", bf(B, HQ, N)), ("v", bf(B, HK, NK, D, dtype=torch.float32)),
])
def test_fwd_rejects_mismatched_tensors(no_library, name, bad):
    a = fwd_args()
    a[name] = bad
    with pytest.raises(ValueError, match=name):
        cowa.fwd(a["q"], a["k"], a["v"], 4, 16, 64, 64, out=a.get("out"), lse=a.get("lse"))


def test_fwd_rejects_host_tensors(no_library):
    a = fwd_args()
    with pytest.raises(ValueError, match="device"):
        cowa.fwd(a["q"], a["k"], a["v"], 4, 16, 64, 64)


def bwd_args():
    return dict(q=bf(B, HQ, N, D), k=bf(B, HK, NK, D), v=bf(B, HK, NK, D), o=bf(B, HQ, N, D),
                lse=bf(B, HQ, N, dtype=torch.float32), do=bf(B, HQ, N, D))


@pytest.mark.parametrize("name,bad", [
    ("v", bf(B, HK, NK - 1, D)), ("o", bf(B, HQ, N, D + 1)), ("do", bf(B, HQ - 1, N, D)),
    ("lse", bf(B, HQ, N + 1, dtype=torch.float32)), ("dq", bf(B, HQ, N - 1, D)), ("dk", bf(B, HK, N, D)),
    ("dv", bf(B, HQ, NK, D)), ("k", bf(B, HK, NK, D + 64)),
])
def test_bwd_rejects_mismatched_tensors(no_library, name, bad):
    a = bwd_args()
    a[name] = bad
    with pytest.raises(ValueError, match=name):
        cowa.bwd(a["q"], a["k"], a["v"], a["o"], a["lse"], a["do"], 4, 16, 64, 64, dq=a.get("dq"), dk=a.get("dk"),
                 dv=a.get("dv"))


def dec_args():
    return dict(q=bf(B, HQ, D), k_cache=bf(B, HK, NK, D), v_cache=bf(B, HK, NK, D),
                seqlens_k=torch.zeros(B, dtype=torch.int32))


@pytest.mark.parametrize("name,bad", [
    ("v_cache", bf(B, HK, NK + 1, D)), ("k_cache", bf(B + 1, HK, NK, D)), ("seqlens_k", torch.zeros(B + 1, dtype=torch.int32)),
    ("seqlens_k", torch.zeros(B, dtype=torch.int64)), ("out", bf(B, HQ, D + 1)), ("lse", bf(B, HQ + 1, dtype=torch.float32)),
])
def test_decode_rejects_mismatched_tensors(no_library, name, bad):
    a = dec_args()
    a[name] = bad
    with pytest.raises(ValueError, match=name):
        cowa.decode(a["q"], a["k_cache"], a["v_cache"], a["seqlens_k"], 4, 16, out=a.get("out"), lse=a.get("lse"))


def test_noncontiguous_rejected(no_library):
    a = fwd_args()
    k = bf(B, HK, D, NK).transpose(2, 3)
    with pytest.raises(ValueError, match="contiguous"):
        cowa.fwd(a["q"], k, a["v"], 4, 16, 64, 64)
