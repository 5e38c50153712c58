"""The Python front end checks every tensor's dtype, shape, layout and
device before it allocates or launches anything (CPU only: the tensors here
live on the host, so any call that got past the checks would fail on the
device test instead).  The C ABI cannot see buffer sizes, so these checks are
what keeps a short K, V, dOut, idx or output buffer from being read or
written out of bounds."""
import pytest

torch = pytest.importorskip("torch")
kmip = pytest.importorskip("paper_2604_03815_amd")

N, H, d, k = 40, 2, 16, 4


def bf(*shape):
    return torch.zeros(shape, dtype=torch.bfloat16)


def f32(*shape):
    return torch.zeros(shape, dtype=torch.float32)


def i32(*shape):
    return torch.zeros(shape, dtype=torch.int32)


def good():
    return dict(q=bf(N, H, d), k_=bf(N, H, d), v=bf(N, H, d), dout=bf(N, H, d), idx=i32(N, H, k),
                lse=f32(N, H))


@pytest.mark.parametrize("name,bad", [
    ("k_", bf(N - 1, H, d)), ("k_", bf(N, H, 2 * d)), ("v", bf(N, H + 1, d)),
    ("v", f32(N, H, d)), ("idx", i32(N - 1, H, k)),
])
def test_attend_rejects_mismatch(name, bad):
    a = good()
    a[name] = bad
    with pytest.raises((ValueError, TypeError)) as e:
        kmip.attend(a["q"], a["k_"], a["v"], a["idx"], 0.25)
    assert "CUDA" not in str(e.value)


@pytest.mark.parametrize("name,bad", [
    ("out", f32(N, H, d + 1)), ("lse", f32(N, H, 1)), ("out", bf(N, H, d)),
])
def test_attend_rejects_bad_outputs(name, bad):
    a = good()
    kw = {name: bad}
    with pytest.raises((ValueError, TypeError)) as e:
        kmip.attend(a["q"], a["k_"], a["v"], a["idx"], 0.25, **kw)
    assert "CUDA" not in str(e.value)


@pytest.mark.parametrize("name,bad", [
    ("k_", bf(N, H, d)[:, :, :8]), ("dout", bf(N - 3, H, d)), ("lse", f32(N)),
    ("idx", i32(N, H, k)[:, :, ::2]), ("idx", torch.zeros((N, H, k), dtype=torch.int64)),
])
def test_bwd_rejects_mismatch(name, bad):
    a = good()
    a[name] = bad
    with pytest.raises((ValueError, TypeError)) as e:
        kmip.bwd(a["q"], a["k_"], a["v"], a["dout"], a["idx"], a["lse"], 0.25)
    assert "CUDA" not in str(e.value)


@pytest.mark.parametrize("name", ["dq", "dk", "dv"])
def test_bwd_rejects_short_gradient_buffers(name):
    a = good()
    with pytest.raises(ValueError):
        kmip.bwd(a["q"], a["k_"], a["v"], a["dout"], a["idx"], a["lse"], 0.25,
                 **{name: f32(N // 2, H, d)})


def test_topk_and_fwd_reject_mismatch():
    a = good()
    with pytest.raises(ValueError):
        kmip.topk(a["q"], bf(N + 1, H, d), k)
    with pytest.raises(ValueError):
        kmip.topk(a["q"], a["k_"], k, idx=i32(N, H, k + 1))
    with pytest.raises(ValueError):
        kmip.fwd(a["q"], a["k_"], bf(N, H + 1, d), k, 0.25)
    with pytest.raises(ValueError):
        kmip.fwd(bf(N, H * d), a["k_"], a["v"], k, 0.25)


def test_value_width_of_its_own():
    # V (and dOut, out, dV) may be wider or narrower than Q and K: only the
    # device check is left to fail on host tensors; a dOut or dV whose width
    # differs from V's is a mismatch
    a = good()
    wide = bf(N, H, 2 * d)
    with pytest.raises(TypeError, match="CUDA"):
        kmip.attend(a["q"], a["k_"], wide, a["idx"], 0.25)
    with pytest.raises(TypeError, match="CUDA"):
        kmip.bwd(a["q"], a["k_"], wide, bf(N, H, 2 * d), a["idx"], a["lse"], 0.25)
    with pytest.raises(ValueError):
        kmip.bwd(a["q"], a["k_"], wide, a["dout"], a["idx"], a["lse"], 0.25)
    with pytest.raises(ValueError):
        kmip.bwd(a["q"], a["k_"], wide, bf(N, H, 2 * d), a["idx"], a["lse"], 0.25, dv=f32(N, H, d))
    with pytest.raises(ValueError):
        kmip.attend(a["q"], a["k_"], wide, a["idx"], 0.25, out=f32(N, H, d))


def test_matching_host_tensors_are_refused_as_not_on_the_gpu():
    a = good()
    with pytest.raises(TypeError, match="CUDA"):
        kmip.attend(a["q"], a["k_"], a["v"], a["idx"], 0.25)
    with pytest.raises(TypeError, match="CUDA"):
        kmip.bwd(a["q"], a["k_"], a["v"], a["dout"], a["idx"], a["lse"], 0.25)
