"""kmip_fwd_noalloc (the forward that allocates nothing) against kmip_fwd.

Both run the same kernels; the no-allocation entry point keeps its working
data in the library's fixed per-device array instead of a caller workspace.
Two calls in a row, the second on a smaller graph (the array then holds the
first call's data), must each give kmip_fwd's index sets bit for bit and
its out and lse; the index sets also pass the oracle protocol.
"""
import ctypes

import numpy as np
import pytest

import oracle
import workloads
from parity import allclose_report, check_sets_all, check_structure

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2604_03815_amd as kmip  # noqa: E402
from paper_2604_03815_amd import _lib  # noqa: E402

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def _noalloc_via_abi(q, k, v, kk, scale):
    """Calls kmip_fwd_noalloc through the C ABI into freshly allocated outputs."""
    N, H, d = q.shape
    out = torch.full((N, H, d), float("nan"), dtype=torch.float32, device=DEV)
    idx = torch.full((N, H, kk), -77, dtype=torch.int32, device=DEV)
    lse = torch.full((N, H), float("nan"), dtype=torch.float32, device=DEV)
    P = ctypes.c_void_p
    st = _lib.load().kmip_fwd_noalloc(P(q.data_ptr()), P(k.data_ptr()), P(v.data_ptr()), N, H, d, kk,
                                      ctypes.c_float(scale), P(out.data_ptr()), P(idx.data_ptr()),
                                      P(lse.data_ptr()), P(torch.cuda.current_stream().cuda_stream))
    _lib.check(st)
    return out, idx, lse


@pytest.mark.parametrize("first,second", [
    ((4, 60_000, 16, 32), (4, 3_000, 16, 32)),        # grouped + key order, then the plain path
    ((5, 40_000, None, None), (1, None, None, None)),  # d = 64, k = 128, then config 1 (d = 32)
])
def test_noalloc_matches_fwd_twice(first, second):
    for cfg, n, _, _ in (first, second):
        w = workloads.make(cfg, n=n)
        print(f"[case] noalloc c{cfg} N={w.N} H={w.H} d={w.d} k={w.k}", flush=True)
        q, k, v = _dev(w.q), _dev(w.kk), _dev(w.v)
        o1, i1, l1 = _noalloc_via_abi(q, k, v, w.k, w.scale)
        o2, i2, l2 = kmip.fwd(q, k, v, w.k, w.scale)
        torch.cuda.synchronize()
        assert torch.equal(i1, i2)
        assert torch.equal(o1, o2)
        assert torch.equal(l1, l2)
        idx = i1.cpu().numpy()
        check_structure(idx, None, w.N, w.H, w.k)
        Qd, Kd, Vd = (oracle.from_bf16(getattr(w, x)) for x in ("q", "kk", "v"))
        check_sets_all(w, Qd, Kd, idx, sel=np.arange(0, w.N * w.H, max(1, w.N * w.H // 4096)))
        ref_out, ref_lse = oracle.attend(Qd, Kd, Vd, idx, w.scale)
        allclose_report("out", o1.cpu().numpy().reshape(-1, w.d), ref_out)
        allclose_report("lse", l1.cpu().numpy().reshape(-1), ref_lse)


def test_noalloc_rejects_oversize_without_writing():
    N, H, d, kk = 1_000_000, 4, 16, 32
    assert kmip.topk_workspace_size(N, H, d, kk) > kmip.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((N, H, d), dtype=torch.bfloat16, device=DEV)
    out = torch.full((N, H, d), 3.0, dtype=torch.float32, device=DEV)
    idx = torch.full((N, H, kk), -5, dtype=torch.int32, device=DEV)
    lse = torch.full((N, H), 4.0, dtype=torch.float32, device=DEV)
    with pytest.raises(kmip.KmipError) as e:
        kmip.fwd_noalloc(q, q, q, kk, 0.25, out, idx, lse)
    assert e.value.status == 2 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (idx == -5).all() and (out == 3.0).all() and (lse == 4.0).all()
