"""The allocation-free backward (lr_attnres_route_bwd_noalloc) through the C
ABI: its dV, dK and dq equal those of lr_attnres_route_bwd, which takes the
dq partials in a caller workspace, bit for bit (the same kernels in the same
order).  Two calls in a row, the second smaller, check that the device array
the partials live in carries nothing over from one call to the next."""
import ctypes

import numpy as np
import pytest

import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import FULL, PROJECTED, SLICED, make_host_problem

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def to_dev(x, dev):
    if x is None:
        return None
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(x).to(dev)


def ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def both_backwards(lib, dev, mode, S, N, d, r, dtype, seed):
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=seed, with_dH=True)
    V, K, q, dH = (to_dev(x, dev) for x in (p.V, p.K, p.q, p.dH))
    code = 1 if dtype == "bf16" else 0
    st = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    outs = []
    for noalloc in (False, True):
        # Fill the outputs with NaN so that a value not written shows.
        dV = torch.full_like(V, float("nan"))
        dK = torch.full_like(K, float("nan")) if K is not None else None
        dq = torch.full((r,), float("nan"), dtype=torch.float32, device=dev)
        if noalloc:
            print(f"noalloc call: mode={mode} S={S} N={N} d={d} r={r} {dtype} seed={seed}",
                  flush=True)
            rc = lib.lr_attnres_route_bwd_noalloc(ptr(V), ptr(K), ptr(q), ptr(dH), ptr(dV),
                                                  ptr(dK), ptr(dq), S, N, d, r, mode, code,
                                                  1e-6, st)
        else:
            need = lib.lr_attnres_route_bwd_workspace_bytes(S, N, d, r, mode, code)
            ws = torch.empty((max(need, 16),), dtype=torch.uint8, device=dev)
            rc = lib.lr_attnres_route_bwd(ptr(V), ptr(K), ptr(q), ptr(dH), ptr(dV), ptr(dK),
                                          ptr(dq), ptr(ws), ws.numel(), S, N, d, r, mode, code,
                                          1e-6, st)
        assert rc == 0, lib.lr_attnres_last_error().decode()
        torch.cuda.synchronize()
        outs.append((dV, dK, dq))
    return outs


def same_bits(a, b):
    if a is None:
        return b is None
    return torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                       b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32))


CASES = [
    # (mode, first call, second call (smaller), storage)
    (PROJECTED, (12, 1500, 2048, 32), (5, 37, 512, 16), "bf16"),
    (SLICED, (9, 777, 1024, 64), (3, 5, 256, 8), "bf16"),
    (FULL, (6, 300, 256, 256), (2, 17, 128, 128), "f32"),
]


@pytest.mark.parametrize("mode,big,small,dtype", CASES,
                         ids=["projected_bf16", "sliced_bf16", "full_f32"])
def test_noalloc_matches_workspace_backward(dev, mode, big, small, dtype):
    lib = lr.load_library()
    for k, (S, N, d, r) in enumerate((big, small)):
        (dV0, dK0, dq0), (dV1, dK1, dq1) = both_backwards(lib, dev, mode, S, N, d, r, dtype,
                                                          seed=100 + k)
        assert torch.isfinite(dq1).all()
        assert torch.isfinite(dV1.float()).all()
        assert same_bits(dV0, dV1), "dV"
        assert same_bits(dK0, dK1), "dK"
        assert same_bits(dq0, dq1), "dq"


def test_noalloc_no_tokens_writes_zero_dq(dev):
    lib = lr.load_library()
    st = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    q = torch.ones((8,), dtype=torch.float32, device=dev)
    dq = torch.full((8,), float("nan"), dtype=torch.float32, device=dev)
    rc = lib.lr_attnres_route_bwd_noalloc(None, None, ptr(q), None, None, None, ptr(dq),
                                          4, 0, 64, 8, SLICED, 1, 1e-6, st)
    assert rc == 0, lib.lr_attnres_last_error().decode()
    torch.cuda.synchronize()
    assert torch.equal(dq, torch.zeros_like(dq))
