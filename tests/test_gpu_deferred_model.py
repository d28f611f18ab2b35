"""GPU parity of the full-source reverse pass in deferred form (each site
records per-source coefficients, one gather per source then forms its whole
gradient) through the C ABI, against the fp64 oracle's backward of every
site of the pass (Sec. 3.1, Eq. full_attnres_source_set: site t reads the
sources 0 .. t-1).

Every source's dV (and dK), and every site's dq, are compared: sliced and
projected keys, a ragged column tail, key lengths that are not a multiple of
8, the paper's 49-source pass at small N, and a stack with sources that no
site reads.
"""
import numpy as np
import pytest

import oracle
import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import PROJECTED, SLICED, bf16_bits_from_f32, make_host_problem
from parity import check_bf16_grown, check_bf16_key_grad, check_dq
from test_gpu_all_sites_bwd import _queries, _upstream, to_dev, to_host

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lr.load_library()
    return torch.device("cuda:0")


def deferred_reverse_pass(V, K, Q, dH, mode):
    """Sites t = T .. 1 (site t reads sources 0 .. t-1 with Q[t-1], dH[t-1]):
    the site's coefficients, then source t-1's gradient from sites t .. T."""
    S, N, d = V.shape
    T, r = Q.shape
    coefs = torch.empty((T, S, 3, N), dtype=torch.float32, device=V.device)
    dV = torch.zeros_like(V)
    dK = torch.zeros_like(K) if K is not None else None
    dq = torch.empty((T, r), dtype=torch.float32, device=V.device)
    ws = torch.empty((max(16, lr.route_bwd_workspace_bytes(S, N, d, r, mode, V.dtype)),),
                     dtype=torch.uint8, device=V.device)
    for t in range(T, 0, -1):
        lr.route_bwd_deferred(V[:t], K[:t] if K is not None else None, Q[t - 1], dH[t - 1], mode,
                              coefs[t - 1, :t], dq=dq[t - 1], workspace=ws)
        i = t - 1
        lr.route_gather_bwd(V, K, i, dH[i:], Q[i:], coefs[i:, i], mode,
                            out=(dV[i], dK[i] if dK is not None else None))
    return dV, dK, dq


# (mode, S, T, N, d, r)
CASES = [
    (PROJECTED, 9, 9, 37, 256, 16),
    (SLICED, 12, 10, 33, 200, 24),     # ragged columns; two sources no site reads
    (PROJECTED, 10, 8, 17, 96, 12),    # r % 8 != 0
    (SLICED, 6, 6, 20, 64, 8),
    (PROJECTED, 49, 49, 24, 1024, 16),  # the paper's pass
    (SLICED, 49, 49, 12, 1024, 64),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "{}-S{}-T{}-N{}-d{}-r{}".format(
    "P" if c[0] == PROJECTED else "S", *c[1:]))
def test_deferred_reverse_pass_matches_oracle(dev, case):
    mode, S, T, N, d, r = case
    p = make_host_problem(mode, S, N, d, r, dtype="bf16", seed=S + T + N)
    Q = _queries(T, r, seed=S + 1)
    dH = _upstream(T, N, d, seed=S + 2)
    dV, dK, dq = deferred_reverse_pass(to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Q, dev),
                                       to_dev(dH, dev), mode)
    torch.cuda.synchronize()
    rV, rK, rQ = oracle.route_all_bwd(p.V, p.K, Q.astype(np.float64), dH, mode, 1, r=r)
    gV = to_host(dV)
    if mode == SLICED:
        check_bf16_grown("dV", gV[..., :-r], rV[..., :-r])
        check_bf16_key_grad("dV key columns", gV[..., -r:], rV[..., -r:])
    else:
        check_bf16_grown("dV", gV, rV)
        check_bf16_key_grad("dK", to_host(dK), rK)
    check_dq("dq", to_host(dq), rQ)


def test_gather_over_no_sites_writes_zeros(dev):
    S, N, d, r = 4, 9, 64, 8
    p = make_host_problem(PROJECTED, S, N, d, r, dtype="bf16", seed=3)
    V, K = to_dev(p.V, dev), to_dev(p.K, dev)
    dV = torch.full((N, d), 5.0, dtype=torch.bfloat16, device=dev)
    dK = torch.full((N, r), 5.0, dtype=torch.bfloat16, device=dev)
    empty = torch.empty((0, N, d), dtype=torch.bfloat16, device=dev)
    lr.route_gather_bwd(V, K, 3, empty, torch.empty((0, r), device=dev),
                        torch.empty((0, 3, N), device=dev), PROJECTED, out=(dV, dK))
    torch.cuda.synchronize()
    assert not bool(dV.float().abs().max() > 0) and not bool(dK.float().abs().max() > 0)


def test_deferred_is_closer_to_the_oracle_than_accumulating(dev):
    """The same gradients as the accumulating single-site backward, which
    rounds every source's partial sum to bf16 at each later site; the
    deferred pass rounds each gradient once, so its error against the oracle
    is the smaller one (relative L2 over all sources)."""
    mode, S, T, N, d, r = PROJECTED, 20, 20, 300, 512, 16
    p = make_host_problem(mode, S, N, d, r, dtype="bf16", seed=9)
    Qh = _queries(T, r, seed=10)
    dHh = _upstream(T, N, d, seed=11)
    V, K, Q, dH = to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Qh, dev), to_dev(dHh, dev)
    dV, dK, dq = deferred_reverse_pass(V, K, Q, dH, mode)
    aV = torch.zeros_like(V)
    aK = torch.zeros_like(K)
    aq = torch.zeros((T, r), device=dev)
    ws = torch.empty((lr.route_bwd_workspace_bytes(S, N, d, r, mode, V.dtype),),
                     dtype=torch.uint8, device=dev)
    for t in range(T, 0, -1):
        lr.route_bwd(V[:t], K[:t], Q[t - 1], dH[t - 1], mode, out=(aV[:t], aK[:t], aq[t - 1]),
                     workspace=ws, accumulate=True)
    torch.cuda.synchronize()
    rV, rK, rQ = oracle.route_all_bwd(p.V, p.K, Qh.astype(np.float64), dHh, mode, 1, r=r)

    def rel_l2(got, ref):
        return np.linalg.norm((got - ref).ravel()) / np.linalg.norm(ref.ravel())

    check_bf16_grown("deferred dV", to_host(dV), rV)
    assert rel_l2(to_host(dV), rV) < rel_l2(to_host(aV), rV)
    assert rel_l2(to_host(dK), rK) < rel_l2(to_host(aK), rK)
    check_dq("deferred dq", to_host(dq), rQ)
