"""Reverse passes whose fp32 gradients cancel, held to the error bound of
their terms (tests/term_bounds.py, parity.check_sum_by_terms) against the
fp64 oracle.

Two kinds of configuration cancel for any fp32 computation:
  - rank-one keys (r = 1): a normalised key is k / sqrt(k^2 + eps), about
    +-1, so the key gradient (ds/rho)(q - kbar s / r) is O(eps) while its
    terms are O(1) (Sec. 3.2 Eq. lr_key_norm);
  - one to three tokens: dq sums ds_i kbar_i over the tokens, and the ds of
    each token sum to zero (the softmax of Eq. lr_attnres_weight).
Each is run through the four reverse passes of a model: the accumulating
and the deferred pass over block sources (Sec. 3.1 Block AttnRes), and the
accumulating and the deferred pass over all earlier sources (Sec. 3.1 Eq.
full_attnres_source_set).  Every member's (source's) gradient and every
site's dq is checked, in fp32 storage."""
import numpy as np
import pytest

import oracle
import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import PROJECTED, SLICED, make_host_problem
from parity import check_sum_by_terms
from term_bounds import pass_magnitudes
from test_gpu_all_sites_bwd import to_dev, to_host
from test_gpu_block import drive_deferred_reverse_pass, drive_model_pass, site_args
from test_gpu_deferred_model import deferred_reverse_pass

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

# Per-term relative error budget: a product of a few fp32 factors, each
# with a few roundings (the weights' own error is a term of its own).
TERM_REL = 16 * 2.0 ** -24


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lr.load_library()
    return torch.device("cuda:0")


def host_inputs(mode, T, N, d, r, seed):
    p = make_host_problem(mode, T, N, d, r, dtype="f32", seed=seed)
    rng = np.random.default_rng(seed + 1)
    Q = (rng.standard_normal((T, r)) * 2.0 / np.sqrt(r)).astype(np.float32)
    dH = rng.standard_normal((T, N, d)).astype(np.float32)
    return p.V, p.K, Q, dH


def n_terms(T, d, r):
    """Longest fp32 sum: a d-long dot, T sources of r-long keys, T sites."""
    return d + T * (r + 2) + T


def check_by_terms(label, mode, got, ref, mags, n):
    (gO, gK, gq), (rO, rK, rq), (MO, MK, Mq) = got, ref, mags
    check_sum_by_terms(f"{label} dO", gO, rO, MO, n, TERM_REL)
    if mode == PROJECTED:
        check_sum_by_terms(f"{label} dK", gK, rK, MK, n, TERM_REL)
    check_sum_by_terms(f"{label} dq", gq, rq, Mq, n, TERM_REL)


# (mode, T, N, d, r, c): rank-one keys, then one, two and three tokens
CASES = [
    (PROJECTED, 10, 33, 128, 1, 3),
    (SLICED, 10, 33, 128, 1, 3),
    (PROJECTED, 13, 1, 256, 16, 4),
    (SLICED, 9, 2, 64, 8, 2),
    (PROJECTED, 7, 3, 512, 32, 1),
    (SLICED, 8, 1, 96, 1, 2),
]
IDS = ["{}-T{}-N{}-d{}-r{}-c{}".format("P" if c[0] == PROJECTED else "S", *c[1:]) for c in CASES]


def block_reference(O, KO, Q, dH, c, mode, r):
    T, N, d = O.shape
    rO = np.zeros((T, N, d))
    rK = np.zeros((T, N, r)) if mode == PROJECTED else None
    rq = np.zeros((T, r))
    for t in range(1, T + 1):
        gO, gK, gq = oracle.block_route_bwd(O, KO, Q[t - 1], dH[t - 1], t, c, mode, r=r)
        rO[:t] += gO
        if rK is not None:
            rK[:t] += gK
        rq[t - 1] = gq
    return rO, rK, rq


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_block_reverse_passes_within_term_bounds(dev, case):
    """The accumulating block reverse pass (fp32 slot gradients, one retire
    per site) and the deferred one (completed slots gathered once)."""
    mode, T, N, d, r, c = case
    Oh, KOh, Qh, dHh = host_inputs(mode, T, N, d, r, seed=T * 7 + N + r)
    ref = block_reference(Oh, KOh, Qh, dHh, c, mode, r)
    mags = pass_magnitudes(Oh, KOh, Qh, dHh, c, mode, r)
    n = n_terms(T, d, r)
    O, KO, Q, dHs = to_dev(Oh, dev), to_dev(KOh, dev), to_dev(Qh, dev), to_dev(dHh, dev)

    _, B, KB = drive_model_pass(dev, O, KO, Q, c, mode, [T])
    dB = torch.zeros_like(B)
    dKB = torch.zeros_like(KB) if KB is not None else None
    dO = torch.empty_like(O)
    dK = torch.empty_like(KO) if KO is not None else None
    dq = torch.empty((T, r), dtype=torch.float32, device=dev)
    for t in range(T, 0, -1):
        n_src, _ = site_args(t, c)
        lr.block_route_bwd(B, KB, dB, dKB, O[t - 1], KO[t - 1] if KO is not None else None,
                           Q[t - 1], dHs[t - 1], n_src, mode,
                           out=(dO[t - 1], dK[t - 1] if dK is not None else None, dq[t - 1]))
    torch.cuda.synchronize()
    check_by_terms("accumulating", mode, (to_host(dO), None if dK is None else to_host(dK),
                                          to_host(dq)), ref, mags, n)

    _, B, KB = drive_model_pass(dev, O, KO, Q, c, mode, [T])
    dO, dK, dq = drive_deferred_reverse_pass(dev, B, KB, O, KO, Q, dHs, c, mode)
    check_by_terms("deferred", mode, (to_host(dO), None if dK is None else to_host(dK),
                                      to_host(dq)), ref, mags, n)


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_full_source_reverse_passes_within_term_bounds(dev, case):
    """Site t reads sources 0 .. t-1: the pass as T accumulating single-site
    backward calls, and in deferred form (per-site coefficients, one gather
    per source)."""
    mode, T, N, d, r, _ = case
    Vh, Kh, Qh, dHh = host_inputs(mode, T, N, d, r, seed=T * 5 + N + r)
    rV, rK, rQ = oracle.route_all_bwd(Vh, Kh, Qh.astype(np.float64), dHh, mode, 1, r=r)
    mags = pass_magnitudes(Vh, Kh, Qh, dHh, 1, mode, r)
    n = n_terms(T, d, r)
    V, K, Q, dH = to_dev(Vh, dev), to_dev(Kh, dev), to_dev(Qh, dev), to_dev(dHh, dev)

    aV = torch.zeros_like(V)
    aK = torch.zeros_like(K) if K is not None else None
    aq = torch.zeros((T, r), dtype=torch.float32, device=dev)
    ws = torch.empty((max(16, lr.route_bwd_workspace_bytes(T, N, d, r, mode, V.dtype)),),
                     dtype=torch.uint8, device=dev)
    for t in range(T, 0, -1):
        lr.route_bwd(V[:t], K[:t] if K is not None else None, Q[t - 1], dH[t - 1], mode,
                     out=(aV[:t], aK[:t] if aK is not None else None, aq[t - 1]), workspace=ws,
                     accumulate=True)
    torch.cuda.synchronize()
    check_by_terms("accumulating", mode, (to_host(aV), None if aK is None else to_host(aK),
                                          to_host(aq)), (rV, rK, rQ), mags, n)

    dV, dK, dq = deferred_reverse_pass(V, K, Q, dH, mode)
    torch.cuda.synchronize()
    check_by_terms("deferred", mode, (to_host(dV), None if dK is None else to_host(dK),
                                      to_host(dq)), (rV, rK, rQ), mags, n)
