"""Pins of the oracle's all-sites backward: the gradient of every read site
of a pass (Sec. 3.1, Eq. full_attnres_source_set; Sec. 3.2) for the loss
L = sum_j sum_n dH[j, n] . h_j[n].

The paper states no backward.  The oracle forms it as the sum over sites of
the single-site backward over each site's prefix; these tests pin it against
fp64 central differences of the oracle's all-sites forward (so a prefix off
by one, a query taken from the wrong site or a dropped site fails), and
against closed forms of the value path.
"""
import itertools

import numpy as np
import pytest

from paper_2607_09694_amd.inputs import FULL, PROJECTED, SLICED

STEP = 1e-6


def _loss(orc, V, K, Q, dH, mode, first, r, eps):
    H, _ = orc.route_all_fwd(V, K, Q, mode, first, r=r, eps=eps)
    return float((H * dH).sum())


def _fd(orc, x, V, K, Q, dH, mode, first, r, eps):
    g = np.empty_like(x)
    for idx in np.ndindex(x.shape):
        saved = x[idx]
        x[idx] = saved + STEP
        lp = _loss(orc, V, K, Q, dH, mode, first, r, eps)
        x[idx] = saved - STEP
        lm = _loss(orc, V, K, Q, dH, mode, first, r, eps)
        x[idx] = saved
        g[idx] = (lp - lm) / (2 * STEP)
    return g


# (S, N, d, r, first, T)
SHAPES = [(3, 2, 4, 2, 1, 3), (5, 2, 6, 3, 2, 3), (4, 1, 5, 1, 3, 2), (6, 2, 4, 4, 1, 4)]
CASES = [(mode, *shape, eps) for mode, shape, eps in
         itertools.product([PROJECTED, SLICED, FULL], SHAPES, [0.0, 0.3])]


@pytest.mark.parametrize("mode,S,N,d,r,first,T,eps", CASES)
def test_all_sites_backward_matches_central_differences(orc, mode, S, N, d, r, first, T, eps):
    rng = np.random.default_rng(100 * S + 10 * first + T)
    if mode == FULL:
        r = d
    if mode == SLICED:
        r = min(r, d)
    V = rng.standard_normal((S, N, d))
    K = rng.standard_normal((S, N, r)) if mode == PROJECTED else None
    Q = rng.standard_normal((T, r)) * 1.5
    dH = rng.standard_normal((T, N, d))
    dV, dK, dQ = orc.route_all_bwd(V, K, Q, dH, mode, first, r=r, eps=eps)
    np.testing.assert_allclose(dV, _fd(orc, V, V, K, Q, dH, mode, first, r, eps),
                               rtol=1e-6, atol=1e-7)
    if mode == PROJECTED:
        np.testing.assert_allclose(dK, _fd(orc, K, V, K, Q, dH, mode, first, r, eps),
                                   rtol=1e-6, atol=1e-7)
    else:
        assert dK is None
    np.testing.assert_allclose(dQ, _fd(orc, Q, V, K, Q, dH, mode, first, r, eps),
                               rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("first,T", [(1, 6), (2, 4), (4, 3)])
def test_value_gradient_sums_to_every_sites_upstream(orc, first, T):
    """Projected keys: each site's weights sum to 1 and its value gradient is
    alpha_{j,i} dH_j, so sum_i dV[i, n] = sum_j dH[j, n]."""
    rng = np.random.default_rng(first + T)
    S, N, d, r = 7, 5, 6, 3
    V, K = rng.standard_normal((S, N, d)), rng.standard_normal((S, N, r))
    Q, dH = rng.standard_normal((T, r)), rng.standard_normal((T, N, d))
    dV, _, _ = orc.route_all_bwd(V, K, Q, dH, PROJECTED, first)
    np.testing.assert_allclose(dV.sum(axis=0), dH.sum(axis=0), rtol=0, atol=1e-13)


@pytest.mark.parametrize("first,T", [(1, 5), (3, 3)])
def test_zero_queries_spread_each_site_uniformly(orc, first, T):
    """Q = 0: site j weighs its first+j sources equally, so with projected keys
    dV[i] = sum over the sites j that read source i of dH[j] / (first + j)."""
    rng = np.random.default_rng(5)
    S, N, d, r = first + T - 1, 4, 5, 2
    V, K = rng.standard_normal((S, N, d)), rng.standard_normal((S, N, r))
    dH = rng.standard_normal((T, N, d))
    dV, _, _ = orc.route_all_bwd(V, K, np.zeros((T, r)), dH, PROJECTED, first)
    want = np.zeros_like(dV)
    for j in range(T):
        want[:first + j] += dH[j] / (first + j)
    np.testing.assert_allclose(dV, want, rtol=1e-14, atol=1e-15)


@pytest.mark.parametrize("mode", [PROJECTED, SLICED])
def test_sources_no_site_reads_get_no_gradient(orc, mode):
    """Sources at or past first + T - 1 are read by no site: exactly zero."""
    rng = np.random.default_rng(6)
    S, N, d, r, first, T = 9, 3, 8, 4, 2, 4
    V = rng.standard_normal((S, N, d))
    K = rng.standard_normal((S, N, r)) if mode == PROJECTED else None
    dV, dK, _ = orc.route_all_bwd(V, K, rng.standard_normal((T, r)),
                                  rng.standard_normal((T, N, d)), mode, first, r=r)
    assert not dV[first + T - 1:].any()
    assert (np.abs(dV[:first + T - 1]).max(axis=(1, 2)) > 0).all()
    if dK is not None:
        assert not dK[first + T - 1:].any()


def test_key_gradient_orthogonal_to_key_at_zero_eps(orc):
    """At eps = 0 every site's score is invariant to a key's scale, so each
    site's key gradient, and their sum, is orthogonal to the key."""
    rng = np.random.default_rng(9)
    S, N, d, r, first, T = 6, 4, 5, 4, 1, 6
    V, K = rng.standard_normal((S, N, d)), rng.standard_normal((S, N, r))
    Q, dH = rng.standard_normal((T, r)), rng.standard_normal((T, N, d))
    _, dK, _ = orc.route_all_bwd(V, K, Q, dH, PROJECTED, first, eps=0.0)
    dots = (dK[:S - 1] * K[:S - 1]).sum(axis=-1)
    np.testing.assert_allclose(dots, 0.0, atol=1e-12)
    assert np.abs(dK[:S - 1]).max() > 1e-3


@pytest.mark.parametrize("mode", [PROJECTED, SLICED, FULL])
def test_one_site_is_the_single_site_backward(orc, mode):
    """T = 1 is the single-site backward over the first `first` sources."""
    rng = np.random.default_rng(11)
    S, N, d, r, first = 5, 3, 6, 3, 4
    if mode == FULL:
        r = d
    V = rng.standard_normal((S, N, d))
    K = rng.standard_normal((S, N, r)) if mode == PROJECTED else None
    q, dH = rng.standard_normal(r), rng.standard_normal((N, d))
    dV, dK, dQ = orc.route_all_bwd(V, K, q[None], dH[None], mode, first, r=r)
    sV, sK, sq = orc.route_bwd(V[:first], None if K is None else K[:first], q, dH, mode, r=r)
    np.testing.assert_array_equal(dV[:first], sV)
    assert not dV[first:].any()
    if mode == PROJECTED:
        np.testing.assert_array_equal(dK[:first], sK)
    np.testing.assert_array_equal(dQ[0], sq)


def test_token_ranges_split_the_pass(orc):
    """Token ranges give the rows of the whole pass; dQ sums over the range."""
    rng = np.random.default_rng(12)
    S, N, d, r, first, T = 6, 7, 8, 2, 2, 5
    V, K = rng.standard_normal((S, N, d)), rng.standard_normal((S, N, r))
    Q, dH = rng.standard_normal((T, r)), rng.standard_normal((T, N, d))
    dV, dK, dQ = orc.route_all_bwd(V, K, Q, dH, PROJECTED, first)
    a = orc.route_all_bwd(V, K, Q, dH, PROJECTED, first, n0=0, n1=3)
    b = orc.route_all_bwd(V, K, Q, dH, PROJECTED, first, n0=3, n1=N)
    np.testing.assert_allclose(np.concatenate([a[0], b[0]], axis=1), dV, rtol=0, atol=1e-15)
    np.testing.assert_allclose(np.concatenate([a[1], b[1]], axis=1), dK, rtol=0, atol=1e-15)
    np.testing.assert_allclose(a[2] + b[2], dQ, rtol=1e-13, atol=1e-14)


def test_rejects_bad_sites_and_upstream(orc):
    V = np.zeros((4, 2, 8))
    with pytest.raises(ValueError):
        orc.route_all_bwd(V, None, np.zeros((4, 2)), np.zeros((4, 2, 8)), SLICED, 2, r=2)
    with pytest.raises(ValueError):
        orc.route_all_bwd(V, None, np.zeros((2, 2)), np.zeros((3, 2, 8)), SLICED, 1, r=2)
    with pytest.raises(ValueError):
        orc.route_all_bwd(V, None, np.zeros((2, 2)), np.zeros((2, 2, 8), dtype=np.float32),
                          SLICED, 1, r=2)
