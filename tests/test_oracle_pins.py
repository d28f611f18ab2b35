"""Pins of the fp64 oracle's forward against closed forms and invariants.

Each check is chosen so that a plausible slip in the oracle (sum instead of
mean in the RMSNorm, eps outside the root, head instead of tail slice, a sign
in the softmax, a transposed [S][N] layout, a dropped normalisation) fails at
least one of them.  Equations cited are those of Sec. 3 of the paper.
"""
import numpy as np
import pytest

import golden_fixtures
from paper_2607_09694_amd.inputs import (FULL, PROJECTED, SLICED, bf16_bits_from_f32,
                                         f32_from_bf16_bits, make_host_problem)

MODES = [PROJECTED, SLICED, FULL]


def _problem(mode, S, N, d, r, seed=0, dtype="f32", q_scale=1.0):
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=seed, q_scale=q_scale,
                          with_dH=True)
    return p


@pytest.mark.parametrize("fx", golden_fixtures.all_fixtures(), ids=lambda f: f["name"])
def test_hand_derived_worked_examples(orc, fx):
    """Hand-derived cases (tests/golden): exact q gives the derivation's numbers
    to fp64 rounding; q rounded to fp32 (as the library receives it) to 1e-6."""
    for store in (np.float64, np.float32):
        V = fx["V"].astype(store)
        K = None if fx["K"] is None else fx["K"].astype(store)
        r = fx["r"]
        for q, tol in ((fx["q"], 1e-12), (fx["q"].astype(np.float32), 1e-6)):
            H = orc.route_fwd(V, K, q, fx["mode"], r=r, eps=fx["eps"])
            a = orc.route_weights(V, K, q, fx["mode"], r=r, eps=fx["eps"])
            np.testing.assert_allclose(a, fx["alpha"], rtol=0, atol=tol)
            np.testing.assert_allclose(H, fx["H"], rtol=0, atol=tol * max(1.0, np.abs(fx["H"]).max()))


@pytest.mark.parametrize("mode", MODES)
def test_weights_are_a_distribution(orc, mode):
    """Eq. lr_attnres_weight: alpha is a softmax, so it sums to 1 and lies in (0, 1]."""
    p = _problem(mode, S=7, N=33, d=24, r=6, q_scale=3.0)
    a = orc.route_weights(p.V, p.K, p.q, mode, r=p.r)
    assert a.shape == (33, 7)
    np.testing.assert_allclose(a.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert (a > 0).all() and (a <= 1).all()


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_source_is_exact_copy(orc, mode, dtype):
    """S = 1: the softmax over one source is exactly 1, so h = o_0 bit for bit."""
    p = _problem(mode, S=1, N=19, d=40, r=8, dtype=dtype)
    H = orc.route_fwd(p.V, p.K, p.q, mode, r=p.r)
    V0 = p.V[0] if dtype == "f32" else f32_from_bf16_bits(p.V[0])
    assert np.array_equal(H, V0.astype(np.float64))


@pytest.mark.parametrize("mode", MODES)
def test_zero_query_gives_uniform_mean(orc, mode):
    """q = 0 (the paper's initialisation, Sec. 4.1): every score is 0 and h is
    the plain mean of the sources, i.e. the standard residual sum divided by S."""
    p = _problem(mode, S=5, N=11, d=16, r=4)
    q = np.zeros_like(p.q)
    H = orc.route_fwd(p.V, p.K, q, mode, r=p.r)
    np.testing.assert_allclose(H, p.V.astype(np.float64).mean(axis=0), rtol=0, atol=1e-14)


def test_equal_keys_give_uniform_mean(orc):
    """Identical keys for every source give identical scores and the mean."""
    p = _problem(PROJECTED, S=6, N=9, d=12, r=5, q_scale=4.0)
    K = np.repeat(p.K[:1], 6, axis=0)
    H = orc.route_fwd(p.V, K, p.q, PROJECTED)
    np.testing.assert_allclose(H, p.V.astype(np.float64).mean(axis=0), rtol=0, atol=1e-14)


def test_dominant_source_is_selected_per_token(orc):
    """A score gap of about 141 makes one source take all the weight (the rest
    is below e^-141).  The winning source differs per token, which pins the
    [S][N][d] layout of values and keys."""
    S, N, d, r = 5, 7, 6, 2
    rng = np.random.default_rng(3)
    V = rng.standard_normal((S, N, d))
    K = np.tile(np.array([-1.0, 0.0]), (S, N, 1))
    winners = [(3 * n + 1) % S for n in range(N)]
    for n, j in enumerate(winners):
        K[j, n] = [1.0, 0.0]
    q = np.array([50.0, 0.0])  # kbar = (+-sqrt 2, 0) -> scores +-70.7
    H = orc.route_fwd(V, K, q, PROJECTED, eps=0.0)
    for n, j in enumerate(winners):
        np.testing.assert_allclose(H[n], V[j, n], rtol=0, atol=1e-15)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sliced_with_full_rank_equals_attnres(orc, dtype):
    """Sec. 3.4: sliced keys with r = d reduce to full-rank AttnRes (fwd and bwd)."""
    p = _problem(SLICED, S=6, N=10, d=12, r=12, dtype=dtype)
    Hs = orc.route_fwd(p.V, None, p.q, SLICED, r=12)
    Hf = orc.route_fwd(p.V, None, p.q, FULL)
    assert np.array_equal(Hs, Hf)
    bs = orc.route_bwd(p.V, None, p.q, p.dH, SLICED, r=12)
    bf = orc.route_bwd(p.V, None, p.q, p.dH, FULL)
    assert np.array_equal(bs[0], bf[0]) and np.array_equal(bs[2], bf[2])


def test_projected_with_tail_copy_equals_sliced(orc):
    """A projected key that happens to equal tail_r(o_i) routes exactly like the
    sliced key (Eq. sliced_key); in the backward, the sliced dV carries the
    projected dK in its last r coordinates."""
    p = _problem(SLICED, S=4, N=8, d=10, r=3, q_scale=2.0)
    K = np.ascontiguousarray(p.V[:, :, -3:])
    Hs = orc.route_fwd(p.V, None, p.q, SLICED, r=3)
    Hp = orc.route_fwd(p.V, K, p.q, PROJECTED)
    assert np.array_equal(Hs, Hp)
    dVs, _, dqs = orc.route_bwd(p.V, None, p.q, p.dH, SLICED, r=3)
    dVp, dKp, dqp = orc.route_bwd(p.V, K, p.q, p.dH, PROJECTED)
    expect = dVp.copy()
    expect[:, :, -3:] += dKp
    np.testing.assert_allclose(dVs, expect, rtol=0, atol=1e-15)
    np.testing.assert_allclose(dqs, dqp, rtol=0, atol=1e-13)


def test_key_scale_invariance(orc):
    """Eq. lr_key_norm with eps = 0: RMSNorm(c k) = RMSNorm(k) for c > 0."""
    p = _problem(PROJECTED, S=5, N=6, d=8, r=4, q_scale=2.0)
    K = p.K.astype(np.float64)
    H1 = orc.route_fwd(p.V, K.astype(np.float32), p.q, PROJECTED, eps=0.0)
    H2 = orc.route_fwd(p.V, (K * 8.0).astype(np.float32), p.q, PROJECTED, eps=0.0)
    np.testing.assert_allclose(H1, H2, rtol=0, atol=1e-14)
    # With eps > 0 the scale matters (pins that eps is used at all).
    H3 = orc.route_fwd(p.V, (K * 0.01).astype(np.float32), p.q, PROJECTED, eps=1e-2)
    assert np.abs(H3 - H1).max() > 1e-3


@pytest.mark.parametrize("mode", MODES)
def test_source_permutation_equivariance(orc, mode):
    """The source set is a set (Eq. lr_attnres_output): permuting the sources
    jointly (values and keys) leaves h unchanged."""
    p = _problem(mode, S=6, N=7, d=9, r=3, q_scale=2.0)
    perm = np.array([4, 0, 5, 2, 1, 3])
    K2 = None if p.K is None else np.ascontiguousarray(p.K[perm])
    H1 = orc.route_fwd(p.V, p.K, p.q, mode, r=p.r)
    H2 = orc.route_fwd(np.ascontiguousarray(p.V[perm]), K2, p.q, mode, r=p.r)
    np.testing.assert_allclose(H1, H2, rtol=0, atol=1e-13)


@pytest.mark.parametrize("mode", MODES)
def test_output_in_convex_hull(orc, mode):
    """h is a convex combination of the sources, coordinate by coordinate."""
    p = _problem(mode, S=5, N=13, d=11, r=4, q_scale=3.0)
    H = orc.route_fwd(p.V, p.K, p.q, mode, r=p.r)
    V = p.V.astype(np.float64)
    assert (H >= V.min(axis=0) - 1e-14).all() and (H <= V.max(axis=0) + 1e-14).all()


def test_linear_in_values_for_fixed_keys(orc):
    """Projected keys: h is linear in the values (Eq. lr_attnres_output)."""
    p1 = _problem(PROJECTED, S=4, N=5, d=6, r=3, seed=1)
    p2 = _problem(PROJECTED, S=4, N=5, d=6, r=3, seed=2)
    V1, V2 = p1.V.astype(np.float64), p2.V.astype(np.float64)
    H1 = orc.route_fwd(V1, p1.K.astype(np.float64), p1.q, PROJECTED)
    H2 = orc.route_fwd(V2, p1.K.astype(np.float64), p1.q, PROJECTED)
    H12 = orc.route_fwd(2.0 * V1 - 3.0 * V2, p1.K.astype(np.float64), p1.q, PROJECTED)
    np.testing.assert_allclose(H12, 2.0 * H1 - 3.0 * H2, rtol=0, atol=1e-13)


@pytest.mark.parametrize("mode", MODES)
def test_token_ranges_compose(orc, mode):
    """Tokens are independent: computing [n0, n1) pieces gives the same rows."""
    p = _problem(mode, S=3, N=20, d=8, r=4)
    H = orc.route_fwd(p.V, p.K, p.q, mode, r=p.r)
    parts = [orc.route_fwd(p.V, p.K, p.q, mode, r=p.r, n0=a, n1=b)
             for a, b in ((0, 7), (7, 8), (8, 20))]
    assert np.array_equal(H, np.concatenate(parts))
    dV, dK, dq = orc.route_bwd(p.V, p.K, p.q, p.dH, mode, r=p.r)
    dV2, _, dq2 = orc.route_bwd(p.V, p.K, p.q, p.dH, mode, r=p.r, n0=5, n1=12)
    assert np.array_equal(dV[:, 5:12], dV2)


def test_bf16_storage_is_widened_exactly(orc):
    """bf16 inputs are read exactly: the same (bf16-representable) numbers
    stored as bf16 and as fp32 give identical results."""
    p = _problem(SLICED, S=4, N=6, d=16, r=8, dtype="bf16", q_scale=2.0)
    Vf = f32_from_bf16_bits(p.V)
    assert np.array_equal(bf16_bits_from_f32(Vf), p.V)
    H16 = orc.route_fwd(p.V, None, p.q, SLICED, r=8)
    H32 = orc.route_fwd(Vf, None, p.q, SLICED, r=8)
    assert np.array_equal(H16, H32)


def test_rejects_invalid_problems(orc):
    p = _problem(SLICED, S=2, N=3, d=4, r=2)
    with pytest.raises(ValueError):
        orc.route_fwd(p.V, None, np.zeros(5), SLICED, r=5)  # r > d
    with pytest.raises(ValueError):
        orc.route_fwd(p.V, None, p.q, SLICED, r=2, n0=2, n1=9)
