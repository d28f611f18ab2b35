"""Pins of the oracle's online-softmax state (Sec. 3.5: the two-phase
inference merges inter-block and intra-block routing with an online-softmax
update)."""
import numpy as np
import pytest

from paper_2607_09694_amd.inputs import FULL, PROJECTED, SLICED, make_host_problem


@pytest.mark.parametrize("mode", [PROJECTED, SLICED, FULL])
def test_state_normalises_to_the_routing(orc, mode):
    p = make_host_problem(mode, 7, 9, 12, 4, dtype="f32", seed=1, q_scale=3.0)
    M, L, A = orc.route_state(p.V, p.K, p.q, mode, r=p.r)
    np.testing.assert_allclose(A / L[:, None], orc.route_fwd(p.V, p.K, p.q, mode, r=p.r),
                               rtol=0, atol=1e-14)
    a = orc.route_weights(p.V, p.K, p.q, mode, r=p.r)
    # the largest weight belongs to the maximum score: exp(0) / Lsum
    np.testing.assert_allclose(a.max(axis=1), 1.0 / L, rtol=1e-14, atol=0)
    assert (L >= 1.0).all()


@pytest.mark.parametrize("mode", [PROJECTED, SLICED])
@pytest.mark.parametrize("split", [1, 3, 6])
def test_merging_two_states_gives_the_whole_routing(orc, mode, split):
    """Route over sources [0, split) and [split, S) separately, merge the two
    states with the online-softmax update, and get the routing over all S."""
    p = make_host_problem(mode, 7, 11, 10, 5, dtype="f32", seed=split, q_scale=2.5)
    K1 = None if p.K is None else p.K[:split]
    K2 = None if p.K is None else p.K[split:]
    M1, L1, A1 = orc.route_state(np.ascontiguousarray(p.V[:split]), K1, p.q, mode, r=p.r)
    M2, L2, A2 = orc.route_state(np.ascontiguousarray(p.V[split:]), K2, p.q, mode, r=p.r)
    M = np.maximum(M1, M2)
    e1, e2 = np.exp(M1 - M), np.exp(M2 - M)
    H = (e1[:, None] * A1 + e2[:, None] * A2) / (e1 * L1 + e2 * L2)[:, None]
    np.testing.assert_allclose(H, orc.route_fwd(p.V, p.K, p.q, mode, r=p.r), rtol=0, atol=1e-14)
