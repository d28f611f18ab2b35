"""The error bound of block routing over bf16-stored completed summaries
(tests/block_bounds.py) checked on the CPU: a numpy model of that storage
(fp32 member-order sums rounded once to bf16, h rounded to bf16) stays
within the bound around the exact oracle at every site, the copies at exact
rounding ties included, and the bound is not vacuous."""
import numpy as np
import pytest

import oracle
from block_bounds import routed_bound, summary_bounds, ulp_bf16
from paper_2607_09694_amd.inputs import (PROJECTED, SLICED, bf16_bits_from_f32,
                                         f32_from_bf16_bits, make_host_problem)


def stored_slots(Xf, t, c):
    """The storage model: per slot the fp32 sum of its members in order;
    every slot but the last rounded to bf16."""
    S = oracle.block_num_sources(t, c)
    out = []
    for j in range(S):
        idx = [0] if j == 0 else list(range((j - 1) * c + 1, min(j * c, t - 1) + 1))
        acc = Xf[idx[0]].astype(np.float32)
        for i in idx[1:]:
            acc = (acc + Xf[i]).astype(np.float32)
        if j < S - 1:
            acc = f32_from_bf16_bits(bf16_bits_from_f32(acc))
        out.append(acc.astype(np.float64))
    return np.stack(out)


@pytest.mark.parametrize("mode,T,N,d,r,c", [(PROJECTED, 13, 30, 64, 16, 3),
                                             (SLICED, 11, 20, 48, 10, 2),
                                             (SLICED, 16, 9, 40, 32, 5),
                                             (PROJECTED, 9, 12, 24, 7, 1)])
def test_storage_model_stays_within_the_bound(orc, mode, T, N, d, r, c):
    p = make_host_problem(mode, T, N, d, r, dtype="bf16", seed=T + c)
    Q = (np.random.default_rng(c).standard_normal((T, r)) * 2.0 / np.sqrt(r)).astype(np.float32)
    Of = f32_from_bf16_bits(p.V)
    Kf = None if p.K is None else f32_from_bf16_bits(p.K)
    for t in range(1, T + 1):
        B, KB, eB, eK = summary_bounds(p.V, p.K, t, c, mode, r)
        ref, bound = routed_bound(B, KB, eB, eK, Q[t - 1], mode, r)
        assert np.array_equal(ref, oracle.block_route_fwd(p.V, p.K, Q[t - 1], t, c, mode, r=r))
        Bs = stored_slots(Of, t, c)
        assert (np.abs(Bs - B) <= eB * (1 + 1e-12)).all()
        KBs = None
        if Kf is not None:
            KBs = stored_slots(Kf, t, c)
            assert (np.abs(KBs - KB) <= eK * (1 + 1e-12)).all()
        h = oracle.route_fwd(Bs, KBs, Q[t - 1].astype(np.float64), mode, r=r)
        h = f32_from_bf16_bits(bf16_bits_from_f32(h.astype(np.float32)))
        assert (np.abs(h - ref) <= bound).all(), t
        assert bound.max() < 0.25 * max(1.0, np.abs(ref).max())


def test_copy_bound_is_half_an_ulp_at_a_tie(orc):
    """1 + 2^-8 (two members, exact in fp32) is a bf16 tie: it rounds to 1,
    an error of exactly half an ulp, which the bound admits with equality."""
    O = bf16_bits_from_f32(np.array([[[0.5]], [[1.0]], [[2.0 ** -8]]], dtype=np.float32))
    B, _, eB, _ = summary_bounds(O, None, 3, 2, SLICED, 1, all_rounded=True)
    assert B[1, 0, 0] == 1.0 + 2.0 ** -8
    stored = f32_from_bf16_bits(bf16_bits_from_f32(np.float32(1.0 + 2.0 ** -8)))
    assert stored == 1.0
    assert abs(stored - B[1, 0, 0]) == 2.0 ** -8 == 0.5 * ulp_bf16(1.0)
    assert abs(stored - B[1, 0, 0]) <= eB[1, 0, 0] < 2.0 ** -8 * (1 + 1e-4)
