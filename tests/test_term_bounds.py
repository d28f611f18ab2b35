"""The cancelling cases of test_gpu_cancelling_passes.py, checked on the
CPU: each is the cancelling case it is meant to be (its rank-one key
gradient, or its dq over one to three tokens, is far below the size of its
terms, so that no normwise bar could hold), and the term magnitudes bound the
result itself (|ref| <= M, which any sum of those terms satisfies)."""
import numpy as np

from paper_2607_09694_amd.inputs import PROJECTED
from term_bounds import pass_magnitudes
from test_gpu_cancelling_passes import CASES, block_reference, host_inputs


def test_cases_cancel(orc):
    """The cases are the cancelling ones they are meant to be: in each, the
    largest rank-one key gradient (r = 1) or the largest dq (few tokens) is
    far below the size of its terms."""
    for mode, T, N, d, r, c in CASES:
        Oh, KOh, Qh, dHh = host_inputs(mode, T, N, d, r, seed=T * 7 + N + r)
        rO, rK, rq = block_reference(Oh, KOh, Qh, dHh, c, mode, r)
        MO, MK, Mq = pass_magnitudes(Oh, KOh, Qh, dHh, c, mode, r)
        if r == 1:
            grad, mag = (rK, MK) if mode == PROJECTED else (rO[..., -1:], MO[..., -1:])
        else:
            grad, mag = rq, Mq
        assert np.abs(grad).max() < 0.2 * mag.max(), (mode, T, N, d, r, c)
        assert (np.abs(rO) <= MO * (1 + 1e-9)).all() and (np.abs(rq) <= Mq * (1 + 1e-9)).all()
        if rK is not None:
            assert (np.abs(rK) <= MK * (1 + 1e-9)).all()
