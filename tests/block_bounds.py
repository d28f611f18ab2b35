"""Error bounds of block routing whose completed summaries are stored in
bf16 (the library's storage option for Sec. 3.1 Block AttnRes), against the
exact fp64 routing of the oracle.

Stored summary.  A completed slot holds the fp32 sum of its m members, in
member order, rounded once to bf16 (nearest even).  With u = 2^-24 and
g = (m - 1) u / (1 - (m - 1) u), the fp32 sum s' of the exact sum s obeys
|s' - s| <= g sum|o|, and the rounding adds at most half a bf16 ulp of the
larger of |s'| and the result, which is at most half an ulp of
(|s| + g sum|o|)(1 + 2^-8).  So

    |stored - s| <= e = ulp16((|s| + g A)(1 + 2^-8)) / 2 + g A,   A = sum|o|.

The slot a site's newest output joins is read from fp32 (e = g A).
Projected keys are summed and stored the same way; a sliced key is the tail
of its stored summary.

Routed output.  With stored summaries b_j + delta_j (|delta_j| <= e_j) and
keys k_j + kappa_j, the weights become alpha'_j and

    h' - h = sum_j alpha'_j delta_j + sum_j (alpha'_j - alpha_j)(b_j - h),

the second form because the weight changes sum to zero.  The first term is
at most max_j e_j per coordinate.  For the score s = q . k / rho with
rho = sqrt(|k|^2 / r + eps), |grad_k s| = |q - kbar s / r| / rho <= 2|q| / rho
(|kbar| <= sqrt(r), |s| <= |q| sqrt(r)), and rho is 1/sqrt(r)-Lipschitz in
k, so a key moved by kappa moves its score by at most
sigma_j = 2 |q| |kappa_j| / (rho_j - |kappa_j| / sqrt(r)).  A softmax whose
scores move by at most sigma scales every weight by a factor within
exp(+-2 sigma), so |alpha'_j - alpha_j| <= alpha_j (exp(2 sigma) - 1).
The kernel's own fp32 arithmetic and the bf16 rounding of h are added on
top: 2^-18 (1 + |q| sqrt(r)) to sigma and 2^-18 (sum alpha |b| + max|b|)
for the accumulation (both far above the fp32 rounding they cover), then
half a bf16 ulp of the result.
"""
import numpy as np

import oracle

U32 = 2.0 ** -24


def ulp_bf16(x):
    """Spacing of bf16 values at |x| (2^-133 at zero)."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    _, e = np.frexp(x)
    return np.where(x > 0, np.maximum(np.ldexp(1.0, e - 8), 2.0 ** -133), 2.0 ** -133)


def _gamma(k):
    k = np.asarray(k, dtype=np.float64)
    return k * U32 / (1.0 - k * U32)


def _abs_bits(x):
    """|x| of bf16 bits (the sign bit cleared); fp32 / fp64 through np.abs."""
    if x is None:
        return None
    return x & np.uint16(0x7FFF) if x.dtype == np.uint16 else np.abs(x)


def slot_members(t, c):
    """Members of each slot at site t: 1 for the embedding, then
    min(jc, t - 1) - (j - 1)c for block j."""
    S = oracle.block_num_sources(t, c)
    return np.array([1] + [min(j * c, t - 1) - (j - 1) * c for j in range(1, S)])


def summary_bounds(O, KO, t, c, mode, r, n0=0, n1=None, all_rounded=False):
    """Exact summaries (B, KB) of site t and elementwise bounds (eB, eK) on
    the error of the stored ones: every slot but the last rounded to bf16
    (all of them with all_rounded)."""
    B, KB = oracle.block_summaries(O, KO, t, c, mode, r=r, n0=n0, n1=n1)
    A, KA = oracle.block_summaries(_abs_bits(O), _abs_bits(KO), t, c, mode, r=r, n0=n0, n1=n1)
    g = _gamma(slot_members(t, c) - 1)[:, None, None]
    nround = B.shape[0] if all_rounded else B.shape[0] - 1

    def bound(X, XA):
        e = g * XA
        e[:nround] += 0.5 * ulp_bf16((np.abs(X[:nround]) + e[:nround]) * (1 + 2.0 ** -8))
        return e

    return B, KB, bound(B, A), None if KB is None else bound(KB, KA)


def routed_bound(B, KB, eB, eK, q, mode, r, eps=1e-6):
    """Elementwise bound on |h' - h| for the routing over summaries B (keys
    KB, or the tails of B) whose stored values are within eB (eK)."""
    q = np.asarray(q, dtype=np.float64)
    alpha = oracle.route_weights(B, KB, q, mode, r=r, eps=eps)       # [nt, S]
    H = oracle.route_fwd(B, KB, q, mode, r=r, eps=eps)               # [nt, d]
    keys = KB if KB is not None else B[:, :, -r:]
    kap = eK if eK is not None else eB[:, :, -r:]
    rho = np.sqrt((keys ** 2).mean(axis=2) + float(np.float32(eps)))  # [S, nt]
    kn = np.sqrt((kap ** 2).sum(axis=2))
    qn = np.linalg.norm(q)
    sigma = 2.0 * qn * kn / np.maximum(rho - kn / np.sqrt(r), 1e-300)
    sig = sigma.max(axis=0) + 2.0 ** -18 * (1.0 + qn * np.sqrt(r))   # [nt]
    spread = np.einsum("ns,snd->nd", alpha, np.abs(B - H[None]))
    mag = np.einsum("ns,snd->nd", alpha, np.abs(B)) + np.abs(B).max(axis=0)
    e = eB.max(axis=0) + np.expm1(2.0 * sig)[:, None] * spread + 2.0 ** -18 * mag
    return H, e + 0.5 * ulp_bf16((np.abs(H) + e) * (1 + 2.0 ** -8))
