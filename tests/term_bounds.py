"""Term magnitudes of the routing backward over a whole reverse pass, for
holding cancelling fp32 gradients to the error bound of their terms.

Where a gradient cancels (a rank-one key, whose gradient (ds/rho)(q - kbar
s / r) is O(eps); dq over one to three tokens, where the ds of each token sum
to zero), a normwise bar relative to the result cannot hold for any fp32
computation.  The bound that does hold is relative to the sizes of the terms
the result is computed from: |err| <= 2 (u_t + n 2^-24) M, M being the sum of
the absolute values of every product that enters the result, u_t a per-term
relative error and n the length of the longest fp32 sum (parity.
check_sum_by_terms).

This module computes M for every output of a reverse pass over block
sources (Sec. 3.1 Eqs. block_attnres_sum / block_attnres_partial_sum; blocks
of one output are full routing, Eq. full_attnres_source_set), from the exact
fp64 summaries and weights of the oracle.  Per site t, slot j and token n
(alpha the weights, b the summaries, k their keys):
  g_j = dH . b_j                  M_g = sum_c |dH_c b_jc|
  s_j = q . kbar_j                M_s = sum_e |q_e kbar_je|
  an fp32 weight has relative error of the order of u (M_s + max M_s + 1),
      which enters every product with a weight as E_a = alpha (M_s + max M_s + 1)
  ds_j = alpha_j (g_j - sum_l alpha_l g_l)
                                  M_ds = alpha_j (M_g + sum_l alpha_l M_g,l)
                                         + E_a,j (|g_j| + |gbar|) + alpha_j sum_l E_a,l |g_l|
  value path of slot j, column c: (alpha_j + E_a,j) |dH_c|
  key path, key column e: (M_ds + |ds|) / rho (|q_e| + |kbar_je| (M_s + |s|) / r)
                          + |ds| / rho (|q_e| + |kbar_je| |s| / r)
  dq_e of the site: sum_n sum_j (M_ds + 2 |ds|) |kbar_je|
A member's gradient adds its slot's terms over every site that reads it.
"""
import numpy as np

import oracle

U32 = 2.0 ** -24


def _f64(x):
    """Values of a host array in fp32 storage (or bf16 bits) as fp64."""
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def block_slot(i, c):
    return 0 if i == 0 else (i - 1) // c + 1


def pass_magnitudes(O, KO, Q, dH, c, mode, r, eps=1e-6):
    """Term magnitudes of a reverse pass whose site t (1-based) reads the
    block summaries of o_0 .. o_{t-1} with query Q[t-1] and upstream dH[t-1].
    Returns (M_dO [T, N, d], M_dK [T, N, r] or None, M_dq [T, r])."""
    T, N, d = O.shape
    eps32 = float(np.float32(eps))
    MdO = np.zeros((T, N, d))
    MdK = np.zeros((T, N, r)) if KO is not None else None
    Mdq = np.zeros((T, r))
    for t in range(1, T + 1):
        q = Q[t - 1].astype(np.float64)
        dh = _f64(dH[t - 1])                                        # [N, d]
        B, KB = oracle.block_summaries(O, KO, t, c, mode, r=r)      # [S, N, d]
        a = oracle.route_weights(B, KB, q, mode, r=r, eps=eps).T    # [S, N]
        keys = KB if KB is not None else B[:, :, d - r:]
        rho = np.sqrt((keys ** 2).mean(axis=2) + eps32)            # [S, N]
        kb = keys / rho[..., None]
        s = (kb * q).sum(axis=2)
        Ms = (np.abs(kb) * np.abs(q)).sum(axis=2)
        g = np.einsum("snd,nd->sn", B, dh)
        Mg = np.einsum("snd,nd->sn", np.abs(B), np.abs(dh))
        gb = (a * g).sum(axis=0)
        ds = a * (g - gb)
        Ea = a * (Ms + Ms.max(axis=0) + 1.0)
        Mds = (a * (Mg + (a * Mg).sum(axis=0)) + Ea * (np.abs(g) + np.abs(gb))
               + a * (Ea * np.abs(g)).sum(axis=0))
        Mv = (a + Ea)[..., None] * np.abs(dh)[None]                 # [S, N, d]
        coef = ((Mds + np.abs(ds)) / rho)[..., None]
        Mk = (coef * (np.abs(q) + np.abs(kb) * ((Ms + np.abs(s)) / r)[..., None])
              + (np.abs(ds) / rho)[..., None] * (np.abs(q) + np.abs(kb) * (np.abs(s) / r)[..., None]))
        Mdq[t - 1] = ((Mds + 2.0 * np.abs(ds))[..., None] * np.abs(kb)).sum(axis=(0, 1))
        if KB is None:
            Mv[:, :, d - r:] += Mk
        for i in range(t):
            j = block_slot(i, c)
            MdO[i] += Mv[j]
            if MdK is not None:
                MdK[i] += Mk[j]
    return MdO, MdK, Mdq
