"""ctypes front end of the fp64 CPU oracle (``lr_attnres_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the test suite, by the smoke check and
by the CPU-baseline leg of the benchmark.  The product library never imports
it.  Arrays are numpy; bf16 data is passed as its raw ``uint16`` bits, exactly
the bytes the GPU consumes.

Every function follows Section 3 of the paper (Eqs. lr_key_norm,
lr_attnres_weight, lr_attnres_output; sliced keys Eq. sliced_key; full-rank
AttnRes Eqs. attnres_weight / attnres_output).  The backward is derived in the
C file's header and pinned by finite differences in the tests.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lr_attnres_oracle.c")
LIB = os.path.join(HERE, "liblrattnres_oracle.so")

PROJECTED, SLICED, FULL = 0, 1, 2
_STORE = {np.dtype(np.float32): 0, np.dtype(np.uint16): 1, np.dtype(np.float64): 2}

_lib = None


def build() -> str:
    """Compile the oracle with gcc (no fast-math: IEEE double throughout)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
           SRC, "-o", LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        build()
    lib = ctypes.CDLL(LIB)
    vp, ll, i, d = ctypes.c_void_p, ctypes.c_longlong, ctypes.c_int, ctypes.c_double
    lib.orc_route_weights.argtypes = [vp, vp, vp, vp, ll, ll, ll, ll, i, i, d, ll, ll]
    lib.orc_route_fwd.argtypes = [vp, vp, vp, vp, ll, ll, ll, ll, i, i, d, ll, ll]
    lib.orc_route_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, ll, ll, ll, ll, i, i, d, ll, ll]
    for f in (lib.orc_route_weights, lib.orc_route_fwd, lib.orc_route_bwd):
        f.restype = ctypes.c_int
    lib.orc_num_threads.restype = ctypes.c_int
    lib.orc_set_num_threads.argtypes = [i]
    lib.orc_set_num_threads.restype = None
    lib.orc_block_num_sources.argtypes = [ll, ll]
    lib.orc_block_num_sources.restype = ll
    lib.orc_block_route_fwd.argtypes = [vp, vp, vp, vp, ll, ll, ll, ll, ll, i, i, d, ll, ll]
    lib.orc_block_route_fwd.restype = ctypes.c_int
    lib.orc_block_summaries.argtypes = [vp, vp, vp, vp, ll, ll, ll, ll, ll, i, i, ll, ll]
    lib.orc_block_summaries.restype = ctypes.c_int
    lib.orc_block_route_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, ll, ll, ll, ll, ll, i, i, d,
                                        ll, ll]
    lib.orc_block_route_bwd.restype = ctypes.c_int
    lib.orc_route_state.argtypes = [vp, vp, vp, vp, vp, vp, ll, ll, ll, ll, i, i, d, ll, ll]
    lib.orc_route_state.restype = ctypes.c_int
    lib.orc_effective_sources.argtypes = [vp, vp, vp, vp, ll, ll, ll, ll, i, i, d, ll, ll]
    lib.orc_effective_sources.restype = ctypes.c_int
    lib.orc_route_all_fwd.argtypes = [vp, vp, vp, vp, vp, ll, ll, ll, ll, ll, ll, i, i, d, ll,
                                      ll]
    lib.orc_route_all_fwd.restype = ctypes.c_int
    lib.orc_route_all_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, ll, ll, ll, ll, ll, ll, i, i,
                                      d, ll, ll]
    lib.orc_route_all_bwd.restype = ctypes.c_int
    lib.orc_key_projection.argtypes = [vp, vp, vp, vp, ll, ll, ll, ll, i, ll, ll]
    lib.orc_key_projection.restype = ctypes.c_int
    lib.orc_key_projection_bwd.argtypes = [vp, vp, vp, vp, vp, vp, ll, ll, ll, ll, i]
    lib.orc_key_projection_bwd.restype = ctypes.c_int
    _lib = lib
    return lib


def num_threads() -> int:
    return _load().orc_num_threads()


def set_num_threads(n: int) -> None:
    """Threads of the oracle's later parallel regions (timing only)."""
    _load().orc_set_num_threads(int(n))


def _eps(eps):
    """eps as the kernels receive it: an fp32 value, widened exactly."""
    return float(np.float32(eps))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _prep(V, K, q, mode, r):
    V = np.ascontiguousarray(V)
    if V.dtype not in _STORE:
        raise TypeError(f"oracle: unsupported value storage {V.dtype}")
    if V.ndim != 3:
        raise ValueError("oracle: V must be [S, N, d]")
    S, N, d = V.shape
    if mode == PROJECTED:
        K = np.ascontiguousarray(K)
        if K.dtype != V.dtype or K.shape[:2] != (S, N):
            raise ValueError("oracle: K must be [S, N, r] in V's storage")
        r = K.shape[2]
    else:
        if K is not None:
            raise ValueError("oracle: K is only used with projected keys")
        if mode == FULL:
            r = d
        elif r is None:
            raise ValueError("oracle: sliced keys need r")
    q = np.ascontiguousarray(np.asarray(q, dtype=np.float64))
    if q.shape != (r,):
        raise ValueError(f"oracle: q must have shape ({r},)")
    return V, K, q, S, N, d, r


def route_weights(V, K, q, mode, r=None, eps=1e-6, n0=0, n1=None):
    """alpha[n, i] (Eq. lr_attnres_weight) for tokens [n0, n1)."""
    V, K, q, S, N, d, r = _prep(V, K, q, mode, r)
    n1 = N if n1 is None else n1
    out = np.empty((n1 - n0, S), dtype=np.float64)
    rc = _load().orc_route_weights(_ptr(V), _ptr(K), _ptr(q), _ptr(out), S, N, d, r, mode,
                                   _STORE[V.dtype], _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid problem")
    return out


def route_fwd(V, K, q, mode, r=None, eps=1e-6, n0=0, n1=None):
    """H[n, :] = sum_i alpha_i V[i, n, :] (Eq. lr_attnres_output), fp64."""
    V, K, q, S, N, d, r = _prep(V, K, q, mode, r)
    n1 = N if n1 is None else n1
    out = np.empty((n1 - n0, d), dtype=np.float64)
    rc = _load().orc_route_fwd(_ptr(V), _ptr(K), _ptr(q), _ptr(out), S, N, d, r, mode,
                               _STORE[V.dtype], _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid problem")
    return out


def route_bwd(V, K, q, dH, mode, r=None, eps=1e-6, n0=0, n1=None):
    """(dV, dK, dq) of L = sum(dH * H) for tokens [n0, n1), fp64.

    dV is [S, n1-n0, d], dK is [S, n1-n0, r] (projected keys, else None),
    dq is [r] summed over the token range.
    """
    V, K, q, S, N, d, r = _prep(V, K, q, mode, r)
    dH = np.ascontiguousarray(dH)
    if dH.dtype != V.dtype or dH.shape != (N, d):
        raise ValueError("oracle: dH must be [N, d] in V's storage")
    n1 = N if n1 is None else n1
    nt = n1 - n0
    dV = np.empty((S, nt, d), dtype=np.float64)
    dK = np.empty((S, nt, r), dtype=np.float64) if mode == PROJECTED else None
    dq = np.empty((r,), dtype=np.float64)
    rc = _load().orc_route_bwd(_ptr(V), _ptr(K), _ptr(q), _ptr(dH), _ptr(dV), _ptr(dK),
                               _ptr(dq), S, N, d, r, mode, _STORE[V.dtype], _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid problem")
    return dV, dK, dq


def block_num_sources(t: int, c: int) -> int:
    """Sources read at site t with blocks of c outputs (Sec. 3.1 Block AttnRes)."""
    return _load().orc_block_num_sources(t, c)


def _block_prep(O, KO, t, mode, r):
    O = np.ascontiguousarray(O)
    if O.dtype not in _STORE or O.ndim != 3 or O.shape[0] < t:
        raise ValueError("oracle: O must be [>=t, N, d] in a supported storage")
    O = np.ascontiguousarray(O[:t])
    if mode == PROJECTED:
        KO = np.ascontiguousarray(np.ascontiguousarray(KO)[:t])
        r = KO.shape[2]
    elif r is None:
        raise ValueError("oracle: sliced keys need r")
    return O, KO, r


def block_route_fwd(O, KO, q, t, c, mode, r=None, eps=1e-6, n0=0, n1=None):
    """Block-source forward at site t (Sec. 3.1 Eqs. block_attnres_sum /
    block_attnres_partial_sum with the routing of Sec. 3.2).

    O [t, N, d] holds o_0 .. o_{t-1}; KO [t, N, r] their projected keys (or
    None for sliced keys).  Returns H [n1-n0, d] in fp64.
    """
    O, KO, r = _block_prep(O, KO, t, mode, r)
    _, N, d = O.shape
    q = np.ascontiguousarray(np.asarray(q, dtype=np.float64))
    n1 = N if n1 is None else n1
    out = np.empty((n1 - n0, d), dtype=np.float64)
    rc = _load().orc_block_route_fwd(_ptr(O), _ptr(KO if mode == PROJECTED else None), _ptr(q),
                                     _ptr(out), t, c, N, d, r, mode, _STORE[O.dtype],
                                     _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid block problem")
    return out


def block_summaries(O, KO, t, c, mode, r=None, n0=0, n1=None):
    """The block summaries site t reads (Sec. 3.1 Eqs. block_attnres_sum /
    block_attnres_partial_sum), exact in fp64: slot 0 the embedding, slot j
    the sum of block j's outputs written before site t.  Returns
    (B [S, n1-n0, d], KB [S, n1-n0, r] or None), S = block_num_sources(t, c);
    a projected summary's key is the sum of its members' keys."""
    O, KO, r = _block_prep(O, KO, t, mode, r)
    _, N, d = O.shape
    S = block_num_sources(t, c)
    n1 = N if n1 is None else n1
    B = np.empty((S, n1 - n0, d), dtype=np.float64)
    KB = np.empty((S, n1 - n0, r), dtype=np.float64) if mode == PROJECTED else None
    rc = _load().orc_block_summaries(_ptr(O), _ptr(KO if mode == PROJECTED else None), _ptr(B),
                                     _ptr(KB), t, c, N, d, r, mode, _STORE[O.dtype], n0, n1)
    if rc:
        raise ValueError("oracle: invalid block problem")
    return B, KB


def block_route_bwd(O, KO, q, dH, t, c, mode, r=None, eps=1e-6, n0=0, n1=None):
    """Gradients (dO, dKO, dq) of L = sum(dH * h_t) for the block-source
    forward at site t: every member of a block receives its summary's
    gradient.  dO [t, n1-n0, d], dKO [t, n1-n0, r] (projected, else None),
    dq [r] summed over the token range; all fp64."""
    O = np.ascontiguousarray(np.ascontiguousarray(O)[:t])
    _, N, d = O.shape
    if mode == PROJECTED:
        KO = np.ascontiguousarray(np.ascontiguousarray(KO)[:t])
        r = KO.shape[2]
    elif r is None:
        raise ValueError("oracle: sliced keys need r")
    dH = np.ascontiguousarray(dH)
    if dH.dtype != O.dtype or dH.shape != (N, d):
        raise ValueError("oracle: dH must be [N, d] in O's storage")
    q = np.ascontiguousarray(np.asarray(q, dtype=np.float64))
    n1 = N if n1 is None else n1
    nt = n1 - n0
    dO = np.empty((t, nt, d), dtype=np.float64)
    dKO = np.empty((t, nt, r), dtype=np.float64) if mode == PROJECTED else None
    dq = np.empty((r,), dtype=np.float64)
    rc = _load().orc_block_route_bwd(_ptr(O), _ptr(KO if mode == PROJECTED else None), _ptr(q),
                                     _ptr(dH), _ptr(dO), _ptr(dKO), _ptr(dq), t, c, N, d, r,
                                     mode, _STORE[O.dtype], _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid block problem")
    return dO, dKO, dq


def route_state(V, K, q, mode, r=None, eps=1e-6, n0=0, n1=None):
    """Online-softmax state (M, Lsum, ACC) of the routing over the sources of
    V (Sec. 3.5): M = max score, Lsum = sum exp(s - M), ACC = sum exp(s - M) o.
    Returns fp64 arrays [n1-n0], [n1-n0], [n1-n0, d]."""
    V, K, q, S, N, d, r = _prep(V, K, q, mode, r)
    n1 = N if n1 is None else n1
    M = np.empty((n1 - n0,), dtype=np.float64)
    L = np.empty((n1 - n0,), dtype=np.float64)
    A = np.empty((n1 - n0, d), dtype=np.float64)
    rc = _load().orc_route_state(_ptr(V), _ptr(K), _ptr(q), _ptr(M), _ptr(L), _ptr(A), S, N, d,
                                 r, mode, _STORE[V.dtype], _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid problem")
    return M, L, A


def effective_sources(V, K, q, mode, r=None, eps=1e-6, n0=0, n1=None):
    """N_eff[n] = exp(-sum_i alpha_i log alpha_i) of the routing over the
    sources of V (Sec. 4.5, Eq. effective_sources), fp64 [n1-n0]."""
    V, K, q, S, N, d, r = _prep(V, K, q, mode, r)
    n1 = N if n1 is None else n1
    out = np.empty((n1 - n0,), dtype=np.float64)
    rc = _load().orc_effective_sources(_ptr(V), _ptr(K), _ptr(q), _ptr(out), S, N, d, r, mode,
                                       _STORE[V.dtype], _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid problem")
    return out


def route_all_fwd(V, K, Q, mode, first, r=None, eps=1e-6, n0=0, n1=None):
    """Every site of a pass over one source stack (Sec. 3.1, Eq.
    full_attnres_source_set): site j = 0..T-1 reads the first first+j
    sources with query Q[j].  Returns (H [T, n1-n0, d], NEFF [T, n1-n0]),
    both fp64; NEFF per Eq. effective_sources."""
    Q = np.ascontiguousarray(np.asarray(Q, dtype=np.float64))
    if Q.ndim != 2:
        raise ValueError("oracle: Q must be [T, r]")
    T = Q.shape[0]
    V, K, _, S, N, d, r = _prep(V, K, Q[0], mode, r)
    if first < 1 or first + T - 1 > S:
        raise ValueError("oracle: sites need 1 <= first and first + T - 1 <= S")
    n1 = N if n1 is None else n1
    H = np.empty((T, n1 - n0, d), dtype=np.float64)
    NEFF = np.empty((T, n1 - n0), dtype=np.float64)
    rc = _load().orc_route_all_fwd(_ptr(V), _ptr(K), _ptr(Q), _ptr(H), _ptr(NEFF), S, N, d, r,
                                   first, T, mode, _STORE[V.dtype], _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid problem")
    return H, NEFF


def route_all_bwd(V, K, Q, dH, mode, first, r=None, eps=1e-6, n0=0, n1=None):
    """Gradient of route_all_fwd for the loss sum_j sum_n dH[j, n] . h_j[n]:
    the sum over sites of each site's single-site backward over its prefix.
    dH is [T, N, d] in the storage of V.  Returns (dV [S, n1-n0, d],
    dK [S, n1-n0, r] or None, dQ [T, r]), all fp64; dQ sums the token range."""
    Q = np.ascontiguousarray(np.asarray(Q, dtype=np.float64))
    if Q.ndim != 2:
        raise ValueError("oracle: Q must be [T, r]")
    T = Q.shape[0]
    V, K, _, S, N, d, r = _prep(V, K, Q[0], mode, r)
    if first < 1 or first + T - 1 > S:
        raise ValueError("oracle: sites need 1 <= first and first + T - 1 <= S")
    dH = np.ascontiguousarray(dH)
    if dH.dtype != V.dtype or dH.shape != (T, N, d):
        raise ValueError("oracle: dH must be [T, N, d] in the storage of V")
    n1 = N if n1 is None else n1
    dV = np.empty((S, n1 - n0, d), dtype=np.float64)
    dK = np.empty((S, n1 - n0, r), dtype=np.float64) if mode == PROJECTED else None
    dQ = np.empty((T, r), dtype=np.float64)
    rc = _load().orc_route_all_bwd(_ptr(V), _ptr(K), _ptr(Q), _ptr(dH), _ptr(dV), _ptr(dK),
                                   _ptr(dQ), S, N, d, r, first, T, mode, _STORE[V.dtype],
                                   _eps(eps), n0, n1)
    if rc:
        raise ValueError("oracle: invalid problem")
    return dV, dK, dQ


def key_projection(A, W, d, n0=0, n1=None):
    """[o_n; k_n] = [W^O; W^K] a_n (Sec. 3.3, Eq. fused_projection) in fp64.

    A [N, m] activations, W [d + r, m] (rows of W^O, then of W^K), both in
    one storage.  Returns (O [n1-n0, d] or None when d = 0,
    K [n1-n0, r] or None when r = 0)."""
    A = np.ascontiguousarray(A)
    W = np.ascontiguousarray(W)
    if A.dtype not in _STORE or W.dtype != A.dtype or A.ndim != 2 or W.ndim != 2:
        raise ValueError("oracle: A [N, m] and W [d + r, m] in one supported storage")
    N, m = A.shape
    if W.shape[1] != m or not 0 <= d <= W.shape[0]:
        raise ValueError("oracle: W must be [d + r, m] with 0 <= d <= d + r")
    r = W.shape[0] - d
    n1 = N if n1 is None else n1
    O = np.empty((n1 - n0, d), dtype=np.float64) if d > 0 else None
    K = np.empty((n1 - n0, r), dtype=np.float64) if r > 0 else None
    rc = _load().orc_key_projection(_ptr(A), _ptr(W), _ptr(O), _ptr(K), N, m, d, r,
                                    _STORE[A.dtype], n0, n1)
    if rc:
        raise ValueError("oracle: invalid projection")
    return O, K


def key_projection_bwd(A, W, dO, dK):
    """Backward of [o_n; k_n] = [W^O; W^K] a_n (Sec. 3.3, Eq.
    fused_projection) in fp64, by the chain rule through the linear map:
    dA = [dO, dK] W and dW = [dO, dK]^T A.

    A [N, m], W [d + r, m], dO [N, d] or None (d = 0), dK [N, r] or None
    (r = 0), all in one storage.  Returns (dA [N, m], dW [d + r, m])."""
    A = np.ascontiguousarray(A)
    W = np.ascontiguousarray(W)
    if A.dtype not in _STORE or W.dtype != A.dtype or A.ndim != 2 or W.ndim != 2:
        raise ValueError("oracle: A [N, m] and W [d + r, m] in one supported storage")
    N, m = A.shape
    d = 0 if dO is None else dO.shape[1]
    r = 0 if dK is None else dK.shape[1]
    if W.shape != (d + r, m):
        raise ValueError("oracle: W must be [d + r, m]")
    for g, w in ((dO, d), (dK, r)):
        if g is not None and (g.dtype != A.dtype or g.shape != (N, w)):
            raise ValueError("oracle: dO [N, d] and dK [N, r] in A's storage")
    dO = None if dO is None else np.ascontiguousarray(dO)
    dK = None if dK is None else np.ascontiguousarray(dK)
    dA = np.empty((N, m), dtype=np.float64)
    dW = np.empty((d + r, m), dtype=np.float64)
    rc = _load().orc_key_projection_bwd(_ptr(A), _ptr(W), _ptr(dO), _ptr(dK), _ptr(dA),
                                        _ptr(dW), N, m, d, r, _STORE[A.dtype])
    if rc:
        raise ValueError("oracle: invalid projection backward")
    return dA, dW
