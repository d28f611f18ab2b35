"""LR-AttnRes depth routing on MI355X (gfx950): Python binding.

Thin ctypes layer over the C ABI of ``liblrattnres.so`` (declared in
``include/lr_attnres.h``).  It only checks and marshals torch tensors
(device, dtype, contiguity) and passes their device pointers and the current
HIP stream; every step of the routing runs in the library's HIP kernels.
There is no fallback: without the built library every call raises.

Routing at one residual site (Sec. 3.2 of arXiv 2607.09694):
    kbar_i = RMSNorm(k_i), alpha_i = softmax_i(q . kbar_i), h = sum_i alpha_i o_i
with keys projected (separate K), sliced (last r coordinates of each value)
or full-rank (the value itself, r = d).
"""
from __future__ import annotations

import ctypes
import os

PROJECTED, SLICED, FULL = 0, 1, 2
MODES = {"projected": PROJECTED, "sliced": SLICED, "full": FULL}
_F32, _BF16 = 0, 1
_STATUS = {1: "EINVAL", 2: "EUNSUPPORTED", 3: "EHIP"}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblrattnres.so")
_lib = None


class RoutingError(RuntimeError):
    """A non-zero status from the C ABI; ``status`` holds its name."""

    def __init__(self, status: int, message: str):
        self.status = _STATUS.get(status, str(status))
        super().__init__(f"lr_attnres {self.status}: {message}")


def load_library(path: str | None = None) -> ctypes.CDLL:
    """Load the HIP routing library (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"HIP routing library not built: {path} is missing "
                           "(run paper_2607_09694_amd/build.py or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    vp, i64, i, f = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    lib.lr_attnres_route_fwd.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i, i, f, vp]
    lib.lr_attnres_route_fwd.restype = ctypes.c_int
    lib.lr_attnres_route_bwd_workspace_bytes.argtypes = [i64, i64, i64, i64, i, i]
    lib.lr_attnres_route_bwd_workspace_bytes.restype = ctypes.c_size_t
    lib.lr_attnres_route_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t,
                                         i64, i64, i64, i64, i, i, f, vp]
    lib.lr_attnres_route_bwd.restype = ctypes.c_int
    lib.lr_attnres_route_bwd_accumulate.argtypes = lib.lr_attnres_route_bwd.argtypes
    lib.lr_attnres_route_bwd_accumulate.restype = ctypes.c_int
    lib.lr_attnres_route_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64,
                                                 i, i, f, vp]
    lib.lr_attnres_route_bwd_noalloc.restype = ctypes.c_int
    lib.lr_attnres_block_route_fwd.argtypes = [vp, vp, vp, vp, vp, vp, i64, i, i64, i64, i64,
                                               i, i, f, vp]
    lib.lr_attnres_block_route_fwd.restype = ctypes.c_int
    lib.lr_attnres_block_route_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                               ctypes.c_size_t, i64, i64, i64, i64, i, i, f, vp]
    lib.lr_attnres_block_route_bwd.restype = ctypes.c_int
    lib.lr_attnres_block_route_fwd_bf16c.argtypes = [vp] * 8 + [i64, i, i, i64, i64, i64, i, f,
                                                                vp]
    lib.lr_attnres_block_route_fwd_bf16c.restype = ctypes.c_int
    lib.lr_attnres_block_inter_fwd.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64,
                                               i, f, vp]
    lib.lr_attnres_block_inter_fwd.restype = ctypes.c_int
    lib.lr_attnres_block_merge_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i, i64,
                                               i64, i64, i, i, f, vp]
    lib.lr_attnres_block_merge_fwd.restype = ctypes.c_int
    lib.lr_attnres_route_all_fwd.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64,
                                             i, i, f, vp]
    lib.lr_attnres_route_all_fwd.restype = ctypes.c_int
    lib.lr_attnres_route_bwd_deferred.argtypes = [vp] * 7 + [ctypes.c_size_t, i64, i64, i64, i64,
                                                             i, i, f, vp]
    lib.lr_attnres_route_bwd_deferred.restype = ctypes.c_int
    lib.lr_attnres_route_gather_bwd.argtypes = [vp, vp, i64, vp, vp, vp, i64, i64, vp, vp, i64, i64,
                                                i64, i64, i, i, f, vp]
    lib.lr_attnres_route_gather_bwd.restype = ctypes.c_int
    lib.lr_attnres_route_all_bwd_workspace_bytes.argtypes = [i64, i64, i64, i64, i64, i64, i, i]
    lib.lr_attnres_route_all_bwd_workspace_bytes.restype = ctypes.c_size_t
    lib.lr_attnres_route_all_bwd.argtypes = [vp] * 8 + [ctypes.c_size_t, i64, i64, i64, i64, i64,
                                                        i64, i, i, f, i, vp]
    lib.lr_attnres_route_all_bwd.restype = ctypes.c_int
    lib.lr_attnres_block_route_bwd_deferred.argtypes = [vp] * 13 + [ctypes.c_size_t, i64, i64,
                                                                    i64, i64, i, i, f, vp]
    lib.lr_attnres_block_route_bwd_deferred.restype = ctypes.c_int
    lib.lr_attnres_block_gather_bwd.argtypes = [vp, vp, i64, vp, vp, vp, i64, i64, vp, vp, i64,
                                                i64, i64, i, i, f, vp]
    lib.lr_attnres_block_gather_bwd.restype = ctypes.c_int
    lib.lr_attnres_route_state_fwd.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64,
                                               i, i, f, vp]
    lib.lr_attnres_route_state_fwd.restype = ctypes.c_int
    lib.lr_attnres_route_merge_fwd.argtypes = [vp, vp, vp, vp, i64, i64, i64, i, vp]
    lib.lr_attnres_route_merge_fwd.restype = ctypes.c_int
    lib.lr_attnres_route_neff.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i, i, f, vp]
    lib.lr_attnres_route_neff.restype = ctypes.c_int
    lib.lr_attnres_key_proj_fwd.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i, vp]
    lib.lr_attnres_key_proj_fwd.restype = ctypes.c_int
    lib.lr_attnres_key_proj_bwd_workspace_bytes.argtypes = [i64, i64, i64, i64, i]
    lib.lr_attnres_key_proj_bwd_workspace_bytes.restype = ctypes.c_size_t
    lib.lr_attnres_key_proj_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, i64,
                                            i64, i64, i64, i, vp]
    lib.lr_attnres_key_proj_bwd.restype = ctypes.c_int
    lib.lr_attnres_last_error.argtypes = []
    lib.lr_attnres_last_error.restype = ctypes.c_char_p
    lib.lr_attnres_abi_version.argtypes = []
    lib.lr_attnres_abi_version.restype = ctypes.c_int
    if path == LIB_PATH:
        _lib = lib
    return lib


def _check(lib, rc):
    if rc != 0:
        raise RoutingError(rc, lib.lr_attnres_last_error().decode())


def _mode(mode) -> int:
    return MODES[mode] if isinstance(mode, str) else int(mode)


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.bfloat16:
        return _BF16
    if t.dtype == torch.float32:
        return _F32
    raise TypeError(f"values must be bfloat16 or float32, got {t.dtype}")


def _dev(t, name, dtype=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(t):
    import torch

    return torch.cuda.current_stream(t.device).cuda_stream


def _shape(V, K, q, mode):
    if V.dim() != 3:
        raise ValueError("V must be [S, N, d]")
    S, N, d = V.shape
    r = K.shape[2] if mode == PROJECTED else q.shape[0]
    if q.dim() != 1 or q.shape[0] != r:
        raise ValueError(f"q must have shape ({r},)")
    if mode == PROJECTED and (K is None or K.dim() != 3 or tuple(K.shape[:2]) != (S, N)):
        raise ValueError("K must be [S, N, r] for projected keys")
    return S, N, d, r


def route_fwd(V, K, q, mode, eps: float = 1e-6, out=None):
    """h[n] = sum_i alpha_i V[i, n] (Eq. lr_attnres_output) on V's device.

    V [S,N,d] bf16/fp32; K [S,N,r] (projected) or None; q [r] fp32 (full-rank:
    r = d); returns H [N,d] in V's dtype (written into ``out`` if given).
    """
    import torch

    lib = load_library()
    mode = _mode(mode)
    S, N, d, r = _shape(V, K, q, mode)
    H = out if out is not None else torch.empty((N, d), dtype=V.dtype, device=V.device)
    rc = lib.lr_attnres_route_fwd(_dev(V, "V"), _dev(K, "K", V.dtype),
                                  _dev(q, "q", torch.float32), _dev(H, "H", V.dtype),
                                  S, N, d, r, mode, _dtype_code(V), float(eps), _stream(V))
    _check(lib, rc)
    return H


def route_state_fwd(V, K, q, mode, chunk: int, eps: float = 1e-6, out=None):
    """Online-softmax states of one site's routing over the sources cut into
    chunks of ``chunk`` (Sec. 3.5's merge form): returns (M [P,N], L [P,N],
    ACC [P,N,d]) fp32, P = ceil(S / chunk); ACC[p] / L[p] routes over chunk p.
    ``out`` = (M, L, ACC) writes into given tensors of those shapes.
    """
    import torch

    lib = load_library()
    mode = _mode(mode)
    S, N, d, r = _shape(V, K, q, mode)
    P = -(-S // int(chunk)) if chunk >= 1 else 1
    if out is not None:
        M, L, ACC = out
        if tuple(M.shape) != (P, N) or tuple(L.shape) != (P, N) or tuple(ACC.shape) != (P, N, d):
            raise ValueError(f"out must be ({P},{N}), ({P},{N}), ({P},{N},{d}) tensors")
    else:
        M = torch.empty((P, N), dtype=torch.float32, device=V.device)
        L = torch.empty((P, N), dtype=torch.float32, device=V.device)
        ACC = torch.empty((P, N, d), dtype=torch.float32, device=V.device)
    rc = lib.lr_attnres_route_state_fwd(_dev(V, "V"), _dev(K, "K", V.dtype),
                                        _dev(q, "q", torch.float32),
                                        _dev(M, "M", torch.float32), _dev(L, "L", torch.float32),
                                        _dev(ACC, "ACC", torch.float32), S, N, d, r, int(chunk), mode,
                                        _dtype_code(V), float(eps), _stream(V))
    _check(lib, rc)
    return M, L, ACC


def route_merge_fwd(M, L, ACC, dtype=None, out=None):
    """h from P online-softmax states (M, L [P,N], ACC [P,N,d] fp32): the
    routing over the union of their sources, in ``dtype`` (default bf16)."""
    import torch

    lib = load_library()
    if ACC.dim() != 3 or tuple(M.shape) != tuple(ACC.shape[:2]) or tuple(L.shape) != tuple(M.shape):
        raise ValueError("need M, L [P, N] and ACC [P, N, d]")
    P, N, d = ACC.shape
    if out is not None:
        dtype = out.dtype
    dtype = dtype or torch.bfloat16
    H = out if out is not None else torch.empty((N, d), dtype=dtype, device=ACC.device)
    code = _BF16 if dtype == torch.bfloat16 else _F32
    rc = lib.lr_attnres_route_merge_fwd(_dev(M, "M", torch.float32), _dev(L, "L", torch.float32),
                                        _dev(ACC, "ACC", torch.float32), _dev(H, "H", dtype),
                                        P, N, d, code, _stream(ACC))
    _check(lib, rc)
    return H


def route_neff(V, K, q, mode, eps: float = 1e-6, out=None):
    """N_eff[n] = exp(-sum alpha log alpha) of one site's routing weights
    (Sec. 4.5, Eq. effective_sources), from the keys alone; [N] fp32."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    S, N, d, r = _shape(V, K, q, mode)
    ne = out if out is not None else torch.empty((N,), dtype=torch.float32, device=V.device)
    rc = lib.lr_attnres_route_neff(_dev(V, "V"), _dev(K, "K", V.dtype),
                                   _dev(q, "q", torch.float32), _dev(ne, "neff", torch.float32),
                                   S, N, d, r, mode, _dtype_code(V), float(eps), _stream(V))
    _check(lib, rc)
    return ne


def route_all_fwd(V, K, Q, mode, first: int, eps: float = 1e-6, with_neff: bool = True,
                  out=None):
    """Every read site of a pass over the stack V in one call (Sec. 3.1):
    site j = 0..T-1 reads the first first+j sources with query Q[j].

    V [S,N,d] bf16/fp32; K [S,N,r] (projected) or None (sliced, full-rank);
    Q [T,r] fp32 (full-rank: r = d).  Returns (H [T,N,d] in V's dtype, neff
    [T,N] fp32 or None), neff per Eq. effective_sources.  ``out`` may supply
    (H, neff).  Problems outside the fused kernel run site by site inside
    the library.
    """
    import torch

    lib = load_library()
    mode = _mode(mode)
    if Q.dim() != 2:
        raise ValueError("Q must be [T, r]")
    S, N, d, r = _shape(V, K, Q[0], mode)
    T = Q.shape[0]
    if out is not None:
        H, neff = out
    else:
        H = torch.empty((T, N, d), dtype=V.dtype, device=V.device)
        neff = torch.empty((T, N), dtype=torch.float32, device=V.device) if with_neff else None
    rc = lib.lr_attnres_route_all_fwd(_dev(V, "V"), _dev(K, "K", V.dtype),
                                      _dev(Q, "Q", torch.float32), _dev(H, "H", V.dtype),
                                      _dev(neff, "neff", torch.float32), S, N, d, r, first, T,
                                      mode, _dtype_code(V), float(eps), _stream(V))
    _check(lib, rc)
    return H, neff


def route_bwd_deferred(V, K, q, dH, mode, coef, eps: float = 1e-6, dq=None, workspace=None):
    """One site of the full-source deferred reverse pass: writes the site's
    coefficients for its S sources into coef [S, 3, N] fp32 (alpha, ds/rho,
    ds s/(rho r)) and returns its dq [r] fp32.  V [S,N,d] and K (projected)
    are the site's prefix of the stacks."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    S, N, d, r = _shape(V, K, q, mode)
    if tuple(coef.shape) != (S, 3, N) or coef.dtype != torch.float32:
        raise ValueError("coef must be fp32 [S, 3, N]")
    if dq is None:
        dq = torch.empty((r,), dtype=torch.float32, device=V.device)
    code = _dtype_code(V)
    need = lib.lr_attnres_route_bwd_workspace_bytes(S, N, d, r, mode, code)
    if workspace is None:
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=V.device)
    rc = lib.lr_attnres_route_bwd_deferred(_dev(V, "V"), _dev(K, "K", V.dtype),
                                           _dev(q, "q", torch.float32), _dev(dH, "dH", V.dtype),
                                           _dev(coef, "coef", torch.float32),
                                           _dev(dq, "dq", torch.float32), _dev(workspace, "workspace"),
                                           workspace.numel(), S, N, d, r, mode, code, float(eps),
                                           _stream(V))
    _check(lib, rc)
    return dq


def route_gather_bwd(V, K, source: int, dHs, Q, coef, mode, eps: float = 1e-6, out=None):
    """Gradient of one source from the sites that read it (deferred reverse
    pass).  dHs [n_sites, N, d] and Q [n_sites, r] of those sites; coef a
    view whose row u is site u's [3, N] coefficients for this source (e.g.
    coefs[t0:, source] of a [T, S, 3, N] array).  Returns (dV [N, d],
    dK [N, r] or None)."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    if V.dim() != 3 or Q.dim() != 2 or dHs.dim() != 3:
        raise ValueError("V must be [S, N, d], Q [n_sites, r] and dHs [n_sites, N, d]")
    S, N, d = V.shape
    r = K.shape[2] if mode == PROJECTED else Q.shape[1]
    n_sites = dHs.shape[0]
    if Q.shape[0] != n_sites or Q.shape[1] != r or tuple(dHs.shape[1:]) != (N, d):
        raise ValueError("Q must be [n_sites, r] and dHs [n_sites, N, d]")
    if coef.dim() != 3 or tuple(coef.shape[1:]) != (3, N) or coef.shape[0] != n_sites:
        raise ValueError("coef must be [n_sites, 3, N]")
    if not coef.is_cuda or coef.dtype != torch.float32 or (
            n_sites > 0 and (coef.stride(1) != N or coef.stride(2) != 1)):
        raise ValueError("coef must be fp32 on the device, each site's 3 rows of N contiguous")
    if out is not None:
        dV, dK = out
    else:
        dV = torch.empty((N, d), dtype=V.dtype, device=V.device)
        dK = torch.empty((N, r), dtype=V.dtype, device=V.device) if mode == PROJECTED else None
    rc = lib.lr_attnres_route_gather_bwd(_dev(V, "V"), _dev(K, "K", V.dtype), source,
                                         _dev(dHs, "dHs", V.dtype), _dev(Q, "Q", torch.float32),
                                         coef.data_ptr(), coef.stride(0) if n_sites > 0 else 3 * N,
                                         n_sites,
                                         _dev(dV, "dV", V.dtype), _dev(dK, "dK", V.dtype),
                                         S, N, d, r, mode, _dtype_code(V), float(eps), _stream(V))
    _check(lib, rc)
    return dV, dK


def route_all_bwd(V, K, Q, dH, mode, first: int, eps: float = 1e-6, out=None,
                  workspace=None, accumulate: bool = False):
    """Gradients of every read site of a pass (the backward of route_all_fwd)
    for L = sum_j sum(dH[j] * H[j]).

    dH [T,N,d] in V's dtype.  Returns (dV [S,N,d], dK [S,N,r] or None,
    dQ [T,r] fp32 summed over the tokens); dV includes the key path for
    sliced keys.  ``out`` may supply (dV, dK, dQ); with ``accumulate`` the
    gradients are added into them.  ``workspace`` is a uint8 device buffer of
    at least route_all_bwd_workspace_bytes(...) bytes.
    """
    import torch

    lib = load_library()
    mode = _mode(mode)
    if Q.dim() != 2:
        raise ValueError("Q must be [T, r]")
    S, N, d, r = _shape(V, K, Q[0], mode)
    T = Q.shape[0]
    if dH.dim() != 3 or tuple(dH.shape) != (T, N, d):
        raise ValueError("dH must be [T, N, d]")
    if out is not None:
        dV, dK, dQ = out
    elif accumulate:
        raise ValueError("accumulate needs the out=(dV, dK, dQ) buffers to add into")
    else:
        dV = torch.empty_like(V)
        dK = torch.empty_like(K) if mode == PROJECTED else None
        dQ = torch.empty((T, r), dtype=torch.float32, device=V.device)
    code = _dtype_code(V)
    need = lib.lr_attnres_route_all_bwd_workspace_bytes(S, N, d, r, first, T, mode, code)
    if workspace is None:
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=V.device)
    rc = lib.lr_attnres_route_all_bwd(_dev(V, "V"), _dev(K, "K", V.dtype),
                                      _dev(Q, "Q", torch.float32), _dev(dH, "dH", V.dtype),
                                      _dev(dV, "dV", V.dtype), _dev(dK, "dK", V.dtype),
                                      _dev(dQ, "dQ", torch.float32), _dev(workspace, "workspace"),
                                      workspace.numel(), S, N, d, r, first, T, mode, code,
                                      float(eps), int(accumulate), _stream(V))
    _check(lib, rc)
    return dV, dK, dQ


def route_all_bwd_workspace_bytes(S, N, d, r, first, T, mode, dtype) -> int:
    """Workspace bytes of route_all_bwd (per-workgroup dQ partials)."""
    import torch

    code = _BF16 if dtype == torch.bfloat16 else _F32
    return load_library().lr_attnres_route_all_bwd_workspace_bytes(S, N, d, r, first, T,
                                                                   _mode(mode), code)


def key_proj_fwd(A, W, d: int, out=None):
    """[o_n; k_n] = [W^O; W^K] a_n (Sec. 3.3, Eq. fused_projection).

    A [N,m] bf16; W [d+r,m] bf16 (rows of W^O, then of W^K).  Returns
    (O [N,d] or None when d = 0, K [N,r] or None when r = 0); ``out`` may
    supply (O, K), e.g. planes of the value and key stacks.
    """
    import torch

    lib = load_library()
    if A.dim() != 2 or W.dim() != 2 or W.shape[1] != A.shape[1]:
        raise ValueError("A must be [N, m] and W [d + r, m]")
    N, m = A.shape
    r = W.shape[0] - d
    if d < 0 or r < 0:
        raise ValueError("0 <= d <= W.shape[0] required")
    if out is not None:
        O, K = out
    else:
        O = torch.empty((N, d), dtype=A.dtype, device=A.device) if d > 0 else None
        K = torch.empty((N, r), dtype=A.dtype, device=A.device) if r > 0 else None
    rc = lib.lr_attnres_key_proj_fwd(_dev(A, "A"), _dev(W, "W", A.dtype), _dev(O, "O", A.dtype),
                                     _dev(K, "K", A.dtype), N, m, d, r, _dtype_code(A),
                                     _stream(A))
    _check(lib, rc)
    return O, K


def key_proj_bwd(A, W, dO, dK, out=None, workspace=None):
    """Backward of [o_n; k_n] = [W^O; W^K] a_n (Sec. 3.3, Eq.
    fused_projection): dA = dO W^O + dK W^K and dW = [dO^T A; dK^T A].

    A [N,m] bf16; W [d+r,m] bf16; dO [N,d] or None (d = 0); dK [N,r] or
    None (r = 0), bf16.  Returns (dA [N,m] bf16, dW [d+r,m] fp32); ``out``
    may supply (dA, dW), ``workspace`` a uint8 device buffer of at least
    key_proj_bwd_workspace_bytes(...) bytes.
    """
    import torch

    lib = load_library()
    if A.dim() != 2 or W.dim() != 2 or W.shape[1] != A.shape[1]:
        raise ValueError("A must be [N, m] and W [d + r, m]")
    N, m = A.shape
    d = 0 if dO is None else dO.shape[1]
    r = 0 if dK is None else dK.shape[1]
    if W.shape[0] != d + r:
        raise ValueError("W must have d + r rows")
    for g, w, name in ((dO, d, "dO"), (dK, r, "dK")):
        if g is not None and (g.dim() != 2 or g.shape[0] != N or g.shape[1] != w):
            raise ValueError(f"{name} must be [N, {w}]")
    if out is not None:
        dA, dW = out
    else:
        dA = torch.empty((N, m), dtype=A.dtype, device=A.device)
        dW = torch.empty((d + r, m), dtype=torch.float32, device=A.device)
    code = _dtype_code(A)
    need = lib.lr_attnres_key_proj_bwd_workspace_bytes(N, m, d, r, code)
    if workspace is None:
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=A.device)
    rc = lib.lr_attnres_key_proj_bwd(_dev(A, "A"), _dev(W, "W", A.dtype), _dev(dO, "dO", A.dtype),
                                     _dev(dK, "dK", A.dtype), _dev(dA, "dA", A.dtype),
                                     _dev(dW, "dW", torch.float32), _dev(workspace, "workspace"),
                                     workspace.numel() * workspace.element_size(), N, m, d, r, code,
                                     _stream(A))
    _check(lib, rc)
    return dA, dW


def key_proj_bwd_workspace_bytes(N, m, d, r, dtype) -> int:
    """Workspace of key_proj_bwd: the fp32 partials of dW's token splits."""
    import torch

    code = _BF16 if dtype == torch.bfloat16 else _F32
    return load_library().lr_attnres_key_proj_bwd_workspace_bytes(N, m, d, r, code)


def route_bwd_workspace_bytes(S, N, d, r, mode, dtype) -> int:
    import torch

    code = _BF16 if dtype == torch.bfloat16 else _F32
    return load_library().lr_attnres_route_bwd_workspace_bytes(S, N, d, r, _mode(mode), code)


def route_bwd(V, K, q, dH, mode, eps: float = 1e-6, out=None, workspace=None,
              accumulate: bool = False):
    """Gradients (dV, dK, dq) of L = sum(dH * H) for the forward above.

    dV [S,N,d] includes the key path for sliced / full-rank keys; dK [S,N,r]
    for projected keys (else None); dq [r] fp32 summed over all tokens.
    ``out`` may supply (dV, dK, dq) buffers, ``workspace`` a uint8 device
    buffer of at least route_bwd_workspace_bytes(...) bytes.  With
    ``accumulate`` the gradients are added into ``out`` (required).
    """
    import torch

    lib = load_library()
    mode = _mode(mode)
    S, N, d, r = _shape(V, K, q, mode)
    if out is not None:
        dV, dK, dq = out
    elif accumulate:
        raise ValueError("accumulate needs the out=(dV, dK, dq) buffers to add into")
    else:
        dV = torch.empty_like(V)
        dK = torch.empty_like(K) if mode == PROJECTED else None
        dq = torch.empty((r,), dtype=torch.float32, device=V.device)
    code = _dtype_code(V)
    need = lib.lr_attnres_route_bwd_workspace_bytes(S, N, d, r, mode, code)
    if workspace is None:
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=V.device)
    fn = lib.lr_attnres_route_bwd_accumulate if accumulate else lib.lr_attnres_route_bwd
    rc = fn(_dev(V, "V"), _dev(K, "K", V.dtype),
            _dev(q, "q", torch.float32), _dev(dH, "dH", V.dtype),
            _dev(dV, "dV", V.dtype), _dev(dK, "dK", V.dtype),
            _dev(dq, "dq", torch.float32), _dev(workspace, "workspace"),
            workspace.numel(), S, N, d, r, mode, code, float(eps), _stream(V))
    _check(lib, rc)
    return dV, dK, dq


def route_bwd_noalloc(V, K, q, dH, mode, out, eps: float = 1e-6):
    """route_bwd into the caller's ``out`` = (dV, dK, dq) buffers with no
    workspace: the library keeps the dq partials in its own device array
    (at most 8 MiB of them; see lr_attnres_route_bwd_noalloc), so the call
    allocates nothing.  Calls that may overlap on one device race."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    S, N, d, r = _shape(V, K, q, mode)
    dV, dK, dq = out
    rc = lib.lr_attnres_route_bwd_noalloc(_dev(V, "V"), _dev(K, "K", V.dtype),
                                          _dev(q, "q", torch.float32), _dev(dH, "dH", V.dtype),
                                          _dev(dV, "dV", V.dtype), _dev(dK, "dK", V.dtype),
                                          _dev(dq, "dq", torch.float32), S, N, d, r, mode,
                                          _dtype_code(V), float(eps), _stream(V))
    _check(lib, rc)
    return dV, dK, dq


def block_route_fwd(B, KB, o_new, k_new, q, n_src: int, start: bool, mode, eps: float = 1e-6,
                    out=None):
    """One residual site of block-source routing (Sec. 3.1 Block AttnRes
    summaries with the low-rank keys of Sec. 3.2).

    B [>=n_src, N, d] fp32 summary slots (slot 0 = embedding); slot n_src-1
    becomes (0 if start else itself) + o_new.  KB [>=n_src, N, r] fp32 key
    summaries for projected keys (else None), updated with k_new.  o_new
    [N, d] and k_new [N, r] in the model dtype (bf16 / fp32); q [r] fp32.
    Returns H [N, d] in o_new's dtype.
    """
    import torch

    lib = load_library()
    mode = _mode(mode)
    if B.dtype != torch.float32 or (KB is not None and KB.dtype != torch.float32):
        raise TypeError("summary slots must be float32")
    if B.dim() != 3 or B.shape[0] < n_src:
        raise ValueError("B must be [>= n_src, N, d]")
    _, N, d = B.shape
    r = KB.shape[2] if mode == PROJECTED else q.shape[0]
    if tuple(o_new.shape) != (N, d):
        raise ValueError("o_new must be [N, d]")
    H = out if out is not None else torch.empty((N, d), dtype=o_new.dtype, device=B.device)
    rc = lib.lr_attnres_block_route_fwd(
        _dev(B, "B"), _dev(KB, "KB"), _dev(o_new, "o_new"), _dev(k_new, "k_new", o_new.dtype),
        _dev(q, "q", torch.float32), _dev(H, "H", o_new.dtype), int(n_src), int(bool(start)),
        N, d, r, mode, _dtype_code(o_new), float(eps), _stream(B))
    _check(lib, rc)
    return H


def block_route_fwd_bf16c(B, KB, BC, KBC, o_new, k_new, q, n_src: int, start: bool,
                          finish: bool, mode, eps: float = 1e-6, out=None):
    """block_route_fwd with the completed block summaries stored in bf16:
    slots 0..n_src-2 are read from BC [>=n_src, N, d] bf16 (KBC [>=n_src,
    N, r] bf16 for projected keys, else None); slot n_src-1 is updated in
    the fp32 B / KB as in block_route_fwd and, when ``finish`` (o_new is its
    block's last member, or the embedding), also rounded into BC / KBC.
    bf16 storage only.  Returns H [N, d] bf16."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    if B.dtype != torch.float32 or (KB is not None and KB.dtype != torch.float32):
        raise TypeError("summary slots must be float32")
    if B.dim() != 3 or B.shape[0] < n_src or BC.dim() != 3 or BC.shape[0] < n_src:
        raise ValueError("B and BC must be [>= n_src, N, d]")
    _, N, d = B.shape
    if tuple(BC.shape[1:]) != (N, d):
        raise ValueError("BC must match B's [N, d]")
    r = KB.shape[2] if mode == PROJECTED else q.shape[0]
    if tuple(o_new.shape) != (N, d):
        raise ValueError("o_new must be [N, d]")
    bf = torch.bfloat16
    H = out if out is not None else torch.empty((N, d), dtype=bf, device=B.device)
    rc = lib.lr_attnres_block_route_fwd_bf16c(
        _dev(B, "B"), _dev(KB, "KB"), _dev(BC, "BC", bf), _dev(KBC, "KBC", bf),
        _dev(o_new, "o_new", bf), _dev(k_new, "k_new", bf), _dev(q, "q", torch.float32),
        _dev(H, "H", bf), int(n_src), int(bool(start)), int(bool(finish)), N, d, r, mode,
        float(eps), _stream(B))
    _check(lib, rc)
    return H


def block_route_bwd(B, KB, dB, dKB, o_new, k_new, q, dH, n_src: int, mode, eps: float = 1e-6,
                    out=None, workspace=None):
    """One site of the block-source reverse pass (see lr_attnres_block_route_bwd).

    Adds the site's slot gradients into dB / dKB (fp32), removes o_new (and
    k_new) from slot n_src-1 of B / KB, and returns (dO, dK, dq): the
    gradient of o_new (= dB[n_src-1]), of k_new (projected keys, else None)
    and of this site's query.
    """
    import torch

    lib = load_library()
    mode = _mode(mode)
    _, N, d = B.shape
    r = KB.shape[2] if mode == PROJECTED else q.shape[0]
    if out is not None:
        dO, dK, dq = out
    else:
        dO = torch.empty((N, d), dtype=o_new.dtype, device=B.device)
        dK = (torch.empty((N, r), dtype=o_new.dtype, device=B.device)
              if mode == PROJECTED else None)
        dq = torch.empty((r,), dtype=torch.float32, device=B.device)
    # full-rank block keys run as sliced keys over the whole row
    wmode = SLICED if mode == FULL else mode
    need = lib.lr_attnres_route_bwd_workspace_bytes(n_src, N, d, r, wmode, _F32)
    if workspace is None:
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=B.device)
    rc = lib.lr_attnres_block_route_bwd(
        _dev(B, "B", torch.float32), _dev(KB, "KB", torch.float32),
        _dev(dB, "dB", torch.float32), _dev(dKB, "dKB", torch.float32),
        _dev(o_new, "o_new"), _dev(k_new, "k_new", o_new.dtype), _dev(q, "q", torch.float32),
        _dev(dH, "dH", o_new.dtype), _dev(dO, "dO", o_new.dtype), _dev(dK, "dK", o_new.dtype),
        _dev(dq, "dq", torch.float32), _dev(workspace, "workspace"), workspace.numel(),
        int(n_src), N, d, r, mode, _dtype_code(o_new), float(eps), _stream(B))
    _check(lib, rc)
    return dO, dK, dq


def block_route_bwd_deferred(B, KB, dP, dKP, coef, o_new, k_new, q, dH, n_src: int, mode,
                             eps: float = 1e-6, out=None, workspace=None):
    """One site of the deferred block reverse pass (see
    lr_attnres_block_route_bwd_deferred): dP / dKP (the running gradient of
    the block in progress) grow by this site's contribution, coef
    [n_src-1, 3, N] receives the completed slots' coefficients, and the
    member o_new retires with gradient dP.  Returns (dO, dK, dq)."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    _, N, d = B.shape
    r = KB.shape[2] if mode == PROJECTED else q.shape[0]
    if out is not None:
        dO, dK, dq = out
    else:
        dO = torch.empty((N, d), dtype=o_new.dtype, device=B.device)
        dK = (torch.empty((N, r), dtype=o_new.dtype, device=B.device)
              if mode == PROJECTED else None)
        dq = torch.empty((r,), dtype=torch.float32, device=B.device)
    wmode = SLICED if mode == FULL else mode
    need = lib.lr_attnres_route_bwd_workspace_bytes(n_src, N, d, r, wmode, _F32)
    if workspace is None:
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=B.device)
    rc = lib.lr_attnres_block_route_bwd_deferred(
        _dev(B, "B", torch.float32), _dev(KB, "KB", torch.float32),
        _dev(dP, "dP", torch.float32), _dev(dKP, "dKP", torch.float32),
        _dev(coef, "coef", torch.float32) if n_src > 1 else None,
        _dev(o_new, "o_new"), _dev(k_new, "k_new", o_new.dtype), _dev(q, "q", torch.float32),
        _dev(dH, "dH", o_new.dtype), _dev(dO, "dO", o_new.dtype), _dev(dK, "dK", o_new.dtype),
        _dev(dq, "dq", torch.float32), _dev(workspace, "workspace"), workspace.numel(),
        int(n_src), N, d, r, mode, _dtype_code(o_new), float(eps), _stream(B))
    _check(lib, rc)
    return dO, dK, dq


def block_gather_bwd(B, KB, slot: int, dHs, Q, coef, first: int, mode, eps: float = 1e-6,
                     out=None):
    """The gradient of completed slot `slot` from sites first..T-1 (0-based
    indices into dHs [T, N, d], Q [T, r] and coef [T, nslots, 3, N]), the
    sites that read it as completed (see lr_attnres_block_gather_bwd).
    Overwrites and returns (dP [N, d] fp32, dKP [N, r] fp32 or None)."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    _, N, d = B.shape
    T = dHs.shape[0]
    r = KB.shape[2] if mode == PROJECTED else Q.shape[1]
    n_sites = max(0, T - first)
    if out is not None:
        dP, dKP = out
    else:
        dP = torch.empty((N, d), dtype=torch.float32, device=B.device)
        dKP = (torch.empty((N, r), dtype=torch.float32, device=B.device)
               if mode == PROJECTED else None)
    for t, name in ((dHs, "dHs"), (Q, "Q"), (coef, "coef")):
        _dev(t, name)
    f0 = first if n_sites > 0 else 0
    rc = lib.lr_attnres_block_gather_bwd(
        _dev(B, "B", torch.float32), _dev(KB, "KB", torch.float32), int(slot),
        dHs[f0].data_ptr(), Q[f0].data_ptr(), coef[f0, slot].data_ptr(), coef.stride(0),
        n_sites, _dev(dP, "dP", torch.float32), _dev(dKP, "dKP", torch.float32), N, d, r, mode,
        _dtype_code(dHs), float(eps), _stream(B))
    _check(lib, rc)
    return dP, dKP


def block_inter_fwd(B, KB, Q, n_prev: int, mode, eps: float = 1e-6, out=None):
    """Phase 1 of the two-phase block inference (Sec. 3.5): for each query of
    Q [nq, r], the online-softmax state over the completed fp32 slots
    B[:n_prev] (KB[:n_prev] for projected keys).  Returns (M [nq, N],
    L [nq, N], ACC [nq, N, d]), fp32."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    _, N, d = B.shape
    nq, r = Q.shape
    if out is not None:
        M, L, ACC = out
    else:
        M = torch.empty((nq, N), dtype=torch.float32, device=B.device)
        L = torch.empty((nq, N), dtype=torch.float32, device=B.device)
        ACC = torch.empty((nq, N, d), dtype=torch.float32, device=B.device)
    rc = lib.lr_attnres_block_inter_fwd(
        _dev(B, "B", torch.float32), _dev(KB, "KB", torch.float32), _dev(Q, "Q", torch.float32),
        _dev(M, "M", torch.float32), _dev(L, "L", torch.float32), _dev(ACC, "ACC", torch.float32),
        int(n_prev), nq, N, d, r, mode, float(eps), _stream(B))
    _check(lib, rc)
    return M, L, ACC


def block_merge_fwd(B, KB, o_new, k_new, q, state, slot: int, start: bool, mode,
                    eps: float = 1e-6, out=None):
    """Phase 2 at one site: add o_new into slot `slot` (as block_route_fwd with
    n_src = slot + 1) and merge its score into the site's phase-1 state
    (M [N], L [N], ACC [N, d]; None when slot = 0).  Returns H [N, d]."""
    import torch

    lib = load_library()
    mode = _mode(mode)
    _, N, d = B.shape
    r = KB.shape[2] if mode == PROJECTED else q.shape[0]
    M, L, ACC = state if state is not None else (None, None, None)
    H = out if out is not None else torch.empty((N, d), dtype=o_new.dtype, device=B.device)
    rc = lib.lr_attnres_block_merge_fwd(
        _dev(B, "B", torch.float32), _dev(KB, "KB", torch.float32), _dev(o_new, "o_new"),
        _dev(k_new, "k_new", o_new.dtype), _dev(q, "q", torch.float32),
        _dev(M, "M", torch.float32), _dev(L, "L", torch.float32),
        _dev(ACC, "ACC", torch.float32), _dev(H, "H", o_new.dtype), int(slot), int(bool(start)),
        N, d, r, mode, _dtype_code(o_new), float(eps), _stream(B))
    _check(lib, rc)
    return H
