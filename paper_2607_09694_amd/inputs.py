"""Seeded synthetic inputs for the depth-routing workloads.

This module only draws random numbers and stores them; it holds none of the
routing arithmetic.  Both the GPU library's tests/benchmark and the CPU oracle
consume exactly the bytes produced here (bf16 data travels as its raw 16 bits).

Workload shapes follow the paper's experimental model (Sec. 4.1): d = 1024,
L = 24 blocks with two residual-writing sub-layers each plus the embedding, so
full routing reads at most 2L + 1 = 49 sources (Sec. 4.7), context 2048.  The
paper trains on Ultra-FineWeb; that data and the trained weights are not
available, so Gaussian tensors of the same shapes stand in for the cached
sub-layer outputs, keys and upstream gradients.  Pseudo-queries are drawn
~ N(0, 1/r) (full-rank: 1/d) so that scores have unit variance; the paper
initialises them to zero (Sec. 4.1), which is the uniform-mean special case
the tests cover separately.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

PROJECTED, SLICED, FULL = 0, 1, 2
MODE_NAMES = {PROJECTED: "projected", SLICED: "sliced", FULL: "full"}


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest even) and return the raw bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bits to fp32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass
class HostProblem:
    """One routing problem in host memory, in the storage the kernels read.

    V  [S, N, d]  float32 or uint16 (bf16 bits)
    K  [S, N, r]  same storage as V, projected keys only (else None)
    q  [r]        float32
    dH [N, d]     same storage as V (None unless requested)
    """
    mode: int
    S: int
    N: int
    d: int
    r: int
    dtype: str
    V: np.ndarray
    K: np.ndarray | None
    q: np.ndarray
    dH: np.ndarray | None


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_from_f32(x)
    raise ValueError(dtype)


def make_host_problem(mode: int, S: int, N: int, d: int, r: int, dtype: str = "bf16",
                      seed: int = 0, q_scale: float = 1.0, with_dH: bool = False,
                      value_std: float = 1.0) -> HostProblem:
    """Gaussian problem drawn with numpy PCG64(seed) in the order V, K, q, dH.

    Values and keys ~ N(0, value_std^2); q ~ N(0, q_scale^2 / r) (full-rank
    keys: r = d).  fp32 draws are rounded to bf16 when dtype is 'bf16'.
    """
    if mode == FULL:
        r = d
    rng = np.random.Generator(np.random.PCG64(seed))
    V = rng.standard_normal((S, N, d), dtype=np.float32) * np.float32(value_std)
    K = None
    if mode == PROJECTED:
        K = rng.standard_normal((S, N, r), dtype=np.float32) * np.float32(value_std)
    q = (rng.standard_normal((r,), dtype=np.float32)
         * np.float32(q_scale / np.sqrt(r))).astype(np.float32)
    dH = rng.standard_normal((N, d), dtype=np.float32) if with_dH else None
    return HostProblem(mode, S, N, d, r, dtype, _store(V, dtype),
                       None if K is None else _store(K, dtype), q,
                       None if dH is None else _store(dH, dtype))


# The five measured workloads.  Each entry names what it is; sizes in tokens
# (N), model width (d), key rank (r) and number of sources (S).
WORKLOADS = {
    "sliced_fp32_small": dict(mode=SLICED, dtype="f32", N=256, d=64, r=8, S=8),
    "projected_model_pass_d1024": dict(mode=PROJECTED, dtype="bf16", N=8 * 2048, d=1024, r=16,
                                        S_sites=list(range(1, 50))),
    "sliced_model_pass_d1024": dict(mode=SLICED, dtype="bf16", N=16384, d=1024,
                                    r_sweep=[8, 16, 32, 64], S_sites=list(range(1, 50))),
    "full_rank_s49_d1024": dict(mode=FULL, dtype="bf16", N=16384, d=1024, S=49),
    "projected_fwd_bwd_d2048": dict(mode=PROJECTED, dtype="bf16", N=4 * 4096, d=2048, r=32,
                                    S=64),
}


def make_device_problem(mode: int, S: int, N: int, d: int, r: int, device, seed: int = 0,
                        with_dH: bool = False, n_queries: int = 1):
    """Large bf16 problem drawn on the device with torch.Generator(seed).

    Draw order V, K, q (n_queries of them, one per residual site), dH; fp32
    normal draws rounded to bf16 by torch.  Returns a dict of device tensors:
    V [S,N,d] bf16, K [S,N,r] bf16 or None, q [n_queries, r] fp32, dH [N,d] bf16.
    """
    import torch

    if mode == FULL:
        r = d
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    V = torch.empty((S, N, d), dtype=torch.bfloat16, device=device)
    # Draw source by source so the fp32 staging buffer stays small.
    for i in range(S):
        V[i].copy_(torch.randn((N, d), generator=g, device=device, dtype=torch.float32))
    K = None
    if mode == PROJECTED:
        K = torch.randn((S, N, r), generator=g, device=device,
                        dtype=torch.float32).to(torch.bfloat16)
    q = torch.randn((n_queries, r), generator=g, device=device,
                    dtype=torch.float32) / float(np.sqrt(r))
    dH = None
    if with_dH:
        dH = torch.randn((N, d), generator=g, device=device,
                         dtype=torch.float32).to(torch.bfloat16)
    return dict(V=V, K=K, q=q, dH=dH)


def bf16_tensor_to_bits(t) -> np.ndarray:
    """Host copy of a bf16 torch tensor as raw uint16 bits (no rounding)."""
    import torch

    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
