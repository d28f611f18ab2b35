"""GPU parity of the all-sites backward (the gradient of every read site of
a pass over one source stack, in one call) through the C ABI, against the
fp64 oracle.

Small cases cover both low-rank key modes, one to four 16-site tiles (one
and two 32-site groups in the dV contraction), one to four 16-column key
tiles, ragged column slabs, a sliced-key tail that straddles two slabs, key
lengths that are not a multiple of 8, a single site, many tokens per
workgroup, accumulation and bitwise reruns.  The full-size cases run the
paper's model pass (49 sources, 48 sites reading 2..49 of them, d = 1024,
N = 16384) and compare sampled tokens; their dQ is checked against the sum
of the single-site backward over every site.
"""
import numpy as np
import pytest

import oracle
import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import (FULL, PROJECTED, SLICED, bf16_bits_from_f32,
                                         bf16_tensor_to_bits, f32_from_bf16_bits,
                                         make_host_problem)
from parity import check_bf16_grown, check_bf16_key_grad, check_dq, check_f32, check_sum_by_terms

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lr.load_library()
    return torch.device("cuda:0")


def to_dev(x, dev):
    if x is None:
        return None
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def to_host(t):
    if t.dtype == torch.bfloat16:
        return f32_from_bf16_bits(bf16_tensor_to_bits(t)).astype(np.float64)
    return t.detach().cpu().numpy().astype(np.float64)


def _queries(T, r, seed, scale=2.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, r)) * scale / np.sqrt(r)).astype(np.float32)


def _upstream(T, N, d, seed):
    rng = np.random.default_rng(seed)
    return bf16_bits_from_f32(rng.standard_normal((T, N, d)).astype(np.float32))


def _problem(mode, S, T, first, N, d, r, seed):
    p = make_host_problem(mode, S, N, d, r, dtype="bf16", seed=seed)
    return p, _queries(T, r, seed + 1), _upstream(T, N, d, seed + 2)


def _check(name_prefix, mode, got, ref):
    """dV is a sum over every site that reads a source, so it grows past
    |x| = 8, where the bf16 half-ulp alone exceeds 2e-2: the bar for grown
    sums.  With sliced keys its last r columns carry the key gradient and
    take the key-gradient bar, as dK does."""
    dV, dK, dQ = got
    rV, rK, rQ = ref
    gV = to_host(dV)
    if mode == SLICED:
        r = rQ.shape[1]
        check_bf16_grown(name_prefix + "dV", gV[..., :-r], rV[..., :-r])
        check_bf16_key_grad(name_prefix + "dV key columns", gV[..., -r:], rV[..., -r:])
    else:
        check_bf16_grown(name_prefix + "dV", gV, rV)
    if mode == PROJECTED:
        check_bf16_key_grad(name_prefix + "dK", to_host(dK), rK)
    else:
        assert dK is None
    if dQ is not None:
        check_dq(name_prefix + "dQ", to_host(dQ), rQ)


def oracle_dQ_all_tokens(V, K, Q, dH, mode, first, r, chunk=1024):
    """The oracle's dQ over every token of device tensors V, K, dH: token
    chunks of the oracle's all-sites backward, summed in fp64."""
    Vh = bf16_tensor_to_bits(V)
    Kh = bf16_tensor_to_bits(K) if K is not None else None
    dHh = bf16_tensor_to_bits(dH)
    Qh = Q.cpu().numpy().astype(np.float64)
    N = Vh.shape[1]
    total = np.zeros(Qh.shape)
    for n0 in range(0, N, chunk):
        _, _, part = oracle.route_all_bwd(Vh, Kh, Qh, dHh, mode, first, r=r, n0=n0,
                                          n1=min(N, n0 + chunk))
        total += part
    return total


# (mode, S, T, first, N, d, r)
CASES = [
    (PROJECTED, 9, 8, 1, 37, 256, 16),      # one site tile, one key tile, two slabs
    (SLICED, 20, 19, 2, 33, 200, 24),       # ragged slab; tail inside the last slab
    (SLICED, 12, 10, 3, 21, 136, 16),       # tail straddles the two slabs
    (PROJECTED, 49, 48, 1, 70, 1024, 16),   # the paper's sites: 3 tiles, 2 site groups
    (SLICED, 49, 48, 2, 40, 1024, 64),      # S-LR r = 64: 4 key tiles
    (PROJECTED, 64, 64, 1, 20, 64, 64),     # every limit: 4 site tiles, half a slab
    (PROJECTED, 10, 8, 3, 17, 96, 12),      # r % 8 != 0: keys read element by element
    (SLICED, 33, 30, 4, 26, 520, 32),       # group boundary, ragged slab, 2 key tiles
    (PROJECTED, 5, 1, 5, 9, 128, 8),        # a single site reading every source
    (SLICED, 12, 11, 1, 1100, 128, 16),     # several tokens per workgroup
    (PROJECTED, 8, 8, 1, 16, 2048, 32),     # the widest rows (16 slabs)
    (SLICED, 17, 16, 2, 13, 2048, 64),
    (SLICED, 64, 60, 2, 1100, 136, 40),     # 4 site tiles, several tokens per workgroup
]


def _ids(c):
    return "{}-S{}-T{}-f{}-N{}-d{}-r{}".format("P" if c[0] == PROJECTED else "S", *c[1:])


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_all_sites_backward_matches_oracle(dev, case):
    mode, S, T, first, N, d, r = case
    p, Q, dH = _problem(mode, S, T, first, N, d, r, seed=S + T + N)
    got = lr.route_all_bwd(to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Q, dev), to_dev(dH, dev),
                           mode, first)
    torch.cuda.synchronize()
    ref = oracle.route_all_bwd(p.V, p.K, Q.astype(np.float64), dH, mode, first, r=r)
    _check("", mode, got, ref)


@pytest.mark.parametrize("mode", [PROJECTED, SLICED])
def test_all_sites_backward_accumulates(dev, mode):
    """accumulate: the gradients are added to what dV, dK and dQ hold."""
    S, T, first, N, d, r = 14, 12, 2, 45, 264, 16
    p, Q, dH = _problem(mode, S, T, first, N, d, r, seed=31)
    V, K = to_dev(p.V, dev), to_dev(p.K, dev)
    rng = np.random.default_rng(32)
    dV0 = bf16_bits_from_f32(rng.standard_normal((S, N, d)).astype(np.float32))
    dK0 = bf16_bits_from_f32(rng.standard_normal((S, N, r)).astype(np.float32))
    dQ0 = rng.standard_normal((T, r)).astype(np.float32)
    out = (to_dev(dV0, dev), to_dev(dK0, dev) if mode == PROJECTED else None, to_dev(dQ0, dev))
    got = lr.route_all_bwd(V, K, to_dev(Q, dev), to_dev(dH, dev), mode, first, out=out,
                           accumulate=True)
    torch.cuda.synchronize()
    rV, rK, rQ = oracle.route_all_bwd(p.V, p.K, Q.astype(np.float64), dH, mode, first, r=r)
    ref = (rV + f32_from_bf16_bits(dV0), None if rK is None else rK + f32_from_bf16_bits(dK0),
           rQ + dQ0)
    _check("acc ", mode, got, ref)


def test_all_sites_backward_is_deterministic(dev):
    S, T, first, N, d, r = 49, 48, 1, 700, 256, 32
    p, Q, dH = _problem(PROJECTED, S, T, first, N, d, r, seed=41)
    args = (to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Q, dev), to_dev(dH, dev), PROJECTED, first)
    a = lr.route_all_bwd(*args)
    b = lr.route_all_bwd(*args)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y)


def test_sources_no_site_reads_get_zero(dev):
    """Sources at or past first + T - 1 receive exactly zero (overwrite)."""
    S, T, first, N, d, r = 20, 6, 3, 30, 128, 16
    p, Q, dH = _problem(PROJECTED, S, T, first, N, d, r, seed=51)
    dV, dK, _ = lr.route_all_bwd(to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Q, dev),
                                 to_dev(dH, dev), PROJECTED, first)
    torch.cuda.synchronize()
    assert not bool(dV[first + T - 1:].float().abs().max() > 0)
    assert not bool(dK[first + T - 1:].float().abs().max() > 0)


def test_empty_token_range(dev):
    """N = 0: nothing is launched over tokens; dQ is zero (overwrite) or
    unchanged (accumulate)."""
    V = torch.empty((4, 0, 64), dtype=torch.bfloat16, device=dev)
    dH = torch.empty((3, 0, 64), dtype=torch.bfloat16, device=dev)
    Q = torch.ones((3, 8), device=dev)
    _, _, dQ = lr.route_all_bwd(V, None, Q, dH, SLICED, 2)
    torch.cuda.synchronize()
    assert bool((dQ == 0).all())
    dQ1 = torch.full((3, 8), 2.5, device=dev)
    lr.route_all_bwd(V, None, Q, dH, SLICED, 2, out=(torch.empty_like(V), None, dQ1),
                     accumulate=True)
    torch.cuda.synchronize()
    assert bool((dQ1 == 2.5).all())


@pytest.mark.parametrize("mode,r", [(PROJECTED, 16), (SLICED, 64)], ids=["P-r16", "S-r64"])
def test_model_pass_full_size(dev, mode, r):
    """The paper's model (Sec. 4.1: d = 1024, 48 sub-layers plus the
    embedding) at N = 16384 tokens: sites 1..48 read 2..49 sources.  Sampled
    tokens against the oracle; dQ over all N tokens against the oracle
    (token chunks), and against the sum over sites of the single-site
    backward of each prefix."""
    S, T, first, N, d = 49, 48, 2, 16384, 1024
    g = torch.Generator(device=dev)
    g.manual_seed(7 + r)
    V = torch.randn((S, N, d), generator=g, device=dev).to(torch.bfloat16)
    K = torch.randn((S, N, r), generator=g, device=dev).to(torch.bfloat16) if mode == PROJECTED \
        else None
    Q = torch.randn((T, r), generator=g, device=dev) * (2.0 / r ** 0.5)
    dH = torch.randn((T, N, d), generator=g, device=dev).to(torch.bfloat16)
    dV, dK, dQ = lr.route_all_bwd(V, K, Q, dH, mode, first)
    torch.cuda.synchronize()
    toks = np.unique(np.concatenate([[0, 511, 512, N - 1],
                                     np.random.default_rng(r).integers(0, N, 12)]))
    idx = torch.as_tensor(toks, device=dev)
    Vs = bf16_tensor_to_bits(V[:, idx].contiguous())
    Ks = bf16_tensor_to_bits(K[:, idx].contiguous()) if K is not None else None
    dHs = bf16_tensor_to_bits(dH[:, idx].contiguous())
    Qh = Q.cpu().numpy().astype(np.float64)
    rV, rK, rQ = oracle.route_all_bwd(Vs, Ks, Qh, dHs, mode, first, r=r)
    # dQ sums over every token, which the sampled oracle does not see.
    _check("", mode, (dV[:, idx].contiguous(), dK[:, idx].contiguous() if K is not None else None,
                      None), (rV, rK, rQ))
    check_dq("dQ", to_host(dQ), oracle_dQ_all_tokens(V, K, Q, dH, mode, first, r))
    # dQ row j is site j's dq: the single-site backward over its prefix.
    ws = torch.empty((lr.route_bwd_workspace_bytes(S, N, d, r, mode, torch.bfloat16),),
                     dtype=torch.uint8, device=dev)
    sdV = torch.empty_like(V)
    sdK = torch.empty_like(K) if K is not None else None
    want = torch.empty_like(dQ)
    for j in range(T):
        s = first + j
        _, _, dq = lr.route_bwd(V[:s], K[:s] if K is not None else None, Q[j], dH[j], mode,
                                out=(sdV[:s], sdK[:s] if sdK is not None else None, want[j]),
                                workspace=ws)
    torch.cuda.synchronize()
    check_dq("dQ", to_host(dQ), to_host(want))


def test_cancelling_query_gradient_within_its_term_bound(dev):
    """dQ_j = sum over tokens and sources of (ds/rho) k: the ds of a token sum
    to zero, so with one-dimensional sliced keys (every normalised key is
    about +-1) the terms cancel several hundredfold.  The normwise bar does
    not apply there; the error is held to the bound of the terms instead:
    each product has the relative error of the hi + lo bf16 split of ds /
    rho (2^-16), and the sum is accumulated in fp32."""
    mode, S, T, first, N, d, r = SLICED, 25, 2, 24, 7, 16, 1
    p, Q, dH = _problem(mode, S, T, first, N, d, r, seed=S + T + N)
    got = lr.route_all_bwd(to_dev(p.V, dev), None, to_dev(Q, dev), to_dev(dH, dev), mode, first)
    torch.cuda.synchronize()
    ref = oracle.route_all_bwd(p.V, None, Q.astype(np.float64), dH, mode, first, r=r)
    # sum |(ds / rho) k| per site, from the oracle's weights and fp64 dots
    Vw = f32_from_bf16_bits(p.V).astype(np.float64)
    dHw = f32_from_bf16_bits(dH).astype(np.float64)
    abs_terms = np.zeros((T, r))
    for j in range(T):
        Sj = first + j
        a = oracle.route_weights(p.V[:Sj], None, Q[j], mode, r=r)          # [N, Sj]
        g = np.einsum("snd,nd->ns", Vw[:Sj], dHw[j])                       # [N, Sj]
        ds = a * (g - (a * g).sum(axis=1, keepdims=True))
        k = Vw[:Sj, :, d - r:]                                             # [Sj, N, r]
        rho = np.sqrt((k ** 2).mean(axis=2) + 1e-6)                        # [Sj, N]
        abs_terms[j] = np.abs(ds.T[:, :, None] * k / rho[:, :, None]).sum(axis=(0, 1))
    dQ = to_host(got[2])
    kappa = abs_terms.max() / np.abs(ref[2]).max()
    assert kappa > 100  # the case is the cancelling one it is meant to be
    check_sum_by_terms("dQ", dQ, ref[2], abs_terms, N * S, 2.0 ** -16)


def test_stack_beyond_2_31_elements(dev):
    """A stack of more than 2^31 elements (S = 64, N = 33000, d = 1024), so
    that plane offsets need 64 bits, through the all-sites forward and
    backward; sampled tokens, the last ones included, against the oracle,
    and dQ over all tokens."""
    mode, r = PROJECTED, 16
    S, T, first, N, d = 64, 48, 17, 33000, 1024
    assert S * N * d > 2 ** 31
    g = torch.Generator(device=dev)
    g.manual_seed(99)
    V = torch.empty((S, N, d), dtype=torch.bfloat16, device=dev)
    for i in range(S):
        V[i].copy_(torch.randn((N, d), generator=g, device=dev))
    K = torch.randn((S, N, r), generator=g, device=dev).to(torch.bfloat16)
    Q = torch.randn((T, r), generator=g, device=dev) * (2.0 / r ** 0.5)
    dH = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)
    for j in range(T):
        dH[j].copy_(torch.randn((N, d), generator=g, device=dev))
    H, ne = lr.route_all_fwd(V, K, Q, mode, first)
    dV, dK, dQ = lr.route_all_bwd(V, K, Q, dH, mode, first)
    torch.cuda.synchronize()
    toks = np.unique(np.concatenate([[0, N // 2, N - 2, N - 1],
                                     np.random.default_rng(3).integers(0, N, 8)]))
    idx = torch.as_tensor(toks, device=dev)
    Vs = bf16_tensor_to_bits(V[:, idx].contiguous())
    Ks = bf16_tensor_to_bits(K[:, idx].contiguous())
    dHs = bf16_tensor_to_bits(dH[:, idx].contiguous())
    Qh = Q.cpu().numpy().astype(np.float64)
    rH, rne = oracle.route_all_fwd(Vs, Ks, Qh, mode, first, r=r)
    check_bf16_grown("H", to_host(H[:, idx].contiguous()), rH)
    got_ne = ne[:, idx].contiguous().cpu().numpy()
    assert np.abs(got_ne - rne).max() <= 1e-5 * np.abs(rne).max()
    rV, rK, rQ = oracle.route_all_bwd(Vs, Ks, Qh, dHs, mode, first, r=r)
    # dQ sums over all N tokens: the oracle walks them in chunks.
    _check("", mode, (dV[:, idx].contiguous(), dK[:, idx].contiguous(), None), (rV, rK, rQ))
    del H, ne, dV, dK
    check_dq("dQ", to_host(dQ), oracle_dQ_all_tokens(V, K, Q, dH, mode, first, r))


# ---------------------------------------------------------------------------
# Site by site: full-rank keys, fp32 storage, and S, T or r above 64 (or
# d % 8 != 0) run as one accumulating single-site backward per site.  The
# running gradient of a source is rounded to the storage after every site
# that reads it, so the bf16 bar is the bound of those roundings: one
# half-ulp (2^-9 relative) of each running sum, with a factor 2 (2^-8), plus
# 1e-3 for the fp32 sums, floored at the value bar 2e-2.  fp32 storage keeps
# the fp32 bar (48 roundings of 2^-24 stay far below 1e-5).
# ---------------------------------------------------------------------------

def _host(t):
    if t.dtype == torch.bfloat16:
        return bf16_tensor_to_bits(t)
    return t.detach().contiguous().cpu().numpy()


def _widen(x):
    return f32_from_bf16_bits(x).astype(np.float64) if x.dtype == np.uint16 else \
        x.astype(np.float64)


def _sbs_problem(mode, dtype, S, T, first, N, d, r, seed):
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=seed)
    rng = np.random.default_rng(seed + 2)
    dH = rng.standard_normal((T, p.N, p.d)).astype(np.float32)
    if dtype == "bf16":
        dH = bf16_bits_from_f32(dH)
    return p, _queries(T, p.r, seed + 1), dH


def _site_parts(V, K, Q, dH, mode, first, r):
    """Each site's oracle gradient of its prefix, in site order."""
    return [oracle.route_bwd(V[:first + j], None if K is None else K[:first + j], Q[j], dH[j],
                             mode, r=r)
            for j in range(Q.shape[0])]


def _check_accumulated(name, dtype, got, parts, start):
    """got = start + parts[0] + parts[1] + ..., part j covering the first
    parts[j].shape[0] sources, rounded to the storage after each part."""
    P = start.astype(np.float64).copy()
    bsum = np.zeros_like(P)
    for G in parts:
        s = G.shape[0]
        P[:s] += G
        bsum[:s] += np.abs(P[:s])
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all()
    if dtype == "f32":
        check_f32(name, got, P)
        return
    bar = np.maximum(2e-2, 2.0 ** -8 * bsum + 1e-3)
    worst = (np.abs(got - P) / bar).max(initial=0.0)
    assert worst <= 1.0, f"{name}: max error / rounding bound {worst:.3f}"


def _check_site_by_site(mode, dtype, got, p, Q, dH, first, start=None):
    dV, dK, dQ = got
    Qh = Q.astype(np.float64)
    parts = _site_parts(p.V, p.K, Qh, dH, mode, first, p.r)
    S = p.V.shape[0]
    zV = np.zeros((S, p.N, p.d)) if start is None else start[0]
    _check_accumulated("dV", dtype, to_host(dV), [g[0] for g in parts], zV)
    if mode == PROJECTED:
        zK = np.zeros((S, p.N, p.r)) if start is None else start[1]
        _check_accumulated("dK", dtype, to_host(dK), [g[1] for g in parts], zK)
    else:
        assert dK is None
    rQ = np.stack([g[2] for g in parts]) + (0.0 if start is None else start[2])
    check_dq("dQ", to_host(dQ), rQ, tol=1e-5 if dtype == "f32" else 1e-4)


# (mode, storage, S, T, first, N, d, r)
SITE_BY_SITE = [
    (FULL, "bf16", 9, 8, 1, 21, 256, 256),
    (FULL, "f32", 7, 5, 2, 13, 136, 136),
    (PROJECTED, "f32", 12, 10, 2, 17, 264, 16),
    (SLICED, "f32", 20, 17, 3, 19, 200, 12),
    (SLICED, "bf16", 70, 6, 65, 9, 128, 16),     # S > 64
    (PROJECTED, "bf16", 10, 8, 2, 15, 128, 80),  # r > 64
    (SLICED, "bf16", 10, 9, 1, 11, 68, 8),       # d % 8 != 0
    (FULL, "bf16", 20, 6, 3, 600, 128, 128),     # sources 8..19 read by no site
]


def _sbs_ids(c):
    return "{}-{}-S{}-T{}-f{}-N{}-d{}-r{}".format({PROJECTED: "P", SLICED: "S", FULL: "F"}[c[0]],
                                                  *c[1:])


@pytest.mark.parametrize("case", SITE_BY_SITE, ids=_sbs_ids)
def test_all_sites_backward_site_by_site(dev, case):
    """The site-by-site path against the oracle's per-site gradients; a
    source no site reads gets exactly zero; dQ row j is bit for bit the
    single-site backward's dq of site j."""
    mode, dtype, S, T, first, N, d, r = case
    p, Q, dH = _sbs_problem(mode, dtype, S, T, first, N, d, r, seed=S + 3 * T + N)
    V, K, Qd, dHd = to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Q, dev), to_dev(dH, dev)
    got = lr.route_all_bwd(V, K, Qd, dHd, mode, first)
    torch.cuda.synchronize()
    _check_site_by_site(mode, dtype, got, p, Q, dH, first)
    last = first + T - 1
    if last < S:
        assert not bool(got[0][last:].float().abs().max() > 0)
    for j in sorted({0, T - 1}):
        s = first + j
        _, _, dq = lr.route_bwd(V[:s], None if K is None else K[:s], Qd[j].contiguous(), dHd[j],
                                mode)
        torch.cuda.synchronize()
        assert torch.equal(got[2][j], dq), f"dQ row {j}"


@pytest.mark.parametrize("mode,dtype", [(FULL, "bf16"), (PROJECTED, "f32")], ids=["F-bf16",
                                                                                 "P-f32"])
def test_all_sites_backward_site_by_site_accumulates(dev, mode, dtype):
    S, T, first, N, d, r = 11, 9, 2, 23, 136, 16
    p, Q, dH = _sbs_problem(mode, dtype, S, T, first, N, d, r, seed=61)
    rng = np.random.default_rng(62)
    dV0 = rng.standard_normal((S, N, p.d)).astype(np.float32)
    dK0 = rng.standard_normal((S, N, p.r)).astype(np.float32)
    dQ0 = rng.standard_normal((T, p.r)).astype(np.float32)
    if dtype == "bf16":
        dV0, dK0 = bf16_bits_from_f32(dV0), bf16_bits_from_f32(dK0)
    out = (to_dev(dV0, dev), to_dev(dK0, dev) if mode == PROJECTED else None, to_dev(dQ0, dev))
    got = lr.route_all_bwd(to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Q, dev), to_dev(dH, dev),
                           mode, first, out=out, accumulate=True)
    torch.cuda.synchronize()
    start = (_widen(dV0), _widen(dK0) if mode == PROJECTED else None, dQ0.astype(np.float64))
    _check_site_by_site(mode, dtype, got, p, Q, dH, first, start=start)


def test_all_sites_backward_site_by_site_overwrites(dev):
    """Overwrite mode clears what the outputs held before the sites add in
    (a kernel fill, no memset): a second call on dirty buffers matches the
    first bit for bit."""
    mode, S, T, first, N, d = FULL, 10, 7, 2, 40, 72
    p, Q, dH = _sbs_problem(mode, "bf16", S, T, first, N, d, d, seed=71)
    args = (to_dev(p.V, dev), None, to_dev(Q, dev), to_dev(dH, dev), mode, first)
    a = lr.route_all_bwd(*args)
    out = (torch.full_like(a[0], 3.0), None, torch.full_like(a[2], -7.0))
    b = lr.route_all_bwd(*args, out=out)
    torch.cuda.synchronize()
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert torch.equal(a[2], b[2])


def test_all_sites_backward_full_rank_model_pass_full_size(dev):
    """Full-rank keys at the paper's model pass (49 sources, 48 sites reading
    2..49, d = 1024, N = 16384), site by site: sampled tokens against the
    oracle's per-site gradients; dQ rows bit for bit the single-site
    backward's dq of their sites (whose full-size parity with the oracle the
    single-site tests hold)."""
    mode, S, T, first, N, d = FULL, 49, 48, 2, 16384, 1024
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    V = torch.empty((S, N, d), dtype=torch.bfloat16, device=dev)
    for i in range(S):
        V[i].copy_(torch.randn((N, d), generator=g, device=dev))
    Q = torch.randn((T, d), generator=g, device=dev) * (2.0 / d ** 0.5)
    dH = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)
    for j in range(T):
        dH[j].copy_(torch.randn((N, d), generator=g, device=dev))
    dV, _, dQ = lr.route_all_bwd(V, None, Q, dH, mode, first)
    torch.cuda.synchronize()
    toks = np.unique(np.concatenate([[0, N - 1], np.random.default_rng(4).integers(0, N, 8)]))
    idx = torch.as_tensor(toks, device=dev)
    Vs = _host(V[:, idx].contiguous())
    dHs = _host(dH[:, idx].contiguous())
    Qh = Q.cpu().numpy().astype(np.float64)
    parts = _site_parts(Vs, None, Qh, dHs, mode, first, d)
    _check_accumulated("dV", "bf16", to_host(dV[:, idx].contiguous()), [g[0] for g in parts],
                       np.zeros((S, len(toks), d)))
    del dV
    for j in (0, 23, 47):
        s = first + j
        _, _, dq = lr.route_bwd(V[:s], None, Q[j].contiguous(), dH[j], mode)
        torch.cuda.synchronize()
        assert torch.equal(dQ[j], dq), f"dQ row {j}"
