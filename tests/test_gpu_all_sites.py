"""GPU parity of the all-sites forward (every read site of a pass over one
source stack in one call) and of its effective number of sources, through
the C ABI, against the fp64 oracle.

Small cases cover both storages, both low-rank key modes, one and several
16-site tiles, one and two 32-source groups, ragged column slabs, key
lengths that need padding and the limits (64 sources, 64 sites, r = 64).
The full-size cases run the paper's model pass (49 sources, sites reading
2..49 of them, d = 1024, N = 16384) and compare sampled tokens.
"""
import numpy as np
import pytest

import oracle
import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import (FULL, PROJECTED, SLICED, bf16_tensor_to_bits,
                                         f32_from_bf16_bits, make_device_problem,
                                         make_host_problem)
from parity import check_bf16_value, check_f32

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
        return f32_from_bf16_bits(bf16_tensor_to_bits(t))
    return t.detach().cpu().numpy()


def host_bits(t):
    if t.dtype == torch.bfloat16:
        return bf16_tensor_to_bits(t)
    return t.detach().contiguous().cpu().numpy()


def check_h(name, dtype, got, ref):
    (check_f32 if dtype == "f32" else check_bf16_value)(name, got, ref)


def check_neff(name, got, ref):
    check_f32(name, got, ref, tol=1e-5)


def _queries(T, r, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, r)) * scale / np.sqrt(r)).astype(np.float32)


# (mode, storage, S, T, first, N, d, r)
CASES = [
    (PROJECTED, "bf16", 49, 48, 2, 37, 256, 16),   # the paper's sites, 3 tiles, 2 groups
    (SLICED, "bf16", 49, 48, 2, 21, 1024, 64),     # full width, r = 64
    (PROJECTED, "f32", 8, 8, 1, 33, 64, 8),        # half a slab
    (SLICED, "f32", 20, 17, 4, 19, 200, 12),       # ragged slab, r padded to 32
    (PROJECTED, "bf16", 64, 64, 1, 9, 136, 64),    # every limit, 4 tiles
    (SLICED, "bf16", 33, 30, 4, 50, 520, 32),      # group boundary, ragged slab
    (PROJECTED, "bf16", 17, 5, 13, 12, 384, 20),   # few sites late in the stack
    (SLICED, "f32", 64, 49, 16, 7, 128, 64),       # fp32 at the limits
    (PROJECTED, "bf16", 1, 1, 1, 5, 8, 1),         # one source, one site
    # above 48 sites the workgroups are persistent and load the next token's
    # keys during the current token's mix: several tokens per workgroup
    (SLICED, "bf16", 64, 60, 2, 700, 136, 40),
    (PROJECTED, "bf16", 57, 55, 3, 530, 256, 16),
]


def _ids(c):
    return "{}-{}-S{}-T{}-f{}-N{}-d{}-r{}".format("P" if c[0] == PROJECTED else "S", *c[1:])


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_all_sites_match_oracle(dev, case):
    mode, dtype, S, T, first, N, d, r = case
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=11)
    Q = _queries(T, r, seed=12, scale=2.0)
    V, K = to_dev(p.V, dev), to_dev(p.K, dev)
    H, ne = lr.route_all_fwd(V, K, to_dev(Q, dev), mode, first)
    torch.cuda.synchronize()
    Hr, NEr = oracle.route_all_fwd(p.V, p.K, Q.astype(np.float64), mode, first, r=r)
    check_h("H", dtype, to_host(H), Hr)
    check_neff("neff", to_host(ne), NEr)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_all_sites_single_source_site_is_a_copy(dev, dtype):
    """first = 1: site 0 reads o_0 alone; its weight is exactly 1, so its
    state is o_0 bit for bit, and N_eff is 1."""
    p = make_host_problem(SLICED, 40, 23, 264, 16, dtype=dtype, seed=3)
    Q = _queries(40, 16, seed=4, scale=3.0)
    V = to_dev(p.V, dev)
    H, ne = lr.route_all_fwd(V, None, to_dev(Q, dev), SLICED, 1)
    torch.cuda.synchronize()
    assert np.array_equal(host_bits(H[0]), host_bits(V[0]))
    assert np.array_equal(to_host(ne[0]), np.ones(23, dtype=np.float32))


def test_all_sites_zero_queries_average_prefixes(dev):
    """Q = 0: site j is the mean of its first+j rows and N_eff = first + j."""
    S, T, first, N, d = 49, 48, 2, 13, 512
    p = make_host_problem(PROJECTED, S, N, d, 16, dtype="bf16", seed=5)
    V, K = to_dev(p.V, dev), to_dev(p.K, dev)
    H, ne = lr.route_all_fwd(V, K, torch.zeros((T, 16), device=dev), PROJECTED, first)
    torch.cuda.synchronize()
    Vh = f32_from_bf16_bits(p.V).astype(np.float64)
    ref = np.stack([Vh[:first + j].mean(axis=0) for j in range(T)])
    check_bf16_value("H", to_host(H), ref)
    want = np.repeat(np.arange(first, first + T, dtype=np.float64)[:, None], N, axis=1)
    check_neff("neff", to_host(ne), want)


def test_all_sites_unaligned_projected_keys(dev):
    """K only element-aligned (r % 8 == 0 but the tensor starts 2 bytes past a
    16-byte boundary): the scores read the keys element by element."""
    S, T, first, N, d, r = 12, 11, 2, 17, 256, 16
    p = make_host_problem(PROJECTED, S, N, d, r, dtype="bf16", seed=13)
    Q = _queries(T, r, seed=14, scale=2.0)
    flat = torch.empty((S * N * r + 1,), dtype=torch.bfloat16, device=dev)
    K = flat[1:].view(S, N, r)
    K.copy_(to_dev(p.K, dev))
    assert K.data_ptr() % 16 != 0
    H, ne = lr.route_all_fwd(to_dev(p.V, dev), K, to_dev(Q, dev), PROJECTED, first)
    torch.cuda.synchronize()
    Hr, NEr = oracle.route_all_fwd(p.V, p.K, Q.astype(np.float64), PROJECTED, first)
    check_bf16_value("H", to_host(H), Hr)
    check_neff("neff", to_host(ne), NEr)


def test_all_sites_without_neff_and_empty(dev):
    p = make_host_problem(SLICED, 10, 6, 64, 8, dtype="bf16", seed=6)
    Q = _queries(9, 8, seed=7)
    V = to_dev(p.V, dev)
    H, ne = lr.route_all_fwd(V, None, to_dev(Q, dev), SLICED, 2, with_neff=False)
    torch.cuda.synchronize()
    assert ne is None
    Hr, _ = oracle.route_all_fwd(p.V, None, Q.astype(np.float64), SLICED, 2, r=8)
    check_bf16_value("H", to_host(H), Hr)
    # N = 0: nothing to do, no launch.
    E = torch.empty((10, 0, 64), dtype=torch.bfloat16, device=dev)
    H0, ne0 = lr.route_all_fwd(E, None, to_dev(Q, dev), SLICED, 2)
    assert H0.shape == (9, 0, 64) and ne0.shape == (9, 0)


def test_all_sites_agree_with_per_site_routing(dev):
    """Each site of the all-sites call against the single-site forward on its
    prefix (both on the GPU): same routed state to the bf16 bar."""
    S, T, first, N, d, r = 49, 48, 2, 300, 1024, 16
    prob = make_device_problem(PROJECTED, S, N, d, r, dev, seed=8, n_queries=T)
    H, _ = lr.route_all_fwd(prob["V"], prob["K"], prob["q"], PROJECTED, first)
    for j in (0, 1, 15, 16, 31, 32, 47):
        s = first + j
        h = lr.route_fwd(prob["V"][:s], prob["K"][:s], prob["q"][j].contiguous(), PROJECTED)
        torch.cuda.synchronize()
        check_bf16_value(f"site {j}", to_host(H[j]), to_host(h).astype(np.float64))


# Problems the fused kernel does not take run site by site inside the
# library: (mode, storage, S, T, first, N, d, r).
SITE_BY_SITE = [
    (FULL, "bf16", 9, 8, 2, 13, 256, 256),     # full-rank keys
    (FULL, "f32", 12, 10, 3, 7, 200, 200),
    (FULL, "bf16", 1, 1, 1, 6, 64, 64),        # one source: a copy
    (SLICED, "bf16", 70, 8, 63, 9, 136, 16),   # S > 64
    (PROJECTED, "f32", 20, 5, 3, 11, 128, 80),  # r > 64
    (SLICED, "bf16", 10, 9, 2, 11, 68, 8),     # d % 8 != 0
    (PROJECTED, "bf16", 66, 65, 2, 5, 64, 8),  # T > 64
]


def _sbs_ids(c):
    return "{}-{}-S{}-T{}-f{}-N{}-d{}-r{}".format({PROJECTED: "P", SLICED: "S", FULL: "F"}[c[0]],
                                                  *c[1:])


@pytest.mark.parametrize("case", SITE_BY_SITE, ids=_sbs_ids)
def test_all_sites_site_by_site_match_oracle(dev, case):
    """Each site of the site-by-site path is the single-site forward of its
    prefix (bit for bit) and matches the oracle to the storage's bar."""
    mode, dtype, S, T, first, N, d, r = case
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=21)
    Q = _queries(T, r, seed=22, scale=2.0)
    V, K, Qd = to_dev(p.V, dev), to_dev(p.K, dev), to_dev(Q, dev)
    H, ne = lr.route_all_fwd(V, K, Qd, mode, first)
    torch.cuda.synchronize()
    Hr, NEr = oracle.route_all_fwd(p.V, p.K, Q.astype(np.float64), mode, first, r=r)
    check_h("H", dtype, to_host(H), Hr)
    check_neff("neff", to_host(ne), NEr)
    for j in sorted({0, T // 2, T - 1}):
        s = first + j
        h = lr.route_fwd(V[:s], None if K is None else K[:s], Qd[j].contiguous(), mode)
        torch.cuda.synchronize()
        assert np.array_equal(host_bits(H[j]), host_bits(h)), f"site {j}"


def test_all_sites_full_rank_model_pass_full_size(dev):
    """Full-rank keys at the paper's model pass (49 sources, sites reading
    2..49, d = 1024, N = 16384), site by site; sampled tokens against the
    oracle token by token."""
    S, T, first, N, d = 49, 48, 2, 16384, 1024
    prob = make_device_problem(FULL, S, N, d, d, dev, seed=0, n_queries=T)
    H, ne = lr.route_all_fwd(prob["V"], None, prob["q"], FULL, first)
    torch.cuda.synchronize()
    toks = np.unique(np.concatenate([[0, N - 1], np.random.default_rng(1).integers(0, N, 10)]))
    idx = torch.as_tensor(toks, device=dev)
    Vs = host_bits(prob["V"][:, idx].contiguous())
    Q = prob["q"].cpu().numpy().astype(np.float64)
    ref, ref_ne = oracle.route_all_fwd(Vs, None, Q, FULL, first, r=d)
    check_bf16_value("H", to_host(H[:, idx].contiguous()), ref)
    check_neff("neff", to_host(ne[:, idx].contiguous()), ref_ne)


def test_all_sites_rejected_outside_limits(dev):
    p = make_host_problem(PROJECTED, 4, 3, 64, 8, dtype="bf16", seed=9)
    V, K = to_dev(p.V, dev), to_dev(p.K, dev)
    with pytest.raises(lr.RoutingError):
        lr.route_all_fwd(V, K, torch.zeros((4, 8), device=dev), PROJECTED, 2)
    # site by site, the last site past the single-site forward's 1024 sources
    big = torch.zeros((1026, 2, 64), dtype=torch.bfloat16, device=dev)
    with pytest.raises(lr.RoutingError, match="site by site"):
        lr.route_all_fwd(big, None, torch.zeros((2, 8), device=dev), SLICED, 1025)
    wide = torch.zeros((2, 1, 8192), dtype=torch.bfloat16, device=dev)
    with pytest.raises(lr.RoutingError, match="site by site"):
        lr.route_all_fwd(wide, None, torch.zeros((1, 8192), device=dev), FULL, 1)


FULL_SIZE = [(PROJECTED, 16), (SLICED, 64)]


@pytest.mark.parametrize("mode,r", FULL_SIZE, ids=["P-r16", "S-r64"])
def test_all_sites_model_pass_full_size(dev, mode, r):
    """The paper's model pass (49 sources, sites reading 2..49, d = 1024,
    N = 16384) in the benchmark's launch configuration; sampled tokens
    against the oracle token by token, every site."""
    S, T, first, N, d = 49, 48, 2, 16384, 1024
    prob = make_device_problem(mode, S, N, d, r, dev, seed=0, n_queries=T)
    H, ne = lr.route_all_fwd(prob["V"], prob["K"], prob["q"], mode, first)
    torch.cuda.synchronize()
    Vb = host_bits(prob["V"])
    Kb = None if prob["K"] is None else host_bits(prob["K"])
    Q = prob["q"].cpu().numpy().astype(np.float64)
    toks = np.unique(np.concatenate([[0, 1, N - 1], np.random.default_rng(0).integers(0, N, 29)]))
    Hh = H[:, torch.as_tensor(toks, device=dev)]
    got = to_host(Hh.contiguous())
    got_ne = to_host(ne[:, torch.as_tensor(toks, device=dev)].contiguous())
    ref = np.empty(got.shape)
    ref_ne = np.empty(got_ne.shape)
    for k, n in enumerate(toks):
        h, e = oracle.route_all_fwd(Vb, Kb, Q, mode, first, r=r, n0=int(n), n1=int(n) + 1)
        ref[:, k] = h[:, 0]
        ref_ne[:, k] = e[:, 0]
    check_bf16_value("H", got, ref)
    check_neff("neff", got_ne, ref_ne)


# (mode, storage, S, N, d, r): the single-site N_eff from the keys alone.
NEFF_CASES = [
    (PROJECTED, "bf16", 49, 300, 1024, 16),
    (SLICED, "bf16", 64, 129, 1024, 64),
    (FULL, "bf16", 13, 77, 256, 256),
    (PROJECTED, "f32", 7, 50, 64, 12),
    (SLICED, "f32", 300, 33, 96, 5),
    (FULL, "f32", 5, 20, 40, 40),
]


@pytest.mark.parametrize("case", NEFF_CASES,
                         ids=lambda c: "{}-{}-S{}-N{}-d{}-r{}".format(
                             {PROJECTED: "P", SLICED: "S", FULL: "F"}[c[0]], *c[1:]))
def test_single_site_neff_matches_oracle(dev, case):
    mode, dtype, S, N, d, r = case
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=31, q_scale=3.0)
    ne = lr.route_neff(to_dev(p.V, dev), to_dev(p.K, dev), to_dev(p.q, dev), mode)
    torch.cuda.synchronize()
    ref = oracle.effective_sources(p.V, p.K, p.q.astype(np.float64), mode, r=p.r)
    check_neff("neff", to_host(ne), ref)


def test_single_site_neff_closed_forms(dev):
    """One source: N_eff = 1 exactly; zero query: N_eff = S."""
    p = make_host_problem(SLICED, 1, 40, 64, 8, dtype="bf16", seed=32)
    ne = lr.route_neff(to_dev(p.V, dev), None, to_dev(p.q, dev), SLICED)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(ne), np.ones(40, dtype=np.float32))
    p = make_host_problem(PROJECTED, 23, 40, 64, 8, dtype="bf16", seed=33)
    ne = lr.route_neff(to_dev(p.V, dev), to_dev(p.K, dev), torch.zeros(8, device=dev), PROJECTED)
    torch.cuda.synchronize()
    check_neff("neff", to_host(ne), np.full(40, 23.0))
