"""GPU parity of the block-source forward with the completed block summaries
stored in bf16 (Sec. 3.1 Block AttnRes, Eqs. block_attnres_sum /
block_attnres_partial_sum, with the keys of Sec. 3.2; the bf16 storage of
completed summaries is the library's option, not the paper's).  The oracle
computes only the paper's definition, exact in fp64; the test holds:
  - every bf16 copy to its rounding bound around the exact member sum (half
    a bf16 ulp plus the fp32 summation error of its members);
  - every site's h to the bound that those roundings imply through Eqs.
    lr_key_norm, lr_attnres_weight and lr_attnres_output (derived in
    tests/block_bounds.py), element by element, and to the bf16 relative-L2
    bar of 5e-3.

Cases: both key modes, blocks of one (every copy is a single output), a
single partial block, scalar key paths (r or the sliced key offset not a
multiple of 4), the widest row, and the paper's 8-block pass at full size
(sampled tokens)."""
import numpy as np
import pytest

import oracle
import paper_2607_09694_amd as lr
from block_bounds import routed_bound, summary_bounds
from paper_2607_09694_amd.inputs import (PROJECTED, SLICED, bf16_tensor_to_bits,
                                         f32_from_bf16_bits, make_host_problem)
from parity import check_bf16_key_grad, rel_errors

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
    return torch.from_numpy(x).to(dev)


def to_host(t):
    return f32_from_bf16_bits(bf16_tensor_to_bits(t))


def site_args(t, c):
    """Slot count, start and finish flags of site t (1-based), blocks of c:
    o_{t-1} starts its block when (t-2) mod c == 0 and completes it when
    (t-1) mod c == 0; the embedding (site 1) is a block of its own."""
    if t == 1:
        return 1, True, True
    return (t - 2) // c + 2, (t - 2) % c == 0, (t - 1) % c == 0


def drive_pass(dev, O, KO, Q, c, mode, sites):
    T, N, d = O.shape
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    BC = torch.zeros((nslots, N, d), dtype=torch.bfloat16, device=dev)
    KB = KBC = None
    if mode == PROJECTED:
        r = KO.shape[2]
        KB = torch.zeros((nslots, N, r), dtype=torch.float32, device=dev)
        KBC = torch.zeros((nslots, N, r), dtype=torch.bfloat16, device=dev)
    out = {}
    for t in range(1, max(sites) + 1):
        n_src, start, finish = site_args(t, c)
        knew = KO[t - 1] if mode == PROJECTED else None
        H = lr.block_route_fwd_bf16c(B, KB, BC, KBC, O[t - 1], knew, Q[t - 1], n_src, start,
                                     finish, mode)
        if t in sites:
            out[t] = H
    torch.cuda.synchronize()
    return out, BC, KBC


def check_site(name, got, O, KO, q, t, c, mode, r):
    """h of site t against the exact routing: the derived bound element by
    element, and rel-L2 <= 5e-3."""
    B, KB, eB, eK = summary_bounds(O, KO, t, c, mode, r)
    ref, bound = routed_bound(B, KB, eB, eK, q, mode, r)
    got = np.asarray(got, dtype=np.float64)
    _, _, nl2 = rel_errors(got, ref)
    worst = (np.abs(got - ref) / bound).max(initial=0.0)
    assert worst <= 1.0 + 1e-12 and nl2 <= 5e-3, \
        f"{name}: max error / bound {worst:.3f}, rel-L2 {nl2:.3e} (bar 5e-3)"
    return ref


def check_copies(BC, KBC, O, KO, T, c, mode, r):
    """The copies of the slots completed by the end of a T-site pass: each
    within its rounding bound of the exact member sum."""
    nfin = 1 + (T - 1) // c
    B, KB, eB, eK = summary_bounds(O, KO, T, c, mode, r, all_rounded=True)
    for name, got, ref, e in (("BC", BC, B, eB), ("KBC", KBC, KB, eK)):
        if ref is None:
            continue
        got = f32_from_bf16_bits(got[:nfin])
        worst = (np.abs(got - ref[:nfin]) / e[:nfin]).max(initial=0.0)
        assert worst <= 1.0 + 1e-12, f"{name}: max error / rounding bound {worst:.4f}"


# (mode, T, N, d, r, c)
CASES = [
    (PROJECTED, 13, 70, 256, 16, 3),
    (SLICED, 13, 70, 256, 16, 3),
    (SLICED, 9, 21, 2048, 8, 1),     # blocks of one: each copy is one output
    (PROJECTED, 9, 24, 100, 7, 20),  # one partial block; r = 7 scalar key loads
    (SLICED, 11, 33, 256, 10, 2),    # sliced key offset 246: scalar key loads
    (PROJECTED, 17, 40, 1024, 32, 4),
    (SLICED, 16, 19, 520, 64, 5),    # last site completes its block; ragged slab
    (PROJECTED, 6, 54, 2048, 8, 3),  # the embedding holds a -0.0, which its copy keeps
]


@pytest.mark.parametrize("case", CASES,
                         ids=lambda c: f"{'P' if c[0] == 0 else 'S'}-T{c[1]}-N{c[2]}-d{c[3]}-r{c[4]}-c{c[5]}")
def test_bf16_copies_model_pass_matches_oracle(dev, case):
    mode, T, N, d, r, c = case
    p = make_host_problem(mode, T, N, d, r, dtype="bf16", seed=T * 31 + c)
    rng = np.random.default_rng(T + c)
    Qh = (rng.standard_normal((T, r)) * 2.0 / np.sqrt(r)).astype(np.float32)
    O, KO, Q = to_dev(p.V, dev), to_dev(p.K, dev), torch.from_numpy(Qh).to(dev)
    sites = list(range(1, T + 1))
    out, BC, KBC = drive_pass(dev, O, KO, Q, c, mode, sites)
    for t in sites:
        check_site(f"H at site {t}", to_host(out[t]), p.V, p.K, Qh[t - 1], t, c, mode, r)
    check_copies(bf16_tensor_to_bits(BC), None if KBC is None else bf16_tensor_to_bits(KBC),
                 p.V, p.K, T, c, mode, r)


def test_bf16_copies_differ_from_fp32_slots_only_by_rounding(dev):
    """The same pass with fp32 completed slots: the two outputs differ by
    less than the bf16 bar of either against its own oracle."""
    mode, T, N, d, r, c = SLICED, 13, 40, 512, 32, 3
    p = make_host_problem(mode, T, N, d, r, dtype="bf16", seed=4)
    Qh = (np.random.default_rng(2).standard_normal((T, r)) / np.sqrt(r)).astype(np.float32)
    O, Q = to_dev(p.V, dev), torch.from_numpy(Qh).to(dev)
    out16, _, _ = drive_pass(dev, O, None, Q, c, mode, [T])
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    for t in range(1, T + 1):
        n_src, start, _ = site_args(t, c)
        H32 = lr.block_route_fwd(B, None, O[t - 1], None, Q[t - 1], n_src, start, mode)
    torch.cuda.synchronize()
    a, b = to_host(out16[T]), to_host(H32)
    check_site("bf16 copies", a, p.V, None, Qh[T - 1], T, c, mode, r)
    check_bf16_key_grad("fp32 slots", b, oracle.block_route_fwd(p.V, None, Qh[T - 1], T, c, mode, r=r))
    assert np.abs(a - b).max() < 0.1 and np.abs(a - b).max() > 0.0


@pytest.mark.parametrize("mode,r", [(SLICED, 64), (PROJECTED, 32)], ids=["S-r64", "P-r32"])
def test_bf16_copies_full_size(dev, mode, r):
    """The paper's 8-block pass (d = 1024, 49 sites, blocks of 6, N = 16384)
    with bf16 completed summaries: sampled tokens at sites around block
    boundaries against the oracle with the same reading."""
    T, N, d, c = 49, 16384, 1024, 6
    g = torch.Generator(device=dev).manual_seed(3)
    O = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)
    for i in range(T):
        O[i].copy_(torch.randn((N, d), generator=g, device=dev))
    KO = (torch.randn((T, N, r), generator=g, device=dev).to(torch.bfloat16)
          if mode == PROJECTED else None)
    Q = torch.randn((T, r), generator=g, device=dev) / r ** 0.5
    sites = [1, 2, 7, 8, 13, 25, 49]
    out, BC, KBC = drive_pass(dev, O, KO, Q, c, mode, sites)
    idx = np.sort(np.concatenate([[0, 1, N - 1], np.random.default_rng(5).choice(N, 29, replace=False)]))
    ti = torch.from_numpy(idx).to(dev)
    Os = bf16_tensor_to_bits(O.index_select(1, ti))
    Ks = bf16_tensor_to_bits(KO.index_select(1, ti)) if KO is not None else None
    for t in sites:
        check_site(f"H at site {t}", to_host(out[t].index_select(0, ti)), Os, Ks,
                   Q[t - 1].cpu().numpy(), t, c, mode, r)
    check_copies(bf16_tensor_to_bits(BC.index_select(1, ti)),
                 None if KBC is None else bf16_tensor_to_bits(KBC.index_select(1, ti)),
                 Os, Ks, T, c, mode, r)


def test_block_slots_beyond_2_31_elements(dev):
    """A 13-site pass (blocks of 3, 5 slots) over N = 220000 tokens at
    d = 2048: the fp32 slot stack and the bf16 copies each hold more than
    2^31 values (64-bit slot offsets).  fp32 slots and bf16 copies both;
    sampled tokens, the last included, at the last site."""
    mode, T, N, d, r, c = SLICED, 13, 220000, 2048, 64, 3
    nslots = (T - 2) // c + 2
    assert nslots * N * d > 2 ** 31
    g = torch.Generator(device=dev).manual_seed(21)
    O = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)
    for i in range(T):
        O[i].copy_(torch.randn((N, d), generator=g, device=dev))
    Q = torch.randn((T, r), generator=g, device=dev) / r ** 0.5
    out16, BC, _ = drive_pass(dev, O, None, Q, c, mode, [T])
    H16 = out16[T]
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    for t in range(1, T + 1):
        n_src, start, _ = site_args(t, c)
        H32 = lr.block_route_fwd(B, None, O[t - 1], None, Q[t - 1], n_src, start, mode)
    torch.cuda.synchronize()
    idx = np.sort(np.concatenate([[0, N - 2, N - 1], np.random.default_rng(6).choice(N, 13, replace=False)]))
    ti = torch.from_numpy(idx).to(dev)
    Os = bf16_tensor_to_bits(O.index_select(1, ti))
    qh = Q[T - 1].cpu().numpy()
    check_site("H bf16 copies", to_host(H16.index_select(0, ti)), Os, None, qh, T, c, mode, r)
    check_bf16_key_grad("H fp32 slots", to_host(H32.index_select(0, ti)),
                        oracle.block_route_fwd(Os, None, qh, T, c, mode, r=r))
    check_copies(bf16_tensor_to_bits(BC.index_select(1, ti)), None, Os, None, T, c, mode, r)
    del O, B, BC, out16
    torch.cuda.empty_cache()
