"""GPU parity of the fused block-source forward (Sec. 3.1 Block AttnRes with
the low-rank keys of Sec. 3.2): a whole model pass is driven site by site,
exactly as a model calls it, and every site's h is checked against the fp64
oracle, which forms the block summaries from the raw outputs."""
import numpy as np
import pytest

import oracle
import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import (FULL, PROJECTED, SLICED, bf16_tensor_to_bits,
                                         f32_from_bf16_bits, make_host_problem)
from parity import check_bf16_key_grad, check_dq, check_f32

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
    if t.dtype == torch.bfloat16:
        return f32_from_bf16_bits(bf16_tensor_to_bits(t))
    return t.detach().cpu().numpy()


def site_args(t, c):
    """Slot count and start flag of site t (1-based) with blocks of c."""
    if t == 1:
        return 1, True
    return (t - 2) // c + 2, (t - 2) % c == 0


def drive_model_pass(dev, O, KO, Q, c, mode, sites):
    """Call the fused op at sites 1..max(sites); return {t: H_t}."""
    T, N, d = O.shape
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    KB = (torch.zeros((nslots, N, KO.shape[2]), dtype=torch.float32, device=dev)
          if mode == PROJECTED else None)
    out = {}
    for t in range(1, max(sites) + 1):
        n_src, start = site_args(t, c)
        knew = KO[t - 1] if mode == PROJECTED else None
        H = lr.block_route_fwd(B, KB, O[t - 1], knew, Q[t - 1], n_src, start, mode)
        if t in sites:
            out[t] = H
    torch.cuda.synchronize()
    return out, B, KB


CASES = [
    (PROJECTED, "bf16", 13, 70, 256, 16, 3),
    (SLICED, "bf16", 13, 70, 256, 16, 3),
    (PROJECTED, "f32", 10, 33, 1024, 32, 4),
    (SLICED, "f32", 10, 33, 1000, 64, 2),
    (SLICED, "bf16", 9, 21, 2048, 8, 1),     # blocks of one: full routing
    (PROJECTED, "bf16", 9, 24, 100, 7, 20),  # one partial block; masked columns
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{'P' if c[0] == 0 else 'S'}-{c[1]}-T{c[2]}-N{c[3]}-d{c[4]}-r{c[5]}-c{c[6]}")
def test_block_model_pass_matches_oracle(dev, case):
    mode, dtype, T, N, d, r, c = case
    p = make_host_problem(mode, T, N, d, r, dtype=dtype, seed=T * 100 + N)
    rng = np.random.default_rng(T)
    Qh = (rng.standard_normal((T, r)) / np.sqrt(r)).astype(np.float32)
    O, KO, Q = to_dev(p.V, dev), to_dev(p.K, dev), torch.from_numpy(Qh).to(dev)
    sites = list(range(1, T + 1))
    out, B, KB = drive_model_pass(dev, O, KO, Q, c, mode, sites)
    # Block summaries are sums of up to c outputs, so h reaches |h| >= 8 where
    # the bf16 half-ulp alone exceeds an absolute 2e-2: the scaled bar applies.
    check = check_f32 if dtype == "f32" else check_bf16_key_grad
    for t in sites:
        ref = oracle.block_route_fwd(p.V, p.K, Qh[t - 1], t, c, mode, r=r)
        check(f"H at site {t}", to_host(out[t]), ref)
    # the slots end as the exact block sums (fp32 accumulation of the outputs)
    Ow = p.V.astype(np.float64) if dtype == "f32" else f32_from_bf16_bits(p.V).astype(np.float64)
    last = (T - 2) // c + 1
    for j in range(0, last + 1):
        members = [0] if j == 0 else list(range((j - 1) * c + 1, min(j * c, T - 1) + 1))
        check_f32(f"slot {j}", B[j].cpu().numpy(), Ow[members].sum(axis=0), tol=1e-6)


@pytest.mark.parametrize("mode,r", [(SLICED, 64), (PROJECTED, 32)], ids=["S-r64", "P-r32"])
def test_block_model_pass_full_size(dev, mode, r):
    """The paper's best block settings (8 blocks, Table 1): d = 1024, 48
    sub-layers plus the embedding, N = 8 x 2048 tokens; sampled tokens at
    sites around block boundaries."""
    T, N, d, c = 49, 16384, 1024, 6
    g = torch.Generator(device=dev).manual_seed(0)
    O = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)
    for i in range(T):
        O[i].copy_(torch.randn((N, d), generator=g, device=dev))
    KO = (torch.randn((T, N, r), generator=g, device=dev).to(torch.bfloat16)
          if mode == PROJECTED else None)
    Q = torch.randn((T, r), generator=g, device=dev) / r ** 0.5
    sites = [1, 2, 7, 8, 25, 49]
    out, _, _ = drive_model_pass(dev, O, KO, Q, c, mode, sites)
    idx = np.sort(np.concatenate([[0, 1, N - 1], np.random.default_rng(1).choice(N, 29, replace=False)]))
    ti = torch.from_numpy(idx).to(dev)
    Os = bf16_tensor_to_bits(O.index_select(1, ti))
    Ks = bf16_tensor_to_bits(KO.index_select(1, ti)) if KO is not None else None
    for t in sites:
        ref = oracle.block_route_fwd(Os, Ks, Q[t - 1].cpu().numpy(), t, c, mode, r=r)
        check_bf16_key_grad(f"H at site {t}", to_host(out[t].index_select(0, ti)), ref)


TRAIN_CASES = [
    (PROJECTED, "bf16", 13, 70, 256, 16, 3),
    (SLICED, "bf16", 13, 70, 256, 16, 3),
    (PROJECTED, "f32", 10, 33, 1024, 32, 4),
    (SLICED, "f32", 10, 33, 1000, 64, 2),
    (SLICED, "bf16", 7, 21, 512, 8, 1),
]


@pytest.mark.parametrize("case", TRAIN_CASES, ids=lambda c: f"{'P' if c[0] == 0 else 'S'}-{c[1]}-T{c[2]}-N{c[3]}-d{c[4]}-r{c[5]}-c{c[6]}")
def test_block_training_pass_matches_oracle(dev, case):
    """Forward at every site, then the reverse pass site by site: each
    member's gradient (summed over every later site) and each site's dq
    against the oracle's per-site block backward, summed over sites."""
    mode, dtype, T, N, d, r, c = case
    p = make_host_problem(mode, T, N, d, r, dtype=dtype, seed=T * 10 + N)
    rng = np.random.default_rng(N)
    Qh = (rng.standard_normal((T, r)) / np.sqrt(r)).astype(np.float32)
    dHh = make_host_problem(PROJECTED, T, N, d, 1, dtype=dtype, seed=T * 10 + N + 1).V
    O, KO, Q, dHs = to_dev(p.V, dev), to_dev(p.K, dev), torch.from_numpy(Qh).to(dev), to_dev(dHh, dev)
    _, B, KB = drive_model_pass(dev, O, KO, Q, c, mode, [T])
    dB = torch.zeros_like(B)
    dKB = torch.zeros_like(KB) if KB is not None else None
    dO = torch.empty_like(O)
    dK = torch.empty_like(KO) if KO is not None else None
    dq = torch.empty((T, r), dtype=torch.float32, device=dev)
    for t in range(T, 0, -1):
        n_src, _ = site_args(t, c)
        lr.block_route_bwd(B, KB, dB, dKB, O[t - 1], KO[t - 1] if KO is not None else None,
                           Q[t - 1], dHs[t - 1], n_src, mode,
                           out=(dO[t - 1], dK[t - 1] if dK is not None else None, dq[t - 1]))
    torch.cuda.synchronize()
    ref_dO = np.zeros((T, N, d))
    ref_dK = np.zeros((T, N, r)) if mode == PROJECTED else None
    for t in range(1, T + 1):
        gO, gK, gq = oracle.block_route_bwd(p.V, p.K, Qh[t - 1], dHh[t - 1], t, c, mode, r=r)
        ref_dO[:t] += gO
        if mode == PROJECTED:
            ref_dK[:t] += gK
        check_dq(f"dq at site {t}", dq[t - 1].cpu().numpy(), gq,
                 tol=1e-5 if dtype == "f32" else 1e-4)
    check = check_f32 if dtype == "f32" else check_bf16_key_grad
    check("dO", to_host(dO), ref_dO)
    if mode == PROJECTED:
        check("dK", to_host(dK), ref_dK)
    # every member has left its slot again
    assert float(B.abs().max()) < 1e-3 * max(1.0, float(torch.from_numpy(
        np.abs(to_host(O)).sum(axis=0)).max()))


def drive_deferred_reverse_pass(dev, B, KB, O, KO, Q, dHs, c, mode):
    """The reverse pass in deferred form: when a slot becomes the block in
    progress (its last site, in reverse order), its gradient from the sites
    that read it as completed is gathered; then each site adds its own part
    and retires its member.  Returns (dO, dK, dq)."""
    T, N, d = O.shape
    nslots = (T - 2) // c + 2
    r = Q.shape[1]
    coef = torch.full((T, nslots, 3, N), float("nan"), dtype=torch.float32, device=dev)
    dP = torch.empty((N, d), dtype=torch.float32, device=dev)
    dKP = torch.empty((N, r), dtype=torch.float32, device=dev) if mode == PROJECTED else None
    dO = torch.empty_like(O)
    dK = torch.empty_like(KO) if KO is not None else None
    dq = torch.empty((T, r), dtype=torch.float32, device=dev)
    cur = None
    for t in range(T, 0, -1):
        n_src, _ = site_args(t, c)
        p = n_src - 1
        if p != cur:
            first = p * c + 2 if p >= 1 else 2  # first site reading slot p as completed
            lr.block_gather_bwd(B, KB, p, dHs, Q, coef, first - 1, mode, out=(dP, dKP))
            cur = p
        lr.block_route_bwd_deferred(B, KB, dP, dKP, coef[t - 1, :n_src - 1], O[t - 1],
                                    KO[t - 1] if KO is not None else None, Q[t - 1], dHs[t - 1],
                                    n_src, mode,
                                    out=(dO[t - 1], dK[t - 1] if dK is not None else None,
                                         dq[t - 1]))
    torch.cuda.synchronize()
    return dO, dK, dq


@pytest.mark.parametrize("case", TRAIN_CASES, ids=lambda c: f"{'P' if c[0] == 0 else 'S'}-{c[1]}-T{c[2]}-N{c[3]}-d{c[4]}-r{c[5]}-c{c[6]}")
def test_deferred_training_pass_matches_oracle(dev, case):
    """The deferred reverse pass (completed-slot gradients gathered once per
    block) against the oracle's per-site block backward summed over sites:
    every member gradient and every site's dq."""
    mode, dtype, T, N, d, r, c = case
    p = make_host_problem(mode, T, N, d, r, dtype=dtype, seed=T * 10 + N)
    rng = np.random.default_rng(N)
    Qh = (rng.standard_normal((T, r)) / np.sqrt(r)).astype(np.float32)
    dHh = make_host_problem(PROJECTED, T, N, d, 1, dtype=dtype, seed=T * 10 + N + 1).V
    O, KO, Q, dHs = to_dev(p.V, dev), to_dev(p.K, dev), torch.from_numpy(Qh).to(dev), to_dev(dHh, dev)
    _, B, KB = drive_model_pass(dev, O, KO, Q, c, mode, [T])
    dO, dK, dq = drive_deferred_reverse_pass(dev, B, KB, O, KO, Q, dHs, c, mode)
    ref_dO = np.zeros((T, N, d))
    ref_dK = np.zeros((T, N, r)) if mode == PROJECTED else None
    for t in range(1, T + 1):
        gO, gK, gq = oracle.block_route_bwd(p.V, p.K, Qh[t - 1], dHh[t - 1], t, c, mode, r=r)
        ref_dO[:t] += gO
        if mode == PROJECTED:
            ref_dK[:t] += gK
        check_dq(f"dq at site {t}", dq[t - 1].cpu().numpy(), gq,
                 tol=1e-5 if dtype == "f32" else 1e-4)
    check = check_f32 if dtype == "f32" else check_bf16_key_grad
    check("dO", to_host(dO), ref_dO)
    if mode == PROJECTED:
        check("dK", to_host(dK), ref_dK)
    assert float(B.abs().max()) < 1e-3 * max(1.0, float(torch.from_numpy(
        np.abs(to_host(O)).sum(axis=0)).max()))


@pytest.mark.parametrize("mode,nprev,nq,d,r", [(PROJECTED, 5, 6, 1024, 32), (SLICED, 9, 12, 2048, 64),
                                               (SLICED, 1, 3, 100, 4), (PROJECTED, 70, 9, 256, 7)],
                         ids=["P-5x6-d1024", "S-9x12-d2048", "S-1x3-d100", "P-70x9-d256"])
def test_inter_state_matches_oracle(dev, mode, nprev, nq, d, r):
    """Phase 1 (Sec. 3.5): each query's online-softmax state over the
    completed fp32 slots equals the oracle's state over the same sources."""
    N = 37
    p = make_host_problem(mode, nprev, N, d, r, dtype="f32", seed=nprev * 7 + nq, q_scale=2.0)
    Qh = (np.random.default_rng(nq).standard_normal((nq, r)) * 2.0 / np.sqrt(r)).astype(np.float32)
    M, L, ACC = lr.block_inter_fwd(to_dev(p.V, dev), to_dev(p.K, dev), torch.from_numpy(Qh).to(dev),
                                   nprev, mode)
    torch.cuda.synchronize()
    for u in range(nq):
        Mr, Lr, Ar = oracle.route_state(p.V, p.K, Qh[u], mode, r=r)
        check_f32(f"M[{u}]", M[u].cpu().numpy(), Mr)
        check_f32(f"L[{u}]", L[u].cpu().numpy(), Lr)
        check_f32(f"ACC[{u}]", ACC[u].cpu().numpy(), Ar)


def drive_two_phase(dev, O, KO, Q, c, mode):
    """Two-phase inference over a whole model pass; returns {t: H_t}."""
    T, N, d = O.shape
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    KB = (torch.zeros((nslots, N, KO.shape[2]), dtype=torch.float32, device=dev)
          if mode == PROJECTED else None)
    out = {}
    out[1] = lr.block_merge_fwd(B, KB, O[0], KO[0] if KO is not None else None, Q[0], None, 0,
                                True, mode)
    t = 2
    while t <= T:
        j = (t - 2) // c + 1                      # block of o_{t-1}: the partial slot
        span = list(range(t, min(t + c, T + 1)))  # the sites of this block
        M, L, ACC = lr.block_inter_fwd(B, KB, Q[span[0] - 1:span[-1]].contiguous(), j, mode)
        for k, s in enumerate(span):
            out[s] = lr.block_merge_fwd(B, KB, O[s - 1], KO[s - 1] if KO is not None else None,
                                        Q[s - 1], (M[k], L[k], ACC[k]), j, k == 0, mode)
        t = span[-1] + 1
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("case", CASES[:5], ids=lambda c: f"{'P' if c[0] == 0 else 'S'}-{c[1]}-T{c[2]}-N{c[3]}-d{c[4]}-r{c[5]}-c{c[6]}")
def test_two_phase_model_pass_matches_oracle(dev, case):
    """Phase 1 once per block, phase 2 at every site: every site's h equals
    the block-source routing of the oracle."""
    mode, dtype, T, N, d, r, c = case
    p = make_host_problem(mode, T, N, d, r, dtype=dtype, seed=T * 100 + N + 5)
    Qh = (np.random.default_rng(T + 1).standard_normal((T, r)) / np.sqrt(r)).astype(np.float32)
    out = drive_two_phase(dev, to_dev(p.V, dev), to_dev(p.K, dev), torch.from_numpy(Qh).to(dev),
                          c, mode)
    check = check_f32 if dtype == "f32" else check_bf16_key_grad
    for t in range(1, T + 1):
        ref = oracle.block_route_fwd(p.V, p.K, Qh[t - 1], t, c, mode, r=r)
        check(f"H at site {t}", to_host(out[t]), ref)


# Block AttnRes with full-rank keys: the sliced routing with r = d (Sec. 3.4).
FULL_CASES = [(FULL, "bf16", 9, 40, 256, 256, 3), (FULL, "f32", 7, 17, 1024, 1024, 2)]


@pytest.mark.parametrize("case", FULL_CASES, ids=lambda c: f"F-{c[1]}-T{c[2]}-N{c[3]}-d{c[4]}-c{c[6]}")
def test_full_rank_block_forward_and_two_phase(dev, case):
    mode, dtype, T, N, d, r, c = case
    p = make_host_problem(mode, T, N, d, r, dtype=dtype, seed=T + N)
    Qh = (np.random.default_rng(T).standard_normal((T, d)) / np.sqrt(d)).astype(np.float32)
    O, Q = to_dev(p.V, dev), torch.from_numpy(Qh).to(dev)
    out, _, _ = drive_model_pass(dev, O, None, Q, c, mode, list(range(1, T + 1)))
    out2 = drive_two_phase(dev, O, None, Q, c, mode)
    check = check_f32 if dtype == "f32" else check_bf16_key_grad
    for t in range(1, T + 1):
        ref = oracle.block_route_fwd(p.V, None, Qh[t - 1], t, c, SLICED, r=d)
        check(f"H at site {t}", to_host(out[t]), ref)
        check(f"two-phase H at site {t}", to_host(out2[t]), ref)


def test_full_rank_block_training_pass(dev):
    mode, dtype, T, N, d, c = FULL, "bf16", 9, 40, 256, 3
    p = make_host_problem(mode, T, N, d, d, dtype=dtype, seed=3)
    Qh = (np.random.default_rng(4).standard_normal((T, d)) / np.sqrt(d)).astype(np.float32)
    dHh = make_host_problem(PROJECTED, T, N, d, 1, dtype=dtype, seed=5).V
    O, Q, dHs = to_dev(p.V, dev), torch.from_numpy(Qh).to(dev), to_dev(dHh, dev)
    _, B, _ = drive_model_pass(dev, O, None, Q, c, mode, [T])
    dB = torch.zeros_like(B)
    dO = torch.empty_like(O)
    dq = torch.empty((T, d), dtype=torch.float32, device=dev)
    for t in range(T, 0, -1):
        n_src, _ = site_args(t, c)
        lr.block_route_bwd(B, None, dB, None, O[t - 1], None, Q[t - 1], dHs[t - 1], n_src, mode,
                           out=(dO[t - 1], None, dq[t - 1]))
    torch.cuda.synchronize()
    ref_dO = np.zeros((T, N, d))
    for t in range(1, T + 1):
        gO, _, gq = oracle.block_route_bwd(p.V, None, Qh[t - 1], dHh[t - 1], t, c, SLICED, r=d)
        ref_dO[:t] += gO
        check_dq(f"dq at site {t}", dq[t - 1].cpu().numpy(), gq)
    check_bf16_key_grad("dO", to_host(dO), ref_dO)
