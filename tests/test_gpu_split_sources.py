"""GPU parity of the split-sources forward (Sec. 3.5's merge of online-softmax
states, applied to the sources of one site) through the C ABI, against the
fp64 oracle.

Each chunk's state (M, L, ACC) is checked against the oracle's state over the
same sources, and the merge of all chunks against the oracle's routing over
all of them.  Cases cover both storages, all three key modes, ragged last
chunks, a chunk wider than the stack (one state), ragged column slabs, rows
split into column blocks (d = 8192), more sources than the one-call forward
takes (2048), one source, and no tokens.  The merge is checked to be
independent of the order of the states, and the full-size case runs the
paper's deepest site (49 sources, d = 1024, N = 16384) on sampled tokens.
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


def check_h(dtype, got, ref):
    (check_f32 if dtype == "f32" else check_bf16_value)("H", got, ref)


# (mode, storage, S, chunk, N, d, r)
CASES = [
    (PROJECTED, "bf16", 49, 8, 37, 1024, 16),    # 7 chunks, last one holds 1 source
    (SLICED, "bf16", 49, 16, 21, 2048, 64),      # widest single-block row
    (SLICED, "f32", 20, 7, 19, 200, 12),         # ragged slab, ragged chunk
    (FULL, "bf16", 33, 10, 12, 512, 512),        # full-rank keys
    (FULL, "f32", 9, 4, 5, 100, 100),            # full-rank, ragged slab
    (PROJECTED, "bf16", 300, 128, 6, 8192, 32),  # rows in two column blocks
    (SLICED, "bf16", 2048, 512, 3, 64, 8),       # beyond the one-call source limit
    (FULL, "f32", 1100, 300, 3, 64, 64),         # full-rank keys beyond it
    (PROJECTED, "f32", 12, 50, 9, 64, 5),        # one chunk wider than the stack
    (SLICED, "bf16", 1, 1, 4, 136, 8),           # one source
    (PROJECTED, "bf16", 16, 1, 33, 264, 24),     # one source per chunk, ragged slab
]


def _ids(c):
    return f"{'PSF'[c[0]]}-{c[1]}-S{c[2]}c{c[3]}-N{c[4]}-d{c[5]}-r{c[6]}"


@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_states_and_merge_match_oracle(dev, case):
    mode, dtype, S, chunk, N, d, r = case
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=S * 3 + chunk, q_scale=2.0)
    V, K, q = to_dev(p.V, dev), to_dev(p.K, dev), to_dev(p.q, dev)
    M, L, ACC = lr.route_state_fwd(V, K, q, mode, chunk)
    P = -(-S // chunk)
    assert tuple(ACC.shape) == (P, N, d)
    H = lr.route_merge_fwd(M, L, ACC, dtype=V.dtype)
    torch.cuda.synchronize()
    Mh, Lh, Ah = M.cpu().numpy(), L.cpu().numpy(), ACC.cpu().numpy()
    for c in range(P):
        i0, i1 = c * chunk, min(S, (c + 1) * chunk)
        Mr, Lr, Ar = oracle.route_state(p.V[i0:i1], None if p.K is None else p.K[i0:i1], p.q,
                                        mode, r=r)
        check_f32(f"M[{c}]", Mh[c], Mr)
        check_f32(f"L[{c}]", Lh[c], Lr)
        check_f32(f"ACC[{c}]", Ah[c], Ar)
    check_h(dtype, to_host(H), oracle.route_fwd(p.V, p.K, p.q, mode, r=r))


def test_merge_ignores_state_order(dev):
    """The merge is a sum over states: reversing their order changes the
    result only by rounding, and both match the oracle."""
    mode, S, chunk, N, d, r = PROJECTED, 40, 6, 25, 512, 16
    p = make_host_problem(mode, S, N, d, r, dtype="f32", seed=5, q_scale=3.0)
    M, L, ACC = lr.route_state_fwd(to_dev(p.V, dev), to_dev(p.K, dev), to_dev(p.q, dev), mode,
                                   chunk)
    fwd = lr.route_merge_fwd(M, L, ACC, dtype=torch.float32)
    rev = lr.route_merge_fwd(M.flip(0).contiguous(), L.flip(0).contiguous(),
                             ACC.flip(0).contiguous(), dtype=torch.float32)
    torch.cuda.synchronize()
    ref = oracle.route_fwd(p.V, p.K, p.q, mode, r=r)
    check_f32("H", to_host(fwd), ref)
    check_f32("H reversed", to_host(rev), ref)


def test_merge_of_a_subset_routes_over_its_sources(dev):
    """Merging chunks 1 and 2 of 4 routes over their sources alone."""
    mode, S, chunk, N, d, r = SLICED, 32, 8, 11, 256, 32
    p = make_host_problem(mode, S, N, d, r, dtype="bf16", seed=9)
    M, L, ACC = lr.route_state_fwd(to_dev(p.V, dev), None, to_dev(p.q, dev), mode, chunk)
    H = lr.route_merge_fwd(M[1:3].contiguous(), L[1:3].contiguous(), ACC[1:3].contiguous())
    torch.cuda.synchronize()
    check_bf16_value("H", to_host(H), oracle.route_fwd(p.V[8:24], None, p.q, mode, r=r))


def test_empty_tokens(dev):
    V = torch.zeros((5, 0, 64), dtype=torch.bfloat16, device=dev)
    q = torch.zeros((8,), dtype=torch.float32, device=dev)
    M, L, ACC = lr.route_state_fwd(V, None, q, SLICED, 2)
    H = lr.route_merge_fwd(M, L, ACC)
    torch.cuda.synchronize()
    assert tuple(ACC.shape) == (3, 0, 64) and tuple(H.shape) == (0, 64)


def test_unsupported_chunk_raises(dev):
    V = torch.zeros((4, 2, 64), dtype=torch.bfloat16, device=dev)
    q = torch.zeros((8,), dtype=torch.float32, device=dev)
    with pytest.raises(lr.RoutingError, match="EUNSUPPORTED"):
        lr.route_state_fwd(torch.zeros((1100, 2, 64), dtype=torch.bfloat16, device=dev), None,
                           q, SLICED, 1100)
    with pytest.raises(lr.RoutingError, match="EINVAL"):
        lr.route_state_fwd(V, None, q, SLICED, 0)


@pytest.mark.parametrize("mode,r,chunk", [(PROJECTED, 16, 7), (SLICED, 64, 4)],
                         ids=["P-r16-c7", "S-r64-c4"])
def test_deepest_site_full_size(dev, mode, r, chunk):
    """The deepest site of the paper's model pass (49 sources, d = 1024,
    N = 16384), split into chunks; sampled tokens against the oracle."""
    S, N, d = 49, 16384, 1024
    prob = make_device_problem(mode, S, N, d, r, dev, seed=1)
    q = prob["q"][0].contiguous()
    M, L, ACC = lr.route_state_fwd(prob["V"], prob["K"], q, mode, chunk)
    H = lr.route_merge_fwd(M, L, ACC)
    torch.cuda.synchronize()
    toks = np.unique(np.concatenate([[0, 1, N - 1], np.random.default_rng(3).integers(0, N, 29)]))
    idx = torch.as_tensor(toks, device=dev)
    Vb = bf16_tensor_to_bits(prob["V"][:, idx].contiguous())
    Kb = None if prob["K"] is None else bf16_tensor_to_bits(prob["K"][:, idx].contiguous())
    qh = q.cpu().numpy()
    check_bf16_value("H", to_host(H[idx].contiguous()), oracle.route_fwd(Vb, Kb, qh, mode, r=r))
    Mr, Lr, Ar = oracle.route_state(Vb[:chunk], None if Kb is None else Kb[:chunk], qh, mode, r=r)
    check_f32("M[0]", M[0, idx].cpu().numpy(), Mr)
    check_f32("L[0]", L[0, idx].cpu().numpy(), Lr)
    check_f32("ACC[0]", ACC[0, idx].cpu().numpy(), Ar)


def test_states_beyond_2_31_elements(dev):
    """Chunks of one source over a 70-source stack at N = 16384, d = 2048:
    ACC holds more than 2^31 fp32 values (64-bit state offsets).  Sampled
    tokens, the last included, against the oracle."""
    mode, S, N, d, r, chunk = PROJECTED, 70, 16384, 2048, 16, 1
    assert S * N * d > 2 ** 31
    prob = make_device_problem(mode, S, N, d, r, dev, seed=12)
    q = prob["q"][0].contiguous()
    M, L, ACC = lr.route_state_fwd(prob["V"], prob["K"], q, mode, chunk)
    H = lr.route_merge_fwd(M, L, ACC)
    torch.cuda.synchronize()
    toks = np.unique(np.concatenate([[0, N - 2, N - 1], np.random.default_rng(4).integers(0, N, 13)]))
    idx = torch.as_tensor(toks, device=dev)
    Vb = bf16_tensor_to_bits(prob["V"][:, idx].contiguous())
    Kb = bf16_tensor_to_bits(prob["K"][:, idx].contiguous())
    qh = q.cpu().numpy()
    check_bf16_value("H", to_host(H[idx].contiguous()), oracle.route_fwd(Vb, Kb, qh, mode, r=r))
    last = S - 1  # the last chunk's state lies past 2^31 values
    Mr, Lr, Ar = oracle.route_state(Vb[last:], Kb[last:], qh, mode, r=r)
    check_f32("M[last]", M[last, idx].cpu().numpy(), Mr)
    check_f32("L[last]", L[last, idx].cpu().numpy(), Lr)
    check_f32("ACC[last]", ACC[last, idx].cpu().numpy(), Ar)
    del prob, M, L, ACC, H
    torch.cuda.empty_cache()
