"""The routing calls inside a captured HIP graph: the library launches only
kernels on the caller's stream (no memset, no allocation, no host sync), so a
captured step replays bit for bit.  Each replay is separated by eager work
and a synchronisation, and every replay is compared with the eager result."""
import numpy as np
import pytest

import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import FULL, PROJECTED, SLICED, make_host_problem

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


@pytest.mark.parametrize("mode", [PROJECTED, SLICED])
def test_captured_step_replays_bitwise(dev, mode):
    S, N, d, r = 24, 300, 1024, 16
    p = make_host_problem(mode, S, N, d, r, dtype="bf16", seed=31, with_dH=True)
    V, K, q, dH = (to_dev(x, dev) for x in (p.V, p.K, p.q, p.dH))
    H = torch.empty((N, d), dtype=torch.bfloat16, device=dev)
    dV = torch.empty_like(V)
    dK = torch.empty_like(K) if K is not None else None
    dq = torch.empty((r,), dtype=torch.float32, device=dev)
    ws = torch.empty((lr.route_bwd_workspace_bytes(S, N, d, r, mode, torch.bfloat16),),
                     dtype=torch.uint8, device=dev)

    def step():
        lr.route_fwd(V, K, q, mode, out=H)
        lr.route_bwd(V, K, q, dH, mode, out=(dV, dK, dq), workspace=ws)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (H, dV, dq) if t is not None]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for k in range(3):
        for t in (H, dV, dq):
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ref, (H, dV, dq)):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {k}"
        # eager work between replays
        V.mul_(1.0)
        torch.cuda.synchronize()


def test_captured_block_model_pass_replays(dev):
    """All 13 sites of a block-source forward pass in one graph."""
    T, N, d, r, c = 13, 70, 256, 16, 3
    p = make_host_problem(SLICED, T, N, d, r, dtype="bf16", seed=7)
    O = to_dev(p.V, dev)
    Q = torch.randn((T, r), generator=torch.Generator(device=dev).manual_seed(1), device=dev)
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    Hs = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)

    def pass_():
        lr.block_route_fwd(B, None, O[0], None, Q[0], 1, True, SLICED, out=Hs[0])
        for t in range(2, T + 1):
            lr.block_route_fwd(B, None, O[t - 1], None, Q[t - 1], (t - 2) // c + 2,
                               (t - 2) % c == 0, SLICED, out=Hs[t - 1])

    pass_()
    torch.cuda.synchronize()
    ref = Hs.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pass_()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pass_()
    for k in range(3):
        Hs.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(ref.view(torch.int16), Hs.view(torch.int16)), f"replay {k}"


def _replays_match(pass_, outs):
    """Eager result, then a captured graph replayed three times with eager
    work (zeroing the outputs) and host synchronisations between replays."""
    pass_()
    torch.cuda.synchronize()
    refs = [o.clone() for o in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pass_()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pass_()
    for k in range(3):
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for ref, o in zip(refs, outs):
            assert torch.equal(ref.view(torch.uint8), o.view(torch.uint8)), f"replay {k}"


def test_captured_block_pass_with_bf16_copies_replays(dev):
    """A 13-site projected-key block pass with bf16 completed summaries in one
    graph: every site's h and every copy written match the eager pass."""
    T, N, d, r, c = 13, 40, 256, 16, 3
    p = make_host_problem(PROJECTED, T, N, d, r, dtype="bf16", seed=9)
    O, KO = to_dev(p.V, dev), to_dev(p.K, dev)
    Q = torch.randn((T, r), generator=torch.Generator(device=dev).manual_seed(2), device=dev)
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    KB = torch.zeros((nslots, N, r), dtype=torch.float32, device=dev)
    BC = torch.zeros((nslots, N, d), dtype=torch.bfloat16, device=dev)
    KBC = torch.zeros((nslots, N, r), dtype=torch.bfloat16, device=dev)
    Hs = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)

    def pass_():
        for t in range(1, T + 1):
            n_src, start = (1, True) if t == 1 else ((t - 2) // c + 2, (t - 2) % c == 0)
            finish = t == 1 or (t - 1) % c == 0
            lr.block_route_fwd_bf16c(B, KB, BC, KBC, O[t - 1], KO[t - 1], Q[t - 1], n_src, start,
                                     finish, PROJECTED, out=Hs[t - 1])

    _replays_match(pass_, [Hs, BC, KBC])


def test_captured_split_sources_replays(dev):
    """Per-chunk states and their merge (a 49-source site at N = 64) in one
    graph, replays against the eager result."""
    S, N, d, r, chunk = 49, 64, 1024, 16, 7
    p = make_host_problem(PROJECTED, S, N, d, r, dtype="bf16", seed=11)
    V, K, q = to_dev(p.V, dev), to_dev(p.K, dev), to_dev(p.q, dev)
    P = -(-S // chunk)
    st = (torch.empty((P, N), dtype=torch.float32, device=dev),
          torch.empty((P, N), dtype=torch.float32, device=dev),
          torch.empty((P, N, d), dtype=torch.float32, device=dev))
    H = torch.empty((N, d), dtype=torch.bfloat16, device=dev)

    def pass_():
        lr.route_state_fwd(V, K, q, PROJECTED, chunk, out=st)
        lr.route_merge_fwd(*st, out=H)

    _replays_match(pass_, [H, *st])


def test_captured_key_producer_forward_and_backward_replays(dev):
    """The key producer and its backward (token splits and their ordered
    sum included) in one graph: every replay matches the eager call bit for
    bit."""
    N, m, d, r = 700, 256, 128, 16
    g = torch.Generator(device=dev).manual_seed(4)
    A = torch.randn((N, m), generator=g, device=dev).to(torch.bfloat16)
    W = (torch.randn((d + r, m), generator=g, device=dev) / m ** 0.5).to(torch.bfloat16)
    dO = torch.randn((N, d), generator=g, device=dev).to(torch.bfloat16)
    dK = torch.randn((N, r), generator=g, device=dev).to(torch.bfloat16)
    O = torch.empty((N, d), dtype=torch.bfloat16, device=dev)
    K = torch.empty((N, r), dtype=torch.bfloat16, device=dev)
    dA = torch.empty((N, m), dtype=torch.bfloat16, device=dev)
    dW = torch.empty((d + r, m), dtype=torch.float32, device=dev)

    def pass_():
        lr.key_proj_fwd(A, W, d, out=(O, K))
        lr.key_proj_bwd(A, W, dO, dK, out=(dA, dW))

    _replays_match(pass_, [O, K, dA, dW])


@pytest.mark.parametrize("mode,dtype", [(FULL, "bf16"), (SLICED, "f32")],
                         ids=["full-bf16", "sliced-f32"])
def test_captured_all_sites_site_by_site_replays(dev, mode, dtype):
    """The all-sites forward and backward on their site-by-site path (full-rank
    keys; fp32 storage) inside one graph: the overwriting backward clears its
    outputs with a fill kernel, so each replay over outputs left dirty by the
    previous one matches the eager result bit for bit."""
    S, T, first, N, d, r = 9, 7, 3, 40, 136, 16
    p = make_host_problem(mode, S, N, d, r, dtype=dtype, seed=17)
    r = p.r
    V = to_dev(p.V, dev)
    gq = torch.Generator(device=dev).manual_seed(2)
    Q = torch.randn((T, r), generator=gq, device=dev) / r ** 0.5
    dH = torch.randn((T, N, d), generator=gq, device=dev).to(V.dtype)
    H = torch.empty((T, N, d), dtype=V.dtype, device=dev)
    ne = torch.empty((T, N), dtype=torch.float32, device=dev)
    dV = torch.empty_like(V)
    dQ = torch.empty((T, r), dtype=torch.float32, device=dev)
    ws = torch.empty((max(16, lr.route_all_bwd_workspace_bytes(S, N, d, r, first, T, mode,
                                                                 V.dtype)),),
                     dtype=torch.uint8, device=dev)

    def step():
        lr.route_all_fwd(V, None, Q, mode, first, out=(H, ne))
        lr.route_all_bwd(V, None, Q, dH, mode, first, out=(dV, None, dQ), workspace=ws)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (H, ne, dV, dQ)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for k in range(3):
        for t in (H, ne, dV, dQ):
            t.fill_(3.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ref, (H, ne, dV, dQ)):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {k}"
        V.mul_(1.0)
        torch.cuda.synchronize()
