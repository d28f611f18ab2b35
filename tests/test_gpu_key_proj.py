"""GPU parity of the projected-key producer (Sec. 3.3, Eq. fused_projection)
through the C ABI against the fp64 oracle.

The kernel accumulates in fp32 and rounds once to bf16, so each output obeys
|got - ref| <= 2^-8 |ref| + m 2^-24 sum_c |a_c w_c| (nearest-even rounding to
8 significant bits, plus the worst-case fp32 accumulation error of m
products); that bound is checked element by element, next to the bf16 bars
of the rest of the suite.  Shapes cover ragged token, output and k tiles,
the scalar output paths (d or r not a multiple of 8), a key projection alone
(the embedding key, d = 0), an output projection alone (r = 0), and the
paper's attention and SwiGLU output projections at full size (sampled rows).
"""
import numpy as np
import pytest

import oracle
import paper_2607_09694_amd as lr
from paper_2607_09694_amd.inputs import bf16_bits_from_f32, bf16_tensor_to_bits, f32_from_bf16_bits
from parity import check_bf16_value

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lr.load_library()
    return torch.device("cuda:0")


def bits_to_dev(x, dev):
    return torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)


def to_host(t):
    return f32_from_bf16_bits(bf16_tensor_to_bits(t)).astype(np.float64)


def operands(N, m, nout, seed):
    rng = np.random.default_rng(seed)
    A = bf16_bits_from_f32(rng.standard_normal((N, m)).astype(np.float32))
    W = bf16_bits_from_f32((rng.standard_normal((nout, m)) / np.sqrt(m)).astype(np.float32))
    return A, W


def check_projection(name, got, ref, Ab, Wb_rows):
    """Element bound of one rounding to bf16 after an fp32 sum of m terms."""
    a = np.abs(f32_from_bf16_bits(Ab).astype(np.float64))
    w = np.abs(f32_from_bf16_bits(Wb_rows).astype(np.float64))
    m = a.shape[1]
    bound = 2.0 ** -8 * np.abs(ref) + m * 2.0 ** -24 * (a @ w.T)
    worst = (np.abs(got - ref) - bound).max(initial=-1.0)
    assert worst <= 0.0, f"{name}: exceeds the rounding bound by {worst:.3e}"
    check_bf16_value(name, got, ref)


# (N, m, d, r)
CASES = [
    (300, 64, 128, 16),     # ragged token tile, ragged output tile, one k stage
    (257, 1024, 1024, 16),  # attention output projection width, 9 output tiles
    (512, 2816, 1024, 32),  # SwiGLU hidden width
    (100, 72, 40, 12),      # ragged k stage; key rows written element by element
    (50, 40, 20, 6),        # d % 8 != 0: segments straddle the value / key split
    (64, 16, 0, 16),        # the embedding key alone (d = 0)
    (33, 128, 96, 0),       # an output projection alone (r = 0)
    (1, 8, 1, 1),           # one token, one value and one key column
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "N{}-m{}-d{}-r{}".format(*c))
def test_key_projection_matches_oracle(dev, case):
    N, m, d, r = case
    Ab, Wb = operands(N, m, d + r, seed=N + m + d + r)
    O, K = lr.key_proj_fwd(bits_to_dev(Ab, dev), bits_to_dev(Wb, dev), d)
    torch.cuda.synchronize()
    Or, Kr = oracle.key_projection(Ab, Wb, d)
    if d:
        check_projection("O", to_host(O), Or, Ab, Wb[:d])
    else:
        assert O is None
    if r:
        check_projection("K", to_host(K), Kr, Ab, Wb[d:])
    else:
        assert K is None


def test_writes_into_stack_planes_only(dev):
    """O and K as planes i of the value and key stacks: the other planes keep
    their contents bit for bit."""
    S, i, N, m, d, r = 5, 3, 96, 128, 256, 16
    Ab, Wb = operands(N, m, d + r, seed=21)
    V = torch.full((S, N, d), 7.0, dtype=torch.bfloat16, device=dev)
    Ks = torch.full((S, N, r), -3.0, dtype=torch.bfloat16, device=dev)
    lr.key_proj_fwd(bits_to_dev(Ab, dev), bits_to_dev(Wb, dev), d, out=(V[i], Ks[i]))
    torch.cuda.synchronize()
    Or, Kr = oracle.key_projection(Ab, Wb, d)
    check_projection("O", to_host(V[i]), Or, Ab, Wb[:d])
    check_projection("K", to_host(Ks[i]), Kr, Ab, Wb[d:])
    for j in range(S):
        if j != i:
            assert bool((V[j] == 7.0).all()) and bool((Ks[j] == -3.0).all())


def test_deterministic(dev):
    Ab, Wb = operands(700, 512, 300, seed=22)
    A, W = bits_to_dev(Ab, dev), bits_to_dev(Wb, dev)
    O1, K1 = lr.key_proj_fwd(A, W, 280)
    O2, K2 = lr.key_proj_fwd(A, W, 280)
    torch.cuda.synchronize()
    assert torch.equal(O1.view(torch.int16), O2.view(torch.int16))
    assert torch.equal(K1.view(torch.int16), K2.view(torch.int16))


@pytest.mark.parametrize("m,r", [(1024, 16), (2816, 16), (2816, 32)],
                         ids=["attn-r16", "swiglu-r16", "swiglu-r32"])
def test_model_projection_full_size(dev, m, r):
    """The paper's model (d = 1024, SwiGLU width 2816, Sec. 4.1) at
    N = 16384 tokens: sampled rows against the oracle row by row."""
    N, d = 16384, 1024
    g = torch.Generator(device=dev)
    g.manual_seed(m + r)
    A = torch.randn((N, m), generator=g, device=dev).to(torch.bfloat16)
    W = (torch.randn((d + r, m), generator=g, device=dev) / m ** 0.5).to(torch.bfloat16)
    O, K = lr.key_proj_fwd(A, W, d)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 255, 256, N - 1],
                                     np.random.default_rng(m).integers(0, N, 28)]))
    idx = torch.as_tensor(rows, device=dev)
    Ab = bf16_tensor_to_bits(A[idx].contiguous())
    Wb = bf16_tensor_to_bits(W)
    Or, Kr = oracle.key_projection(Ab, Wb, d)
    check_projection("O", to_host(O[idx].contiguous()), Or, Ab, Wb[:d])
    check_projection("K", to_host(K[idx].contiguous()), Kr, Ab, Wb[d:])


def test_rejected_outside_limits(dev):
    A = torch.zeros((4, 12), dtype=torch.bfloat16, device=dev)
    W = torch.zeros((6, 12), dtype=torch.bfloat16, device=dev)
    with pytest.raises(lr.RoutingError, match="m % 8"):
        lr.key_proj_fwd(A, W, 4)
    with pytest.raises(lr.RoutingError, match="bf16"):
        lr.key_proj_fwd(A.float()[:, :8].contiguous(), W.float()[:, :8].contiguous(), 4)


def test_activations_beyond_2_31_elements(dev):
    """N = 770000 tokens at the SwiGLU width m = 2816: the activation holds
    more than 2^31 elements (64-bit row offsets); sampled rows, the last
    included, against the oracle."""
    N, m, d, r = 770000, 2816, 1024, 16
    assert N * m > 2 ** 31
    g = torch.Generator(device=dev)
    g.manual_seed(77)
    A = torch.empty((N, m), dtype=torch.bfloat16, device=dev)
    for n0 in range(0, N, 1 << 17):
        n1 = min(N, n0 + (1 << 17))
        A[n0:n1].copy_(torch.randn((n1 - n0, m), generator=g, device=dev))
    W = (torch.randn((d + r, m), generator=g, device=dev) / m ** 0.5).to(torch.bfloat16)
    O, K = lr.key_proj_fwd(A, W, d)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, N // 2, N - 257, N - 256, N - 1],
                                     np.random.default_rng(8).integers(0, N, 11)]))
    idx = torch.as_tensor(rows, device=dev)
    Ab = bf16_tensor_to_bits(A[idx].contiguous())
    Wb = bf16_tensor_to_bits(W)
    Or, Kr = oracle.key_projection(Ab, Wb, d)
    check_projection("O", to_host(O[idx].contiguous()), Or, Ab, Wb[:d])
    check_projection("K", to_host(K[idx].contiguous()), Kr, Ab, Wb[d:])
    del A, O, K
    torch.cuda.empty_cache()
