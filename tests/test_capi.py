"""The C ABI on the CPU: the library loads, exports what include/lr_attnres.h
declares, and rejects every invalid call during host-side validation, which
runs before any HIP call (so no device is touched; no pointer is
dereferenced on the host)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2607_09694_amd as lr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lr_attnres.h")
EINVAL, EUNSUPPORTED = 1, 2
P, SL, F = lr.PROJECTED, lr.SLICED, lr.FULL
BF16, F32 = 1, 0

# Distinct fake device addresses, far apart and 256-byte aligned.  Validation
# only compares them; nothing reads through them.
A, B, C, D, E, G, W = (0x10_0000_0000 * k for k in range(1, 8))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lr.LIB_PATH):
        from paper_2607_09694_amd.build import build

        build()
    return lr.load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lr_attnres_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert names == sorted(["lr_attnres_route_fwd", "lr_attnres_route_bwd",
                            "lr_attnres_route_bwd_accumulate", "lr_attnres_route_bwd_noalloc",
                            "lr_attnres_block_route_fwd",
                            "lr_attnres_block_route_bwd", "lr_attnres_block_inter_fwd",
                            "lr_attnres_block_merge_fwd", "lr_attnres_route_all_fwd",
                            "lr_attnres_key_proj_fwd", "lr_attnres_key_proj_bwd",
                            "lr_attnres_key_proj_bwd_workspace_bytes", "lr_attnres_route_neff",
                            "lr_attnres_block_route_bwd_deferred", "lr_attnres_block_gather_bwd",
                            "lr_attnres_route_all_bwd", "lr_attnres_route_all_bwd_workspace_bytes",
                            "lr_attnres_route_bwd_deferred", "lr_attnres_route_gather_bwd",
                            "lr_attnres_route_state_fwd", "lr_attnres_route_merge_fwd",
                            "lr_attnres_block_route_fwd_bf16c",
                            "lr_attnres_route_bwd_workspace_bytes", "lr_attnres_last_error",
                            "lr_attnres_abi_version"])
    out = subprocess.run(["nm", "-D", "--defined-only", lr.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s+(\w+)", out))
    for name in names:
        assert name in exported, name
        assert hasattr(lib, name)


def test_abi_version(lib):
    assert lib.lr_attnres_abi_version() == 1


def fwd(lib, V=A, K=None, q=B, H=C, S=4, N=8, d=64, r=8, mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_route_fwd(V, K, q, H, S, N, d, r, mode, dtype, eps, None)


def bwd(lib, V=A, K=None, q=B, dH=C, dV=D, dK=None, dq=E, ws=W, wsb=1 << 30, S=4, N=8, d=64,
        r=8, mode=SL, dtype=BF16, eps=1e-6, accumulate=False):
    fn = lib.lr_attnres_route_bwd_accumulate if accumulate else lib.lr_attnres_route_bwd
    return fn(V, K, q, dH, dV, dK, dq, ws, wsb, S, N, d, r, mode, dtype, eps, None)


def err(lib):
    return lib.lr_attnres_last_error().decode()


FWD_INVALID = [
    ("V NULL", dict(V=None), "V is NULL"),
    ("q NULL", dict(q=None), "q is NULL"),
    ("H NULL", dict(H=None), "H is NULL"),
    ("S zero", dict(S=0), "sizes"),
    ("d zero", dict(d=0), "sizes"),
    ("r zero", dict(r=0), "sizes"),
    ("N negative", dict(N=-1), "sizes"),
    ("sliced r > d", dict(r=65), "r <= d"),
    ("full r != d", dict(mode=F, r=8), "r == d"),
    ("K outside projected", dict(K=G), "K must be NULL"),
    ("projected without K", dict(mode=P, K=None), "K is NULL"),
    ("unknown mode", dict(mode=7), "mode"),
    ("unknown dtype", dict(dtype=5), "storage"),
    ("eps negative", dict(eps=-1.0), "eps"),
    ("eps nan", dict(eps=float("nan")), "eps"),
    ("eps inf", dict(eps=float("inf")), "eps"),
    ("V misaligned", dict(V=A + 2), "aligned"),
    ("H misaligned", dict(H=C + 8), "aligned"),
    ("q misaligned", dict(q=B + 2), "aligned"),
    ("H overlaps V", dict(H=A + 256), "overlaps"),
    ("H overlaps q", dict(H=B - 16), "overlaps"),
    ("overflow", dict(S=1 << 40, N=1 << 20, d=1 << 10), "overflow"),
]


@pytest.mark.parametrize("name,kw,msg", FWD_INVALID, ids=[c[0] for c in FWD_INVALID])
def test_forward_rejects(lib, name, kw, msg):
    assert fwd(lib, **kw) == EINVAL
    assert msg in err(lib)


BWD_INVALID = [
    ("dH NULL", dict(dH=None), "dH is NULL"),
    ("dV NULL", dict(dV=None), "dV is NULL"),
    ("dq NULL", dict(dq=None), "dq is NULL"),
    ("dK outside projected", dict(dK=G), "must be NULL"),
    ("projected without dK", dict(mode=P, K=G, dK=None), "dK is NULL"),
    ("workspace too small", dict(mode=P, K=G, dK=G + 0x1_0000_0000, wsb=4), "workspace"),
    ("workspace NULL", dict(ws=None), "workspace"),
    ("dV overlaps V", dict(dV=A + 64), "overlaps"),
    ("dV overlaps dH", dict(dV=C), "overlaps"),
    ("dq overlaps dV", dict(dq=D + 16), "overlap"),
    ("workspace overlaps dV", dict(ws=D + 64), "overlap"),
    ("dV misaligned", dict(dV=D + 4), "aligned"),
    ("eps nan", dict(eps=float("nan")), "eps"),
    ("full r != d", dict(mode=F, r=8), "r == d"),
]


@pytest.mark.parametrize("name,kw,msg", BWD_INVALID, ids=[c[0] for c in BWD_INVALID])
def test_backward_rejects(lib, name, kw, msg):
    assert bwd(lib, **kw) == EINVAL
    assert msg in err(lib)


@pytest.mark.parametrize("name,kw,msg", BWD_INVALID, ids=[c[0] for c in BWD_INVALID])
def test_accumulating_backward_rejects(lib, name, kw, msg):
    assert bwd(lib, accumulate=True, **kw) == EINVAL
    assert msg in err(lib)


def bwd_noalloc(lib, V=A, K=None, q=B, dH=C, dV=D, dK=None, dq=E, S=4, N=8, d=64, r=8, mode=SL,
                dtype=BF16, eps=1e-6):
    return lib.lr_attnres_route_bwd_noalloc(V, K, q, dH, dV, dK, dq, S, N, d, r, mode, dtype,
                                            eps, None)


NOALLOC_INVALID = [c for c in BWD_INVALID if "workspace" not in c[0]]


@pytest.mark.parametrize("name,kw,msg", NOALLOC_INVALID, ids=[c[0] for c in NOALLOC_INVALID])
def test_noalloc_backward_rejects(lib, name, kw, msg):
    kw = {k: v for k, v in kw.items() if k not in ("ws", "wsb")}
    assert bwd_noalloc(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_noalloc_backward_limit(lib):
    """Problems whose dq partials exceed the 8 MiB device array are refused
    before any HIP call; the workspace query says how much they need."""
    q = lib.lr_attnres_route_bwd_workspace_bytes
    limit = 8 << 20
    # projected r = 32 at d = 2048: two tokens per wave, 8 per workgroup
    assert q(64, 1 << 19, 2048, 32, P, BF16) == limit
    assert q(64, (1 << 19) + 8, 2048, 32, P, BF16) > limit
    big = dict(mode=P, K=G, dK=G + 0x1_0000_0000, S=1, d=2048, r=32, N=(1 << 19) + 8)
    assert bwd_noalloc(lib, **big) == EUNSUPPORTED
    assert "8388608" in err(lib)
    # full rank, d = 1024: four tokens per wave, 16 per workgroup
    assert q(1, 32768, 1024, 1024, F, BF16) == limit
    assert bwd_noalloc(lib, mode=F, S=1, d=1024, r=1024, N=32768 + 16) == EUNSUPPORTED
    assert bwd_noalloc(lib, S=513) == EUNSUPPORTED


def test_unsupported_shapes(lib):
    assert fwd(lib, S=1025) == EUNSUPPORTED
    assert "1024" in err(lib)
    assert bwd(lib, S=513) == EUNSUPPORTED
    assert bwd(lib, mode=P, K=G, dK=G + 0x1_0000_0000, r=257, d=1024) == EUNSUPPORTED
    assert bwd(lib, mode=F, r=8192, d=8192) == EUNSUPPORTED
    assert fwd(lib, mode=F, r=8192, d=8192) == EUNSUPPORTED
    assert fwd(lib, N=(1 << 30) + 1, S=1, d=8, r=8) == EUNSUPPORTED


def test_workspace_query(lib):
    q = lib.lr_attnres_route_bwd_workspace_bytes
    # per-workgroup dq partials: ceil(N / tokens per workgroup) x r fp32
    assert q(64, 16384, 2048, 32, P, BF16) > 0
    assert q(64, 16384, 2048, 32, P, BF16) % 4 == 0
    assert q(49, 16384, 1024, 1024, F, BF16) >= 1024 * 4
    assert q(4, 0, 64, 8, SL, BF16) == 0
    assert q(0, 8, 64, 8, SL, BF16) == 0          # invalid -> 0
    assert q(4, 8, 64, 8, 9, BF16) == 0           # unknown mode -> 0


def test_error_text_is_per_call(lib):
    assert fwd(lib, S=0) == EINVAL
    assert err(lib) != ""
    assert fwd(lib, V=None) == EINVAL
    assert "V is NULL" in err(lib)


def test_python_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError, match="not built"):
        lr.load_library(str(tmp_path / "missing.so"))


def blk(lib, B=A, KB=None, o_new=C, k_new=None, q=E, H=D, n_src=3, start=0, N=8, d=64, r=8,
        mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_block_route_fwd(B, KB, o_new, k_new, q, H, n_src, start, N, d, r,
                                          mode, dtype, eps, None)


BLOCK_INVALID = [
    ("B NULL", dict(B=None), "B is NULL"),
    ("o_new NULL", dict(o_new=None), "o_new is NULL"),
    ("H NULL", dict(H=None), "H is NULL"),
    ("start not 0/1", dict(start=2), "start"),
    ("unknown mode", dict(mode=9), "projected, sliced or full-rank"),
    ("full-rank with r != d", dict(mode=F, r=8), "r == d"),
    ("projected without KB", dict(mode=P, k_new=G), "KB is NULL"),
    ("projected without k_new", dict(mode=P, KB=G), "k_new is NULL"),
    ("KB outside projected", dict(KB=G), "must be NULL"),
    ("n_src zero", dict(n_src=0), "sizes"),
    ("sliced r > d", dict(r=65), "r <= d"),
    ("H overlaps B", dict(H=A + 64), "overlap"),
    ("B overlaps o_new", dict(o_new=A + 4096), "overlaps"),
    ("B misaligned", dict(B=A + 4), "aligned"),
    ("eps negative", dict(eps=-1.0), "eps"),
]


@pytest.mark.parametrize("name,kw,msg", BLOCK_INVALID, ids=[c[0] for c in BLOCK_INVALID])
def test_block_forward_rejects(lib, name, kw, msg):
    assert blk(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_block_forward_unsupported(lib):
    assert blk(lib, d=66) == EUNSUPPORTED
    assert blk(lib, d=4096) == EUNSUPPORTED
    assert blk(lib, n_src=1025) == EUNSUPPORTED


B_, X, Y, Z = (0x10_0000_0000 * k for k in range(8, 12))


def bblk(lib, B=A, KB=None, dB=B_, dKB=None, o_new=C, k_new=None, q=E, dH=D, dO=G, dK=None,
         dq=X, ws=W, wsb=1 << 30, n_src=3, N=8, d=64, r=8, mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_block_route_bwd(B, KB, dB, dKB, o_new, k_new, q, dH, dO, dK, dq, ws,
                                          wsb, n_src, N, d, r, mode, dtype, eps, None)


BLOCK_BWD_INVALID = [
    ("dB NULL", dict(dB=None), "dB is NULL"),
    ("dO NULL", dict(dO=None), "dO is NULL"),
    ("dH NULL", dict(dH=None), "dH is NULL"),
    ("projected without dKB", dict(mode=P, KB=Y, k_new=Z, dK=Z + 0x1000_0000), "dKB is NULL"),
    ("dK outside projected", dict(dK=Y), "must be NULL"),
    ("dB overlaps B", dict(dB=A + 64), "overlap"),
    ("dO overlaps dH", dict(dO=D), "overlaps"),
    ("workspace too small", dict(wsb=4), "workspace"),
    ("unknown mode", dict(mode=9), "projected, sliced or full-rank"),
]


@pytest.mark.parametrize("name,kw,msg", BLOCK_BWD_INVALID, ids=[c[0] for c in BLOCK_BWD_INVALID])
def test_block_backward_rejects(lib, name, kw, msg):
    assert bblk(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_block_backward_unsupported(lib):
    assert bblk(lib, mode=F, r=1024, d=1024) == EUNSUPPORTED  # runs as sliced r = 1024 > 256
    assert bblk(lib, d=66) == EUNSUPPORTED
    assert bblk(lib, n_src=513) == EUNSUPPORTED


def inter(lib, B=A, KB=None, Q=E, M=G, L=X, ACC=Y, n_prev=3, nq=6, N=8, d=64, r=8, mode=SL,
          eps=1e-6):
    return lib.lr_attnres_block_inter_fwd(B, KB, Q, M, L, ACC, n_prev, nq, N, d, r, mode, eps,
                                          None)


def merge(lib, B=A, KB=None, o_new=C, k_new=None, q=E, M=G, L=X, ACC=Y, H=D, slot=2, start=0,
          N=8, d=64, r=8, mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_block_merge_fwd(B, KB, o_new, k_new, q, M, L, ACC, H, slot, start, N,
                                          d, r, mode, dtype, eps, None)


TWO_PHASE_INVALID = [
    (inter, "no queries", dict(nq=0), "n_queries"),
    (inter, "ACC NULL", dict(ACC=None), "ACC is NULL"),
    (inter, "ACC overlaps B", dict(ACC=A + 16), "overlaps"),
    (inter, "KB outside projected", dict(KB=Z), "must be NULL"),
    (merge, "state at slot 0", dict(slot=0), "must be NULL"),
    (merge, "no state at slot 2", dict(M=None), "M is NULL"),
    (merge, "negative slot", dict(slot=-1), "slot"),
    (merge, "H overlaps ACC", dict(H=Y + 64), "overlaps"),
    (merge, "start not 0/1", dict(start=3), "start"),
]


@pytest.mark.parametrize("fn,name,kw,msg", TWO_PHASE_INVALID, ids=[c[1] for c in TWO_PHASE_INVALID])
def test_two_phase_rejects(lib, fn, name, kw, msg):
    assert fn(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_two_phase_unsupported(lib):
    assert inter(lib, mode=F, r=8) == EINVAL  # full rank needs r == d
    assert inter(lib, nq=65) == EUNSUPPORTED
    assert merge(lib, d=4096) == EUNSUPPORTED


def allf(lib, V=A, K=None, Q=B, H=C, neff=D, S=6, N=8, d=64, r=8, first=2, T=5, mode=SL,
         dtype=BF16, eps=1e-6):
    return lib.lr_attnres_route_all_fwd(V, K, Q, H, neff, S, N, d, r, first, T, mode, dtype, eps,
                                        None)


ALL_INVALID = [
    ("first 0", dict(first=0), "first >= 1"),
    ("no sites", dict(T=0), "T >= 1"),
    ("sites past the stack", dict(first=2, T=6), "first + T - 1 <= S"),
    ("V NULL", dict(V=None), "V is NULL"),
    ("Q NULL", dict(Q=None), "Q is NULL"),
    ("H NULL", dict(H=None), "H is NULL"),
    ("K NULL when projected", dict(mode=P), "K is NULL"),
    ("K outside projected", dict(K=E), "must be NULL"),
    ("H misaligned", dict(H=C + 8), "16-byte aligned"),
    ("neff misaligned", dict(neff=D + 2), "4-byte aligned"),
    ("H overlaps V", dict(H=A + 64), "overlaps"),
    ("neff overlaps H", dict(neff=C + 128), "overlap"),
    ("sliced r > d", dict(r=65), "r <= d"),
    ("negative eps", dict(eps=-1.0), "eps"),
]


@pytest.mark.parametrize("name,kw,msg", ALL_INVALID, ids=[c[0] for c in ALL_INVALID])
def test_all_sites_rejects(lib, name, kw, msg):
    assert allf(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_all_sites_unsupported(lib):
    # Beyond the fused kernel the sites run one by one, so the limits are
    # those of the single-site forward at the last site (first + T - 1
    # sources).
    assert allf(lib, S=1026, first=1025, T=2) == EUNSUPPORTED
    assert "site by site" in err(lib)
    assert allf(lib, mode=F, r=8192, d=8192) == EUNSUPPORTED
    assert allf(lib, N=(1 << 30) + 1, S=2, first=1, T=1, d=8, r=8) == EUNSUPPORTED


def allb_ws(lib, S=6, N=8, d=64, r=8, first=2, T=5, mode=SL, dtype=BF16):
    return lib.lr_attnres_route_all_bwd_workspace_bytes(S, N, d, r, first, T, mode, dtype)


def allb(lib, V=A, K=None, Q=B, dH=C, dV=D, dK=None, dQ=E, ws=G, ws_bytes=1 << 20, S=6, N=8,
         d=64, r=8, first=2, T=5, mode=SL, dtype=BF16, eps=1e-6, acc=0):
    return lib.lr_attnres_route_all_bwd(V, K, Q, dH, dV, dK, dQ, ws, ws_bytes, S, N, d, r, first,
                                        T, mode, dtype, eps, acc, None)


def test_all_sites_backward_workspace(lib):
    # fused: one fp32 partial row of T x r per workgroup, at most 512 workgroups
    assert allb_ws(lib) == 8 * 5 * 8 * 4
    assert allb_ws(lib, N=100000, S=49, first=1, T=48, r=16, d=1024) == 512 * 48 * 16 * 4
    assert allb_ws(lib, N=0) == 0
    assert allb_ws(lib, first=0) == 0
    assert allb_ws(lib, first=2, T=6) == 0
    # site by site (full rank, fp32 storage, S > 64): the single-site
    # backward's workspace, reused by every site
    single = lib.lr_attnres_route_bwd_workspace_bytes
    assert allb_ws(lib, mode=F, r=64) == single(6, 8, 64, 64, F, BF16) > 0
    assert allb_ws(lib, dtype=F32) == single(6, 8, 64, 8, SL, F32) > 0
    assert allb_ws(lib, S=100, first=30, T=71, N=5000, d=1024, r=16, mode=P) == \
        single(100, 5000, 1024, 16, P, BF16)


ALLB_INVALID = [
    ("first 0", dict(first=0), "first >= 1"),
    ("sites past the stack", dict(T=6), "first + T - 1 <= S"),
    ("accumulate 2", dict(acc=2), "accumulate"),
    ("dH NULL", dict(dH=None), "dH is NULL"),
    ("dV NULL", dict(dV=None), "dV is NULL"),
    ("dQ NULL", dict(dQ=None), "dQ is NULL"),
    ("dK NULL when projected", dict(mode=P, K=W), "dK is NULL"),
    ("dK outside projected", dict(dK=W), "must be NULL"),
    ("dV misaligned", dict(dV=D + 8), "16-byte aligned"),
    ("dH misaligned", dict(dH=C + 4), "16-byte aligned"),
    ("dQ misaligned", dict(dQ=E + 2), "4-byte aligned"),
    ("workspace NULL", dict(ws=None), "workspace too small"),
    ("workspace too small", dict(ws_bytes=16), "workspace too small"),
    ("dV overlaps V", dict(dV=A + 256), "overlaps"),
    ("dQ overlaps dH", dict(dQ=C + 64), "overlaps"),
    ("workspace overlaps dV", dict(ws=D + 1024), "overlap"),
    ("negative eps", dict(eps=-1.0), "eps"),
]


@pytest.mark.parametrize("name,kw,msg", ALLB_INVALID, ids=[c[0] for c in ALLB_INVALID])
def test_all_sites_backward_rejects(lib, name, kw, msg):
    assert allb(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_all_sites_backward_unsupported(lib):
    # Beyond the fused kernel (full rank, fp32 storage, S, T or r above 64,
    # d % 8 != 0) the sites run one by one: the limits are the single-site
    # backward's at the last site.
    assert allb(lib, S=514, first=513, T=2) == EUNSUPPORTED
    assert "site by site" in err(lib)
    assert allb(lib, mode=P, K=W, dK=W + 0x1_0000_0000, r=257, d=1024) == EUNSUPPORTED
    assert allb(lib, mode=F, r=8192, d=8192) == EUNSUPPORTED
    assert allb(lib, dtype=F32, mode=F, r=8192, d=8192) == EUNSUPPORTED


def sdef(lib, V=A, K=None, q=B, dH=C, coef=D, dq=E, ws=G, ws_bytes=1 << 20, S=6, N=8, d=64, r=8,
         mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_route_bwd_deferred(V, K, q, dH, coef, dq, ws, ws_bytes, S, N, d, r, mode,
                                             dtype, eps, None)


def sgat(lib, V=A, K=None, source=2, dHs=C, Q=B, coef=D, stride=3 * 8 * 6, n_sites=4, dV=E,
         dK=None, S=6, N=8, d=64, r=8, mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_route_gather_bwd(V, K, source, dHs, Q, coef, stride, n_sites, dV, dK, S,
                                           N, d, r, mode, dtype, eps, None)


SDEF_INVALID = [
    ("coef NULL", dict(coef=None), "coef is NULL"),
    ("dq NULL", dict(dq=None), "dq is NULL"),
    ("K outside projected", dict(K=W), "must be NULL"),
    ("coef misaligned", dict(coef=D + 2), "4-byte aligned"),
    ("coef overlaps V", dict(coef=A + 64), "overlaps"),
    ("coef overlaps the workspace", dict(ws=D + 64), "overlap"),
    ("workspace too small", dict(ws_bytes=4), "workspace too small"),
]


@pytest.mark.parametrize("name,kw,msg", SDEF_INVALID, ids=[c[0] for c in SDEF_INVALID])
def test_deferred_site_rejects(lib, name, kw, msg):
    assert sdef(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_deferred_site_rejects_full_rank(lib):
    assert sdef(lib, mode=F, r=64) == EUNSUPPORTED
    assert "projected or sliced" in err(lib)


SGAT_INVALID = [
    ("negative source", dict(source=-1), "source and n_sites"),
    ("source past the stack", dict(source=6), "source must be < S"),
    ("negative n_sites", dict(n_sites=-1), "source and n_sites"),
    ("short stride", dict(stride=3 * 8 - 1), "coef_site_stride"),
    ("dV NULL", dict(dV=None), "dV is NULL"),
    ("dHs NULL", dict(dHs=None), "dHs is NULL"),
    ("dK NULL when projected", dict(mode=P, K=W), "dK is NULL"),
    ("dV misaligned", dict(dV=E + 8), "16-byte aligned"),
    ("dV overlaps dHs", dict(dV=C + 64), "overlaps"),
    ("dV overlaps coef", dict(dV=D + 256), "overlaps"),
]


@pytest.mark.parametrize("name,kw,msg", SGAT_INVALID, ids=[c[0] for c in SGAT_INVALID])
def test_source_gather_rejects(lib, name, kw, msg):
    assert sgat(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_source_gather_unsupported(lib):
    assert sgat(lib, mode=F, r=64) == EUNSUPPORTED
    assert sgat(lib, d=4104, r=8) == EUNSUPPORTED


def kproj(lib, A_=A, W=B, O=C, K=D, N=8, m=64, d=32, r=16, dtype=BF16):
    return lib.lr_attnres_key_proj_fwd(A_, W, O, K, N, m, d, r, dtype, None)


KPROJ_INVALID = [
    ("no outputs", dict(d=0, r=0), "d + r >= 1"),
    ("negative N", dict(N=-1), "N >= 0"),
    ("m zero", dict(m=0), "m >= 1"),
    ("A NULL", dict(A_=None), "A is NULL"),
    ("W misaligned", dict(W=B + 8), "16-byte aligned"),
    ("O NULL with d", dict(O=None), "O is NULL"),
    ("K NULL with r", dict(K=None), "K is NULL"),
    ("O given with d = 0", dict(d=0), "O must be NULL"),
    ("K given with r = 0", dict(r=0), "K must be NULL"),
    ("O misaligned", dict(O=C + 1), "2-byte aligned"),
    ("O overlaps A", dict(O=A + 32), "overlaps"),
    ("K overlaps O", dict(K=C + 64), "overlap"),
    ("unknown storage", dict(dtype=7), "storage"),
]


@pytest.mark.parametrize("name,kw,msg", KPROJ_INVALID, ids=[c[0] for c in KPROJ_INVALID])
def test_key_projection_rejects(lib, name, kw, msg):
    assert kproj(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_key_projection_unsupported(lib):
    assert kproj(lib, dtype=F32) == EUNSUPPORTED
    assert "bf16" in err(lib)
    assert kproj(lib, m=60) == EUNSUPPORTED
    assert kproj(lib, N=(1 << 30) + 1, m=8, d=8, r=8) == EUNSUPPORTED


def kproj_bwd(lib, A_=A, W=B, dO=C, dK=D, dA=E, dW=G, ws=None, wsb=0, N=8, m=64, d=32, r=16,
              dtype=BF16):
    return lib.lr_attnres_key_proj_bwd(A_, W, dO, dK, dA, dW, ws, wsb, N, m, d, r, dtype, None)


KPROJ_BWD_INVALID = [
    ("no outputs", dict(d=0, r=0), "d + r >= 1"),
    ("negative N", dict(N=-1), "N >= 0"),
    ("A NULL", dict(A_=None), "A is NULL"),
    ("dA NULL", dict(dA=None), "dA is NULL"),
    ("dW NULL", dict(dW=None), "dW is NULL"),
    ("dK misaligned", dict(dK=D + 8), "16-byte aligned"),
    ("dO given with d = 0", dict(d=0), "dO must be NULL"),
    ("dK given with r = 0", dict(r=0), "dK must be NULL"),
    ("dA overlaps A", dict(dA=A + 64), "overlaps"),
    ("dW overlaps dA", dict(dW=E + 256), "overlap"),
    ("workspace too small", dict(N=4096, m=512, d=512, r=16), "workspace too small"),
    ("unknown storage", dict(dtype=7), "storage"),
]


@pytest.mark.parametrize("name,kw,msg", KPROJ_BWD_INVALID, ids=[c[0] for c in KPROJ_BWD_INVALID])
def test_key_projection_bwd_rejects(lib, name, kw, msg):
    assert kproj_bwd(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_key_projection_bwd_unsupported(lib):
    assert kproj_bwd(lib, dtype=F32) == EUNSUPPORTED
    assert "bf16" in err(lib)
    assert kproj_bwd(lib, m=60) == EUNSUPPORTED
    assert kproj_bwd(lib, r=12) == EUNSUPPORTED
    assert kproj_bwd(lib, N=(1 << 30) + 1, m=8, d=8, r=8) == EUNSUPPORTED


def test_key_projection_bwd_workspace(lib):
    """Token splits only when the dW tile grid alone is small: the paper's
    projection shape (72 tiles) splits 16384 tokens 7 ways, 504 workgroups
    resident at once; a 512-tile grid and no tokens need none; unsupported
    inputs report 0."""
    ws = lib.lr_attnres_key_proj_bwd_workspace_bytes
    assert ws(16384, 1024, 1024, 16, BF16) == 7 * 1040 * 1024 * 4
    assert ws(16384, 2816, 1024, 16, BF16) == 2 * 1040 * 2816 * 4
    assert ws(100, 8192, 1024, 0, BF16) == 0
    assert ws(0, 1024, 1024, 16, BF16) == 0
    assert ws(64, 64, 32, 16, F32) == 0


def neff_call(lib, V=A, K=None, q=B, ne=C, S=4, N=8, d=64, r=8, mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_route_neff(V, K, q, ne, S, N, d, r, mode, dtype, eps, None)


def test_neff_rejects(lib):
    assert neff_call(lib, ne=None) == EINVAL and "neff is NULL" in err(lib)
    assert neff_call(lib, ne=A + 4) == EINVAL and "overlaps" in err(lib)
    assert neff_call(lib, K=E) == EINVAL and "must be NULL" in err(lib)
    assert neff_call(lib, mode=P) == EINVAL and "K is NULL" in err(lib)
    assert neff_call(lib, mode=F, r=8) == EINVAL
    assert neff_call(lib, S=1025, N=2) == EUNSUPPORTED


def dbwd(lib, B=A, KB=None, dP=B_, dKP=None, coef=X, o_new=C, k_new=None, q=E, dH=D, dO=G,
         dK=None, dq=Y, ws=W, wsb=1 << 30, n_src=3, N=8, d=64, r=8, mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_block_route_bwd_deferred(B, KB, dP, dKP, coef, o_new, k_new, q, dH, dO,
                                                   dK, dq, ws, wsb, n_src, N, d, r, mode, dtype,
                                                   eps, None)


def gath(lib, B=A, KB=None, slot=1, dHs=C, Q=E, coef=X, stride=3 * 8, n_sites=4, dP=B_, dKP=None,
         N=8, d=64, r=8, mode=SL, dtype=BF16, eps=1e-6):
    return lib.lr_attnres_block_gather_bwd(B, KB, slot, dHs, Q, coef, stride, n_sites, dP, dKP, N,
                                           d, r, mode, dtype, eps, None)


DEFERRED_INVALID = [
    (dbwd, "coef NULL with completed slots", dict(coef=None), "coef is NULL"),
    (dbwd, "dP NULL", dict(dP=None), "dP is NULL"),
    (dbwd, "dKP outside projected", dict(dKP=Z), "must be NULL"),
    (dbwd, "coef overlaps dH", dict(coef=D + 64), "overlaps"),
    (dbwd, "dP overlaps coef", dict(dP=X + 16), "overlap"),
    (gath, "negative slot", dict(slot=-1), "slot"),
    (gath, "coef stride too small", dict(stride=8), "coef_site_stride"),
    (gath, "dP overlaps dHs", dict(dP=C + 16), "overlaps"),
    (gath, "dHs NULL", dict(dHs=None), "dHs is NULL"),
    (gath, "KB outside projected", dict(KB=Z), "must be NULL"),
]


@pytest.mark.parametrize("fn,name,kw,msg", DEFERRED_INVALID, ids=[c[1] for c in DEFERRED_INVALID])
def test_deferred_reverse_pass_rejects(lib, fn, name, kw, msg):
    assert fn(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_deferred_reverse_pass_unsupported(lib):
    assert dbwd(lib, d=66) == EUNSUPPORTED
    assert gath(lib, n_sites=1025, stride=24) == EUNSUPPORTED
    assert gath(lib, d=4096) == EUNSUPPORTED


def state_call(lib, V=A, K=None, q=B, M=C, L=D, ACC=G, S=10, N=8, d=64, r=8, chunk=4, mode=SL,
               dtype=BF16, eps=1e-6):
    return lib.lr_attnres_route_state_fwd(V, K, q, M, L, ACC, S, N, d, r, chunk, mode, dtype, eps,
                                          None)


def merge_call(lib, M=C, L=D, ACC=G, H=A, P=3, N=8, d=64, dtype=BF16):
    return lib.lr_attnres_route_merge_fwd(M, L, ACC, H, P, N, d, dtype, None)


STATE_INVALID = [
    (state_call, "chunk zero", dict(chunk=0), "chunk"),
    (state_call, "M NULL", dict(M=None), "M is NULL"),
    (state_call, "ACC misaligned", dict(ACC=G + 4), "16-byte aligned"),
    (state_call, "K outside projected", dict(K=E), "must be NULL"),
    (state_call, "K NULL when projected", dict(mode=P), "K is NULL"),
    # 3 chunks x 8 tokens x 4 bytes of M reach into L 64 bytes on.
    (state_call, "L overlaps M", dict(L=C + 64), "overlap"),
    (state_call, "ACC overlaps V", dict(ACC=A + 256), "overlaps"),
    (merge_call, "P zero", dict(P=0), "P must be"),
    (merge_call, "H NULL", dict(H=None), "H is NULL"),
    (merge_call, "unknown dtype", dict(dtype=5), "dtype"),
    (merge_call, "H overlaps ACC", dict(H=G + 256), "overlaps"),
    (merge_call, "ACC misaligned", dict(ACC=G + 8), "16-byte aligned"),
]


@pytest.mark.parametrize("fn,name,kw,msg", STATE_INVALID, ids=[c[1] for c in STATE_INVALID])
def test_split_sources_rejects(lib, fn, name, kw, msg):
    assert fn(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_split_sources_unsupported(lib):
    assert state_call(lib, S=2000, chunk=1025) == EUNSUPPORTED and "1024" in err(lib)
    assert state_call(lib, S=70000, chunk=1, N=2) == EUNSUPPORTED and "65535" in err(lib)
    assert state_call(lib, mode=F, d=8192, r=8192) == EUNSUPPORTED
    assert merge_call(lib, P=1025) == EUNSUPPORTED and "1024" in err(lib)


def bfc_call(lib, B=A, KB=None, BC=C, KBC=None, o_new=D, k_new=None, q=E, H=G, n_src=3, start=0,
             finish=0, N=8, d=64, r=8, mode=SL, eps=1e-6):
    return lib.lr_attnres_block_route_fwd_bf16c(B, KB, BC, KBC, o_new, k_new, q, H, n_src, start,
                                                finish, N, d, r, mode, eps, None)


BFC_INVALID = [
    ("finish not 0/1", dict(finish=2), "finish"),
    ("BC NULL with completed slots", dict(BC=None), "BC is NULL"),
    ("BC NULL when finishing", dict(BC=None, n_src=1, finish=1), "BC is NULL"),
    ("BC misaligned", dict(BC=C + 8), "16-byte aligned"),
    ("KBC outside projected", dict(KBC=W), "must be NULL"),
    ("KBC NULL when projected", dict(mode=P, KB=W, k_new=B_, KBC=None), "KBC is NULL"),
    ("BC overlaps B", dict(BC=A + 64), "overlap"),
    ("H overlaps BC", dict(H=C + 16), "overlap"),
    ("BC overlaps o_new", dict(BC=D - 64), "overlap"),
]


@pytest.mark.parametrize("name,kw,msg", BFC_INVALID, ids=[c[0] for c in BFC_INVALID])
def test_block_bf16_copies_rejects(lib, name, kw, msg):
    assert bfc_call(lib, **kw) == EINVAL
    assert msg in err(lib)


def test_block_bf16_copies_unsupported(lib):
    assert bfc_call(lib, d=66) == EUNSUPPORTED
    assert bfc_call(lib, d=4096) == EUNSUPPORTED


def test_last_error_is_per_thread(lib):
    """Two threads make different invalid calls, interleaved; each reads back
    its own message afterwards (the error string is thread-local)."""
    import threading

    step = threading.Barrier(2)
    seen = {}

    def first():
        assert fwd(lib, V=None) == EINVAL       # "V is NULL"
        step.wait()                             # the other thread fails now
        step.wait()
        seen["first"] = err(lib)

    def second():
        step.wait()
        assert fwd(lib, N=-1) == EINVAL         # "N >= 0"
        step.wait()
        seen["second"] = err(lib)

    threads = [threading.Thread(target=first), threading.Thread(target=second)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=30)
    assert "V is NULL" in seen["first"]
    assert "N >= 0" in seen["second"]
