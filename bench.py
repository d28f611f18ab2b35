"""Benchmark of the LR-AttnRes depth-routing path on one MI355X.

One step = one pass of the whole routing hot path (scores, depth softmax,
value mix; then the backward's recomputation, value-gradient dots, dV, dK and
dq) over one batch: projected low-rank keys, d = 2048, r = 32, N = 4 x 4096
tokens, S = 64 sources, bf16 values and keys, fp32 arithmetic, fp32 q / dq.
Inputs are synthetic Gaussians resident in HBM before the timed region.

Prints ONE JSON line: tokens/s of the step, the HBM roofline of the dominant
kernel (the backward) from HIP events on its stream, the fp64 CPU oracle
timed on a bounded token sample, and the other measured workloads (the
49-site model pass with projected and sliced keys, the full-rank baseline at
S = 49, the forward alone) under "extra".
"""
from __future__ import annotations

import argparse
import platform
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak
METRIC = "depth-routing tokens/s and achieved HBM TB/s (% of peak), fwd and fwd+bwd"
KERNEL_DIR = os.path.join(ROOT, "paper_2607_09694_amd", "csrc")
COUNTERS = os.path.join(ROOT, "profiles", "route_bwd_lr_d2048_counters.txt")

# Main workload: projected keys, forward + backward.
S5, N5, D5, R5 = 64, 16384, 2048, 32


def fwd_bytes(S, N, d, r, mode):
    """Algorithmic HBM bytes of one forward call (bf16): every value row once,
    projected keys once (sliced keys are a view of the values), H written."""
    key = r if mode == 0 else 0
    return S * N * (d + key) * 2 + N * d * 2


def bwd_bytes(S, N, d, r):
    """Projected-key backward (bf16): V and K read, dV and dK written, dH read."""
    return 2 * S * N * (d + r) * 2 + N * d * 2


# The sources that define the measured backward and forward kernels; the
# committed counter summary is valid only while these are unchanged.
KERNEL_FILES = ("route_bwd.hip", "route_fwd.hip", "route_common.h", "route_device.h")


def kernel_source_hash():
    h = hashlib.sha256()
    for name in KERNEL_FILES:
        with open(os.path.join(KERNEL_DIR, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(algo_bytes):
    """HBM bytes per launch of the backward kernel from committed rocprofv3
    counter summaries, if they were taken on the current kernel sources."""
    try:
        with open(COUNTERS) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("kernel_source_hash") != kernel_source_hash():
        return None
    return c.get("hbm_bytes_per_launch")


def load_probe():
    """Streaming copy / read / fill kernels of known traffic (benchmark helper)."""
    import ctypes

    path = os.path.join(ROOT, "paper_2607_09694_amd", "libhbmprobe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build the package first")
    lib = ctypes.CDLL(path)
    vp, ll, i = ctypes.c_void_p, ctypes.c_longlong, ctypes.c_int
    for f in (lib.hbm_probe_copy, lib.hbm_probe_read):
        f.argtypes = [vp, vp, ll, i, vp]
        f.restype = i
    for f in (lib.hbm_probe_copy_u, lib.hbm_probe_read_u):
        f.argtypes = [vp, vp, ll, i, i, vp]
        f.restype = i
    lib.hbm_probe_fill_u.argtypes = [vp, ll, i, i, vp]
    lib.hbm_probe_fill_u.restype = i
    return lib


def probe_ceilings(torch, dev, reps, warmup):
    """HBM ceilings measured on this GPU with 4 GiB streams: read only, read +
    write (copy) and write only (fill), each the best over grid sizes and
    loads in flight per lane (1-8 independent 16-byte loads)."""
    probe = load_probe()
    nbytes = 4 << 30
    src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream().cuda_stream
    best = {"read_GBps": 0.0, "copy_GBps": 0.0, "fill_GBps": 0.0}
    how = {}
    runs = []
    for u in (2, 4, 8):
        for blocks in (1024, 4096, 16384, 65536):
            runs.append(("copy_GBps", u, blocks, 2, lambda u=u, b=blocks: probe.hbm_probe_copy_u(
                src.data_ptr(), dst.data_ptr(), nbytes, b, u, st)))
    for u in (4, 8):
        for blocks in (256, 512, 2048):
            runs.append(("read_GBps", u, blocks, 1, lambda u=u, b=blocks: probe.hbm_probe_read_u(
                src.data_ptr(), sink.data_ptr(), nbytes, b, u, st)))
    for blocks in (4096, 65536):
        runs.append(("fill_GBps", 4, blocks, 1, lambda b=blocks: probe.hbm_probe_fill_u(
            dst.data_ptr(), nbytes, b, 4, st)))
    for key, u, blocks, mult, fn in runs:
        ts = time_calls(torch, lambda: check_probe(fn()), reps, warmup)
        rate = round(mult * nbytes / (np.median(ts) * 1e-3) / 1e9, 1)
        if rate > best[key]:
            best[key] = rate
            how[key] = f"{u} loads in flight per lane, {blocks} workgroups"
    best["best_config"] = how
    del src, dst
    return best


def check_probe(rc):
    if rc != 0:
        raise RuntimeError(f"hbm probe launch failed ({rc})")


class Flusher:
    """Untimed read of a 1 GiB buffer between timed calls, so that the 256 MB
    memory-side cache (MALL) holds none of the data a previous call left in
    it.  A read, not a write: a written flush buffer leaves dirty lines whose
    write-back then overlaps the timed call (measured: 4-5% slower forward
    calls on MI355X)."""

    def __init__(self, torch, dev):
        self.torch = torch
        self.buf = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        self.out = torch.empty((), dtype=torch.float32, device=dev)

    def __call__(self):
        self.torch.sum(self.buf, dim=0, out=self.out)


def time_calls(torch, fn, reps, warmup, flush=None):
    """Per-call device time (ms) from HIP events on the current stream."""
    st = torch.cuda.current_stream()
    for _ in range(warmup):
        fn()
    ts = []
    for _ in range(reps):
        if flush:
            flush()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        fn()
        b.record(st)
        ts.append((a, b))
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ts]


def cpu_baseline(g, q, target_s=10.0, chunk=1024, single_s=4.0):
    """fp64 oracle (as it stands) on the host: fwd + bwd of the main workload
    in 1024-token chunks, in order, repeated over the whole token set until
    about target_s seconds have passed, on every host thread; then the same
    on one thread for about single_s seconds.  Host copies of the inputs are
    made before timing."""
    import oracle
    from paper_2607_09694_amd.inputs import bf16_tensor_to_bits

    V, K, dH = (bf16_tensor_to_bits(g[k]) for k in ("V", "K", "dH"))

    def run(limit, step):
        done, spent = 0, 0.0
        while spent < limit:
            n0 = done % N5
            n1 = min(N5, n0 + step)
            t0 = time.perf_counter()
            oracle.route_fwd(V, K, q, oracle.PROJECTED, n0=n0, n1=n1)
            oracle.route_bwd(V, K, q, dH, oracle.PROJECTED, n0=n0, n1=n1)
            spent += time.perf_counter() - t0
            done += n1 - n0
        return done, spent

    cores = oracle.num_threads()
    done, spent = run(target_s, chunk)
    oracle.set_num_threads(1)
    done1, spent1 = run(single_s, 64)
    oracle.set_num_threads(cores)
    cpu = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    per_token = (fwd_bytes(S5, N5, D5, R5, 0) + bwd_bytes(S5, N5, D5, R5)) / N5
    return {"value": round(done / spent, 1), "unit": "tokens/s", "cores": cores,
            "kind": "oracle",
            "algo_GBps": round(done / spent * per_token / 1e9, 2),
            "sample": f"{done} tokens ({done / N5:.2f} passes over all {N5} tokens) of the main "
                      f"workload, fwd+bwd in fp64, {spent:.1f} s",
            "single_thread_value": round(done1 / spent1, 1),
            "single_thread_sample": f"{done1} tokens in 64-token chunks, {spent1:.1f} s",
            "cpu": cpu}


def device_state(torch, dev):
    """Clock levels and power of the GPU, read from its sysfs entries
    (read-only; empty where the files are not readable)."""
    import glob

    p = torch.cuda.get_device_properties(dev)
    out = {"name": p.name, "arch": p.gcnArchName, "compute_units": p.multi_processor_count}
    bdf = f"{p.pci_domain_id:04x}:{p.pci_bus_id:02x}:{p.pci_device_id:02x}.0"
    base = f"/sys/bus/pci/devices/{bdf}"
    for key, fname in (("sclk", "pp_dpm_sclk"), ("mclk", "pp_dpm_mclk"),
                       ("fclk", "pp_dpm_fclk")):
        try:
            with open(f"{base}/{fname}") as f:
                cur = [l.split(":", 1)[1].strip() for l in f if l.rstrip().endswith("*")]
            if cur:
                out[key] = cur[0].rstrip("*").strip()
        except OSError:
            pass
    try:
        with open(f"{base}/power_dpm_force_performance_level") as f:
            out["perf_level"] = f.read().strip()
    except OSError:
        pass
    for hw in glob.glob(f"{base}/hwmon/hwmon*"):
        for name in ("power1_average", "power1_input"):
            try:
                with open(f"{hw}/{name}") as f:
                    out["power_W"] = round(int(f.read().strip()) / 1e6, 1)
                break
            except (OSError, ValueError):
                continue
        try:
            with open(f"{hw}/power1_cap") as f:
                out["power_cap_W"] = round(int(f.read().strip()) / 1e6, 1)
        except (OSError, ValueError):
            pass
    return out


def all_sites_bytes(S, T, N, d, r, mode, es=2):
    """Bytes one all-sites call must move: the stack once (keys too when
    projected), every site's state written once, N_eff in fp32."""
    keys = S * N * r * es if mode == 0 else 0
    return S * N * d * es + keys + T * N * d * es + T * N * 4


def all_sites_bwd_bytes(S, T, N, d, r, mode, es=2):
    """Bytes one all-sites backward must move: the stack and the keys read
    once, every site's upstream gradient read once, dV (and dK) written once."""
    keys = 2 * S * N * r * es if mode == 0 else 0
    return 2 * S * N * d * es + keys + T * N * d * es


def all_sites_backward(torch, lr, dev, mode, r, V, K, queries, reps, warmup, flush,
                       per_site=True):
    """Backward of sites 2..49 of the 49-source pass (prefixes of 2..49
    sources) in one call, cold; beside it, the same gradients as 48
    accumulating single-site backward calls (warm, once)."""
    S, N, d = V.shape
    T = 48
    gen = torch.Generator(device=dev).manual_seed(300 + r)
    dH = torch.randn((T, N, d), generator=gen, device=dev).to(torch.bfloat16)
    Qa = queries[1:].contiguous()
    dV = torch.empty_like(V)
    dK = torch.empty_like(K) if K is not None else None
    dQ = torch.empty((T, r), dtype=torch.float32, device=dev)
    ws = torch.empty((max(16, lr.route_all_bwd_workspace_bytes(S, N, d, r, 2, T, mode,
                                                               V.dtype)),),
                     dtype=torch.uint8, device=dev)
    ts = time_calls(torch, lambda: lr.route_all_bwd(V, K, Qa, dH, mode, 2, out=(dV, dK, dQ),
                                                    workspace=ws), reps, warmup, flush)
    med = float(np.median(ts))
    nbytes = all_sites_bwd_bytes(S, T, N, d, r, mode)
    res = {"median_ms": med, "min_ms": float(np.min(ts)), "max_ms": float(np.max(ts)),
           "tokens_per_s": N / (med * 1e-3), "algo_bytes": nbytes,
           "algo_GBps": nbytes / (med * 1e-3) / 1e9,
           "frac_of_peak": nbytes / (med * 1e-3) / 1e9 / HBM_PEAK_GBS}
    if per_site:
        # The same gradients from the single-site backward: site j reads the
        # first j + 2 sources and adds into their gradient rows.
        wsb = torch.empty((lr.route_bwd_workspace_bytes(S, N, d, r, mode, V.dtype),),
                          dtype=torch.uint8, device=dev)
        dq = torch.empty((T, r), dtype=torch.float32, device=dev)
        dV.zero_()
        if dK is not None:
            dK.zero_()
        dq.zero_()

        def sweep():
            for j in range(T - 1, -1, -1):
                s = j + 2
                lr.route_bwd(V[:s], K[:s] if K is not None else None, Qa[j], dH[j], mode,
                             out=(dV[:s], dK[:s] if dK is not None else None, dq[j]),
                             workspace=wsb, accumulate=True)
        tp = time_calls(torch, sweep, 1, 0, flush)
        res["per_site_accumulating_calls_ms"] = float(tp[0])
        res["speedup_vs_per_site_calls"] = float(tp[0]) / med
        del wsb, dq
    del dH, dV, dK, dQ, ws
    return res


def model_training_pass(torch, lr, dev, V, K, mode, r, reps, warmup):
    """A whole full-source training pass over the 49-source stack V [49, N, d]
    (site t reads sources 0 .. t-1): the forward at every site, then the
    reverse pass in two forms, each timed end to end with HIP events, warm:
    48 + 1 accumulating single-site backward calls, and the deferred form
    (per site its coefficients, then one gather for the source that became
    final)."""
    T, N, d = V.shape
    gen = torch.Generator(device=dev).manual_seed(400 + r)
    Q = torch.randn((T, r), generator=gen, device=dev) / r ** 0.5
    dH = torch.randn((T, N, d), generator=gen, device=dev).to(torch.bfloat16)
    H = torch.empty((N, d), dtype=V.dtype, device=dev)
    dV = torch.empty_like(V)
    dK = torch.empty_like(K) if K is not None else None
    dq = torch.empty((T, r), dtype=torch.float32, device=dev)
    ws = torch.empty((lr.route_bwd_workspace_bytes(T, N, d, r, mode, V.dtype),),
                     dtype=torch.uint8, device=dev)
    coefs = torch.empty((T, T, 3, N), dtype=torch.float32, device=dev)

    def fwd():
        for t in range(1, T + 1):
            lr.route_fwd(V[:t], K[:t] if K is not None else None, Q[t - 1], mode, out=H)

    def bwd():
        dV.zero_()
        if dK is not None:
            dK.zero_()
        for t in range(T, 0, -1):
            lr.route_bwd(V[:t], K[:t] if K is not None else None, Q[t - 1], dH[t - 1], mode,
                         out=(dV[:t], dK[:t] if dK is not None else None, dq[t - 1]),
                         workspace=ws, accumulate=True)

    def bwd_deferred():
        for t in range(T, 0, -1):
            lr.route_bwd_deferred(V[:t], K[:t] if K is not None else None, Q[t - 1], dH[t - 1],
                                  mode, coefs[t - 1, :t], dq=dq[t - 1], workspace=ws)
            i = t - 1
            lr.route_gather_bwd(V, K, i, dH[i:], Q[i:], coefs[i:, i], mode,
                                out=(dV[i], dK[i] if dK is not None else None))

    st = torch.cuda.current_stream()
    res = {}
    for name, back in (("accumulating_", bwd), ("deferred_", bwd_deferred)):
        for _ in range(warmup):
            fwd()
            back()
        tf, tb = [], []
        for _ in range(reps):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record(st)
            fwd()
            e[1].record(st)
            back()
            e[2].record(st)
            torch.cuda.synchronize()
            tf.append(e[0].elapsed_time(e[1]))
            tb.append(e[1].elapsed_time(e[2]))
        f, b = float(np.median(tf)), float(np.median(tb))
        res.update({"fwd_pass_ms": f, name + "bwd_pass_ms": b, name + "step_ms": f + b,
                    name + "tokens_per_s": N / ((f + b) * 1e-3)})
    del dH, dV, dK, ws, coefs
    return res


def block_pass_bytes(t, c, N, d, r, mode, es=2, completed_bf16=False):
    """Algorithmic HBM bytes of the fused block call at site t: the earlier
    fp32 slots (with their fp32 key slots for projected keys) read once, the
    updated slot read (unless it starts) and written, o_{t-1} read, h written.
    completed_bf16: the earlier slots are bf16 copies (2 bytes), and a call
    that completes its block also writes the slot's bf16 copy."""
    if t == 1:
        j, start, finish = 0, True, True
    else:
        j, start, finish = (t - 2) // c + 1, (t - 2) % c == 0, (t - 1) % c == 0
    row = d + (r if mode == 0 else 0)
    eb = 2 if completed_bf16 else 4
    b = j * N * row * eb + (0 if start else N * row * 4) + N * row * 4
    if completed_bf16 and finish:
        b += N * row * 2
    return b + N * row * es + N * d * es


def block_deferred_bwd_bytes(T, c, N, d, r, mode, es=2):
    """Algorithmic HBM bytes of the deferred block reverse pass over T sites
    with blocks of c outputs.  Site step with j completed slots: the j + 1
    fp32 slot rows read, the partial slot's gradient rows read and written,
    dH read, 3 fp32 coefficients per completed slot written, and the fused
    retire (slot row written back, o_new / k_new read, dO / dK written).
    Gather of slot p read as completed by u sites: their dH and
    coefficients read, the slot's fp32 key read, its gradient written."""
    row = d + (r if mode == 0 else 0)
    nsrc = [1] + [(t - 2) // c + 2 for t in range(2, T + 1)]
    total = 0
    for n_src in nsrc:
        j = n_src - 1
        total += (j + 1) * N * row * 4 + N * row * 8 + N * d * es + j * 3 * N * 4 \
            + N * row * (4 + es + es)
    for p in sorted(set(n - 1 for n in nsrc)):
        u = sum(1 for n in nsrc if n - 1 > p)
        total += u * N * d * es + u * 3 * N * 4 + N * r * 4 + N * row * 4
    return total


def block_pass(torch, lr, dev, O, mode, r, c, reps, warmup, flush, completed_bf16=False):
    """49-site block-source forward pass over the output stack O [49, N, d].
    Each site's real call (with its own start flag) is timed `reps` times;
    before each, untimed, the updated slot is restored and the MALL flushed.
    completed_bf16: the completed summaries are read from bf16 copies."""
    T, N, d = O.shape
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    KB = torch.zeros((nslots, N, r), dtype=torch.float32, device=dev) if mode == 0 else None
    BC = KBC = None
    if completed_bf16:
        BC = torch.zeros((nslots, N, d), dtype=torch.bfloat16, device=dev)
        KBC = torch.zeros((nslots, N, r), dtype=torch.bfloat16, device=dev) if mode == 0 else None
    gen = torch.Generator(device=dev).manual_seed(100 + r)
    KO = (torch.randn((T, N, r), generator=gen, device=dev).to(torch.bfloat16)
          if mode == 0 else None)
    Q = torch.randn((T, r), generator=gen, device=dev) / r ** 0.5
    H = torch.empty((N, d), dtype=O.dtype, device=dev)
    st = torch.cuda.current_stream()
    total, nbytes = 0.0, 0
    for t in range(1, T + 1):
        n_src, start = (1, True) if t == 1 else ((t - 2) // c + 2, (t - 2) % c == 0)
        j = n_src - 1
        kn = KO[t - 1] if KO is not None else None
        saved = B[j].clone()
        ksaved = KB[j].clone() if KB is not None else None

        def restore():
            B[j].copy_(saved)
            if KB is not None:
                KB[j].copy_(ksaved)

        finish = t == 1 or (t - 1) % c == 0

        def call():
            if completed_bf16:
                lr.block_route_fwd_bf16c(B, KB, BC, KBC, O[t - 1], kn, Q[t - 1], n_src, start,
                                         finish, mode, out=H)
            else:
                lr.block_route_fwd(B, KB, O[t - 1], kn, Q[t - 1], n_src, start, mode, out=H)

        for _ in range(warmup):
            restore()
            call()
        ev = []
        for _ in range(reps):
            restore()
            flush()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            call()
            b.record(st)
            ev.append((a, b))
        torch.cuda.synchronize()
        total += float(np.median([a.elapsed_time(b) for a, b in ev]))
        nbytes += block_pass_bytes(t, c, N, d, r, mode, completed_bf16=completed_bf16)
        del saved, ksaved
    del B, KB, KO, BC, KBC
    return {"total_ms": total, "tokens_per_s": N / (total * 1e-3),
            "algo_GBps": nbytes / (total * 1e-3) / 1e9,
            "frac_of_peak": nbytes / (total * 1e-3) / 1e9 / HBM_PEAK_GBS}


def block_training_pass(torch, lr, dev, O, mode, r, c, reps, warmup):
    """A whole block-source training pass: the forward at all 49 sites, then
    the reverse pass (slot gradients zeroed first, then one fused backward
    call per site, last site first).  Timed end to end with HIP events; the
    MALL is not flushed between sites (a real step runs them back to back)."""
    T, N, d = O.shape
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    dB = torch.zeros_like(B)
    KB = torch.zeros((nslots, N, r), dtype=torch.float32, device=dev) if mode == 0 else None
    dKB = torch.zeros_like(KB) if KB is not None else None
    gen = torch.Generator(device=dev).manual_seed(200 + r)
    KO = (torch.randn((T, N, r), generator=gen, device=dev).to(torch.bfloat16)
          if mode == 0 else None)
    Q = torch.randn((T, r), generator=gen, device=dev) / r ** 0.5
    dHs = torch.randn((T, N, d), generator=gen, device=dev).to(torch.bfloat16)
    H = torch.empty((N, d), dtype=O.dtype, device=dev)
    dO = torch.empty((N, d), dtype=O.dtype, device=dev)
    dK = torch.empty((N, r), dtype=O.dtype, device=dev) if mode == 0 else None
    dq = torch.empty((r,), dtype=torch.float32, device=dev)
    ws = torch.empty((lr.route_bwd_workspace_bytes(nslots, N, d, r, mode, torch.float32),),
                     dtype=torch.uint8, device=dev)
    sites = [(1, True)] + [((t - 2) // c + 2, (t - 2) % c == 0) for t in range(2, T + 1)]

    def fwd():
        for t in range(1, T + 1):
            n_src, start = sites[t - 1]
            lr.block_route_fwd(B, KB, O[t - 1], KO[t - 1] if KO is not None else None,
                               Q[t - 1], n_src, start, mode, out=H)

    def bwd():
        dB.zero_()
        if dKB is not None:
            dKB.zero_()
        for t in range(T, 0, -1):
            lr.block_route_bwd(B, KB, dB, dKB, O[t - 1], KO[t - 1] if KO is not None else None,
                               Q[t - 1], dHs[t - 1], sites[t - 1][0], mode,
                               out=(dO, dK, dq), workspace=ws)

    # The deferred form: a completed slot's gradient is gathered once, when
    # the reverse pass reaches its block, from the coefficients the later
    # sites recorded; only the block in progress keeps a running gradient.
    coef = torch.empty((T, nslots, 3, N), dtype=torch.float32, device=dev)
    dP = dB[0]
    dKP = dKB[0] if dKB is not None else None

    def bwd_deferred():
        cur = None
        for t in range(T, 0, -1):
            n_src = sites[t - 1][0]
            p = n_src - 1
            if p != cur:
                first = p * c + 2 if p >= 1 else 2
                lr.block_gather_bwd(B, KB, p, dHs, Q, coef, first - 1, mode, out=(dP, dKP))
                cur = p
            lr.block_route_bwd_deferred(B, KB, dP, dKP, coef[t - 1, :n_src - 1], O[t - 1],
                                        KO[t - 1] if KO is not None else None, Q[t - 1],
                                        dHs[t - 1], n_src, mode, out=(dO, dK, dq), workspace=ws)

    st = torch.cuda.current_stream()
    res = {}
    for name, back in (("", bwd), ("deferred_", bwd_deferred)):
        for _ in range(warmup):
            fwd()
            back()
        tf, tb = [], []
        for _ in range(reps):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record(st)
            fwd()
            e[1].record(st)
            back()
            e[2].record(st)
            torch.cuda.synchronize()
            tf.append(e[0].elapsed_time(e[1]))
            tb.append(e[1].elapsed_time(e[2]))
        f, b = float(np.median(tf)), float(np.median(tb))
        res.update({name + "fwd_pass_ms": f, name + "bwd_pass_ms": b, name + "step_ms": f + b,
                    name + "tokens_per_s": N / ((f + b) * 1e-3)})
    # Roofline of the forward pass and of the deferred reverse pass and step
    # on their algorithmic bytes (warm: the sites run back to back).
    fb = sum(block_pass_bytes(t, c, N, d, r, mode) for t in range(1, T + 1))
    bb = block_deferred_bwd_bytes(T, c, N, d, r, mode)
    f, b = res["deferred_fwd_pass_ms"], res["deferred_bwd_pass_ms"]
    res.update({"fwd_pass_algo_bytes": fb, "deferred_bwd_pass_algo_bytes": bb,
                "fwd_pass_frac_of_peak": fb / (f * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "deferred_bwd_pass_frac_of_peak": bb / (b * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "deferred_step_frac_of_peak": (fb + bb) / ((f + b) * 1e-3) / 1e9 / HBM_PEAK_GBS})
    del B, dB, KB, dKB, KO, dHs, ws, coef
    return res


def block_inference_passes(torch, lr, dev, O, mode, r, c, reps, warmup):
    """Warm, back-to-back 49-site block-source inference: one fused call per
    site, against the two-phase form of Sec. 3.5 (phase 1 once per block over
    the completed slots for all of its sites' queries, then one merge call per
    site).  Both produce the same h."""
    T, N, d = O.shape
    nslots = (T - 2) // c + 2
    B = torch.zeros((nslots, N, d), dtype=torch.float32, device=dev)
    KB = torch.zeros((nslots, N, r), dtype=torch.float32, device=dev) if mode == 0 else None
    gen = torch.Generator(device=dev).manual_seed(300 + r)
    KO = (torch.randn((T, N, r), generator=gen, device=dev).to(torch.bfloat16)
          if mode == 0 else None)
    Q = torch.randn((T, r), generator=gen, device=dev) / r ** 0.5
    H = torch.empty((N, d), dtype=O.dtype, device=dev)
    M = torch.empty((c, N), dtype=torch.float32, device=dev)
    L = torch.empty((c, N), dtype=torch.float32, device=dev)
    ACC = torch.empty((c, N, d), dtype=torch.float32, device=dev)
    kn = (lambda t: KO[t - 1]) if KO is not None else (lambda t: None)

    def per_site():
        lr.block_route_fwd(B, KB, O[0], kn(1), Q[0], 1, True, mode, out=H)
        for t in range(2, T + 1):
            lr.block_route_fwd(B, KB, O[t - 1], kn(t), Q[t - 1], (t - 2) // c + 2,
                               (t - 2) % c == 0, mode, out=H)

    def two_phase():
        lr.block_merge_fwd(B, KB, O[0], kn(1), Q[0], None, 0, True, mode, out=H)
        t = 2
        while t <= T:
            j = (t - 2) // c + 1
            span = list(range(t, min(t + c, T + 1)))
            nq = len(span)
            lr.block_inter_fwd(B, KB, Q[span[0] - 1:span[-1]], j, mode,
                               out=(M[:nq], L[:nq], ACC[:nq]))
            for k, s_ in enumerate(span):
                lr.block_merge_fwd(B, KB, O[s_ - 1], kn(s_), Q[s_ - 1], (M[k], L[k], ACC[k]), j,
                                   k == 0, mode, out=H)
            t = span[-1] + 1

    st = torch.cuda.current_stream()
    res = {}
    for name, fn in (("per_site_ms", per_site), ("two_phase_ms", two_phase)):
        for _ in range(warmup):
            fn()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            fn()
            b.record(st)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        res[name] = float(np.median(ts))
    res["tokens_per_s_two_phase"] = N / (res["two_phase_ms"] * 1e-3)
    del B, KB, KO, ACC
    return res


def decode_model_pass(torch, lr, dev, reps, warmup, N=128, d=1024, r=16):
    """A decode-sized model pass (N = 128 tokens, 49 sites, P-LR r = 16):
    49 launches of a few microseconds each, eager and replayed from one
    captured HIP graph."""
    from paper_2607_09694_amd.inputs import PROJECTED, make_device_problem

    g = make_device_problem(PROJECTED, 49, N, d, r, dev, seed=4, n_queries=49)
    V, K, Q = g["V"], g["K"], g["q"]
    Hs = torch.empty((49, N, d), dtype=torch.bfloat16, device=dev)

    def pass_():
        for t in range(1, 50):
            lr.route_fwd(V[:t], K[:t], Q[t - 1], PROJECTED, out=Hs[t - 1])

    st = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(warmup):
            fn()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            fn()
            b.record(st)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    eager = timed(pass_)
    side = torch.cuda.Stream()
    side.wait_stream(st)
    with torch.cuda.stream(side):
        pass_()
    st.wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pass_()
    replay = timed(graph.replay)
    del g, V, K, Hs, graph
    return {"tokens": N, "eager_ms": eager, "graph_ms": replay,
            "graph_tokens_per_s": N / (replay * 1e-3)}


def split_sources(torch, lr, dev, reps, warmup, flush, S=49, d=1024, r=16):
    """The deepest site (49 sources, d = 1024, P-LR r = 16) at decode-sized
    token counts: the one-call forward against per-chunk states + merge
    (Sec. 3.5's merge form over the sources), cold, for several chunk sizes."""
    from paper_2607_09694_amd.inputs import PROJECTED, make_device_problem

    res = {}
    for N in (16, 128, 1024):
        g = make_device_problem(PROJECTED, S, N, d, r, dev, seed=6)
        V, K, q = g["V"], g["K"], g["q"][0].contiguous()
        H = torch.empty((N, d), dtype=torch.bfloat16, device=dev)
        row = {"one_call_ms": float(np.median(time_calls(
            torch, lambda: lr.route_fwd(V, K, q, PROJECTED, out=H), reps, warmup, flush)))}
        for chunk in (1, 4, 7, 13, 25):
            P = -(-S // chunk)
            st = (torch.empty((P, N), dtype=torch.float32, device=dev),
                  torch.empty((P, N), dtype=torch.float32, device=dev),
                  torch.empty((P, N, d), dtype=torch.float32, device=dev))

            def call():
                lr.route_state_fwd(V, K, q, PROJECTED, chunk, out=st)
                lr.route_merge_fwd(*st, out=H)

            row[f"split_c{chunk}_ms"] = float(np.median(time_calls(torch, call, reps, warmup,
                                                                    flush)))
        res[f"N{N}"] = row
        del g, V, K, H
    return res


def key_producer(torch, lr, dev, reps, warmup, flush):
    """The projected-key producer (Eq. fused_projection) at the paper's
    output projections (d = 1024; attention m = 1024, SwiGLU m = 2816) for
    N = 16384 tokens, writing planes of the value and key stacks.  The
    library GEMM (hipBLASLt through torch) is timed beside it: one fused GEMM
    then a split copy, and two GEMMs written straight into the planes."""
    out = {}
    N, d = 16384, 1024
    for m, r in ((1024, 16), (2816, 16), (2816, 32)):
        g = torch.Generator(device=dev)
        g.manual_seed(m + r)
        A = torch.randn((N, m), generator=g, device=dev).to(torch.bfloat16)
        W = (torch.randn((d + r, m), generator=g, device=dev) / m ** 0.5).to(torch.bfloat16)
        V = torch.empty((2, N, d), dtype=torch.bfloat16, device=dev)
        K = torch.empty((2, N, r), dtype=torch.bfloat16, device=dev)
        C = torch.empty((N, d + r), dtype=torch.bfloat16, device=dev)
        Wt, Wo, Wk = W.t(), W[:d].t(), W[d:].t()

        def lib_fused():
            torch.matmul(A, Wt, out=C)
            V[0].copy_(C[:, :d])
            K[0].copy_(C[:, d:])

        def lib_two():
            torch.matmul(A, Wo, out=V[0])
            torch.matmul(A, Wk, out=K[0])

        flops = 2.0 * N * m * (d + r)
        res = {}
        for name, fn in (("fused_key_producer", lambda: lr.key_proj_fwd(A, W, d, out=(V[1], K[1]))),
                         ("library_gemm_then_split", lib_fused),
                         ("library_two_gemms", lib_two)):
            ts = time_calls(torch, fn, reps, warmup, flush)
            med = float(np.median(ts))
            res[name] = {"median_ms": med, "min_ms": float(np.min(ts)),
                         "TFLOPs": flops / (med * 1e-3) / 1e12,
                         "frac_of_bf16_peak": flops / (med * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS}
        # Warm: the activation was just written by the previous kernel, as in
        # a model, so the memory-side cache may still hold it.
        ts = time_calls(torch, lambda: lr.key_proj_fwd(A, W, d, out=(V[1], K[1])), reps, warmup)
        res["fused_key_producer_warm"] = {"median_ms": float(np.median(ts)),
                                          "TFLOPs": flops / (float(np.median(ts)) * 1e-3) / 1e12}
        ts = time_calls(torch, lib_two, reps, warmup)
        res["library_two_gemms_warm"] = {"median_ms": float(np.median(ts)),
                                         "TFLOPs": flops / (float(np.median(ts)) * 1e-3) / 1e12}
        torch.matmul(A, Wt, out=C)
        torch.cuda.synchronize()
        res["bitwise_equal_to_library_fused_gemm"] = bool(torch.equal(V[1], C[:, :d]) and
                                                          torch.equal(K[1], C[:, d:]))
        # Backward: dA = [dO, dK] W (bf16) and dW = [dO, dK]^T A (fp32), against
        # the library's two GEMMs on the concatenated gradient (dW in bf16).
        dO = torch.randn((N, d), generator=g, device=dev).to(torch.bfloat16)
        dK = torch.randn((N, r), generator=g, device=dev).to(torch.bfloat16)
        dA = torch.empty((N, m), dtype=torch.bfloat16, device=dev)
        dW = torch.empty((d + r, m), dtype=torch.float32, device=dev)
        Gc = torch.cat([dO, dK], dim=1)
        Gt = Gc.t().contiguous()
        dA2 = torch.empty_like(dA)
        dW2 = torch.empty((d + r, m), dtype=torch.bfloat16, device=dev)

        def lib_bwd():
            torch.matmul(Gc, W, out=dA2)
            torch.matmul(Gt, A, out=dW2)

        for name, fn in (("backward", lambda: lr.key_proj_bwd(A, W, dO, dK, out=(dA, dW))),
                         ("library_backward_two_gemms", lib_bwd)):
            ts = time_calls(torch, fn, reps, warmup, flush)
            med = float(np.median(ts))
            res[name] = {"median_ms": med, "min_ms": float(np.min(ts)),
                         "TFLOPs": 2 * flops / (med * 1e-3) / 1e12,
                         "frac_of_bf16_peak": 2 * flops / (med * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS}
        del dO, dK, dA, dW, Gc, Gt, dA2, dW2
        out[f"m{m}_r{r}"] = res
        del A, W, V, K, C
        torch.cuda.empty_cache()
    return out


def extras(torch, lr, dev, reps, warmup):
    """The other workloads: the 49-site forward model pass (projected r=16 and
    sliced r in {8,16,32,64}), full-rank vs low-rank at S = 49, and a copy
    kernel ceiling.  Cold: the MALL is flushed before every timed call."""
    from paper_2607_09694_amd.inputs import FULL, PROJECTED, SLICED, make_device_problem

    out = {}
    flush = Flusher(torch, dev)
    N, d = 16384, 1024
    g = make_device_problem(PROJECTED, 49, N, d, 16, dev, seed=0, n_queries=49)
    V, K, Q = g["V"], g["K"], g["q"]
    H = torch.empty((N, d), dtype=torch.bfloat16, device=dev)

    def model_pass(mode, r, queries):
        per_site, nbytes = [], 0
        for t in range(1, 50):
            Kt = K[:t] if mode == PROJECTED else None
            qt = queries[t - 1]
            ts = time_calls(torch, lambda: lr.route_fwd(V[:t], Kt, qt, mode, out=H),
                            reps, warmup, flush)
            per_site.append(float(np.median(ts)))
            nbytes += fwd_bytes(t, N, d, r, mode)
        total_ms = sum(per_site)
        return {"total_ms": total_ms, "tokens_per_s": N / (total_ms * 1e-3),
                "algo_GBps": nbytes / (total_ms * 1e-3) / 1e9,
                "frac_of_peak": nbytes / (total_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "site49_ms": per_site[-1], "sites_2_to_49_ms": total_ms - per_site[0]}

    def all_sites(mode, r, Vs, Ks, queries, per_site):
        """Sites 2..49 (prefixes of 2..49 sources) in one call, with N_eff."""
        T = 48
        Ha = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)
        ne = torch.empty((T, N), dtype=torch.float32, device=dev)
        Qa = queries[1:].contiguous()
        ts = time_calls(torch, lambda: lr.route_all_fwd(Vs, Ks, Qa, mode, 2, out=(Ha, ne)),
                        reps, warmup, flush)
        med = float(np.median(ts))
        nbytes = all_sites_bytes(49, T, N, d, r, mode)
        del Ha, ne
        return {"median_ms": med, "min_ms": float(np.min(ts)), "max_ms": float(np.max(ts)),
                "tokens_per_s": N / (med * 1e-3), "algo_GBps": nbytes / (med * 1e-3) / 1e9,
                "frac_of_peak": nbytes / (med * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "per_site_calls_ms": per_site["sites_2_to_49_ms"],
                "speedup_vs_per_site_calls": per_site["sites_2_to_49_ms"] / med}

    out["model_pass_projected_r16"] = model_pass(PROJECTED, 16, Q)
    out["all_sites_pass_projected_r16"] = all_sites(PROJECTED, 16, V, K, Q,
                                                    out["model_pass_projected_r16"])
    out["all_sites_backward_projected_r16"] = all_sites_backward(
        torch, lr, dev, PROJECTED, 16, V, K, Q, reps, warmup, flush)
    gen = torch.Generator(device=dev)
    for r in (8, 16, 32, 64):
        gen.manual_seed(r)
        qs = torch.randn((49, r), generator=gen, device=dev) / r ** 0.5
        out[f"model_pass_sliced_r{r}"] = model_pass(SLICED, r, qs)
        if r == 64:
            out["all_sites_pass_sliced_r64"] = all_sites(SLICED, 64, V, None, qs,
                                                         out["model_pass_sliced_r64"])
            out["all_sites_backward_sliced_r64"] = all_sites_backward(
                torch, lr, dev, SLICED, 64, V, None, qs, reps, warmup, flush)

    # Head to head at S = 49: full rank vs low rank, forward and backward.
    # The full-rank forward reads every row once (online softmax); its
    # backward must read the rows twice (the key path needs o_i after every
    # g_j is known).
    gen.manual_seed(1024)
    qf = torch.randn((d,), generator=gen, device=dev) / d ** 0.5
    dH = torch.randn((N, d), generator=gen, device=dev).to(torch.bfloat16)
    dV = torch.empty_like(V)
    dK = torch.empty_like(K)
    ws = torch.empty((lr.route_bwd_workspace_bytes(49, N, d, d, FULL, V.dtype),),
                     dtype=torch.uint8, device=dev)
    dqf = torch.empty((d,), dtype=torch.float32, device=dev)
    dq16 = torch.empty((16,), dtype=torch.float32, device=dev)
    head = {}
    cases = (
        ("full_rank", FULL, None, qf, dqf, fwd_bytes(49, N, d, d, FULL),
         2 * 49 * N * d * 2 + N * d * 2),
        ("projected_r16", PROJECTED, K, Q[48], dq16, fwd_bytes(49, N, d, 16, PROJECTED),
         bwd_bytes(49, N, d, 16)),
        ("sliced_r16", SLICED, None, Q[48], dq16, fwd_bytes(49, N, d, 16, SLICED),
         2 * 49 * N * d * 2 + N * d * 2))
    # 3x the reps of the other workloads, so that the min-max ranges are
    # those of the kernels and not of a few outliers.
    for name, mode, Kc, qc, dqc, fb, bb in cases:
        dKc = dK if mode == PROJECTED else None
        tf = time_calls(torch, lambda: lr.route_fwd(V, Kc, qc, mode, out=H), 3 * reps, warmup,
                        flush)
        tb = time_calls(torch, lambda: lr.route_bwd(V, Kc, qc, dH, mode, out=(dV, dKc, dqc),
                                                     workspace=ws), 3 * reps, warmup, flush)
        head[name] = {"fwd_median_ms": float(np.median(tf)), "fwd_min_ms": float(np.min(tf)),
                      "fwd_max_ms": float(np.max(tf)),
                      "fwd_algo_GBps": fb / (np.median(tf) * 1e-3) / 1e9,
                      "bwd_median_ms": float(np.median(tb)), "bwd_min_ms": float(np.min(tb)),
                      "bwd_max_ms": float(np.max(tb)),
                      "bwd_algo_GBps": bb / (np.median(tb) * 1e-3) / 1e9}
    for name in ("projected_r16", "sliced_r16"):
        for k in ("fwd", "bwd"):
            head[name][f"{k}_clear_of_full_rank"] = bool(
                head[name][f"{k}_max_ms"] < head["full_rank"][f"{k}_min_ms"])
    out["site49_head_to_head"] = head
    del dH, dV, dK, ws

    # Block sources (8 blocks of 6 sub-layer outputs), the paper's best
    # settings: one fused call per site adds o_{t-1} into its fp32 summary
    # slot and routes over the embedding and the block summaries.
    out["block_model_pass_sliced_r64_8blocks"] = block_pass(torch, lr, dev, V, SLICED, 64,
                                                            6, reps, warmup, flush)
    out["block_model_pass_projected_r32_8blocks"] = block_pass(torch, lr, dev, V, PROJECTED,
                                                               32, 6, reps, warmup, flush)
    for mode, r in ((SLICED, 64), (PROJECTED, 32)):
        key = f"block_model_pass_{'sliced' if mode == SLICED else 'projected'}_r{r}_8blocks"
        out[key + "_bf16_completed"] = block_pass(torch, lr, dev, V, mode, r, 6, reps, warmup,
                                                  flush, completed_bf16=True)
    out["model_training_pass_projected_r16"] = model_training_pass(
        torch, lr, dev, V, K, PROJECTED, 16, 3, 1)
    out["model_training_pass_sliced_r64"] = model_training_pass(
        torch, lr, dev, V, None, SLICED, 64, 3, 1)
    out["block_training_pass_sliced_r64_8blocks"] = block_training_pass(
        torch, lr, dev, V, SLICED, 64, 6, 5, 1)
    out["block_training_pass_projected_r32_8blocks"] = block_training_pass(
        torch, lr, dev, V, PROJECTED, 32, 6, 5, 1)
    out["block_inference_sliced_r64_8blocks"] = block_inference_passes(
        torch, lr, dev, V, SLICED, 64, 6, 5, 1)
    out["block_inference_projected_r32_8blocks"] = block_inference_passes(
        torch, lr, dev, V, PROJECTED, 32, 6, 5, 1)
    out["decode_model_pass_projected_r16_N128"] = decode_model_pass(torch, lr, dev, reps, warmup)
    out["key_producer_d1024_N16384"] = key_producer(torch, lr, dev, reps, warmup, flush)
    del g, V, K, H, flush
    torch.cuda.empty_cache()
    return out


def focused(torch, lr, dev, names, reps=20, warmup=3):
    """Only the named workloads (for profiling one kernel at a time):
    'key_producer', 'split_sources' (the deepest site at decode token counts,
    one call against states + merge), 'decode' (a 49-site pass at N = 128,
    eager and as one graph), 'block_forward' (the 8-block forward pass, fp32 and
    bf16 completed summaries), 'block_training', 'model_training' and
    'all_sites' (sites 2..49 of the 49-source pass, P-LR r = 16 and S-LR
    r = 64, cold; with 'per_site', also the per-site accumulating backward)."""
    from paper_2607_09694_amd.inputs import PROJECTED, SLICED, make_device_problem

    flush = Flusher(torch, dev)
    out = {}
    if "key_producer" in names:
        out["key_producer_d1024_N16384"] = key_producer(torch, lr, dev, reps, warmup, flush)
    if "split_sources" in names:
        out["split_sources_49src_d1024_projected_r16"] = split_sources(torch, lr, dev, reps,
                                                                       warmup, flush)
    if "decode" in names:
        out["decode_model_pass_projected_r16_N128"] = decode_model_pass(torch, lr, dev, reps,
                                                                        warmup)
    if "block_forward" in names:
        N, d = 16384, 1024
        g = make_device_problem(PROJECTED, 49, N, d, 16, dev, seed=0, n_queries=1)
        for mode, r in ((SLICED, 64), (PROJECTED, 32)):
            key = f"block_model_pass_{'sliced' if mode == SLICED else 'projected'}_r{r}_8blocks"
            out[key] = block_pass(torch, lr, dev, g["V"], mode, r, 6, reps, warmup, flush)
            out[key + "_bf16_completed"] = block_pass(torch, lr, dev, g["V"], mode, r, 6, reps,
                                                      warmup, flush, completed_bf16=True)
        del g
        torch.cuda.empty_cache()
    if "block_training" in names:
        N, d = 16384, 1024
        g = make_device_problem(PROJECTED, 49, N, d, 16, dev, seed=0, n_queries=1)
        for mode, r in ((SLICED, 64), (PROJECTED, 32)):
            out[f"block_training_pass_{'sliced' if mode == SLICED else 'projected'}_r{r}_8blocks"] = \
                block_training_pass(torch, lr, dev, g["V"], mode, r, 6, 5, 1)
        del g
        torch.cuda.empty_cache()
    if "model_training" in names:
        N, d = 16384, 1024
        for mode, r in ((PROJECTED, 16), (SLICED, 64)):
            g = make_device_problem(mode, 49, N, d, r, dev, seed=0, n_queries=1)
            out[f"model_training_pass_{'projected' if mode == PROJECTED else 'sliced'}_r{r}"] = \
                model_training_pass(torch, lr, dev, g["V"], g["K"], mode, r, 3, 1)
            del g
            torch.cuda.empty_cache()
    if "all_sites" in names:
        N, d, T = 16384, 1024, 48
        for mode, r in ((PROJECTED, 16), (SLICED, 64)):
            g = make_device_problem(mode, 49, N, d, r, dev, seed=0, n_queries=49)
            Ha = torch.empty((T, N, d), dtype=torch.bfloat16, device=dev)
            ne = torch.empty((T, N), dtype=torch.float32, device=dev)
            Qa = g["q"][1:].contiguous()
            ts = time_calls(torch, lambda: lr.route_all_fwd(g["V"], g["K"], Qa, mode, 2,
                                                            out=(Ha, ne)), reps, warmup, flush)
            med = float(np.median(ts))
            nbytes = all_sites_bytes(49, T, N, d, r, mode)
            out[f"all_sites_pass_{'projected' if mode == PROJECTED else 'sliced'}_r{r}"] = {
                "median_ms": med, "algo_GBps": nbytes / (med * 1e-3) / 1e9,
                "frac_of_peak": nbytes / (med * 1e-3) / 1e9 / HBM_PEAK_GBS}
            del Ha, ne
            out[f"all_sites_backward_{'projected' if mode == PROJECTED else 'sliced'}_r{r}"] = \
                all_sites_backward(torch, lr, dev, mode, r, g["V"], g["K"], g["q"], reps, warmup,
                                   flush, per_site="per_site" in names)
            del g
            torch.cuda.empty_cache()
    return out


def key_producer_pass(torch, lr, dev):
    """Untimed calls of the SwiGLU key producer for counter runs: dispatches
    4-13 of the kernel are cold (the memory-side cache flushed by a read
    before each), 14-23 warm (back to back)."""
    N, d, m, r = 16384, 1024, 2816, 16
    g = torch.Generator(device=dev)
    g.manual_seed(m + r)
    A = torch.randn((N, m), generator=g, device=dev).to(torch.bfloat16)
    W = (torch.randn((d + r, m), generator=g, device=dev) / m ** 0.5).to(torch.bfloat16)
    O = torch.empty((N, d), dtype=torch.bfloat16, device=dev)
    K = torch.empty((N, r), dtype=torch.bfloat16, device=dev)
    flush = Flusher(torch, dev)
    for _ in range(3):
        lr.key_proj_fwd(A, W, d, out=(O, K))
    for _ in range(10):
        flush()
        lr.key_proj_fwd(A, W, d, out=(O, K))
    for _ in range(10):
        lr.key_proj_fwd(A, W, d, out=(O, K))
    torch.cuda.synchronize()
    print("bench: key producer pass done", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-extra", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--extra-only", default="",
                    help="comma-separated workloads to run alone, without the main step "
                         "(key_producer, split_sources, decode, all_sites, block_forward, "
                         "block_training, "
                         "model_training; per_site "
                         "adds the per-site backward beside the all-sites one); prints their JSON")
    ap.add_argument("--counters-pass", action="store_true",
                    help="no timing: 3 reference copies of 1 GiB, then 3 forward and 3 "
                         "backward calls of the main workload (for rocprofv3 --pmc runs)")
    ap.add_argument("--key-producer-pass", action="store_true",
                    help="no timing: the SwiGLU key producer (m = 2816, d = 1024, r = 16, "
                         "N = 16384), 3 warm-up calls, 10 cold calls (a 1 GiB read before "
                         "each), then 10 warm calls (for rocprofv3 --pmc runs)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: --gpus must be 1 (tokens are independent, so the "
              "routing shards over tokens with no exchange; one GPU's share is what is timed)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2607_09694_amd as lr
    from paper_2607_09694_amd.inputs import PROJECTED, make_device_problem

    lr.load_library()
    dev = torch.device("cuda:0")
    if args.key_producer_pass:
        key_producer_pass(torch, lr, dev)
        return
    if args.extra_only:
        names = set(args.extra_only.split(","))
        print(json.dumps({"extra_only": focused(torch, lr, dev, names)}), flush=True)
        return
    print(f"bench: generating inputs S={S5} N={N5} d={D5} r={R5}", file=sys.stderr, flush=True)
    g = make_device_problem(PROJECTED, S5, N5, D5, R5, dev, seed=0, with_dH=True)
    V, K, q, dH = g["V"], g["K"], g["q"][0].contiguous(), g["dH"]
    H = torch.empty((N5, D5), dtype=torch.bfloat16, device=dev)
    dV, dK = torch.empty_like(V), torch.empty_like(K)
    dq = torch.empty((R5,), dtype=torch.float32, device=dev)
    ws = torch.empty((lr.route_bwd_workspace_bytes(S5, N5, D5, R5, PROJECTED, V.dtype),),
                     dtype=torch.uint8, device=dev)
    st = torch.cuda.current_stream()

    def step(ev=None):
        lr.route_fwd(V, K, q, PROJECTED, out=H)
        if ev is not None:
            ev[0].record(st)
        lr.route_bwd(V, K, q, dH, PROJECTED, out=(dV, dK, dq), workspace=ws)
        if ev is not None:
            ev[1].record(st)

    if args.counters_pass:
        probe = load_probe()
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            check_probe(probe.hbm_probe_copy(src.data_ptr(), dst.data_ptr(), 1 << 30, 8192,
                                             st.cuda_stream))
        torch.cuda.synchronize()
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        print("bench: counters pass done", file=sys.stderr, flush=True)
        return

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
    print(f"bench: timing {args.steps} steps", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gpu_state = device_state(torch, dev)  # right after the timed steps
    bwd_all = [a.elapsed_time(b) for a, b in events]
    bwd_ms = float(np.mean(bwd_all))
    ms_per_step = elapsed * 1e3 / args.steps

    # Forward alone (same inputs), for the record.
    fwd_ts = time_calls(torch, lambda: lr.route_fwd(V, K, q, PROJECTED, out=H), args.steps, 2)
    fwd_ms = float(np.mean(fwd_ts))

    b_bwd = bwd_bytes(S5, N5, D5, R5)
    achieved = b_bwd / (bwd_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": "route_bwd_lr (+ dq_reduce)",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(b_bwd),
                "algo_bytes_per_launch": b_bwd, "avg_launch_ms": round(bwd_ms, 4),
                "median_launch_ms": round(float(np.median(bwd_all)), 4),
                "min_launch_ms": round(float(np.min(bwd_all)), 4)}

    result = {
        "metric": METRIC,
        "value": round(N5 / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "projected-key LR-AttnRes routing fwd+bwd, d=2048, r=32, "
                               "N=4x4096 tokens, S=64 sources",
                   "global_batch": N5, "seq_len": 4096, "sources": S5, "d": D5, "r": R5,
                   "storage": "bf16", "parallelism": "single GPU"},
        "roofline": roofline,
        "device": gpu_state,
        "fwd": {"avg_ms": round(fwd_ms, 4), "min_ms": round(float(np.min(fwd_ts)), 4),
                "tokens_per_s": round(N5 / (fwd_ms * 1e-3), 1),
                "algo_GBps": round(fwd_bytes(S5, N5, D5, R5, 0) / (fwd_ms * 1e-3) / 1e9, 1)},
    }
    if not args.no_cpu:
        print("bench: CPU oracle baseline", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(g, q.cpu().numpy())
    del g, V, K, dH, dV, dK, H, ws
    torch.cuda.empty_cache()
    # The same fractions against what this GPU's plain streaming kernels
    # reach: the backward reads and writes (copy), the forward reads.
    print("bench: HBM ceilings", file=sys.stderr, flush=True)
    ceil = probe_ceilings(torch, dev, 10, 2)
    result["hbm_ceilings"] = ceil
    roofline["frac_of_measured_copy"] = round(achieved / ceil["copy_GBps"], 4)
    result["fwd"]["frac_of_measured_read"] = round(
        result["fwd"]["algo_GBps"] / ceil["read_GBps"], 4)
    if not args.no_extra:
        print("bench: other workloads", file=sys.stderr, flush=True)
        result["extra"] = extras(torch, lr, dev, reps=20, warmup=3)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
