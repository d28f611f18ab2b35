"""Parity bars between the HIP path and the fp64 oracle.

fp32 storage: normwise relative error <= 1e-5, both max|err| / max|ref| and
||err||_2 / ||ref||_2.
bf16 storage (outputs rounded to bf16): values and value gradients
max|err| <= 2e-2 and ||err||_2 / ||ref||_2 <= 5e-3.  Results that grow past
|x| = 8 (key gradients; h over block summaries, which are sums of several
outputs), where the bf16 half-ulp alone exceeds 2e-2, take
|err| <= 2e-2 * max(1, |ref|) element by element, with the same relative L2.
dq is fp32 accumulated over N*S terms: normwise 1e-4 (the fp32 bar scaled
for the length of the sum), and rel-L2 <= 5e-3.  Where the sum cancels
(sum_i ds_i = 0 per token), a normwise bar cannot hold: such a sum is
checked against the error bound of its terms instead, |err| <= 2 (u_t +
n 2^-24) sum |term| per entry, u_t being the relative error of one term
and n their number.
Value gradients summed over many sites (the all-sites backward) also grow
past |x| = 8; they keep the 2e-2 bar up to |x| = 5.12 and beyond it take one
bf16 half-ulp, |err| <= 2^-8 |ref| (+ 1e-3 for the fp32 sums), which a
correctly rounded result always meets.
"""
import numpy as np


def rel_errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), "non-finite values in the HIP result"
    d = got - ref
    ref_max = max(np.abs(ref).max(initial=0.0), 1e-30)
    ref_l2 = max(np.linalg.norm(ref.ravel()), 1e-30)
    return np.abs(d).max(initial=0.0), np.abs(d).max(initial=0.0) / ref_max, \
        np.linalg.norm(d.ravel()) / ref_l2


def check_f32(name, got, ref, tol=1e-5):
    amax, nmax, nl2 = rel_errors(got, ref)
    assert nmax <= tol and nl2 <= tol, \
        f"{name}: normwise max {nmax:.3e}, rel-L2 {nl2:.3e} (bar {tol:g})"


def check_bf16_value(name, got, ref):
    amax, nmax, nl2 = rel_errors(got, ref)
    assert amax <= 2e-2 and nl2 <= 5e-3, \
        f"{name}: max-abs {amax:.3e} (bar 2e-2), rel-L2 {nl2:.3e} (bar 5e-3)"


def check_bf16_grown(name, got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    _, _, nl2 = rel_errors(got, ref)
    bar = np.maximum(2e-2, 2.0 ** -8 * np.abs(ref) + 1e-3)
    worst = (np.abs(got - ref) / bar).max(initial=0.0)
    assert worst <= 1.0 and nl2 <= 5e-3, \
        f"{name}: max error / bar {worst:.3f} (bar max(2e-2, 2^-8 |ref| + 1e-3)), " \
        f"rel-L2 {nl2:.3e} (bar 5e-3)"


def check_bf16_key_grad(name, got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    _, _, nl2 = rel_errors(got, ref)
    worst = (np.abs(got - ref) / np.maximum(1.0, np.abs(ref))).max(initial=0.0)
    assert worst <= 2e-2 and nl2 <= 5e-3, \
        f"{name}: scaled max {worst:.3e} (bar 2e-2), rel-L2 {nl2:.3e} (bar 5e-3)"


def check_dq(name, got, ref, tol=1e-4):
    _, nmax, nl2 = rel_errors(got, ref)
    assert nmax <= tol and nl2 <= min(tol, 5e-3), \
        f"{name}: normwise max {nmax:.3e}, rel-L2 {nl2:.3e} (bar {tol:g})"


def check_sum_by_terms(name, got, ref, abs_terms, n_terms, term_rel):
    """Elementwise forward error bound of a sum of n_terms terms, each with
    relative error term_rel, accumulated in fp32: |err| <= 2 (term_rel +
    n 2^-24) sum |term| (a factor 2 above the bound)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert np.isfinite(got).all(), "non-finite values in the HIP result"
    bar = 2.0 * (term_rel + n_terms * 2.0 ** -24) * np.asarray(abs_terms, dtype=np.float64)
    worst = (np.abs(got - ref) / bar).max(initial=0.0)
    assert worst <= 1.0, f"{name}: max error / term bound {worst:.3f}"
