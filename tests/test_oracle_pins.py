"""Pins for the fp64 oracle, checked against facts that do not come from it.

Each test names what fixes the expected value: a closed form, a brute-force
enumeration, a finite-difference derivative, a hand-derived fixture in
tests/golden/, an independent numpy formulation of the definition, or an
invariant of the mathematics.  None of them needs a GPU.
"""
import glob
import itertools
import json
import os

import numpy as np
import pytest
from scipy.optimize import brentq

import oracle
import synth

HERE = os.path.dirname(os.path.abspath(__file__))


# ----------------------------------------------------------- closed forms

def sparsemax_sorted(x):
    """Euclidean projection onto the simplex by sorting (alpha = 2)."""
    z = np.sort(x)[::-1]
    cs = np.cumsum(z)
    k = np.arange(1, x.size + 1)
    kstar = k[1 + k * z > cs].max()
    return (cs[kstar - 1] - 1.0) / kstar


def entmax15_sorted(x):
    """Exact alpha = 1.5 threshold on sorted prefixes: for the top-k set,
    sum (x_j - tau)^2 = 1 gives tau_k = M_k - sqrt(1/k - (M2_k - M_k^2)); the
    answer is the k whose tau_k separates x_(k) from x_(k+1)."""
    z = np.sort(x)[::-1]
    n = z.size
    for k in range(1, n + 1):
        M = z[:k].mean()
        M2 = (z[:k] ** 2).mean()
        rad = 1.0 / k - (M2 - M * M)
        if rad < 0:
            continue
        tau = M - np.sqrt(rad)
        nxt = z[k] if k < n else -np.inf
        if z[k - 1] > tau >= nxt:
            return tau
    raise AssertionError("no consistent support")


def brute_force_tau(x, alpha):
    """Enumerate every non-empty support S; on S solve sum_S (x-t)^g = 1 for
    t < min_S x with brentq; keep the S whose t also satisfies t >= max of the
    complement.  Asserts exactly one support is self-consistent."""
    g = 1.0 / (alpha - 1.0)
    n = x.size
    found = []
    for r in range(1, n + 1):
        for S in itertools.combinations(range(n), r):
            xs = x[list(S)]
            rest = np.delete(x, list(S))
            top = xs.min()
            h = lambda t: np.sum((xs - t) ** g) - 1.0  # decreasing on t < top
            lo = top - 1.0 - 1e-9
            if h(lo) < 0 or h(top) > 0:
                continue
            t = brentq(h, lo, top, xtol=1e-15, rtol=1e-15, maxiter=500)
            if rest.size == 0 or t >= rest.max() - 1e-13:
                if t < top:
                    found.append(t)
    assert len(found) >= 1
    found = np.array(found)
    assert np.ptp(found) < 1e-10, found  # ties at the boundary give the same t
    return found[0]


@pytest.mark.parametrize("n", [1, 2, 3, 7, 64, 1000])
def test_sparsemax_closed_form(n):
    rng = np.random.default_rng(n)
    for _ in range(20):
        x = rng.standard_normal(n) * rng.uniform(0.1, 5)
        tau = oracle.entmax_threshold(x, 2.0)
        assert abs(tau - sparsemax_sorted(x)) < 1e-12
        p, _ = oracle.entmax(x, 2.0)
        ref = np.maximum(x - sparsemax_sorted(x), 0)
        assert np.max(np.abs(p - ref)) < 1e-12


@pytest.mark.parametrize("n", [1, 2, 3, 5, 64, 1000, 8192])
def test_entmax15_closed_form(n):
    rng = np.random.default_rng(100 + n)
    for _ in range(10):
        x = 0.5 * rng.standard_normal(n) * rng.uniform(0.05, 8)
        tau = oracle.entmax_threshold(x, 1.5)
        assert abs(tau - entmax15_sorted(x)) < 1e-12 * max(1, abs(tau))


@pytest.mark.parametrize("alpha", [1.1, 1.25, 1.5, 2.0, 3.0])
def test_brute_force_supports(alpha):
    rng = np.random.default_rng(int(alpha * 100))
    for n in (1, 2, 4, 7, 10):
        for _ in range(4):
            x = rng.standard_normal(n) * rng.uniform(0.2, 3)
            ref = brute_force_tau(x, alpha)
            assert abs(oracle.entmax_threshold(x, alpha) - ref) < 1e-11 * max(1, abs(ref))


def test_golden_examples():
    files = sorted(f for f in glob.glob(os.path.join(HERE, "golden", "*.json"))
                   if not os.path.basename(f).startswith("alg1_"))
    assert len(files) >= 6
    for fn in files:
        e = json.load(open(fn))
        x = np.array(e["x"])
        p, tau = oracle.entmax(x, e["alpha"])
        assert abs(tau - e["tau"]) < 1e-12, fn
        assert np.max(np.abs(p - np.array(e["p"]))) < 1e-12, fn


# ------------------------------------------------------------- invariants

@pytest.mark.parametrize("alpha", [1.25, 1.5, 2.0, 1.7])
def test_row_invariants(alpha):
    rng = np.random.default_rng(7)
    n = 300
    for scale in (0.01, 0.3, 1, 10):
        x = rng.standard_normal(n) * scale
        p, tau = oracle.entmax(x, alpha)
        m = x.max()
        # bracket of Algorithm 1
        assert m - 1 - 1e-12 <= tau <= m - n ** (1 - alpha) + 1e-12
        assert np.all(p >= 0)
        assert abs(p.sum() - 1) < 1e-12
        # p > 0 exactly where x > tau (Eq. 2)
        assert np.array_equal(p > 0, x > tau)
        # shift by a constant moves tau by the constant, p unchanged
        p2, tau2 = oracle.entmax(x + 0.37, alpha)
        assert abs(tau2 - tau - 0.37) < 1e-12 and np.max(np.abs(p2 - p)) < 1e-12
        # permutation equivariance
        perm = rng.permutation(n)
        p3, tau3 = oracle.entmax(x[perm], alpha)
        assert abs(tau3 - tau) < 1e-12 and np.max(np.abs(p3 - p[perm])) < 1e-12


@pytest.mark.parametrize("alpha", [1.25, 1.5, 2.0])
def test_special_cases(alpha):
    for n in (1, 2, 5, 100):
        x = np.full(n, 0.42)
        p, tau = oracle.entmax(x, alpha)
        assert abs(tau - (0.42 - n ** (1 - alpha))) < 1e-12
        assert np.max(np.abs(p - 1.0 / n)) < 1e-12
    x = np.array([3.0, 1.5, 0.0, -2.0])  # gap >= 1: one-hot, tau = max - 1
    p, tau = oracle.entmax(x, alpha)
    assert abs(tau - 2.0) < 1e-12 and np.array_equal(p, [1.0, 0, 0, 0])


@pytest.mark.parametrize("name", ["alg1_trace_a15", "alg1_trace_a125"])
def test_halley_bisection_trace_iterates(name):
    """The oracle's fp64 Algorithm 1 iterates against the exact rational ones
    (tests/golden/make_golden.py; the first update is derived by hand there:
    19/106 at alpha 1.5, where a Newton step would give 7/40, and
    4871/64004 at alpha 1.25, which a wrong f'' coefficient would miss)."""
    ex = json.load(open(os.path.join(HERE, "golden", name + ".json")))
    tr = oracle.halley_bisection_trace(np.array(ex["x"]), ex["alpha"], ex["iters"])
    assert np.allclose(tr, ex["tau"], rtol=1e-14, atol=1e-15), (tr, ex["tau"])


def test_halley_bisection_trace_converges():
    rng = np.random.default_rng(3)
    for alpha in (1.25, 1.5, 2.0):
        for c in (0.05, 1, 8):
            x = (alpha - 1) * rng.standard_normal(2048) * c
            tr = oracle.halley_bisection_trace(x, alpha, 30)
            exact = oracle.entmax_threshold(x, alpha)
            m = x.max()
            assert np.all(tr >= m - 1 - 1e-12) and np.all(tr <= m - x.size ** (1 - alpha) + 1e-12)
            assert abs(tr[-1] - exact) < 1e-12 * max(1, abs(exact))


# ---------------------------------------------- attention: independent numpy

def numpy_attention(q, k, v, alpha, scale, causal, dout=None):
    """Dense fp64 numpy formulation of the definitions, with tau from the sort
    closed forms (alpha in {1.5, 2}), for small n."""
    n, d = q.shape
    x = (alpha - 1) * scale * (q @ k.T)
    valid = np.tril(np.ones((n, n), bool)) if causal else np.ones((n, n), bool)
    tau = np.empty(n)
    for i in range(n):
        xi = x[i, valid[i]]
        tau[i] = sparsemax_sorted(xi) if alpha == 2.0 else entmax15_sorted(xi)
    g = 1 / (alpha - 1)
    z = np.where(valid, x - tau[:, None], -1.0)
    P = np.where(z > 0, np.maximum(z, 0) ** g, 0.0)
    U = np.where(z > 0, np.maximum(z, 0) ** (g - 1), 0.0)
    out = {"tau": tau, "o": P @ v, "o2": (U @ v) / U.sum(1, keepdims=True), "P": P}
    if dout is not None:
        dP = dout @ v.T
        delta = (U * dP).sum(1) / U.sum(1)
        dS = U * (dP - delta[:, None])
        out.update(delta=delta, dq=scale * dS @ k, dk=scale * dS.T @ q, dv=P.T @ dout)
    return out


@pytest.mark.parametrize("alpha", [1.5, 2.0])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n", [1, 5, 64, 130])
def test_attention_head_matches_numpy(alpha, causal, n):
    d = 16
    inp = synth.attention_inputs(1, 1, n, d, c=3.0, dtype="f32", with_dout=True, seed=11 + n)
    q, k, v, do = (inp[t].f64()[0, 0] for t in ("q", "k", "v", "dout"))
    scale = 1 / np.sqrt(d)
    got = oracle.attention_head(q, k, v, alpha, scale, causal, dout=do, nthreads=3)
    ref = numpy_attention(q, k, v, alpha, scale, causal, dout=do)
    for key in ("tau", "o", "o2", "delta", "dq", "dk", "dv"):
        err = np.max(np.abs(got[key] - ref[key]))
        assert err < 1e-10 * max(1.0, np.max(np.abs(ref[key]))), (key, err)
    # block mask of Eq. 8: block kept iff some p in it is positive
    T = (n + 63) // 64
    mask_ref = np.zeros((T, T), np.uint8)
    for I in range(T):
        for J in range(T):
            mask_ref[I, J] = np.any(ref["P"][I * 64:(I + 1) * 64, J * 64:(J + 1) * 64] > 0)
    assert np.array_equal(oracle.block_mask_from_margin(got["margin"]), mask_ref)


def test_rows_and_cols_subsets_match_full():
    n, d = 200, 8
    inp = synth.attention_inputs(1, 1, n, d, c=2.0, dtype="f32", with_dout=True, seed=5)
    q, k, v, do = (inp[t].f64()[0, 0] for t in ("q", "k", "v", "dout"))
    full = oracle.attention_head(q, k, v, 1.5, 0.3, True, dout=do)
    rows = np.array([0, 17, 199])
    tau = oracle.head_tau(q, k, 1.5, 0.3, True, rows=rows)
    assert np.array_equal(tau[rows], full["tau"][rows]) and np.isnan(tau[1])
    dk, dv = oracle.head_dkdv_cols(q, k, v, do, 1.5, 0.3, True, full["tau"], full["delta"],
                                   cols=[3, 150])
    assert np.array_equal(dk[[3, 150]], full["dk"][[3, 150]])
    assert np.array_equal(dv[[3, 150]], full["dv"][[3, 150]])


# -------------------------------------------------------------- backward

def _loss(q, k, v, do, alpha, scale, causal):
    tau = oracle.head_tau(q, k, alpha, scale, causal, nthreads=1)
    o, _ = oracle.head_forward_rows(q, k, v, alpha, scale, causal, tau, want_o2=False,
                                    nthreads=1)
    return np.sum(do * o)


@pytest.mark.parametrize("alpha", [1.25, 1.5, 2.0])
@pytest.mark.parametrize("causal", [False, True])
def test_backward_finite_differences(alpha, causal):
    """Central differences of L = sum(dO * O) against the analytic backward."""
    n, d, scale, h = 9, 4, 0.7, 1e-6
    rng = np.random.default_rng(int(alpha * 10) + causal)
    for _ in range(20):  # pick a seed away from support changes (kinks)
        q = rng.standard_normal((n, d)) * 2
        k, v, do = (rng.standard_normal((n, d)) for _ in range(3))
        tau = oracle.head_tau(q, k, alpha, scale, causal)
        x = (alpha - 1) * scale * (q @ k.T)
        valid = np.tril(np.ones((n, n), bool)) if causal else np.ones((n, n), bool)
        if np.min(np.abs(x - tau[:, None])[valid]) > 1e-3:
            break
    out = oracle.attention_head(q, k, v, alpha, scale, causal, dout=do)
    for name, arr, grad in (("q", q, out["dq"]), ("k", k, out["dk"]), ("v", v, out["dv"])):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a0 = arr[idx]
            arr[idx] = a0 + h
            lp = _loss(q, k, v, do, alpha, scale, causal)
            arr[idx] = a0 - h
            lm = _loss(q, k, v, do, alpha, scale, causal)
            arr[idx] = a0
            fd[idx] = (lp - lm) / (2 * h)
        err = np.max(np.abs(fd - grad)) / max(1.0, np.max(np.abs(grad)))
        assert err < 1e-6, (name, err)


def test_backward_row_sum_invariants():
    """sum_j dS_ij = 0 gives sum_j dK_j = 0; sum_j p_ij = 1 gives
    sum_j dV_j = sum_i dO_i; the two delta formulas agree."""
    n, d = 150, 16
    inp = synth.attention_inputs(1, 1, n, d, c=4.0, dtype="bf16", with_dout=True, seed=9)
    q, k, v, do = (inp[t].f64()[0, 0] for t in ("q", "k", "v", "dout"))
    for causal in (False, True):
        out = oracle.attention_head(q, k, v, 1.5, 0.25, causal, dout=do)
        assert np.max(np.abs(out["dk"].sum(0))) < 1e-11 * max(1, np.abs(out["dk"]).max()) * n
        assert np.max(np.abs(out["dv"].sum(0) - do.sum(0))) < 1e-10
        x = 0.5 * 0.25 * (q @ k.T)
        z = x - out["tau"][:, None]
        if causal:
            z = np.where(np.tril(np.ones((n, n), bool)), z, -1)
        U = np.where(z > 0, z, 0.0)
        dP = do @ v.T
        assert np.max(np.abs((U * dP).sum(1) / U.sum(1) - out["delta"])) < 1e-11


@pytest.mark.parametrize("alpha", [1.25, 1.5, 2.0, 3.0])
def test_row_backward_finite_differences(alpha):
    """The row-wise backward (gradient of <g, p> with respect to s, where
    x = (alpha-1) s) against central differences of the oracle's forward."""
    rng = np.random.default_rng(int(alpha * 100))
    n, h = 12, 1e-7
    for _ in range(50):  # a seed whose scores sit away from the support edge
        s = rng.standard_normal(n) * 3
        x = (alpha - 1) * s
        tau = oracle.entmax_threshold(x, alpha)
        if np.min(np.abs(x - tau)) > 1e-3:
            break
    g = rng.standard_normal(n)
    grad = oracle.entmax_bwd(x, alpha, tau, g)
    fd = np.zeros(n)
    for j in range(n):
        sp, sm = s.copy(), s.copy()
        sp[j] += h
        sm[j] -= h
        fd[j] = (g @ oracle.entmax((alpha - 1) * sp, alpha)[0]
                 - g @ oracle.entmax((alpha - 1) * sm, alpha)[0]) / (2 * h)
    assert np.max(np.abs(fd - grad)) <= 1e-6 * max(1.0, np.max(np.abs(grad)))
    # the Jacobian annihilates constants: gradients sum to zero over the row
    assert abs(grad.sum()) <= 1e-12 * max(1.0, np.abs(grad).max()) * n
