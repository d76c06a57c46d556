"""fp64 CPU oracle for alpha-entmax attention (AdaSplash, arXiv 2502.12082).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the bench's CPU
baseline leg may use this package; the product path (the HIP library and its
binding) never imports it and shares no code with it.

The arithmetic lives in ``entmax_oracle.c`` (plain C, double precision); this
module is argument marshalling plus per-head composition of its calls.  See the
C file's header for the definitions and the paper passages each one follows.

Inputs are numpy arrays of shape [B, H, n, d] holding the exact values the GPU
sees (bf16 or fp32 widened to fp64).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "entmax_oracle.c")
_LIB = os.path.join(_HERE, "libentmax_oracle.so")
BLOCK = 64

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain -O2, IEEE fp64, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-o", tmp, _SRC,
                               "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        D = ctypes.POINTER(ctypes.c_double)
        I = ctypes.POINTER(ctypes.c_int32)
        i, d = ctypes.c_int, ctypes.c_double
        lib.eo_entmax_threshold.argtypes = [D, i, d]
        lib.eo_entmax_threshold.restype = d
        lib.eo_entmax_row.argtypes = [D, i, d, D]
        lib.eo_entmax_row.restype = d
        lib.eo_halley_bisection_trace.argtypes = [D, i, d, i, D]
        lib.eo_entmax_row_bwd.argtypes = [D, i, d, d, D, D]
        lib.eo_tau.argtypes = [i, i, D, D, d, d, i, I, i, D, i]
        lib.eo_forward_rows.argtypes = [i, i, D, D, D, d, d, i, D, I, i, D, D, i]
        lib.eo_block_margin.argtypes = [i, i, D, D, d, d, i, D, I, i, D, i]
        lib.eo_delta_rows.argtypes = [i, i, D, D, I, i, D]
        lib.eo_dq_rows.argtypes = [i, i, D, D, D, D, d, d, i, D, D, I, i, D, i]
        lib.eo_dkdv_cols.argtypes = [i, i, D, D, D, D, d, d, i, D, D, I, i, D, D, i]
        for f in ("eo_halley_bisection_trace", "eo_tau", "eo_forward_rows", "eo_block_margin",
                  "eo_delta_rows", "eo_dq_rows", "eo_dkdv_cols", "eo_entmax_row_bwd"):
            getattr(lib, f).restype = None
        _lib = lib
    return _lib


def threads() -> int:
    """Worker threads the oracle uses (every host core this process may run on)."""
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:
        return max(1, os.cpu_count() or 1)


def _dp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _idx(sel, n):
    if sel is None:
        return None, n
    s = np.ascontiguousarray(np.asarray(sel, dtype=np.int32))
    if s.size and (s.min() < 0 or s.max() >= n):
        raise ValueError("index out of range")
    return s, int(s.size)


# --------------------------------------------------------------- single rows

def entmax_threshold(x, alpha: float) -> float:
    """Exact tau of alpha-entmax for one row already in Eq. 2 coordinates."""
    x = _f64(x)
    return _load().eo_entmax_threshold(_dp(x), x.size, float(alpha))


def entmax(x, alpha: float):
    """(p, tau) = alpha-entmax of one row in Eq. 2 coordinates (x = (alpha-1) s)."""
    x = _f64(x)
    p = np.empty_like(x)
    tau = _load().eo_entmax_row(_dp(x), x.size, float(alpha), _dp(p))
    return p, tau


def entmax_bwd(x, alpha: float, tau: float, g):
    """Gradient of <g, p> with respect to x / (alpha-1) for p = entmax(x) (one row)."""
    x, g = _f64(x), _f64(g)
    out = np.empty_like(x)
    _load().eo_entmax_row_bwd(_dp(x), x.size, float(alpha), float(tau), _dp(g), _dp(out))
    return out


def halley_bisection_trace(x, alpha: float, iters: int):
    """tau before each of `iters` Algorithm-1 updates and after the last (fp64)."""
    x = _f64(x)
    out = np.empty(iters + 1)
    _load().eo_halley_bisection_trace(_dp(x), x.size, float(alpha), int(iters), _dp(out))
    return out


# ------------------------------------------------------------- one head ops

def head_tau(q, k, alpha, scale, causal, rows=None, nthreads=None):
    q, k = _f64(q), _f64(k)
    n, d = q.shape
    r, cnt = _idx(rows, n)
    tau = np.full(n, np.nan)
    _load().eo_tau(n, d, _dp(q), _dp(k), alpha, scale, int(causal), _ip(r), cnt, _dp(tau),
                   nthreads or threads())
    return tau


def head_forward_rows(q, k, v, alpha, scale, causal, tau, rows=None, want_o2=True,
                      nthreads=None):
    q, k, v, tau = _f64(q), _f64(k), _f64(v), _f64(tau)
    n, d = q.shape
    r, cnt = _idx(rows, n)
    o = np.full((n, d), np.nan)
    o2 = np.full((n, d), np.nan) if want_o2 else None
    _load().eo_forward_rows(n, d, _dp(q), _dp(k), _dp(v), alpha, scale, int(causal), _dp(tau),
                            _ip(r), cnt, _dp(o), _dp(o2) if want_o2 else None,
                            nthreads or threads())
    return o, o2


def head_block_margin(q, k, alpha, scale, causal, tau, block_rows=None, nthreads=None):
    """[T, T] block margins max (x_ij - tau_i) over valid pairs; rows of blocks
    not in block_rows (when given) are NaN."""
    q, k, tau = _f64(q), _f64(k), _f64(tau)
    n, d = q.shape
    T = (n + BLOCK - 1) // BLOCK
    b, cnt = _idx(block_rows, T)
    m = np.full((T, T), np.nan)
    _load().eo_block_margin(n, d, _dp(q), _dp(k), alpha, scale, int(causal), _dp(tau), _ip(b),
                            cnt, _dp(m), nthreads or threads())
    return m


def head_delta_rows(dout, o2, rows=None):
    dout, o2 = _f64(dout), _f64(o2)
    n, d = dout.shape
    r, cnt = _idx(rows, n)
    delta = np.full(n, np.nan)
    _load().eo_delta_rows(n, d, _dp(dout), _dp(o2), _ip(r), cnt, _dp(delta))
    return delta


def head_dq_rows(q, k, v, dout, alpha, scale, causal, tau, delta, rows=None, nthreads=None):
    q, k, v, dout, tau, delta = map(_f64, (q, k, v, dout, tau, delta))
    n, d = q.shape
    r, cnt = _idx(rows, n)
    dq = np.full((n, d), np.nan)
    _load().eo_dq_rows(n, d, _dp(q), _dp(k), _dp(v), _dp(dout), alpha, scale, int(causal),
                       _dp(tau), _dp(delta), _ip(r), cnt, _dp(dq), nthreads or threads())
    return dq


def head_dkdv_cols(q, k, v, dout, alpha, scale, causal, tau, delta, cols=None, nthreads=None):
    q, k, v, dout, tau, delta = map(_f64, (q, k, v, dout, tau, delta))
    n, d = q.shape
    c, cnt = _idx(cols, n)
    dk = np.full((n, d), np.nan)
    dv = np.full((n, d), np.nan)
    _load().eo_dkdv_cols(n, d, _dp(q), _dp(k), _dp(v), _dp(dout), alpha, scale, int(causal),
                         _dp(tau), _dp(delta), _ip(c), cnt, _dp(dk), _dp(dv),
                         nthreads or threads())
    return dk, dv


# ------------------------------------------------------- full compositions

def attention_head(q, k, v, alpha, scale, causal, dout=None, nthreads=None):
    """Every output of one head: tau, O, O2, block margin and, given dO, delta
    and dQ/dK/dV.  Returns a dict of fp64 arrays."""
    tau = head_tau(q, k, alpha, scale, causal, nthreads=nthreads)
    o, o2 = head_forward_rows(q, k, v, alpha, scale, causal, tau, nthreads=nthreads)
    out = {"tau": tau, "o": o, "o2": o2,
           "margin": head_block_margin(q, k, alpha, scale, causal, tau, nthreads=nthreads)}
    if dout is not None:
        delta = head_delta_rows(dout, o2)
        out["delta"] = delta
        out["dq"] = head_dq_rows(q, k, v, dout, alpha, scale, causal, tau, delta,
                                 nthreads=nthreads)
        out["dk"], out["dv"] = head_dkdv_cols(q, k, v, dout, alpha, scale, causal, tau, delta,
                                              nthreads=nthreads)
    return out


def block_mask_from_margin(margin):
    """Eq. 8 read on the returned tau: a block is kept iff some p in it is > 0."""
    return (margin > 0).astype(np.uint8)
