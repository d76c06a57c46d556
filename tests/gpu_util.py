"""Helpers for the GPU tests: run the HIP path through the C ABI binding and
the fp64 oracle on the same seeded inputs, and compare them."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import synth

BF16_TOL = 2e-2    # max-abs for O, O2, dQ, dK, dV with bf16 inputs
F32_TOL = 1e-4     # max-abs with fp32 inputs
TAU_REL = 1e-3     # |dtau| <= TAU_REL * max(1, |tau|)
MASK_BAND = 1e-4   # blocks with |margin| <= MASK_BAND * max(1, |tau|) may legitimately flip
# Blocks inside that band are few: the band is ~1e-4 |tau| wide while block
# margins spread over O(1), so about 1e-3 of the blocks (15 of the 16384 of
# one n = 8192 head at c = 4).  More than MASK_BAND_FRAC of the checked
# blocks (plus a few) means the band is too wide to be a meaningful check.
MASK_BAND_FRAC = 2e-3
# The GPU's own mask against its own tau (Sec. 3.2.1: a block may be skipped
# only if all its probabilities are zero): fp64 margins at the GPU's tau must
# be <= 0 on every skipped block and > 0 on every kept one, up to the fp32
# rounding of the GPU's scores, SELF_BAND * max(1, |tau|).
SELF_BAND = 2e-5


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(t: synth.Tensor):
    import torch
    if t.dtype == "bf16":
        x = torch.from_numpy(t.raw.view(np.int16)).view(torch.bfloat16)
    else:
        x = torch.from_numpy(t.raw)
    return x.cuda().contiguous()


def run_gpu(inp: dict, alpha: float, scale: float, causal: bool, bwd: bool, max_iter=None,
            tol=None, device_inputs=None, heads=None):
    """All outputs of the HIP path as numpy arrays (float64 for float data).
    heads: copy the [n, d] outputs (O, O2, dQ, dK, dV) of these heads only,
    as a dict {bh: array}; None copies every head."""
    import torch
    import paper_2502_12082_amd as ea
    q, k, v = device_inputs or (to_device(inp["q"]), to_device(inp["k"]), to_device(inp["v"]))
    B, H, n, d = q.shape
    o, res = ea.forward(q, k, v, alpha=alpha, scale=scale, causal=causal, need_bwd=bwd,
                        max_iter=max_iter, tol=tol)
    out = {}
    if bwd:
        do = to_device(inp["dout"])
        dq, dk, dv = ea.backward(q, k, v, do, res)
        out.update(dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    out.update(o=o.float(), tau=res.tau, mask=res.block_mask, q_count=res.q_count,
               q_index=res.q_index, k_count=res.k_count, k_index=res.k_index, stats=res.stats)
    if res.tau_lo is not None:
        out["tau_lo"] = res.tau_lo
    if bwd:
        out["o2"] = res.o2
    host = {}
    BH = B * H
    big = ("o", "o2", "dq", "dk", "dv")
    for key, val in out.items():
        if key in big:
            val = val.reshape(BH, n, d)
            if heads is not None:
                host[key] = {bh: val[bh].cpu().numpy().astype(np.float64) for bh in heads}
                continue
        a = val.cpu().numpy()
        host[key] = a.astype(np.float64) if a.dtype.kind == "f" else a
    host["inputs"] = inp
    host["params"] = (alpha, scale, causal)
    return host


def abi_param(x: float) -> float:
    """The value the C ABI receives for alpha or scale: they are fp32 fields,
    so the oracle computes with the same fp32-rounded numbers."""
    return float(np.float32(x))


def oracle_head(inp: dict, bh: int, alpha, scale, causal, bwd, rows=None, cols=None,
                block_rows=None):
    """Oracle outputs for head bh.  rows/cols=None: every row/column; otherwise
    only those rows (tau, O, O2, dQ) and columns (dK, dV) are computed, plus
    whatever rows the listed columns depend on.  block_rows: 64-row query
    blocks whose mask margins to compute (None with rows=None: all).  alpha
    and scale are taken as the fp32 values the GPU path is given."""
    alpha, scale = abi_param(alpha), abi_param(scale)
    B, H, n, d = inp["q"].shape
    b, h = divmod(bh, H)
    q = inp["q"].f64()[b, h]
    k = inp["k"].f64()[b, h]
    v = inp["v"].f64()[b, h]
    do = inp["dout"].f64()[b, h] if bwd else None
    if rows is None and cols is None and block_rows is None:
        return oracle.attention_head(q, k, v, alpha, scale, causal, dout=do)
    need = set()
    if rows is not None:
        need.update(int(r) for r in rows)
    if block_rows is not None:
        for I in block_rows:
            need.update(range(I * 64, min(n, I * 64 + 64)))
    if cols is not None and bwd:
        lo = int(np.min(cols)) if causal else 0
        need.update(range(lo, n))
    need = np.array(sorted(need), dtype=np.int32)
    tau = oracle.head_tau(q, k, alpha, scale, causal, rows=need)
    o, o2 = oracle.head_forward_rows(q, k, v, alpha, scale, causal, tau, rows=need)
    out = {"tau": tau, "o": o, "o2": o2, "rows": np.array(sorted(rows)) if rows is not None else None}
    if block_rows is not None:
        out["margin"] = oracle.head_block_margin(q, k, alpha, scale, causal, tau,
                                                 block_rows=block_rows)
        out["block_rows"] = list(block_rows)
    if bwd:
        delta = oracle.head_delta_rows(do, o2, rows=need)
        out["delta"] = delta
        if rows is not None:
            out["dq"] = oracle.head_dq_rows(q, k, v, do, alpha, scale, causal, tau, delta,
                                            rows=rows)
        if cols is not None:
            out["dk"], out["dv"] = oracle.head_dkdv_cols(q, k, v, do, alpha, scale, causal, tau,
                                                         delta, cols=cols)
            out["cols"] = np.array(sorted(cols))
    return out


def maxabs(a, b):
    return float(np.max(np.abs(a - b))) if a.size else 0.0


def check_head(gpu: dict, ref: dict, bh: int, dtype: str, label: str, rows=None, cols=None):
    """Asserts parity of one head; returns a dict of the measured errors."""
    tol = BF16_TOL if dtype == "bf16" else F32_TOL
    n = gpu["tau"].shape[1]
    r = np.arange(n) if rows is None else np.asarray(sorted(rows))
    errs = {}
    tr, tg = ref["tau"][r], gpu["tau"][bh][r]
    if "tau_lo" in gpu:
        tg = tg + gpu["tau_lo"][bh][r]
    errs["tau_rel"] = float(np.max(np.abs(tg - tr) / np.maximum(1.0, np.abs(tr))))
    assert errs["tau_rel"] <= TAU_REL, (label, "tau", errs)
    errs["o"] = maxabs(gpu["o"][bh][r], ref["o"][r])
    assert errs["o"] <= tol, (label, "O", errs)
    if "o2" in gpu and ref.get("o2") is not None:
        errs["o2"] = maxabs(gpu["o2"][bh][r], ref["o2"][r])
        assert errs["o2"] <= tol, (label, "O2", errs)
    if "dq" in gpu and "dq" in ref:
        errs["dq"] = maxabs(gpu["dq"][bh][r], ref["dq"][r])
        assert errs["dq"] <= tol, (label, "dQ", errs)
    if "dk" in gpu and "dk" in ref:
        c = np.arange(n) if cols is None else np.asarray(sorted(cols))
        errs["dk"] = maxabs(gpu["dk"][bh][c], ref["dk"][c])
        errs["dv"] = maxabs(gpu["dv"][bh][c], ref["dv"][c])
        assert errs["dk"] <= tol, (label, "dK", errs)
        assert errs["dv"] <= tol, (label, "dV", errs)
    if "margin" in ref:
        errs.update(check_mask(gpu["mask"][bh], ref["margin"], ref["tau"], n,
                               ref.get("block_rows"), label))
        errs.update(check_mask_self(gpu, bh, ref.get("block_rows"), label))
    return errs


def check_mask(mask, margin, tau_ref, n, block_rows, label):
    """Bit-exact outside the guard band |margin| <= MASK_BAND * max(1, |tau|)."""
    T = mask.shape[0]
    rows = range(T) if block_rows is None else block_rows
    flips = band = band_flips = checked = 0
    for I in rows:
        t = tau_ref[I * 64:min(n, I * 64 + 64)]
        g = MASK_BAND * max(1.0, float(np.nanmax(np.abs(t))))
        m = margin[I]
        ref = (m > 0).astype(np.uint8)
        inband = np.abs(m) <= g
        band += int(inband.sum())
        bad = (mask[I] != ref) & ~inband
        flips += int(bad.sum())
        band_flips += int(((mask[I] != ref) & inband).sum())
        checked += int(np.isfinite(m).sum())
    assert flips == 0, (label, "mask differs outside the guard band", flips)
    assert band <= 4 + MASK_BAND_FRAC * checked, (label, "blocks inside the guard band", band,
                                                  checked)
    return {"mask_band_blocks": band, "mask_band_flips": band_flips, "mask_blocks": checked}


def check_mask_self(gpu: dict, bh: int, block_rows, label):
    """The GPU's mask describes exactly the probabilities at the GPU's own
    tau: with the margins max (x_ij - tau_gpu_i) of each block, in fp64 from
    the same input values, a skipped block has margin <= 0 and a kept block
    margin > 0, outside a band that covers the fp32 rounding of the GPU's
    scores (Sec. 3.2.1: only blocks whose probabilities are all zero may be
    skipped).  Returns the number of blocks inside that band."""
    inp = gpu["inputs"]
    alpha, scale, causal = gpu["params"]
    alpha, scale = abi_param(alpha), abi_param(scale)
    B, H, n, d = inp["q"].shape
    b, h = divmod(bh, H)
    tau = gpu["tau"][bh] + (gpu["tau_lo"][bh] if "tau_lo" in gpu else 0.0)
    margin = oracle.head_block_margin(inp["q"].f64()[b, h], inp["k"].f64()[b, h], alpha, scale,
                                      causal, tau, block_rows=block_rows)
    mask = gpu["mask"][bh]
    T = mask.shape[0]
    rows = range(T) if block_rows is None else block_rows
    band = 0
    for I in rows:
        t = tau[I * 64:min(n, I * 64 + 64)]
        g = SELF_BAND * max(1.0, float(np.max(np.abs(t))))
        m = margin[I]
        if causal:  # blocks entirely above the diagonal hold no valid pair
            m = np.where(np.arange(T) > I, -np.inf, m)
        inband = np.abs(m) <= g
        band += int(inband.sum())
        skipped_but_positive = (mask[I] == 0) & (m > g)
        kept_but_empty = (mask[I] == 1) & (m < -g)
        assert not skipped_but_positive.any(), (label, "a skipped block has p > 0 at the GPU tau",
                                                I, np.nonzero(skipped_but_positive)[0])
        assert not kept_but_empty.any(), (label, "a kept block has no p > 0 at the GPU tau",
                                          I, np.nonzero(kept_but_empty)[0])
    return {"self_band_blocks": band}


def check_tables(gpu: dict, causal: bool, columns: bool = True):
    """Integer checks, bit-exact: tables list exactly the mask's nonzeros,
    ascending; every mask row has a block; causal dead blocks are empty.
    columns: also the key-block tables (written by a training forward)."""
    mask = gpu["mask"]
    BH, T, _ = mask.shape
    for bh in range(BH):
        M = mask[bh]
        assert M.max() <= 1
        assert np.all(M.sum(1) >= 1), "a query block with no key block"
        if causal:
            assert not np.any(np.triu(M, 1)), "causally dead block set"
        for i in range(T):
            cols = np.nonzero(M[i])[0]
            assert gpu["q_count"][bh, i] == cols.size
            assert np.array_equal(gpu["q_index"][bh, i, :cols.size], cols)
        for j in range(T if columns else 0):
            rows = np.nonzero(M[:, j])[0]
            assert gpu["k_count"][bh, j] == rows.size
            assert np.array_equal(gpu["k_index"][bh, j, :rows.size], rows)
