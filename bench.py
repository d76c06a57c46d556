"""Benchmark: alpha-entmax flash attention forward + backward on one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1]

Workload (the sparsity-sweep shape): batch 1, 16 heads, n = 8192, d = 128,
bf16 inputs, non-causal, alpha = 1.5, scale = 1/sqrt(d); Q ~ c N(0,1),
K, V, dO ~ N(0,1), seeded synthetic data.  One step = the whole path: tau
solver (with the mask's row tables), sparse forward (with O2 and the column
tables), delta, dK/dV, dQ, each launched through the C ABI stage entry points
on the current stream.

Prints ONE JSON line.  `value` is dense-equivalent TFLOP/s (14 n^2 d per head
for forward + backward, the FlashAttention convention) at the headline
temperature c; `executed_tflops` counts the MFMA work the method actually
performs (solver passes over every valid block, 10 block products per listed
block).  `roofline` is for the kernel with the largest share of the step,
timed with HIP events over the timed region; `cpu_baseline` is the fp64
oracle on a bounded sample (four heads by default), on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fwd+bwd ms & effective TFLOP/s vs sparsity, n=8192 d=128 α=1.5 (1 GPU)"
PEAK_BF16_TFLOPS = 2500.0
KERNELS = ("tau_solve", "fwd_sparse", "bwd_delta", "bwd_dkdv", "bwd_dq")
# MFMA block products (64 x 64 x d each) per listed block, by kernel
PRODUCTS_PER_ACTIVE = {"fwd_sparse": 3, "bwd_dkdv": 4, "bwd_dq": 3}
# kernel name fragment in profiler output, and the sources that define each kernel
PROFILE_NAMES = {"tau_solve": "solve_kernel", "fwd_sparse": "fwd_kernel",
                 "bwd_dkdv": "dkdv2_kernel", "bwd_dq": "dq_kernel"}
KERNEL_SOURCES = {"tau_solve": ["ea_tau.hip"], "fwd_sparse": ["ea_fwd.hip"],
                  "bwd_dkdv": ["ea_bwd.hip"], "bwd_dq": ["ea_bwd.hip"]}
COMMON_SOURCES = ["ea_common.h", "ea_internal.h", "../build.py"]


def sources_sha256(kernel):
    """Hash of the files a kernel's code comes from: traffic counters taken on
    another version of them no longer describe it."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2502_12082_amd", "csrc")
    for f in KERNEL_SOURCES[kernel] + COMMON_SOURCES:
        with open(os.path.normpath(os.path.join(csrc, f)), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_path(kernel):
    return os.path.join(ROOT, "profiles", "traffic_%s.md" % kernel)


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from its committed counter summary, or
    None when there is none or its sources have changed since."""
    f = summary_fields(traffic_path(kernel), kernel)
    return None if f is None else float(f["hbm_bytes_per_launch"])


def mfma_path(kernel):
    return os.path.join(ROOT, "profiles", "mfma_%s.md" % kernel)


def summary_fields(path, kernel):
    """The `- key: value` lines of a committed counter summary, or None when
    there is none or the kernel's sources have changed since it was taken."""
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ": " in line:
            key, val = line[2:].split(": ", 1)
            fields[key.strip().strip("`")] = val.strip().strip("`")
    if fields.get("sources_sha256") != sources_sha256(kernel):
        return None
    return fields


def measured_mfma(kernel):
    """(MFMA-busy fraction, executed MFMA FLOPs per launch) of `kernel` from its
    committed rocprofv3 counter summary, or None."""
    f = summary_fields(mfma_path(kernel), kernel)
    if f is None:
        return None
    return float(f["mfma_busy"]), float(f["mfma_flops_per_launch"])


def write_mfma(pmc_csv, command, head_dim=128):
    """One summary per kernel from a rocprofv3 --pmc run of MfmaUtil and
    SQ_INSTS_VALU_MFMA_MOPS_BF16: MfmaUtil = busy cycles of the MFMA units over
    GRBM_GUI_ACTIVE x SIMDs (rocprofv3's derived counter), and the executed
    bf16 MFMA FLOPs per dispatch (512 per MOPS count)."""
    import csv
    import collections
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for row in csv.DictReader(open(pmc_csv)):
        vals[row["Kernel_Name"]][row["Counter_Name"]].append(float(row["Counter_Value"]))
    for kernel, frag in PROFILE_NAMES.items():
        names = [k for k in vals if frag in k and headline_instance(k, head_dim)]
        if not names:
            continue
        util = [v for k in names for v in vals[k]["MfmaUtil"]]
        mops = [v for k in names for v in vals[k]["SQ_INSTS_VALU_MFMA_MOPS_BF16"]]
        busy = sum(util) / len(util) / 100.0
        flops = sum(mops) / len(mops) * 512.0
        with open(mfma_path(kernel), "w") as fh:
            fh.write("# MFMA utilisation of `%s` (rocprofv3 MfmaUtil, SQ_INSTS_VALU_MFMA_MOPS_BF16)\n\n"
                     % frag)
            fh.write("Commands (repository root on an MI355X; `cd /tmp && export TMPDIR=/tmp` "
                     "first):\n\n```\n%s\n```\n\n" % command)
            fh.write("MfmaUtil is rocprofv3's derived counter: SQ_VALU_MFMA_BUSY_CYCLES summed over "
                     "the SIMDs / (GRBM_GUI_ACTIVE x SIMD count) x 100, i.e. the fraction of the "
                     "dispatch's cycles the matrix units were busy.  Executed FLOPs are "
                     "512 per SQ_INSTS_VALU_MFMA_MOPS_BF16 count (the hi/lo operand splits "
                     "included).\n\n")
            fh.write("| dispatches | MfmaUtil % (mean) | MFMA MOPS (mean) |\n|---|---|---|\n")
            fh.write("| %d | %.2f | %.0f |\n\n" % (len(util), busy * 100.0, sum(mops) / len(mops)))
            fh.write("- mfma_busy: %.4f\n" % busy)
            fh.write("- mfma_flops_per_launch: %.0f\n" % flops)
            fh.write("- sources_sha256: `%s`\n" % sources_sha256(kernel))
        print("wrote %s: MFMA busy %.1f%%, %.3e FLOP per launch" % (mfma_path(kernel),
                                                                    busy * 100, flops))


def write_kernel_stats(stats_csv, bench_json, out_md, command):
    """profiles/<out_md>: rocprofv3's per-kernel statistics of a profiled run
    next to the HIP-event kernel times of an unprofiled run of the same
    command (its JSON line), with the roofline fraction each timing gives."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    line = json.loads(open(bench_json).read().strip().splitlines()[-1])
    flops = {k: v["tflops"] * v["ms"] * 1e9 for k, v in line["kernels"].items()}
    with open(out_md, "w") as fh:
        fh.write("# rocprofv3 kernel statistics: %s\n\n" % line["config"]["workload"])
        fh.write("Commands (repository root on an MI355X; `cd /tmp && export TMPDIR=/tmp` "
                 "first):\n\n```\n%s\n```\n\n" % command)
        fh.write("| kernel | calls | average us | % of GPU time |\n|---|---|---|---|\n")
        avg = {}
        for r in rows:
            name = r["Name"]
            short = name if len(name) < 90 else name[:87] + "..."
            fh.write("| `%s` | %s | %.1f | %.2f |\n" % (short, r["Calls"],
                                                     float(r["AverageNs"]) / 1e3,
                                                     float(r["Percentage"])))
            for kernel, frag in PROFILE_NAMES.items():
                if frag in name and headline_instance(name, line["config"]["head_dim"]):
                    avg[kernel] = float(r["AverageNs"]) / 1e6
        fh.write("\nSame kernels, HIP-event times of the unprofiled run (`python bench.py` with "
                 "the arguments above, no profiler attached), and the fraction of the 2.5 PFLOP/s "
                 "bf16 peak that each timing gives for the kernel's algorithmic FLOPs:\n\n")
        fh.write("| kernel | algorithmic TFLOP per launch | profiled ms | frac | unprofiled ms "
                 "| frac |\n|---|---|---|---|---|---|\n")
        for kernel in PROFILE_NAMES:
            if kernel not in avg:
                continue
            t = line["kernels"][kernel]["ms"]
            f = flops[kernel]
            fh.write("| %s | %.4f | %.4f | %.3f | %.4f | %.3f |\n" % (
                kernel, f / 1e12, avg[kernel], f / (avg[kernel] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                t, f / (t * 1e-3) / 1e12 / PEAK_BF16_TFLOPS))
        fh.write("\nUnprofiled run: %.4f ms per step (p10 %.4f, p90 %.4f).  The profiler's "
                 "kernel trace makes kernels run a few percent slower; the JSON line's "
                 "`roofline.frac` uses the unprofiled timing.\n"
                 % (line["ms_per_step"], line["step_ms"]["p10"], line["step_ms"]["p90"]))
    print("wrote %s" % out_md)


def headline_instance(name, head_dim):
    """Whether a profiled kernel name is a bf16 instantiation for head_dim.
    rocprofv3 prints names with a __bf16 template argument mangled (dtype
    "DF16b", fp32 "If", head_dim "Li<d>E") and the bf16-only kernels'
    demangled ("dkdv2_kernel<128, 2>")."""
    if name.startswith("_Z"):
        return ("Li%dE" % head_dim) in name and "IfLi" not in name
    return ("<%d," % head_dim) in name or ("__bf16, %d," % head_dim) in name


def write_traffic(fetch_csv, write_csv, calib_mib, command, head_dim=128):
    """Scale each kernel's FETCH_SIZE and WRITE_SIZE (KiB per dispatch) by what
    the same counter reads for the plain copy of `calib_mib` MiB, and write
    one summary per kernel into profiles/.  Only the bf16 instantiations for
    `head_dim` (the headline workload's) are counted."""
    import csv
    import collections

    def per_kernel(path, counter):
        vals = collections.defaultdict(list)
        for row in csv.DictReader(open(path)):
            if row["Counter_Name"] != counter:
                continue
            vals[row["Kernel_Name"]].append(float(row["Counter_Value"]))
        return vals

    fetch = per_kernel(fetch_csv, "FETCH_SIZE")
    write = per_kernel(write_csv, "WRITE_SIZE")
    copy_name = [k for k in fetch if "copy" in k.lower()]
    if not copy_name:
        raise SystemExit("no copy dispatch in %s (run with --calib-copy-mib)" % fetch_csv)
    calib_kib = calib_mib * 1024.0
    cname = max(copy_name, key=lambda k: max(fetch[k]))
    f_scale = calib_kib / max(fetch[cname])
    w_scale = calib_kib / max(write[cname])
    for kernel, frag in PROFILE_NAMES.items():
        names = [k for k in fetch if frag in k and headline_instance(k, head_dim)]
        if not names:
            continue
        fk = [v for k in names for v in fetch[k]]
        wk = [v for k in names for v in write.get(k, [])]
        f_b = sum(fk) / len(fk) * 1024.0 * f_scale
        w_b = sum(wk) / len(wk) * 1024.0 * w_scale if wk else 0.0
        with open(traffic_path(kernel), "w") as fh:
            fh.write("# HBM traffic of `%s` (rocprofv3 FETCH_SIZE / WRITE_SIZE)\n\n" % frag)
            fh.write("Commands (repository root on an MI355X; `cd /tmp && export TMPDIR=/tmp` "
                     "first, one counter per run):\n\n```\n%s\n```\n\n" % command)
            fh.write("Scaling: the plain device copy of %d MiB read %.0f KiB (FETCH_SIZE) and "
                     "wrote %.0f KiB (WRITE_SIZE); each counter is multiplied by the ratio of "
                     "the known size to its copy reading (%.4f, %.4f).\n\n"
                     % (calib_mib, max(fetch[cname]), max(write[cname]), f_scale, w_scale))
            fh.write("| dispatches | FETCH_SIZE KiB (mean) | WRITE_SIZE KiB (mean) |\n|---|---|---|\n")
            fh.write("| %d | %.0f | %.0f |\n\n" % (len(fk), sum(fk) / len(fk),
                                                      sum(wk) / len(wk) if wk else 0.0))
            fh.write("- hbm_read_bytes_per_launch: %.0f\n" % f_b)
            fh.write("- hbm_write_bytes_per_launch: %.0f\n" % w_b)
            fh.write("- hbm_bytes_per_launch: %.0f\n" % (f_b + w_b))
            fh.write("- sources_sha256: `%s`\n" % sources_sha256(kernel))
        print("wrote %s: %.3f GB per launch" % (traffic_path(kernel), (f_b + w_b) / 1e9))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--c", type=float, default=1.0, help="headline query temperature")
    ap.add_argument("--sweep", type=str, default="0.0625,0.25,1,2,4,8,16,32",
                    help="temperatures reported in 'sweep' at the headline alpha (empty: none)")
    ap.add_argument("--sweep-alphas", type=str, default="1.25,2",
                    help="further alphas of the sweep, each at the --sweep-alpha-c temperatures")
    ap.add_argument("--sweep-alpha-c", type=str, default="1,2,4,8,16,32")
    ap.add_argument("--long", type=str, default="16384,32768,65536",
                    help="sequence lengths of the long-context report: B1 H8 d64 bf16 causal, "
                         "c 16 (empty: none)")
    ap.add_argument("--sweep-steps", type=int, default=5)
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--heads", type=int, default=16)
    ap.add_argument("--seqlen", type=int, default=8192)
    ap.add_argument("--head-dim", type=int, default=128)
    ap.add_argument("--alpha", type=float, default=1.5)
    ap.add_argument("--causal", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the tiny, encoder and decoder workloads")
    ap.add_argument("--cpu-heads", type=int, default=4, help="heads in the oracle sample")
    ap.add_argument("--no-rows", action="store_true",
                    help="skip the row-wise entmax measurement (materialized 8192 x 8192 scores)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed region, one plain device copy of this many MiB "
                         "(the reference dispatch for HBM counter scaling)")
    ap.add_argument("--kernel-stats-from", nargs=3, metavar=("STATS_CSV", "BENCH_JSON", "OUT_MD"),
                    help="write a kernel-statistics summary from a rocprofv3 --kernel-trace "
                         "--stats run and an unprofiled run's JSON line, then exit")
    ap.add_argument("--mfma-from", metavar="PMC_CSV",
                    help="write profiles/mfma_<kernel>.md from a rocprofv3 --pmc MfmaUtil "
                         "SQ_INSTS_VALU_MFMA_MOPS_BF16 run of this script, then exit")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic_<kernel>.md from two rocprofv3 --pmc runs "
                         "(FETCH_SIZE, WRITE_SIZE) of this script with --calib-copy-mib, then exit")
    return ap.parse_args()


class Runner:
    """Device buffers and the six stage launches of one configuration."""

    def __init__(self, args, c, dtype="bf16", bwd=True):
        import torch
        import synth
        import paper_2502_12082_amd as ea
        self.ea, self.torch = ea, torch
        B, H, n, d = args.batch, args.heads, args.seqlen, args.head_dim
        self.B, self.H, self.n, self.d, self.c = B, H, n, d, c
        self.bwd = bwd
        inp = synth.attention_inputs(B, H, n, d, c=c, dtype=dtype, with_dout=True)
        self.inp = inp
        if dtype == "bf16":
            dev = lambda t: torch.from_numpy(t.raw.view(np.int16)).view(torch.bfloat16).cuda()
        else:
            dev = lambda t: torch.from_numpy(np.ascontiguousarray(t.raw, dtype=np.float32)).cuda()
        self.q, self.k, self.v, self.do = (dev(inp[x]) for x in ("q", "k", "v", "dout"))
        self.shape = ea.make_shape(self.q)
        self.params = ea.make_params(args.alpha, d ** -0.5, args.causal, bwd, head_dim=d)
        self.res = ea.Residuals(self.shape, self.params, self.q.device)
        self.rp = self.res.ptrs()
        self.o = torch.empty_like(self.q)
        f32 = lambda: torch.empty(self.q.shape, dtype=torch.float32, device=self.q.device)
        self.dq, self.dk, self.dv = f32(), f32(), f32()
        self.ws = torch.empty(self.res.sizes.ws_bwd // 4 + 4, dtype=torch.float32,
                              device=self.q.device)
        self.ws_fwd = ea.forward_workspace(self.res, self.q.device)
        self.events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(KERNELS) + 1)]
                       for _ in range(max(1, args.steps))]

    def step(self, ev=None):
        ea, s = self.ea, self.torch.cuda.current_stream().cuda_stream
        q, k, v, do = self.q.data_ptr(), self.k.data_ptr(), self.v.data_ptr(), self.do.data_ptr()
        if ev:
            ev[0].record()
        for st in range(2):
            ea._check(ea.entmax_attn_fwd_stage(st, self.shape, self.params, q, k, v,
                                               self.o.data_ptr(), self.rp, self.ws_fwd.data_ptr(),
                                               self.ws_fwd.numel(), s), "fwd stage")
            if ev:
                ev[1 + st].record()
        if not self.bwd:
            return
        for st in range(3):
            ea._check(ea.entmax_attn_bwd_stage(st, self.shape, self.params, q, k, v, do, self.rp,
                                               self.dq.data_ptr(), self.dk.data_ptr(),
                                               self.dv.data_ptr(), self.ws.data_ptr(),
                                               self.ws.numel() * 4, s), "bwd stage")
            if ev:
                ev[3 + st].record()

    def timed(self, steps, warmup, per_kernel=True, warm_s=0.0):
        """Mean ms per step over `steps` steps after `warmup` untimed ones,
        followed by more untimed steps until `warm_s` seconds have passed
        (sub-millisecond steps: the GPU's clocks ramp up over tens of ms)."""
        torch = self.torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < warm_s:
            for _ in range(5):
                self.step()
            torch.cuda.synchronize()
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        wall0 = time.perf_counter()
        t_start.record()
        for i in range(steps):
            self.step(self.events[i] if per_kernel else None)
        t_end.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        total_ms = t_start.elapsed_time(t_end)
        kern = None
        if per_kernel:
            kern = {name: 0.0 for name in KERNELS}
            per_step = []
            for i in range(steps):
                ev = self.events[i]
                for j, name in enumerate(KERNELS):
                    kern[name] += ev[j].elapsed_time(ev[j + 1])
                per_step.append(ev[0].elapsed_time(ev[len(KERNELS)]))
            kern = {k_: v_ / steps for k_, v_ in kern.items()}
            q = np.percentile(per_step, [10, 50, 90])
            kern["_steps"] = {"p10": round(float(q[0]), 4), "median": round(float(q[1]), 4),
                              "p90": round(float(q[2]), 4)}
        return total_ms / steps, wall, kern

    def work(self):
        """Block counts and FLOPs of the last step (from its mask and stats)."""
        n, d, BH = self.n, self.d, self.B * self.H
        T = (n + 63) // 64
        f_blk = 2.0 * 64 * 64 * d
        mask = self.res.block_mask.cpu().numpy()
        if self.params.causal:
            n_valid = BH * T * (T + 1) // 2
        else:
            n_valid = BH * T * T
        n_act = int(self.res.q_count.sum().item())
        planes = self.res.stats.cpu().numpy().astype(np.int64).reshape(2, BH, T)
        stats, evals = planes[0], planes[1]
        # valid 64x64 blocks each query block streams per solver pass
        per_qb = np.arange(1, T + 1) if self.params.causal else np.full(T, T)
        # The solver's work is its K passes: the max pass and the evaluation
        # passes that streamed K (stats).  The extra stream over the leading
        # key blocks that precedes a candidate collection is an implementation
        # choice, not work of the method, and is left out.
        solver_blocks = float((stats * per_qb[None, :]).sum())
        flops = {"tau_solve": solver_blocks * f_blk, "bwd_delta": 0.0}
        for k_, m in PRODUCTS_PER_ACTIVE.items():
            # the forward without a backward to follow forms S and P V only
            if k_ == "fwd_sparse" and not self.bwd:
                m = 2
            flops[k_] = m * n_act * f_blk
        dense = 14.0 * n * n * d * BH * (0.5 if self.params.causal else 1.0)
        return {"n_valid": n_valid, "n_act": n_act, "block_density": n_act / n_valid,
                "passes_mean": float(stats.mean()), "passes_max": int(stats.max()),
                "evals_mean": float(evals.mean()), "evals_max": int(evals.max()),
                "flops": flops, "dense_flops": dense, "mask_nnz": int(mask.sum())}

    def _sampled_z(self, rows):
        """x - tau (fp64, from the input values and the returned tau) on
        `rows` sampled rows of head 0; invalid pairs hold -1."""
        q = self.inp["q"].f64()[0, 0]
        k = self.inp["k"].f64()[0, 0]
        tau = self.res.tau[0].cpu().numpy().astype(np.float64)
        if self.res.tau_lo is not None:
            tau = tau + self.res.tau_lo[0].cpu().numpy().astype(np.float64)
        idx = np.linspace(0, self.n - 1, rows).astype(int)
        a, sc = float(np.float32(self.params.alpha)), float(np.float32(self.params.scale))
        z = (a - 1) * sc * (q[idx] @ k.T) - tau[idx, None]
        if self.params.causal:
            z = np.where(np.arange(self.n)[None, :] <= idx[:, None], z, -1.0)
        return idx, z

    def zero_fraction(self, rows=64):
        """Fraction of zero probabilities on sampled rows of head 0, from the
        returned tau (host numpy; a statistic, not part of the timed path)."""
        idx, z = self._sampled_z(rows)
        valid = (idx + 1).sum() if self.params.causal else rows * self.n
        return 1.0 - float((z > 0).sum()) / valid

    def sum_p_error(self, rows=64):
        """max |sum_j p_ij - 1| over sampled rows of head 0 at the returned tau:
        f(tau) of Eq. 3, the residual Algorithm 1's output leaves (O is not
        renormalised)."""
        _, z = self._sampled_z(rows)
        g = 1.0 / (float(np.float32(self.params.alpha)) - 1.0)
        p = np.where(z > 0, np.maximum(z, 0.0) ** g, 0.0)
        return float(np.max(np.abs(p.sum(1) - 1.0)))


PEAK_HBM_GBS = 8000.0


def rows_bench(steps=20, warmup=3, rows=8192, n=8192, alpha=1.5):
    """Row-wise alpha-entmax of a materialized [rows, n] fp32 Gaussian score
    matrix (the shape of the paper's Halley-bisection efficiency benchmark):
    forward (p, tau) and backward (ds), each HBM-bound; achieved = bytes one
    launch must move (read s; write p) or (read s, dp; write ds) / time."""
    import torch
    import paper_2502_12082_amd as ea
    gen = torch.Generator(device="cuda")
    gen.manual_seed(20250217 + 7)
    s = torch.randn((rows, n), generator=gen, device="cuda", dtype=torch.float32)
    dp = torch.randn((rows, n), generator=gen, device="cuda", dtype=torch.float32)
    out = {}
    for kind in ("fwd", "bwd"):
        p, tau = ea.rows_forward(s, alpha=alpha)
        fn = (lambda: ea.rows_forward(s, alpha=alpha)) if kind == "fwd" else \
            (lambda: ea.rows_backward(s, tau, dp, alpha=alpha))
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / steps
        nbytes = rows * n * 4 * (2 if kind == "fwd" else 3) + rows * 4
        gbs = nbytes / (ms * 1e-3) / 1e9
        out[kind] = {"ms": round(ms, 4), "GB/s": round(gbs, 1),
                     "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}
    out["shape"] = "%d x %d fp32, alpha %g, N(0,1) scores" % (rows, n, alpha)
    return out


def dense_mode_bench(run, steps=5, warmup=2):
    """The no-mask mode (fused tau + O forward, table-free backward) on the
    headline workload: ms per fwd+bwd step and dense-equivalent TFLOP/s.  All
    buffers are allocated before the timed loop, which makes only the two C
    ABI calls per step."""
    import ctypes
    import torch
    import paper_2502_12082_amd as ea
    q, k, v, do = run.q, run.k, run.v, run.do
    p = run.params
    o = torch.empty_like(q)
    tau = torch.empty((run.B * run.H, run.n), dtype=torch.float32, device=q.device)
    f32 = lambda: torch.empty(q.shape, dtype=torch.float32, device=q.device)
    o2, dq, dk, dv = f32(), f32(), f32(), f32()
    ws = ea.forward_workspace(run.res, q.device)
    wsb = torch.empty(run.res.sizes.ws_bwd // 4 + 4, dtype=torch.float32, device=q.device)
    shape, stream = run.shape, torch.cuda.current_stream().cuda_stream
    ptr = lambda t: t.data_ptr()

    def step():
        ea._check(ea._lib.entmax_attn_fwd_dense(
            ctypes.byref(shape), ctypes.byref(p), ptr(q), ptr(k), ptr(v), ptr(o), ptr(tau),
            None, ptr(o2), ptr(ws), ws.numel(), stream), "entmax_attn_fwd_dense")
        ea._check(ea._lib.entmax_attn_bwd_dense(
            ctypes.byref(shape), ctypes.byref(p), ptr(q), ptr(k), ptr(v), ptr(do), ptr(tau),
            None, ptr(o2), ptr(dq), ptr(dk), ptr(dv), ptr(wsb), wsb.numel() * 4, stream),
            "entmax_attn_bwd_dense")

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        step()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    dense = 14.0 * run.n * run.n * run.d * run.B * run.H * (0.5 if p.causal else 1.0)
    return {"ms_per_step": round(ms, 4), "tflops_dense_equiv": round(dense / (ms * 1e-3) / 1e12, 3)}


def sweep_point(args, alpha, c):
    """One point of the sparsity sweep (its own inputs and buffers)."""
    import torch
    a = argparse.Namespace(**{**vars(args), "alpha": alpha})
    r = Runner(a, c)
    msv, _, _ = r.timed(max(1, args.sweep_steps), 2, per_kernel=False)
    w = r.work()
    out = {"alpha": alpha, "c": c, "ms": round(msv, 4),
           "tflops_dense_equiv": round(w["dense_flops"] / (msv * 1e-3) / 1e12, 3),
           "tflops_executed": round(sum(w["flops"].values()) / (msv * 1e-3) / 1e12, 3),
           "block_density": round(w["block_density"], 4),
           "zero_fraction_sampled": round(r.zero_fraction(), 5),
           "solver_passes_mean": round(w["passes_mean"], 3),
           "solver_evals_mean": round(w["evals_mean"], 3),
           "sum_p_minus_1_max_sampled": r.sum_p_error()}
    del r
    torch.cuda.empty_cache()
    return out


def other_configs(args, steps=20, warmup=5):
    """The other workload shapes, each at its own size: the tiny fp32 forward,
    the encoder-shaped forward at three temperatures and the decoder-shaped
    training step (ms per call and dense-equivalent TFLOP/s).  Each call takes
    0.07-1 ms: 20 timed calls follow at least 50 ms of untimed ones, so that
    the timed region sees the clocks of a busy GPU."""
    import torch
    cases = [("tiny forward", 1, 1, 256, 64, "f32", False, 1.0, False),
             ("encoder forward", 8, 12, 1024, 64, "bf16", False, 1.0, False),
             ("encoder forward", 8, 12, 1024, 64, "bf16", False, 4.0, False),
             ("encoder forward", 8, 12, 1024, 64, "bf16", False, 16.0, False),
             ("decoder step", 4, 12, 4096, 64, "bf16", True, 8.0, True)]
    out = []
    for name, B, H, n, d, dt, causal, c, bwd in cases:
        a = argparse.Namespace(**{**vars(args), "batch": B, "heads": H, "seqlen": n,
                                  "head_dim": d, "alpha": 1.5, "causal": causal, "steps": steps})
        r = Runner(a, c, dtype=dt, bwd=bwd)
        ms, _, _ = r.timed(steps, warmup, per_kernel=False, warm_s=0.05)
        w = r.work()
        flops = (14.0 if bwd else 4.0) * n * n * d * B * H * (0.5 if causal else 1.0)
        executed = sum(v_ for k_, v_ in w["flops"].items()
                       if bwd or k_ in ("tau_solve", "fwd_sparse"))
        out.append({"config": name, "shape": "B%d H%d n%d d%d %s%s" % (
                        B, H, n, d, dt, " causal" if causal else ""),
                    "c": c, "fwd_bwd" if bwd else "fwd": True, "ms": round(ms, 4),
                    "tflops_dense_equiv": round(flops / (ms * 1e-3) / 1e12, 3),
                    "tflops_executed": round(executed / (ms * 1e-3) / 1e12, 3),
                    "block_density": round(w["block_density"], 4),
                    "solver_passes_mean": round(w["passes_mean"], 3)})
        del r
        torch.cuda.empty_cache()
    return out


def long_context(args, lengths, steps=3):
    """The long-context workload (B1 H8 d64 bf16, causal, alpha 1.5, c 16):
    fwd+bwd time and the device memory it holds, per sequence length."""
    import torch
    out = []
    for n in lengths:
        a = argparse.Namespace(**{**vars(args), "batch": 1, "heads": 8, "seqlen": n,
                                  "head_dim": 64, "alpha": 1.5, "causal": True, "steps": steps})
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        r = Runner(a, 16.0)
        ms, _, _ = r.timed(steps, 1, per_kernel=False)
        peak = torch.cuda.max_memory_allocated() - base
        w = r.work()
        z = r.res.sizes
        resid = z.tau + z.o2 + z.block_mask + z.q_count + z.q_index + z.k_count + z.k_index + z.stats
        io = 4 * r.q.numel() * r.q.element_size() + 3 * r.q.numel() * 4  # Q K V dO O, dQ dK dV
        out.append({"seqlen": n, "ms": round(ms, 3),
                    "tflops_dense_equiv": round(w["dense_flops"] / (ms * 1e-3) / 1e12, 3),
                    "tflops_executed": round(sum(w["flops"].values()) / (ms * 1e-3) / 1e12, 3),
                    "block_density": round(w["block_density"], 4),
                    "solver_passes_mean": round(w["passes_mean"], 3),
                    "peak_device_mib": round(peak / 2**20, 1),
                    "library_residual_mib": round(resid / 2**20, 1),
                    "library_workspace_mib": round((z.ws_fwd + z.ws_bwd) / 2**20, 1),
                    "inputs_outputs_mib": round(io / 2**20, 1)})
        del r
    torch.cuda.empty_cache()
    return {"workload": "B1 H8 d64 bf16, causal, alpha 1.5, c 16", "steps": steps, "points": out}


def cpu_baseline(runner, heads):
    """The oracle (fp64, all host cores) on `heads` heads of the same workload:
    tau, O, O2, block margins, delta, dQ, dK, dV of every row and column."""
    import oracle
    inp = runner.inp
    heads = max(1, min(heads, runner.B * runner.H))
    oracle.build()
    sec = 0.0
    for bh in range(heads):
        b, h = divmod(bh, runner.H)
        q, k, v, do = (inp[x].f64()[b, h] for x in ("q", "k", "v", "dout"))
        t0 = time.perf_counter()
        oracle.attention_head(q, k, v, runner.params.alpha, runner.params.scale,
                              bool(runner.params.causal), dout=do)
        sec += time.perf_counter() - t0
    flops = heads * 14.0 * runner.n * runner.n * runner.d * (0.5 if runner.params.causal else 1.0)
    return {"value": flops / sec / 1e12, "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle",
            "sample": "%d of %d heads (all %d rows and columns), fwd+bwd, %.1f s; dense-equivalent "
                      "FLOPs of the sample / time" % (heads, runner.B * runner.H, runner.n, sec)}


def main():
    args = parse()
    if args.kernel_stats_from:
        stats_csv, bench_json, out_md = args.kernel_stats_from
        line = json.loads(open(bench_json).read().strip().splitlines()[-1])
        base = ("python bench.py --steps %d --warmup %d --sweep= --long= --no-configs "
                "--no-cpu-baseline --no-rows" % (line["steps"], line["warmup"]))
        write_kernel_stats(stats_csv, bench_json, out_md,
                           "%s > %s\nrocprofv3 --kernel-trace --stats --output-format csv -d %s -o run "
                           "-- %s\npython bench.py --kernel-stats-from %s %s %s"
                           % (base, bench_json, os.path.dirname(stats_csv), base, stats_csv,
                              bench_json, out_md))
        return
    if args.mfma_from:
        run = ("-- python bench.py --steps 2 --warmup 1 --sweep= --long= --no-configs "
               "--no-cpu-baseline --no-rows")
        write_mfma(args.mfma_from,
                   "rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_BF16 --output-format csv -d %s "
                   "-o run %s\npython bench.py --mfma-from %s"
                   % (os.path.dirname(args.mfma_from), run, args.mfma_from),
                   head_dim=args.head_dim)
        return
    if args.traffic_from:
        mib = args.calib_copy_mib or 1024
        fetch_csv, write_csv = args.traffic_from
        # the counter runs that wrote the two files, as they were run
        run = ("-- python bench.py --steps 2 --warmup 1 --sweep= --long= --no-configs "
               "--no-cpu-baseline --no-rows --calib-copy-mib %d" % mib)
        write_traffic(fetch_csv, write_csv, mib,
                      "rocprofv3 --pmc FETCH_SIZE --output-format csv -d %s -o run %s\n"
                      "rocprofv3 --pmc WRITE_SIZE --output-format csv -d %s -o run %s\n"
                      "python bench.py --traffic-from %s %s --calib-copy-mib %d"
                      % (os.path.dirname(fetch_csv), run, os.path.dirname(write_csv), run,
                         fetch_csv, write_csv, mib), head_dim=args.head_dim)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the alpha-entmax path here is a single-GPU "
              "build (heads would shard across GPUs with no communication); --gpus %d is not "
              "supported" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    steps = max(1, args.steps)
    run = Runner(args, args.c)
    ms, wall, kern = run.timed(steps, args.warmup)
    work = run.work()
    dense_tflops = work["dense_flops"] / (ms * 1e-3) / 1e12
    executed = sum(work["flops"].values())
    kernels = {}
    for name in KERNELS:
        t = kern[name]
        kernels[name] = {"ms": round(t, 4),
                         "tflops": round(work["flops"][name] / (t * 1e-3) / 1e12, 2) if t > 0 else 0.0}
        if name in PROFILE_NAMES:
            mf = measured_mfma(name)
            tr = measured_traffic(name)
            # from the committed counter summaries (null once the sources changed)
            kernels[name]["mfma_busy"] = round(mf[0], 4) if mf else None
            kernels[name]["mfma_executed_tflops"] = (round(mf[1] / (t * 1e-3) / 1e12, 2)
                                                     if mf and t > 0 else None)
            kernels[name]["hbm_GBps"] = round(tr / (t * 1e-3) / 1e9, 1) if tr and t > 0 else None
    dom = max(("tau_solve", "fwd_sparse", "bwd_dkdv", "bwd_dq"), key=lambda k_: kern[k_])
    ach = work["flops"][dom] / (kern[dom] * 1e-3) / 1e12
    traffic = measured_traffic(dom)
    roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                "traffic": round(traffic) if traffic is not None else None,
                "traffic_unit": "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE, "
                                "copy-calibrated)",
                "timing": "HIP events around the kernel's stage launch on the current stream, "
                          "mean over the timed steps (no profiler attached)",
                "mfma_busy": kernels[dom].get("mfma_busy")}
    if args.calib_copy_mib > 0:
        src = torch.empty(args.calib_copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    out = {
        "metric": METRIC, "value": round(dense_tflops, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian Q*c, K, V, dO)",
        "config": {"workload": "alpha-entmax attention fwd+bwd, B%d H%d n%d d%d bf16 %s, "
                               "alpha %g, c %g" % (args.batch, args.heads, args.seqlen,
                                                   args.head_dim,
                                                   "causal" if args.causal else "non-causal",
                                                   args.alpha, args.c),
                   "batch": args.batch, "heads": args.heads, "seqlen": args.seqlen,
                   "head_dim": args.head_dim, "alpha": args.alpha, "c": args.c,
                   "causal": bool(args.causal)},
        "executed_tflops": round(executed / (ms * 1e-3) / 1e12, 3),
        "executed_frac_of_peak": round(executed / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "wall_s_timed": round(wall, 4),
        "step_ms": kern["_steps"],
        "kernels": kernels,
        "sparsity": {"block_density": round(work["block_density"], 4),
                     "zero_fraction_sampled": round(run.zero_fraction(), 5),
                     "solver_passes_mean": round(work["passes_mean"], 3),
                     "solver_passes_max": work["passes_max"],
                     "solver_evals_mean": round(work["evals_mean"], 3),
                     "solver_evals_max": work["evals_max"],
                     "sum_p_minus_1_max_sampled": run.sum_p_error()},
        "roofline": roofline,
    }
    vals = lambda text: [float(x) for x in text.split(",") if x.strip()]
    sweep = [sweep_point(args, args.alpha, cv) for cv in vals(args.sweep)]
    if sweep:
        for av in vals(args.sweep_alphas):
            sweep += [sweep_point(args, av, cv) for cv in vals(args.sweep_alpha_c)]
        out["sweep"] = sweep
    if args.long.strip():
        out["long_context"] = long_context(args, [int(x) for x in vals(args.long)])
    if not args.no_configs:
        out["other_configs"] = other_configs(args)
    if not args.no_rows:
        out["entmax_rows"] = rows_bench()
        out["entmax_rows_short"] = rows_bench(rows=65536, n=1024)
        out["no_mask_mode"] = dense_mode_bench(run)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(run, args.cpu_heads)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
