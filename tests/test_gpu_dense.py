"""GPU parity of the no-mask ("memory-efficient") mode: the fused forward
(tau and O, O2 in one kernel, no block mask or tables) and the backward that
visits every valid block, against the fp64 oracle and against the masked
path on the same inputs."""
import numpy as np
import pytest

import synth
from gpu_util import BF16_TOL, F32_TOL, TAU_REL, log, maxabs, oracle_head, to_device

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_12082_amd  # noqa: F401


def _run_dense(inp, alpha, causal, bwd):
    import paper_2502_12082_amd as ea
    q, k, v = to_device(inp["q"]), to_device(inp["k"]), to_device(inp["v"])
    d = q.shape[-1]
    o, tau, o2, tau_lo = ea.forward_dense(q, k, v, alpha=alpha, scale=d ** -0.5, causal=causal,
                                          need_bwd=bwd)
    out = {"o": o, "tau": tau + tau_lo if tau_lo is not None else tau, "o2": o2}
    if bwd:
        do = to_device(inp["dout"])
        out["dq"], out["dk"], out["dv"] = ea.backward_dense(q, k, v, do, tau, o2, alpha=alpha,
                                                            scale=d ** -0.5, causal=causal,
                                                            tau_lo=tau_lo)
    torch.cuda.synchronize()
    return {key: (val.float().cpu().numpy().astype(np.float64) if val is not None else None)
            for key, val in out.items()}


@pytest.mark.parametrize("n", [1, 63, 64, 65, 300])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128), ("bf16", 64)])
@pytest.mark.parametrize("alpha", [1.5, 2.0, 1.6])
def test_dense_against_oracle(n, causal, dtype, d, alpha):
    B, H = 1, 2
    inp = synth.attention_inputs(B, H, n, d, c=1.0, dtype=dtype, with_dout=True, seed=31)
    gpu = _run_dense(inp, alpha, causal, True)
    tol = BF16_TOL if dtype == "bf16" else F32_TOL
    for bh in range(B * H):
        ref = oracle_head(inp, bh, alpha, d ** -0.5, causal, True)
        errs = {"tau": float(np.max(np.abs(gpu["tau"][bh] - ref["tau"]) / np.maximum(1, np.abs(ref["tau"]))))}
        for key in ("o", "o2", "dq", "dk", "dv"):
            errs[key] = maxabs(gpu[key].reshape(B * H, n, d)[bh], ref[key])
        log("dense n%d causal%d %s d%d alpha %g bh%d: %s" % (n, causal, dtype, d, alpha, bh, errs))
        assert errs["tau"] <= TAU_REL
        for key in ("o", "o2", "dq", "dk", "dv"):
            assert errs[key] <= tol, (key, errs)


def test_dense_matches_masked_path():
    """Bench-shaped heads: the no-mask mode and the masked path agree."""
    import paper_2502_12082_amd as ea
    inp = synth.attention_inputs(1, 4, 2048, 128, c=1.0, dtype="bf16", with_dout=True, seed=5)
    q, k, v, do = (to_device(inp[x]) for x in ("q", "k", "v", "dout"))
    for causal in (False, True):
        o, res = ea.forward(q, k, v, alpha=1.5, causal=causal)
        dq, dk, dv = ea.backward(q, k, v, do, res)
        o_d, tau_d, o2_d, _ = ea.forward_dense(q, k, v, alpha=1.5, causal=causal)
        dq_d, dk_d, dv_d = ea.backward_dense(q, k, v, do, tau_d, o2_d, alpha=1.5, causal=causal)
        torch.cuda.synchronize()
        dt = ((tau_d - res.tau).abs() / res.tau.abs().clamp(min=1)).max().item()
        errs = {"tau": dt}
        for name, a_, b_ in (("o", o_d, o), ("o2", o2_d, res.o2), ("dq", dq_d, dq), ("dk", dk_d, dk),
                             ("dv", dv_d, dv)):
            errs[name] = (a_.float() - b_.float()).abs().max().item()
        log("dense vs masked causal=%d: %s" % (causal, errs))
        assert errs["tau"] <= 1e-5
        for name in ("o", "o2", "dq", "dk", "dv"):
            assert errs[name] <= BF16_TOL, (name, errs)


@pytest.mark.parametrize("n", [1, 63, 65, 257])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("d", [64, 128])
def test_dense_f32_general_alpha(n, causal, d):
    """fp32 inputs at alpha in (1.5, 2), where u = z^(gamma-1) is steep near
    the support edge: the fused forward refines tau in fp64 (tau + tau_lo) and
    takes x - tau in fp64 near the edge, and the backward reads tau_lo."""
    B, H = 1, 2
    for alpha in (1.6, 1.7, 1.75):
        inp = synth.attention_inputs(B, H, n, d, c=2.0, dtype="f32", with_dout=True, seed=100 + n)
        gpu = _run_dense(inp, alpha, causal, True)
        for bh in range(B * H):
            ref = oracle_head(inp, bh, alpha, d ** -0.5, causal, True)
            errs = {"tau": float(np.max(np.abs(gpu["tau"][bh] - ref["tau"])
                                        / np.maximum(1, np.abs(ref["tau"]))))}
            for key in ("o", "o2", "dq", "dk", "dv"):
                errs[key] = maxabs(gpu[key].reshape(B * H, n, d)[bh], ref[key])
            log("dense f32 n%d causal%d d%d alpha %g bh%d: %s" % (n, causal, d, alpha, bh, errs))
            assert errs["tau"] <= TAU_REL
            for key in ("o", "o2", "dq", "dk", "dv"):
                assert errs[key] <= F32_TOL, (key, alpha, errs)
