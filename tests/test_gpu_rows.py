"""GPU parity of the row-wise alpha-entmax entry points (materialized scores)
against the fp64 oracle: tau and p of every row, and the backward.

Scores are seeded standard normals times sigma (the paper's efficiency
benchmark draws unit-variance Gaussians, n = 8192).  The kernels compute in
fp32 from bf16 or fp32 inputs; p is compared max-abs (p <= 1), tau relative.
For alpha > 2 the forward alone is compared (u = z^(gamma-1) is unbounded
near the support edge, so the backward amplifies score rounding without
bound), with a larger iteration budget since convergence is linear at worst.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import TAU_REL, log, to_device

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

P_TOL = 1e-4       # max-abs on p (fp32 arithmetic, p in [0, 1])
GRAD_REL = 1e-3    # max-abs on ds relative to max(1, max |ds|)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_12082_amd  # noqa: F401


def _case(rows, n, dtype, alpha, sigma, seed, scale=1.0, bwd=True):
    import paper_2502_12082_amd as ea
    s = synth.normal((rows, n), seed, scale=sigma, dtype=dtype)
    g = synth.normal((rows, n), seed + 1, scale=1.0, dtype="f32")
    it = 12 if alpha <= 2 else 40
    sd = to_device(s)
    p, tau = ea.rows_forward(sd, alpha=alpha, scale=scale, max_iter=it)
    ds = None
    if bwd:
        ds = ea.rows_backward(sd, tau, to_device(g), alpha=alpha, scale=scale)
    torch.cuda.synchronize()
    p, tau = p.cpu().numpy().astype(np.float64), tau.cpu().numpy().astype(np.float64)
    sf, gf = s.f64(), g.f64()
    worst = {"tau": 0.0, "p": 0.0, "ds": 0.0}
    for r in range(rows):
        x = (alpha - 1) * scale * sf[r]
        pr, tr = oracle.entmax(x, alpha)
        worst["tau"] = max(worst["tau"], abs(tau[r] - tr) / max(1.0, abs(tr)))
        worst["p"] = max(worst["p"], np.max(np.abs(p[r] - pr)))
        if bwd:
            ref = scale * oracle.entmax_bwd(x, alpha, tr, gf[r])
            d = ds[r].cpu().numpy().astype(np.float64)
            worst["ds"] = max(worst["ds"], np.max(np.abs(d - ref)) / max(1.0, np.max(np.abs(ref))))
    log("rows %d n %d %s alpha %g sigma %g: %s" % (rows, n, dtype, alpha, sigma, worst))
    assert worst["tau"] <= TAU_REL
    assert worst["p"] <= P_TOL
    if bwd:
        assert worst["ds"] <= GRAD_REL


@pytest.mark.parametrize("n", [1, 2, 255, 256, 257, 1000, 1024, 2048, 2049, 4096, 8192, 16384, 32768])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rows_shapes(n, dtype):
    _case(5, n, dtype, 1.5, 1.0, synth.SEED_BASE + 10)


@pytest.mark.parametrize("alpha", [1.25, 1.6, 2.0, 3.0])
@pytest.mark.parametrize("sigma", [0.1, 1.0, 6.0])
def test_rows_alpha_sigma(alpha, sigma):
    _case(16, 8192, "f32", alpha, sigma, synth.SEED_BASE + 20, scale=0.5, bwd=alpha <= 2)


def test_rows_special_cases():
    """Constant rows (p uniform) and one dominant score (p one-hot)."""
    import paper_2502_12082_amd as ea
    n = 3000
    s = torch.zeros((2, n), dtype=torch.float32, device="cuda")
    s[1, 17] = 10.0
    p, tau = ea.rows_forward(s, alpha=1.5)
    torch.cuda.synchronize()
    assert (p[0] - 1.0 / n).abs().max().item() <= 1e-6
    assert abs(p[1, 17].item() - 1.0) <= 1e-5 and p[1].sum().item() == pytest.approx(1.0, abs=1e-5)
