"""entmax_attn_bwd_noalloc: the backward whose delta lives in the library's
own scratch array instead of a caller workspace (for callers that cannot
allocate device memory).  Through the C ABI it must return exactly what
entmax_attn_bwd returns for the same residuals (the same kernels run on the
same inputs), call after call on one device, as the scratch array keeps the
previous call's contents."""
import ctypes

import numpy as np
import pytest

import synth
from gpu_util import log, to_device

torch = pytest.importorskip("torch")
ea = pytest.importorskip("paper_2502_12082_amd", reason="HIP library not built")


def _noalloc(q, k, v, do, res):
    dq, dk, dv = (torch.empty(q.shape, dtype=torch.float32, device=q.device) for _ in range(3))
    st = ea.entmax_attn_bwd_noalloc(ea.make_shape(q), res.params, q.data_ptr(), k.data_ptr(),
                                    v.data_ptr(), do.data_ptr(), res.ptrs(), dq.data_ptr(),
                                    dk.data_ptr(), dv.data_ptr(),
                                    torch.cuda.current_stream(q.device).cuda_stream)
    assert st == ea.EA_OK, ea.EntmaxAttnError(st, "entmax_attn_bwd_noalloc")
    return dq, dk, dv


@pytest.mark.gpu
def test_noalloc_matches_bwd_on_consecutive_calls():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # the second and third calls are smaller than the first; the last one
    # fills the whole scratch array (batch * heads * seqlen = the maximum)
    cases = [(2, 3, 700, 64, "bf16", True, 1.5), (1, 2, 300, 128, "bf16", False, 2.0),
             (1, 1, 130, 64, "f32", True, 1.25),
             (1, 16, ea.NOALLOC_MAX_ROWS // 16, 64, "bf16", True, 1.5)]
    for B, H, n, d, dt, causal, alpha in cases:
        log("noalloc B%d H%d n%d d%d %s causal=%d alpha=%g" % (B, H, n, d, dt, causal, alpha))
        inp = synth.attention_inputs(B, H, n, d, c=4.0, dtype=dt, with_dout=True, seed=n)
        q, k, v, do = (to_device(inp[x]) for x in ("q", "k", "v", "dout"))
        o, res = ea.forward(q, k, v, alpha=alpha, scale=d ** -0.5, causal=causal)
        ref = ea.backward(q, k, v, do, res)
        got = _noalloc(q, k, v, do, res)
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv"), ref, got):
            assert torch.equal(a, b), (name, (a - b).abs().max().item())


def test_noalloc_rejects_more_rows_than_the_scratch_holds():
    """Checked on the host before anything is launched (no GPU needed)."""
    shape = ea.Shape(3, 5, 69906, 64, ea.EA_BF16)  # 3 * 5 * 69906 > EA_NOALLOC_MAX_ROWS
    assert 3 * 5 * 69906 > ea.NOALLOC_MAX_ROWS
    params = ea.make_params(head_dim=64)
    fake = 1 << 20  # aligned stand-in pointers: never dereferenced
    res = ea.ResidualPtrs(*([fake] * 8))
    st = ea.entmax_attn_bwd_noalloc(shape, params, fake, fake, fake, fake, res, fake, fake, fake,
                                    None)
    assert st == ea.EA_ERR_UNSUPPORTED
    # bad arguments within the limit are refused as by entmax_attn_bwd
    shape = ea.Shape(1, 1, 100, 64, ea.EA_BF16)
    st = ea.entmax_attn_bwd_noalloc(shape, params, None, fake, fake, fake, res, fake, fake, fake,
                                    None)
    assert st == ea.EA_ERR_INVALID_ARG
