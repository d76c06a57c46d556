"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/entmax_attn.h declares, sizes are right, and invalid
arguments are rejected before anything is launched."""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "entmax_attn.h")

ea = pytest.importorskip("paper_2502_12082_amd", reason="HIP library not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(entmax_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert set(names) == set(ea.SYMBOLS)
    lib = ctypes.CDLL(ea.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    for s in range(5):
        assert ea._lib.entmax_attn_status_string(s)
    assert ea._lib.entmax_attn_status_string(99) == b"unknown status"


def shape(B=2, H=3, n=1000, d=64, dt=0):
    return ea.Shape(B, H, n, d, dt)


def test_default_params():
    p = ea.default_params()
    assert p.alpha == 1.5 and p.causal == 0 and p.need_bwd == 1
    assert p.max_iter > 0 and p.tol > 0


def test_sizes():
    s, p = shape(), ea.default_params()
    z = ea.entmax_attn_sizes(s, p)
    BH, n, d, T = 6, 1000, 64, 16
    assert z.tau == BH * n * 4
    assert z.o2 == BH * n * d * 4
    assert z.block_mask == BH * T * T
    assert z.q_count == z.k_count == BH * T * 4
    assert z.q_index == z.k_index == BH * T * T * 4
    assert z.stats == 2 * BH * T * 4
    # solver cache: one slot per 256-row tile, each 2 lists x 256 threads x
    # 96 quads (16 bytes of scores + 2 bytes of key) and 96 singles (4 bytes
    # of score + 2 bytes of key block), at most 512 slots
    slot = 2 * 256 * 96 * (18 + 6)
    assert z.ws_fwd == BH * ((n + 255) // 256) * slot and z.ws_bwd == BH * n * 4
    big = ea.entmax_attn_sizes(ea.Shape(1, 8, 65536, 64, 0), p)
    assert big.ws_fwd == 512 * slot  # 2048 tiles share 512 slots


@pytest.mark.parametrize("field,value,code", [
    ("batch", 0, ea.EA_ERR_INVALID_ARG),
    ("seqlen", -1, ea.EA_ERR_INVALID_ARG),
    ("head_dim", 96, ea.EA_ERR_UNSUPPORTED),
    ("head_dim", 256, ea.EA_ERR_UNSUPPORTED),
    ("dtype", 7, ea.EA_ERR_UNSUPPORTED),
    ("seqlen", 131073, ea.EA_ERR_UNSUPPORTED),
])
def test_shape_validation(field, value, code):
    s = shape()
    setattr(s, field, value)
    with pytest.raises(ea.EntmaxAttnError) as e:
        ea.entmax_attn_sizes(s, ea.default_params())
    assert e.value.status == code


@pytest.mark.parametrize("field,value", [
    ("alpha", 1.0), ("alpha", 0.5), ("alpha", math.nan), ("alpha", math.inf),
    ("scale", 0.0), ("scale", -0.1), ("scale", math.nan),
    ("causal", 2), ("need_bwd", -1), ("max_iter", -1), ("max_iter", 65),
    ("tol", -1e-3), ("tol", math.nan),
])
def test_param_validation(field, value):
    p = ea.default_params()
    setattr(p, field, value)
    with pytest.raises(ea.EntmaxAttnError) as e:
        ea.entmax_attn_sizes(shape(), p)
    assert e.value.status == ea.EA_ERR_INVALID_ARG


def _fake(addr=0x10000):
    return addr  # never dereferenced: every case below fails validation first


def test_fwd_rejects_bad_pointers_before_launch():
    s, p = shape(), ea.default_params()
    good = ea.ResidualPtrs(*[_fake() for _ in range(7)], None)
    # null q
    assert ea.entmax_attn_fwd(s, p, None, _fake(), _fake(), _fake(), good, None, 0,
                              None) == ea.EA_ERR_INVALID_ARG
    # misaligned v
    assert ea.entmax_attn_fwd(s, p, _fake(), _fake(), _fake() + 2, _fake(), good, None, 0,
                              None) == ea.EA_ERR_INVALID_ARG
    # missing o2 while need_bwd
    r = ea.ResidualPtrs(*[_fake() for _ in range(7)], None)
    r.o2 = None
    assert ea.entmax_attn_fwd(s, p, _fake(), _fake(), _fake(), _fake(), r, None, 0,
                              None) == ea.EA_ERR_INVALID_ARG
    # missing table
    r = ea.ResidualPtrs(*[_fake() for _ in range(7)], None)
    r.k_index = None
    assert ea.entmax_attn_fwd(s, p, _fake(), _fake(), _fake(), _fake(), r, None, 0,
                              None) == ea.EA_ERR_INVALID_ARG
    # bad parameter
    p.alpha = 1.0
    assert ea.entmax_attn_fwd(s, p, _fake(), _fake(), _fake(), _fake(), good, None, 0,
                              None) == ea.EA_ERR_INVALID_ARG


def test_bwd_rejects_small_workspace_and_bad_pointers():
    s, p = shape(), ea.default_params()
    z = ea.entmax_attn_sizes(s, p)
    r = ea.ResidualPtrs(*[_fake() for _ in range(7)], None)
    args = [_fake()] * 4
    assert ea.entmax_attn_bwd(s, p, *args, r, _fake(), _fake(), _fake(), _fake(),
                              z.ws_bwd - 4, None) == ea.EA_ERR_WORKSPACE
    assert ea.entmax_attn_bwd(s, p, *args, r, _fake(), _fake(), _fake(), None,
                              z.ws_bwd, None) == ea.EA_ERR_INVALID_ARG
    assert ea.entmax_attn_bwd(s, p, *args, r, None, _fake(), _fake(), _fake(),
                              z.ws_bwd, None) == ea.EA_ERR_INVALID_ARG
    r.o2 = None
    assert ea.entmax_attn_bwd(s, p, *args, r, _fake(), _fake(), _fake(), _fake(),
                              z.ws_bwd, None) == ea.EA_ERR_INVALID_ARG


def test_last_hip_error_empty_without_failure():
    # only validation failures so far in this process: no HIP error recorded
    assert ea._lib.entmax_attn_last_hip_error() == b""


def test_single_hip_runtime_after_import():
    """Importing the package in a fresh process maps exactly one HIP runtime
    (torch's); a second copy makes every launch fail with no device."""
    import subprocess
    import sys
    code = ("import paper_2502_12082_amd, torch\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "print(len({l.split()[-1] for l in maps if 'libamdhip64' in l}))\n")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True,
                         text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1"


def test_rows_validation():
    p = ea.default_params()
    f = ea.entmax_rows_fwd
    assert f(4, 100, ea.EA_F32, p, None, _fake(), _fake(), None) == ea.EA_ERR_INVALID_ARG
    assert f(0, 100, ea.EA_F32, p, _fake(), _fake(), _fake(), None) == ea.EA_ERR_INVALID_ARG
    assert f(4, 0, ea.EA_F32, p, _fake(), _fake(), _fake(), None) == ea.EA_ERR_INVALID_ARG
    assert f(4, 32769, ea.EA_F32, p, _fake(), _fake(), _fake(), None) == ea.EA_ERR_UNSUPPORTED
    assert f(4, 100, 5, p, _fake(), _fake(), _fake(), None) == ea.EA_ERR_UNSUPPORTED
    assert f(4, 100, ea.EA_F32, p, _fake(), _fake() + 4, _fake(), None) == ea.EA_ERR_INVALID_ARG
    p.alpha = 0.9
    assert f(4, 100, ea.EA_F32, p, _fake(), _fake(), _fake(), None) == ea.EA_ERR_INVALID_ARG
    p = ea.default_params()
    b = ea.entmax_rows_bwd
    assert b(4, 100, ea.EA_BF16, p, _fake(), _fake(), None, _fake(), None) == ea.EA_ERR_INVALID_ARG
    assert b(4, 100, ea.EA_BF16, p, _fake(), _fake(), _fake(), None, None) == ea.EA_ERR_INVALID_ARG


def test_dense_mode_validation():
    s, p = shape(), ea.default_params()
    f = ea._lib.entmax_attn_fwd_dense
    # null tau
    assert f(s, p, _fake(), _fake(), _fake(), _fake(), None, None, _fake(), None, 0, None) == \
        ea.EA_ERR_INVALID_ARG
    # o2 required while need_bwd
    assert f(s, p, _fake(), _fake(), _fake(), _fake(), _fake(), None, None, None, 0, None) == \
        ea.EA_ERR_INVALID_ARG
    # misaligned workspace
    assert f(s, p, _fake(), _fake(), _fake(), _fake(), _fake(), None, _fake(), _fake() + 8, 64,
             None) == ea.EA_ERR_INVALID_ARG
    # fp32 inputs need tau_lo, forward and backward
    s32 = shape(dt=ea.EA_F32)
    assert f(s32, p, _fake(), _fake(), _fake(), _fake(), _fake(), None, _fake(), None, 0, None) == \
        ea.EA_ERR_INVALID_ARG
    b = ea._lib.entmax_attn_bwd_dense
    z = ea.entmax_attn_sizes(s, p)
    args = [_fake()] * 4
    assert b(s, p, *args, _fake(), None, _fake(), _fake(), _fake(), _fake(), _fake(), z.ws_bwd - 4,
             None) == ea.EA_ERR_WORKSPACE
    assert b(s, p, *args, None, None, _fake(), _fake(), _fake(), _fake(), _fake(), z.ws_bwd,
             None) == ea.EA_ERR_INVALID_ARG
    z32 = ea.entmax_attn_sizes(s32, p)
    assert b(s32, p, *args, _fake(), None, _fake(), _fake(), _fake(), _fake(), _fake(), z32.ws_bwd,
             None) == ea.EA_ERR_INVALID_ARG


# ------------------------------------------- binding argument checks (CPU)
#
# The C ABI takes no sizes for the residual buffers, so the binding refuses
# any tensor whose shape, dtype, layout or device does not match before a
# call is made.  CPU tensors exercise every check; the last one (the device
# is a GPU) then refuses them as well.

torch = pytest.importorskip("torch")


def _bf(*shape):
    return torch.zeros(*shape, dtype=torch.bfloat16)


def test_binding_refuses_mismatched_inputs():
    q = _bf(1, 2, 64, 64)
    with pytest.raises(ValueError, match="k has shape"):
        ea.forward(q, _bf(1, 2, 65, 64), q)
    with pytest.raises(ValueError, match="v has dtype"):
        ea.forward(q, q, q.float())
    with pytest.raises(ValueError, match="contiguous"):
        ea.forward(q, _bf(1, 2, 64, 128)[..., ::2], q)
    with pytest.raises(ValueError, match="GPU"):
        ea.forward(q, q, q)
    with pytest.raises(ValueError, match="out has shape"):
        ea.forward(q, q, q, out=_bf(1, 2, 64, 65))


def test_binding_refuses_mismatched_residuals():
    q = _bf(1, 2, 64, 64)
    shape, params = ea.make_shape(q), ea.make_params(head_dim=64)
    res = ea.Residuals(shape, params, "cpu")
    q2 = _bf(1, 2, 128, 64)
    with pytest.raises(ValueError, match="different shape"):
        ea.backward(q2, q2, q2, q2, res)
    with pytest.raises(ValueError, match="dout has shape"):
        ea.backward(q, q, q, q2, res)
    with pytest.raises(ValueError, match="dq has dtype"):
        ea.backward(q, q, q, q, res, dq=q)
    with pytest.raises(ValueError, match="workspace holds"):
        ea.backward(q, q, q, q, res, workspace=torch.zeros(3))
    res.tau = torch.zeros(2, 63)
    with pytest.raises(ValueError, match="res.tau has shape"):
        ea.backward(q, q, q, q, res)
    res = ea.Residuals(shape, params, "cpu")
    res.o2 = None
    with pytest.raises(ValueError, match="no o2"):
        ea.backward(q, q, q, q, res)
    res = ea.Residuals(shape, params, "cpu")
    res.k_index = res.k_index.to(torch.int64)
    with pytest.raises(ValueError, match="res.k_index has dtype"):
        ea.forward(q, q, q, res=res)
    res = ea.Residuals(shape, params, "cpu")
    with pytest.raises(ValueError, match="GPU"):
        ea.backward(q, q, q, q, res)


def test_binding_refuses_mismatched_dense_and_rows():
    q = _bf(1, 2, 64, 64)
    with pytest.raises(ValueError, match="tau has shape"):
        ea.backward_dense(q, q, q, q, torch.zeros(2, 65), torch.zeros(1, 2, 64, 64))
    with pytest.raises(ValueError, match="o2 has dtype"):
        ea.backward_dense(q, q, q, q, torch.zeros(2, 64), q)
    q32 = torch.zeros(1, 2, 64, 64)
    with pytest.raises(ValueError, match="tau_lo"):
        ea.backward_dense(q32, q32, q32, q32, torch.zeros(2, 64), q32)
    with pytest.raises(ValueError, match="tau_lo has shape"):
        ea.backward_dense(q32, q32, q32, q32, torch.zeros(2, 64), q32, tau_lo=torch.zeros(2, 63))
    s = torch.zeros(4, 100)
    with pytest.raises(ValueError, match="tau has shape"):
        ea.rows_backward(s, torch.zeros(5), torch.zeros(4, 100))
    with pytest.raises(ValueError, match="dp has dtype"):
        ea.rows_backward(s, torch.zeros(4), torch.zeros(4, 100, dtype=torch.float64))
    with pytest.raises(ValueError, match="GPU"):
        ea.rows_backward(s, torch.zeros(4), torch.zeros(4, 100))
