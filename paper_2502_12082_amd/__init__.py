"""alpha-entmax flash attention for MI355X (gfx950): Python binding.

Argument marshalling over the C ABI declared in include/entmax_attn.h; every
step of the computation runs in the HIP kernels of libentmax_attn.so.  torch
is used only to own device memory and to name the stream.  There is no CPU
fallback: importing this module without the built library raises.

    import paper_2502_12082_amd as ea
    o, res = ea.forward(q, k, v, alpha=1.5, scale=d ** -0.5, causal=False)
    dq, dk, dv = ea.backward(q, k, v, do, res)
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libentmax_attn.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("libentmax_attn.so is not built; run `python paper_2502_12082_amd/build.py` "
                      "(or __graft_entry__.build()) first")

# torch ships its own HIP and HSA runtimes.  Importing it first lets the
# library's libamdhip64.so.7 dependency resolve to the copy torch already
# loaded; loaded the other way round the process holds two runtimes, and
# launches through the second one find no device.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

EA_OK, EA_ERR_INVALID_ARG, EA_ERR_UNSUPPORTED, EA_ERR_WORKSPACE, EA_ERR_HIP = range(5)
EA_BF16, EA_F32 = 0, 1
SYMBOLS = ("entmax_attn_default_params", "entmax_attn_sizes", "entmax_attn_fwd",
           "entmax_attn_bwd", "entmax_attn_fwd_stage", "entmax_attn_bwd_stage",
           "entmax_attn_status_string", "entmax_attn_last_hip_error", "entmax_rows_fwd",
           "entmax_rows_bwd", "entmax_attn_fwd_dense", "entmax_attn_bwd_dense",
           "entmax_attn_bwd_noalloc")
NOALLOC_MAX_ROWS = 1048576  # EA_NOALLOC_MAX_ROWS of include/entmax_attn.h


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32),
                ("seqlen", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]


class Params(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("scale", ctypes.c_float),
                ("causal", ctypes.c_int32), ("max_iter", ctypes.c_int32),
                ("tol", ctypes.c_float), ("need_bwd", ctypes.c_int32)]


class ResidualPtrs(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f in
                ("tau", "o2", "block_mask", "q_count", "q_index", "k_count", "k_index", "stats",
                 "tau_lo")]


class Sizes(ctypes.Structure):
    _fields_ = [(f, ctypes.c_size_t) for f in
                ("tau", "o2", "block_mask", "q_count", "q_index", "k_count", "k_index", "stats",
                 "ws_fwd", "ws_bwd", "tau_lo")]


_P = ctypes.POINTER
_v = ctypes.c_void_p
_lib.entmax_attn_default_params.argtypes = [_P(Params)]
_lib.entmax_attn_default_params.restype = None
_lib.entmax_attn_sizes.argtypes = [_P(Shape), _P(Params), _P(Sizes)]
_lib.entmax_attn_sizes.restype = ctypes.c_int
_lib.entmax_attn_fwd.argtypes = [_P(Shape), _P(Params), _v, _v, _v, _v, _P(ResidualPtrs), _v,
                                 ctypes.c_size_t, _v]
_lib.entmax_attn_fwd.restype = ctypes.c_int
_lib.entmax_attn_bwd.argtypes = [_P(Shape), _P(Params), _v, _v, _v, _v, _P(ResidualPtrs), _v, _v,
                                 _v, _v, ctypes.c_size_t, _v]
_lib.entmax_attn_bwd.restype = ctypes.c_int
_lib.entmax_attn_fwd_stage.argtypes = [ctypes.c_int, _P(Shape), _P(Params), _v, _v, _v, _v,
                                       _P(ResidualPtrs), _v, ctypes.c_size_t, _v]
_lib.entmax_attn_fwd_stage.restype = ctypes.c_int
_lib.entmax_attn_bwd_stage.argtypes = [ctypes.c_int, _P(Shape), _P(Params), _v, _v, _v, _v,
                                       _P(ResidualPtrs), _v, _v, _v, _v, ctypes.c_size_t, _v]
_lib.entmax_attn_bwd_stage.restype = ctypes.c_int
_lib.entmax_attn_status_string.argtypes = [ctypes.c_int]
_lib.entmax_attn_status_string.restype = ctypes.c_char_p
_lib.entmax_attn_fwd_dense.argtypes = [_P(Shape), _P(Params), _v, _v, _v, _v, _v, _v, _v, _v,
                                       ctypes.c_size_t, _v]
_lib.entmax_attn_fwd_dense.restype = ctypes.c_int
_lib.entmax_attn_bwd_dense.argtypes = [_P(Shape), _P(Params), _v, _v, _v, _v, _v, _v, _v, _v, _v,
                                       _v, _v, ctypes.c_size_t, _v]
_lib.entmax_attn_bwd_dense.restype = ctypes.c_int
_lib.entmax_rows_fwd.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int, _P(Params), _v, _v,
                                 _v, _v]
_lib.entmax_rows_fwd.restype = ctypes.c_int
_lib.entmax_rows_bwd.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int, _P(Params), _v, _v,
                                 _v, _v, _v]
_lib.entmax_rows_bwd.restype = ctypes.c_int
_lib.entmax_attn_bwd_noalloc.argtypes = [_P(Shape), _P(Params), _v, _v, _v, _v, _P(ResidualPtrs),
                                         _v, _v, _v, _v]
_lib.entmax_attn_bwd_noalloc.restype = ctypes.c_int
_lib.entmax_attn_last_hip_error.argtypes = []
_lib.entmax_attn_last_hip_error.restype = ctypes.c_char_p


class EntmaxAttnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = "%s: %s (status %d)" % (
            where, _lib.entmax_attn_status_string(status).decode(), status)
        if status == EA_ERR_HIP:
            msg += ": " + _lib.entmax_attn_last_hip_error().decode()
        super().__init__(msg)


def _check(status: int, where: str):
    if status != EA_OK:
        raise EntmaxAttnError(status, where)


# --------------------------------------------------------- raw C ABI calls

def default_params() -> Params:
    p = Params()
    _lib.entmax_attn_default_params(ctypes.byref(p))
    return p


def entmax_attn_sizes(shape: Shape, params: Params) -> Sizes:
    z = Sizes()
    _check(_lib.entmax_attn_sizes(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(z)),
           "entmax_attn_sizes")
    return z


def entmax_attn_fwd(shape, params, q, k, v, o, res: ResidualPtrs, workspace, ws_bytes, stream):
    """Raw call; pointers are ints (device addresses), stream an int handle."""
    return _lib.entmax_attn_fwd(ctypes.byref(shape), ctypes.byref(params), q, k, v, o,
                                ctypes.byref(res), workspace, ws_bytes, stream)


def entmax_attn_bwd(shape, params, q, k, v, dout, res: ResidualPtrs, dq, dk, dv, workspace,
                    ws_bytes, stream):
    return _lib.entmax_attn_bwd(ctypes.byref(shape), ctypes.byref(params), q, k, v, dout,
                                ctypes.byref(res), dq, dk, dv, workspace, ws_bytes, stream)


def entmax_attn_bwd_noalloc(shape, params, q, k, v, dout, res: ResidualPtrs, dq, dk, dv, stream):
    return _lib.entmax_attn_bwd_noalloc(ctypes.byref(shape), ctypes.byref(params), q, k, v, dout,
                                        ctypes.byref(res), dq, dk, dv, stream)


def entmax_attn_fwd_stage(stage, shape, params, q, k, v, o, res: ResidualPtrs, workspace,
                          ws_bytes, stream):
    return _lib.entmax_attn_fwd_stage(stage, ctypes.byref(shape), ctypes.byref(params), q, k, v,
                                      o, ctypes.byref(res), workspace, ws_bytes, stream)


def entmax_attn_bwd_stage(stage, shape, params, q, k, v, dout, res: ResidualPtrs, dq, dk, dv,
                          workspace, ws_bytes, stream):
    return _lib.entmax_attn_bwd_stage(stage, ctypes.byref(shape), ctypes.byref(params), q, k, v,
                                      dout, ctypes.byref(res), dq, dk, dv, workspace, ws_bytes,
                                      stream)


# ------------------------------------------------------ torch conveniences

def make_shape(q) -> Shape:
    if q.dim() != 4:
        raise ValueError("expected [batch, heads, seqlen, head_dim]")
    if q.dtype == torch.bfloat16:
        dt = EA_BF16
    elif q.dtype == torch.float32:
        dt = EA_F32
    else:
        raise ValueError("dtype must be bfloat16 or float32")
    B, H, n, d = q.shape
    return Shape(B, H, n, d, dt)


def make_params(alpha=1.5, scale=None, causal=False, need_bwd=True, max_iter=None, tol=None,
                head_dim=64) -> Params:
    p = default_params()
    p.alpha = float(alpha)
    p.scale = float(scale if scale is not None else head_dim ** -0.5)
    p.causal = int(bool(causal))
    p.need_bwd = int(bool(need_bwd))
    if max_iter is not None:
        p.max_iter = int(max_iter)
    if tol is not None:
        p.tol = float(tol)
    return p


class Residuals:
    """Device buffers (torch tensors) that the forward fills and the backward
    reads, sized by entmax_attn_sizes."""

    def __init__(self, shape: Shape, params: Params, device, with_stats: bool = True):
        z = entmax_attn_sizes(shape, params)
        BH, n, d = shape.batch * shape.heads, shape.seqlen, shape.head_dim
        T = (n + 63) // 64
        self.shape, self.params, self.sizes = shape, params, z
        self.tau = torch.empty(z.tau // 4, dtype=torch.float32, device=device).view(BH, n)
        self.o2 = (torch.empty(z.o2 // 4, dtype=torch.float32, device=device).view(BH, n, d)
                   if params.need_bwd else None)
        self.block_mask = torch.empty(z.block_mask, dtype=torch.uint8, device=device).view(BH, T, T)
        self.q_count = torch.empty(BH * T, dtype=torch.int32, device=device).view(BH, T)
        self.q_index = torch.empty(BH * T * T, dtype=torch.int32, device=device).view(BH, T, T)
        self.k_count = torch.empty(BH * T, dtype=torch.int32, device=device).view(BH, T)
        self.k_index = torch.empty(BH * T * T, dtype=torch.int32, device=device).view(BH, T, T)
        # [0]: K passes the solver streamed, [1]: its evaluations, per query block
        self.stats = (torch.empty(z.stats // 4, dtype=torch.int32, device=device).view(2, BH, T)
                      if with_stats else None)
        # fp32 inputs: the low part of tau (tau + tau_lo to ~fp64 precision)
        self.tau_lo = (torch.empty(z.tau_lo // 4, dtype=torch.float32, device=device).view(BH, n)
                       if z.tau_lo else None)

    def ptrs(self) -> ResidualPtrs:
        f = lambda t: None if t is None else t.data_ptr()
        return ResidualPtrs(f(self.tau), f(self.o2), f(self.block_mask), f(self.q_count),
                            f(self.q_index), f(self.k_count), f(self.k_index), f(self.stats),
                            f(self.tau_lo))


def _stream_handle(device):
    return torch.cuda.current_stream(device).cuda_stream


# ------------------------------------------------------ argument checks
#
# The C ABI takes bare device pointers and no sizes for the residual buffers,
# so a tensor of the wrong shape, dtype or device would make the kernels read
# or write past its end.  Every tensor is checked here before any call.

def _need(t, name, shape, dtype, device=None):
    """Raises ValueError unless t is a contiguous tensor of this shape and
    dtype (and, given device, on that device).  Whether that device is a GPU
    is checked once per call by _on_gpu, after every tensor's shape."""
    if not isinstance(t, torch.Tensor):
        raise ValueError("%s must be a torch tensor" % name)
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if t.dtype != dtype:
        raise ValueError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))


def _on_gpu(device):
    if device is None or device.type != "cuda":
        raise ValueError("tensors must be on a GPU device, not %s" % device)


def _torch_dtype(shape: Shape):
    return torch.bfloat16 if shape.dtype == EA_BF16 else torch.float32


def _check_qkv(names_tensors, shape: Shape):
    """q, k, v (and dO) against one shape: [B, H, n, d] in the shape's dtype,
    all on the device of the first."""
    dims = (shape.batch, shape.heads, shape.seqlen, shape.head_dim)
    dev = names_tensors[0][1].device if isinstance(names_tensors[0][1], torch.Tensor) else None
    for name, t in names_tensors:
        _need(t, name, dims, _torch_dtype(shape), dev)
    return dev


def _same_shape(a: Shape, b: Shape) -> bool:
    return all(getattr(a, f) == getattr(b, f) for f, _ in Shape._fields_)


def _check_residuals(res, shape: Shape, device, need_o2: bool):
    if not isinstance(res, Residuals):
        raise ValueError("res must be the Residuals of a forward call")
    if not _same_shape(res.shape, shape):
        raise ValueError("res was sized for a different shape or dtype")
    BH, n, d = shape.batch * shape.heads, shape.seqlen, shape.head_dim
    T = (n + 63) // 64
    _need(res.tau, "res.tau", (BH, n), torch.float32, device)
    if need_o2:
        if res.o2 is None:
            raise ValueError("res has no o2 (forward ran with need_bwd=False)")
        _need(res.o2, "res.o2", (BH, n, d), torch.float32, device)
    _need(res.block_mask, "res.block_mask", (BH, T, T), torch.uint8, device)
    _need(res.q_count, "res.q_count", (BH, T), torch.int32, device)
    _need(res.q_index, "res.q_index", (BH, T, T), torch.int32, device)
    _need(res.k_count, "res.k_count", (BH, T), torch.int32, device)
    _need(res.k_index, "res.k_index", (BH, T, T), torch.int32, device)
    if res.stats is not None:
        _need(res.stats, "res.stats", (2, BH, T), torch.int32, device)
    if shape.dtype == EA_F32:
        _need(res.tau_lo, "res.tau_lo", (BH, n), torch.float32, device)


def _check_bytes(ws, name, need_bytes, device):
    if not isinstance(ws, torch.Tensor) or not ws.is_contiguous():
        raise ValueError("%s must be a contiguous tensor" % name)
    if ws.numel() * ws.element_size() < need_bytes:
        raise ValueError("%s holds %d bytes, needs %d" % (
            name, ws.numel() * ws.element_size(), need_bytes))
    if ws.device != device:
        raise ValueError("%s must be on %s" % (name, device))


def forward_workspace(res: Residuals, device):
    """A device buffer of sizes.ws_fwd bytes for the solver's candidate cache."""
    return torch.empty(max(res.sizes.ws_fwd, 16), dtype=torch.uint8, device=device)


def forward(q, k, v, alpha=1.5, scale=None, causal=False, need_bwd=True, max_iter=None,
            tol=None, out=None, res: Residuals | None = None, workspace=None):
    """O and the residuals for Q, K, V ([B, H, n, d] bf16/fp32 CUDA tensors).

    workspace: a uint8 device tensor for the solver's candidate cache (None
    allocates sizes.ws_fwd bytes; False runs the solver without the cache)."""
    shape = make_shape(q)
    dev = _check_qkv([("q", q), ("k", k), ("v", v)], shape)
    params = make_params(alpha, scale, causal, need_bwd, max_iter, tol, head_dim=q.shape[-1])
    if res is None:
        res = Residuals(shape, params, q.device)
    else:
        _check_residuals(res, shape, dev, bool(need_bwd))
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", q.shape, q.dtype, dev)
    if workspace is not None and workspace is not False:
        _check_bytes(workspace, "workspace", 0, dev)
    _on_gpu(dev)
    rp = res.ptrs()
    if workspace is None:
        workspace = forward_workspace(res, q.device)
    ws_ptr, ws_bytes = (None, 0) if workspace is False else (workspace.data_ptr(),
                                                            workspace.numel() * workspace.element_size())
    _check(entmax_attn_fwd(shape, params, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                           out.data_ptr(), rp, ws_ptr, ws_bytes, _stream_handle(q.device)),
           "entmax_attn_fwd")
    res.params = params
    return out, res


def backward(q, k, v, dout, res: Residuals, dq=None, dk=None, dv=None, workspace=None):
    """(dQ, dK, dV) in fp32 for the loss sum(dO * O) of the forward that filled res."""
    shape = make_shape(q)
    dev = _check_qkv([("q", q), ("k", k), ("v", v), ("dout", dout)], shape)
    _check_residuals(res, shape, dev, True)
    if not res.params.need_bwd:
        raise ValueError("res comes from a forward with need_bwd=False")
    mk = lambda t: t if t is not None else torch.empty(q.shape, dtype=torch.float32, device=q.device)
    dq, dk, dv = mk(dq), mk(dk), mk(dv)
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _need(t, name, q.shape, torch.float32, dev)
    if workspace is None:
        workspace = torch.empty(max(res.sizes.ws_bwd, 16) // 4 + 4, dtype=torch.float32,
                                device=q.device)
    else:
        _check_bytes(workspace, "workspace", res.sizes.ws_bwd, dev)
    _on_gpu(dev)
    rp = res.ptrs()
    _check(entmax_attn_bwd(shape, res.params, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                           dout.data_ptr(), rp, dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                           workspace.data_ptr(), workspace.numel() * 4, _stream_handle(q.device)),
           "entmax_attn_bwd")
    return dq, dk, dv


# ------------------------------------------------------- row-wise entmax

def entmax_rows_fwd(rows, n, dtype, params, s, p, tau, stream):
    return _lib.entmax_rows_fwd(rows, n, dtype, ctypes.byref(params), s, p, tau, stream)


def entmax_rows_bwd(rows, n, dtype, params, s, tau, dp, ds, stream):
    return _lib.entmax_rows_bwd(rows, n, dtype, ctypes.byref(params), s, tau, dp, ds, stream)


def _row_params(alpha, scale, max_iter, tol):
    p = default_params()
    p.alpha, p.scale, p.causal, p.need_bwd = float(alpha), float(scale), 0, 0
    if max_iter is not None:
        p.max_iter = int(max_iter)
    if tol is not None:
        p.tol = float(tol)
    return p


def rows_forward(s, alpha=1.5, scale=1.0, max_iter=None, tol=None):
    """(p, tau): alpha-entmax of each row of s ([..., n] bf16/fp32 device tensor)."""
    if not s.is_cuda or not s.is_contiguous() or s.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("s must be a contiguous bf16 or fp32 device tensor")
    n = s.shape[-1]
    rows = s.numel() // n
    p = torch.empty(s.shape, dtype=torch.float32, device=s.device)
    tau = torch.empty(s.shape[:-1], dtype=torch.float32, device=s.device)
    params = _row_params(alpha, scale, max_iter, tol)
    _check(entmax_rows_fwd(rows, n, EA_BF16 if s.dtype == torch.bfloat16 else EA_F32, params,
                           s.data_ptr(), p.data_ptr(), tau.data_ptr(), _stream_handle(s.device)),
           "entmax_rows_fwd")
    return p, tau


def rows_backward(s, tau, dp, alpha=1.5, scale=1.0):
    """Gradient of sum(dp * p) with respect to s, for (p, tau) = rows_forward(s)."""
    if not isinstance(s, torch.Tensor) or s.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("s must be a bf16 or fp32 tensor")
    _need(s, "s", s.shape, s.dtype)
    n = s.shape[-1]
    rows = s.numel() // n
    _need(dp, "dp", s.shape, torch.float32, s.device)
    _need(tau, "tau", s.shape[:-1], torch.float32, s.device)
    _on_gpu(s.device)
    ds = torch.empty(s.shape, dtype=torch.float32, device=s.device)
    params = _row_params(alpha, scale, None, None)
    _check(entmax_rows_bwd(rows, n, EA_BF16 if s.dtype == torch.bfloat16 else EA_F32, params,
                           s.data_ptr(), tau.data_ptr(), dp.data_ptr(), ds.data_ptr(),
                           _stream_handle(s.device)), "entmax_rows_bwd")
    return ds


# ---------------------------------------------------------- no-mask mode

def forward_dense(q, k, v, alpha=1.5, scale=None, causal=False, need_bwd=True, max_iter=None,
                  tol=None, workspace=None):
    """(O, tau, O2 or None, tau_lo or None) without block mask or tables
    (Algorithm 2 as written); tau_lo, the threshold's low part, exists for fp32
    inputs and goes back into backward_dense."""
    shape = make_shape(q)
    dev = _check_qkv([("q", q), ("k", k), ("v", v)], shape)
    _on_gpu(dev)
    params = make_params(alpha, scale, causal, need_bwd, max_iter, tol, head_dim=q.shape[-1])
    B, H, n, d = q.shape
    o = torch.empty_like(q)
    tau = torch.empty((B * H, n), dtype=torch.float32, device=q.device)
    tau_lo = torch.empty_like(tau) if q.dtype == torch.float32 else None
    o2 = torch.empty(q.shape, dtype=torch.float32, device=q.device) if need_bwd else None
    z = entmax_attn_sizes(shape, params)
    if workspace is None:
        workspace = torch.empty(max(z.ws_fwd, 16), dtype=torch.uint8, device=q.device)
    elif workspace is not False:
        _check_bytes(workspace, "workspace", 0, dev)
    _on_gpu(dev)
    ws_ptr, ws_bytes = (None, 0) if workspace is False else (workspace.data_ptr(),
                                                            workspace.numel() * workspace.element_size())
    _check(_lib.entmax_attn_fwd_dense(ctypes.byref(shape), ctypes.byref(params), q.data_ptr(),
                                      k.data_ptr(), v.data_ptr(), o.data_ptr(), tau.data_ptr(),
                                      tau_lo.data_ptr() if tau_lo is not None else None,
                                      o2.data_ptr() if o2 is not None else None, ws_ptr, ws_bytes,
                                      _stream_handle(q.device)), "entmax_attn_fwd_dense")
    return o, tau, o2, tau_lo


def backward_dense(q, k, v, dout, tau, o2, alpha=1.5, scale=None, causal=False, tau_lo=None):
    """(dQ, dK, dV) in fp32 for the no-mask forward that produced tau, o2 and
    (fp32 inputs) tau_lo."""
    shape = make_shape(q)
    dev = _check_qkv([("q", q), ("k", k), ("v", v), ("dout", dout)], shape)
    B, H, n, d = q.shape
    _need(tau, "tau", (B * H, n), torch.float32, dev)
    _need(o2, "o2", q.shape, torch.float32, dev)
    if q.dtype == torch.float32:
        if tau_lo is None:
            raise ValueError("backward_dense: fp32 inputs need the forward's tau_lo")
        _need(tau_lo, "tau_lo", (B * H, n), torch.float32, dev)
    _on_gpu(dev)
    params = make_params(alpha, scale, causal, True, None, None, head_dim=q.shape[-1])
    z = entmax_attn_sizes(shape, params)
    mk = lambda: torch.empty(q.shape, dtype=torch.float32, device=q.device)
    dq, dk, dv = mk(), mk(), mk()
    ws = torch.empty(max(z.ws_bwd, 16) // 4 + 4, dtype=torch.float32, device=q.device)
    _check(_lib.entmax_attn_bwd_dense(ctypes.byref(shape), ctypes.byref(params), q.data_ptr(),
                                      k.data_ptr(), v.data_ptr(), dout.data_ptr(), tau.data_ptr(),
                                      tau_lo.data_ptr() if q.dtype == torch.float32 else None,
                                      o2.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                      ws.data_ptr(), ws.numel() * 4, _stream_handle(q.device)),
           "entmax_attn_bwd_dense")
    return dq, dk, dv
