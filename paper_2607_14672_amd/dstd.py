"""Thin Python binding of the DSTD-LIF C ABI (``include/dstd_lif.h``).

The functions named like the C entry points take plain integers (device
pointers, sizes, stream handles) and return the status code. The tensor
helpers below them only marshal arguments: they allocate outputs and
workspace with PyTorch on the tensors' device, pass ``data_ptr()`` and the
current stream, and raise on a non-OK status. Every step of the layer runs in
the HIP library; if ``libdstd_lif.so`` is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes as C
import math
import os
from typing import Optional, Tuple

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdstd_lif.so")

DSTD_OK = 0
DSTD_ERR_NULL = -1
DSTD_ERR_SHAPE = -2
DSTD_ERR_PARAM = -3
DSTD_ERR_UNSUPPORTED = -4
DSTD_ERR_WORKSPACE = -5
DSTD_ERR_HIP = -6
DSTD_F32 = 0
DSTD_BF16 = 1
DSTD_MAX_M = 256
DSTD_NOALLOC_SCRATCH_BYTES = 32 << 20
DSTD_FLAG_CONTRACT_SPARSE = 0x2
DSTD_FLAG_CONTRACT_MFMA = 0x4
DSTD_FLAG_CONV_KEEP = 0x8
DSTD_FLAG_CONV_REUSE = 0x10


class dstd_lif_params(C.Structure):
    _fields_ = [("tau_m", C.c_float), ("tau_s", C.c_float), ("threshold", C.c_float),
                ("M", C.c_int32), ("t0", C.c_float), ("dt", C.c_float), ("t_max", C.c_float),
                ("flags", C.c_int32)]


class dstd_conv_shape(C.Structure):
    _fields_ = [(k, C.c_int32) for k in ("C_in", "H", "W", "C_out", "KH", "KW", "stride", "pad",
                                         "pool_in")]


class dstd_synfire_params(C.Structure):
    _fields_ = [(k, C.c_float) for k in ("gamma_head", "gamma_tail", "t_head", "t_tail", "gamma_q",
                                         "scale")]


class DSTDError(RuntimeError):
    def __init__(self, fn: str, status: int):
        lib = _load()
        self.status = status
        msg = lib.dstd_status_string(status).decode()
        detail = lib.dstd_last_error().decode()
        super().__init__(f"{fn}: {msg} ({status}): {detail}")


_lib = None
_P = C.c_void_p
_L = C.c_int64
_S = C.c_size_t
_I = C.c_int
_F = C.c_float

# name -> (restype, argtypes)
_SIGS = {
    "dstd_lif_forward_workspace_size": (_S, [_P, _L, _L, _L]),
    "dstd_lif_backward_workspace_size": (_S, [_P, _L, _L, _L]),
    "dstd_lif_forward": (_I, [_P, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P, _S, _P]),
    "dstd_lif_forward_noalloc": (_I, [_P, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P]),
    "dstd_lif_backward": (_I, [_P, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "dstd_lif_conv_forward_workspace_size": (_S, [_P, _P, _L]),
    "dstd_lif_conv_backward_workspace_size": (_S, [_P, _P, _L]),
    "dstd_lif_conv_forward": (_I, [_P, _P, _L, _P, _P, _I, _P, _P, _P, _P, _S, _P]),
    "dstd_lif_conv_backward": (_I, [_P, _P, _L, _P, _P, _I, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "dstd_lif_backward_synfire": (_I, [_P, _P, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P, _P, _P, _P,
                                       _S, _P]),
    "dstd_lif_conv_backward_synfire": (_I, [_P, _P, _P, _L, _P, _P, _I, _P, _P, _P, _P, _P, _P, _P,
                                            _S, _P]),
    "dstd_synfire_penalty_workspace_size": (_S, [_L, _L, _L]),
    "dstd_synfire_penalty": (_I, [_P, _L, _L, _L, _L, _P, _P, _I, _P, _P, _S, _P]),
    "dstd_exact_forward_workspace_size": (_S, [_P, _L, _L, _L]),
    "dstd_exact_backward_workspace_size": (_S, [_P, _L, _L, _L]),
    "dstd_exact_forward": (_I, [_P, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P, _S, _P]),
    "dstd_exact_backward": (_I, [_P, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "dstd_lif_multispike_forward_workspace_size": (_S, [_P, _L, _L, _L, _L, _L]),
    "dstd_lif_multispike_backward_workspace_size": (_S, [_P, _L, _L, _L, _L, _L]),
    "dstd_lif_multispike_forward": (_I, [_P, _L, _L, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P, _P,
                                         _S, _P]),
    "dstd_lif_multispike_backward": (_I, [_P, _L, _L, _L, _L, _L, _P, _P, _I, _P, _P, _P, _P, _P,
                                          _P, _P, _P, _S, _P]),
    "dstd_skip_delay_concat": (_I, [_L, _L, _L, _L, _P, _F, _P, _P, _P]),
    "dstd_skip_delay_concat_backward": (_I, [_L, _L, _L, _L, _P, _P, C.c_int32, _P, _P]),
    "dstd_softmax_ce_grad": (_I, [_L, _L, _P, _P, _F, _F, _P, _P, _P]),
    "dstd_mse_grad": (_I, [_L, _L, _P, _P, _P, _P, _P]),
    "dstd_profile_enable": (C.c_int32, [C.c_int32]),
    "dstd_profile_collect": (_I, []),
    "dstd_profile_count": (C.c_int32, []),
    "dstd_profile_entry": (_I, [C.c_int32, C.POINTER(C.c_char_p), C.POINTER(C.c_int64),
                                C.POINTER(C.c_double)]),
    "dstd_profile_reset": (None, []),
    "dstd_status_string": (C.c_char_p, [_I]),
    "dstd_last_error": (C.c_char_p, []),
    "dstd_version": (C.c_int32, []),
}


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2607_14672_amd.build`")
        lib = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def exported_symbols():
    return list(_SIGS)


def _ref(s):
    return None if s is None else C.addressof(s)


# ------------------------------------------------------------ raw C ABI --
def dstd_lif_forward_workspace_size(p, B, N_in, N_out):
    return _load().dstd_lif_forward_workspace_size(_ref(p), B, N_in, N_out)


def dstd_lif_backward_workspace_size(p, B, N_in, N_out):
    return _load().dstd_lif_backward_workspace_size(_ref(p), B, N_in, N_out)


def dstd_lif_forward(p, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx, ws, ws_bytes, stream):
    return _load().dstd_lif_forward(_ref(p), B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx,
                                    ws, ws_bytes, stream)


def dstd_lif_forward_noalloc(p, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx, stream):
    return _load().dstd_lif_forward_noalloc(_ref(p), B, N_in, N_out, t_in, W, w_dtype, t_out,
                                            slope, q_idx, stream)


def dstd_lif_backward(p, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx, grad_t_out,
                      grad_W, grad_t_in, ws, ws_bytes, stream):
    return _load().dstd_lif_backward(_ref(p), B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx,
                                     grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream)


def dstd_exact_forward_workspace_size(p, B, N_in, N_out):
    return _load().dstd_exact_forward_workspace_size(_ref(p), B, N_in, N_out)


def dstd_exact_backward_workspace_size(p, B, N_in, N_out):
    return _load().dstd_exact_backward_workspace_size(_ref(p), B, N_in, N_out)


def dstd_exact_forward(p, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, k_idx, ws, ws_bytes,
                       stream):
    return _load().dstd_exact_forward(_ref(p), B, N_in, N_out, t_in, W, w_dtype, t_out, slope,
                                      k_idx, ws, ws_bytes, stream)


def dstd_exact_backward(p, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, k_idx, grad_t_out,
                        grad_W, grad_t_in, ws, ws_bytes, stream):
    return _load().dstd_exact_backward(_ref(p), B, N_in, N_out, t_in, W, w_dtype, t_out, slope,
                                       k_idx, grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream)


def dstd_lif_multispike_forward_workspace_size(p, B, N_in, F_in, N_out, F_out):
    return _load().dstd_lif_multispike_forward_workspace_size(_ref(p), B, N_in, F_in, N_out, F_out)


def dstd_lif_multispike_backward_workspace_size(p, B, N_in, F_in, N_out, F_out):
    return _load().dstd_lif_multispike_backward_workspace_size(_ref(p), B, N_in, F_in, N_out, F_out)


def dstd_lif_multispike_forward(p, B, N_in, F_in, N_out, F_out, t_in, W, w_dtype, t_out, slope,
                                q_idx, cur, ws, ws_bytes, stream):
    return _load().dstd_lif_multispike_forward(_ref(p), B, N_in, F_in, N_out, F_out, t_in, W,
                                               w_dtype, t_out, slope, q_idx, cur, ws, ws_bytes,
                                               stream)


def dstd_lif_multispike_backward(p, B, N_in, F_in, N_out, F_out, t_in, W, w_dtype, t_out, slope,
                                 q_idx, cur, grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream):
    return _load().dstd_lif_multispike_backward(_ref(p), B, N_in, F_in, N_out, F_out, t_in, W,
                                                w_dtype, t_out, slope, q_idx, cur, grad_t_out,
                                                grad_W, grad_t_in, ws, ws_bytes, stream)


def dstd_skip_delay_concat(B, C1, C2, HW, t1, delay, t2, out, stream):
    return _load().dstd_skip_delay_concat(B, C1, C2, HW, t1, delay, t2, out, stream)


def dstd_skip_delay_concat_backward(B, C1, C2, HW, g, g1, accumulate, g2, stream):
    return _load().dstd_skip_delay_concat_backward(B, C1, C2, HW, g, g1, accumulate, g2, stream)


def dstd_lif_conv_forward_workspace_size(p, cs, B):
    return _load().dstd_lif_conv_forward_workspace_size(_ref(p), _ref(cs), B)


def dstd_lif_conv_backward_workspace_size(p, cs, B):
    return _load().dstd_lif_conv_backward_workspace_size(_ref(p), _ref(cs), B)


def dstd_lif_conv_forward(p, cs, B, t_in, W, w_dtype, t_out, slope, q_idx, ws, ws_bytes, stream):
    return _load().dstd_lif_conv_forward(_ref(p), _ref(cs), B, t_in, W, w_dtype, t_out, slope, q_idx,
                                         ws, ws_bytes, stream)


def dstd_lif_conv_backward(p, cs, B, t_in, W, w_dtype, t_out, slope, q_idx, grad_t_out, grad_W,
                           grad_t_in, ws, ws_bytes, stream):
    return _load().dstd_lif_conv_backward(_ref(p), _ref(cs), B, t_in, W, w_dtype, t_out, slope,
                                          q_idx, grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream)


def dstd_lif_backward_synfire(p, sp, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx,
                              grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream):
    return _load().dstd_lif_backward_synfire(_ref(p), _ref(sp), B, N_in, N_out, t_in, W, w_dtype,
                                             t_out, slope, q_idx, grad_t_out, grad_W, grad_t_in,
                                             ws, ws_bytes, stream)


def dstd_lif_conv_backward_synfire(p, sp, cs, B, t_in, W, w_dtype, t_out, slope, q_idx,
                                   grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream):
    return _load().dstd_lif_conv_backward_synfire(_ref(p), _ref(sp), _ref(cs), B, t_in, W, w_dtype,
                                                  t_out, slope, q_idx, grad_t_out, grad_W,
                                                  grad_t_in, ws, ws_bytes, stream)


def dstd_synfire_penalty_workspace_size(B, rows, spatial):
    return _load().dstd_synfire_penalty_workspace_size(B, rows, spatial)


def dstd_synfire_penalty(sp, B, rows, spatial, row_len, t_out, W, w_dtype, value, ws, ws_bytes,
                         stream):
    return _load().dstd_synfire_penalty(_ref(sp), B, rows, spatial, row_len, t_out, W, w_dtype,
                                        value, ws, ws_bytes, stream)


def dstd_softmax_ce_grad(B, N, t_out, labels, tau_soft, t_cap, grad_t, loss, stream):
    return _load().dstd_softmax_ce_grad(B, N, t_out, labels, tau_soft, t_cap, grad_t, loss, stream)


def dstd_mse_grad(B, N, t_out, target, grad_t, loss, stream):
    return _load().dstd_mse_grad(B, N, t_out, target, grad_t, loss, stream)


def dstd_status_string(s):
    return _load().dstd_status_string(s).decode()


def dstd_last_error():
    return _load().dstd_last_error().decode()


def dstd_version():
    return _load().dstd_version()


def dstd_profile_enable(on):
    return _load().dstd_profile_enable(1 if on else 0)


def dstd_profile_collect():
    return _load().dstd_profile_collect()


def dstd_profile_count():
    return _load().dstd_profile_count()


def dstd_profile_entry(idx):
    name = C.c_char_p()
    n = C.c_int64()
    ms = C.c_double()
    st = _load().dstd_profile_entry(idx, C.byref(name), C.byref(n), C.byref(ms))
    _check("dstd_profile_entry", st)
    return name.value.decode(), n.value, ms.value


def dstd_profile_reset():
    _load().dstd_profile_reset()


def profile_table():
    """{kernel name: (launches, total ms)} of the library's own timer."""
    dstd_profile_collect()
    return {e[0]: (e[1], e[2]) for e in (dstd_profile_entry(i) for i in range(dstd_profile_count()))}


# -------------------------------------------------------- tensor helpers --
def make_params(tau_m, tau_s, threshold, M, t0, dt, t_max=math.inf, flags=0) -> dstd_lif_params:
    return dstd_lif_params(float(tau_m), float(tau_s), float(threshold), int(M), float(t0),
                           float(dt), float(t_max), int(flags))


def make_synfire(gamma_head, gamma_tail, t_head, t_tail, gamma_q, scale) -> dstd_synfire_params:
    """One layer's synfire-term parameters (window ends t_head, t_tail already
    shifted for the layer; scale = 1/B, conv 1/(B*H_out*W_out))."""
    return dstd_synfire_params(gamma_head, gamma_tail, t_head, t_tail, gamma_q, scale)


def make_conv_shape(C_in, H, W, C_out, KH=3, KW=3, stride=1, pad=1, pool_in=1) -> dstd_conv_shape:
    return dstd_conv_shape(C_in, H, W, C_out, KH, KW, stride, pad, pool_in)


def conv_out_hw(cs: dstd_conv_shape) -> Tuple[int, int]:
    H, W = cs.H, cs.W
    if cs.pool_in == 2:
        H, W = H // 2, W // 2
    elif cs.pool_in == 0:
        H, W = 1, 1
    return (H + 2 * cs.pad - cs.KH) // cs.stride + 1, (W + 2 * cs.pad - cs.KW) // cs.stride + 1


def _torch():
    import torch
    return torch


def _stream(dev):
    return _torch().cuda.current_stream(dev).cuda_stream


def _wdtype(W):
    torch = _torch()
    if W.dtype == torch.float32:
        return DSTD_F32
    if W.dtype == torch.bfloat16:
        return DSTD_BF16
    raise TypeError(f"W must be float32 or bfloat16, got {W.dtype}")


def _check(name, st):
    if st != DSTD_OK:
        raise DSTDError(name, st)


def _cont(x, dtype=None):
    if dtype is not None:
        assert x.dtype == dtype, f"expected {dtype}, got {x.dtype}"
    assert x.is_cuda, "tensors must live on the GPU"
    return x.contiguous()


def _ptr(x):
    return None if x is None else x.data_ptr()


def workspace(nbytes: int, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def forward(p: dstd_lif_params, t_in, W, ws=None):
    """Dense layer forward. t_in [B, N_in] f32, W [N_out, N_in] f32|bf16 (CUDA tensors)."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    assert W.shape[1] == N_in
    dev = t_in.device
    t_out = torch.empty((B, N_out), dtype=torch.float32, device=dev)
    slope = torch.empty_like(t_out)
    q = torch.empty((B, N_out), dtype=torch.int32, device=dev)
    need = dstd_lif_forward_workspace_size(p, B, N_in, N_out)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    _check("dstd_lif_forward",
           dstd_lif_forward(p, B, N_in, N_out, _ptr(t_in), _ptr(W), _wdtype(W), _ptr(t_out),
                            _ptr(slope), _ptr(q), _ptr(ws), ws.numel(), _stream(dev)))
    return t_out, slope, q


def forward_noalloc(p: dstd_lif_params, t_in, W, outputs=None):
    """Dense layer forward through the allocation-free entry point (the
    library's static scratch). `outputs` = (t_out, slope, q) preallocated
    tensors, or None to allocate them here."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    assert W.shape[1] == N_in
    dev = t_in.device
    if outputs is None:
        t_out = torch.empty((B, N_out), dtype=torch.float32, device=dev)
        outputs = (t_out, torch.empty_like(t_out), torch.empty((B, N_out), dtype=torch.int32, device=dev))
    t_out, slope, q = outputs
    _check("dstd_lif_forward_noalloc",
           dstd_lif_forward_noalloc(p, B, N_in, N_out, _ptr(t_in), _ptr(W), _wdtype(W), _ptr(t_out),
                                    _ptr(slope), _ptr(q), _stream(dev)))
    return t_out, slope, q


def backward(p: dstd_lif_params, t_in, W, t_out, slope, q, grad_t_out, need_W=True,
             need_t_in=True, ws=None, synfire: Optional[dstd_synfire_params] = None):
    """Dense layer backward; returns (grad_W or None, grad_t_in or None). With
    `synfire`, the layer's temporal-penalty and dead-neuron gradients are
    included."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    dev = t_in.device
    gW = torch.empty((N_out, N_in), dtype=torch.float32, device=dev) if need_W else None
    gt = torch.empty((B, N_in), dtype=torch.float32, device=dev) if need_t_in else None
    need = dstd_lif_backward_workspace_size(p, B, N_in, N_out)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    args = (B, N_in, N_out, _ptr(t_in), _ptr(W), _wdtype(W), _ptr(_cont(t_out, torch.float32)),
            _ptr(_cont(slope, torch.float32)), _ptr(_cont(q, torch.int32)),
            _ptr(_cont(grad_t_out, torch.float32)), _ptr(gW), _ptr(gt), _ptr(ws), ws.numel(),
            _stream(dev))
    if synfire is None:
        _check("dstd_lif_backward", dstd_lif_backward(p, *args))
    else:
        _check("dstd_lif_backward_synfire", dstd_lif_backward_synfire(p, synfire, *args))
    return gW, gt


def multispike_forward(p: dstd_lif_params, t_in, W, F_out: int, ws=None):
    """Multi-spike dense forward. t_in [B, N_in, F_in]; returns (t_out, slope, q, cur),
    each [B, N_out, F_out]."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B, N_in, F_in = t_in.shape
    N_out = W.shape[0]
    dev = t_in.device
    shp = (B, N_out, F_out)
    t_out = torch.empty(shp, dtype=torch.float32, device=dev)
    slope = torch.empty_like(t_out)
    cur = torch.empty_like(t_out)
    q = torch.empty(shp, dtype=torch.int32, device=dev)
    need = dstd_lif_multispike_forward_workspace_size(p, B, N_in, F_in, N_out, F_out)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    _check("dstd_lif_multispike_forward",
           dstd_lif_multispike_forward(p, B, N_in, F_in, N_out, F_out, _ptr(t_in), _ptr(W),
                                       _wdtype(W), _ptr(t_out), _ptr(slope), _ptr(q), _ptr(cur),
                                       _ptr(ws), ws.numel(), _stream(dev)))
    return t_out, slope, q, cur


def multispike_backward(p: dstd_lif_params, t_in, W, t_out, slope, q, cur, grad_t_out,
                        need_W=True, need_t_in=True, ws=None):
    """Multi-spike dense backward; returns (grad_W or None, grad_t_in [B, N_in, F_in] or None)."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B, N_in, F_in = t_in.shape
    N_out = W.shape[0]
    F_out = t_out.shape[2]
    dev = t_in.device
    gW = torch.empty((N_out, N_in), dtype=torch.float32, device=dev) if need_W else None
    gt = torch.empty((B, N_in, F_in), dtype=torch.float32, device=dev) if need_t_in else None
    need = dstd_lif_multispike_backward_workspace_size(p, B, N_in, F_in, N_out, F_out)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    _check("dstd_lif_multispike_backward",
           dstd_lif_multispike_backward(p, B, N_in, F_in, N_out, F_out, _ptr(t_in), _ptr(W),
                                        _wdtype(W), _ptr(_cont(t_out, torch.float32)),
                                        _ptr(_cont(slope, torch.float32)),
                                        _ptr(_cont(q, torch.int32)), _ptr(_cont(cur, torch.float32)),
                                        _ptr(_cont(grad_t_out, torch.float32)), _ptr(gW), _ptr(gt),
                                        _ptr(ws), ws.numel(), _stream(dev)))
    return gW, gt


def skip_delay_concat(t1, delay: float, t2):
    """SD-block skip input: cat([t1 + delay, t2], channels). t1 [B, C1, H, W], t2 [B, C2, H, W]."""
    torch = _torch()
    t1 = _cont(t1, torch.float32)
    t2 = _cont(t2, torch.float32)
    B, C1 = t1.shape[:2]
    C2 = t2.shape[1]
    assert t2.shape[0] == B and t1.shape[2:] == t2.shape[2:]
    HW = int(math.prod(t1.shape[2:]))
    out = torch.empty((B, C1 + C2) + tuple(t1.shape[2:]), dtype=torch.float32, device=t1.device)
    _check("dstd_skip_delay_concat",
           dstd_skip_delay_concat(B, C1, C2, HW, _ptr(t1), float(delay), _ptr(t2), _ptr(out),
                                  _stream(t1.device)))
    return out


def skip_delay_concat_backward(g, C1: int, g1=None, want_g2=True):
    """Split dL/d(concat) [B, C1 + C2, H, W]: adds the first C1 channels into g1
    (written when g1 is None) and returns (g1, g2)."""
    torch = _torch()
    g = _cont(g, torch.float32)
    B, C = g.shape[:2]
    C2 = C - C1
    HW = int(math.prod(g.shape[2:]))
    acc = 1
    if g1 is None:
        g1 = torch.empty((B, C1) + tuple(g.shape[2:]), dtype=torch.float32, device=g.device)
        acc = 0
    else:
        assert g1.is_contiguous() and g1.dtype == torch.float32 and g1.shape[:2] == (B, C1)
    g2 = torch.empty((B, C2) + tuple(g.shape[2:]), dtype=torch.float32, device=g.device) if want_g2 else None
    _check("dstd_skip_delay_concat_backward",
           dstd_skip_delay_concat_backward(B, C1, C2, HW, _ptr(g), _ptr(g1), acc, _ptr(g2),
                                           _stream(g.device)))
    return g1, g2


def exact_forward(p: dstd_lif_params, t_in, W, ws=None):
    """Exact (sorted-input) forward of a dense layer; returns (t_out, slope,
    k_idx). Only tau_m, tau_s, threshold and t_max of `p` are used."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    assert W.shape[1] == N_in
    dev = t_in.device
    t_out = torch.empty((B, N_out), dtype=torch.float32, device=dev)
    slope = torch.empty_like(t_out)
    k = torch.empty((B, N_out), dtype=torch.int32, device=dev)
    need = dstd_exact_forward_workspace_size(p, B, N_in, N_out)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    _check("dstd_exact_forward",
           dstd_exact_forward(p, B, N_in, N_out, _ptr(t_in), _ptr(W), _wdtype(W), _ptr(t_out),
                              _ptr(slope), _ptr(k), _ptr(ws), ws.numel(), _stream(dev)))
    return t_out, slope, k


def exact_backward(p: dstd_lif_params, t_in, W, t_out, slope, k, grad_t_out, need_W=True,
                   need_t_in=True, ws=None):
    """Exact backward of a dense layer; returns (grad_W or None, grad_t_in or None)."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    dev = t_in.device
    gW = torch.empty((N_out, N_in), dtype=torch.float32, device=dev) if need_W else None
    gt = torch.empty((B, N_in), dtype=torch.float32, device=dev) if need_t_in else None
    need = dstd_exact_backward_workspace_size(p, B, N_in, N_out)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    _check("dstd_exact_backward",
           dstd_exact_backward(p, B, N_in, N_out, _ptr(t_in), _ptr(W), _wdtype(W),
                               _ptr(_cont(t_out, torch.float32)), _ptr(_cont(slope, torch.float32)),
                               _ptr(_cont(k, torch.int32)), _ptr(_cont(grad_t_out, torch.float32)),
                               _ptr(gW), _ptr(gt), _ptr(ws), ws.numel(), _stream(dev)))
    return gW, gt


def conv_forward(p: dstd_lif_params, cs: dstd_conv_shape, t_in, W, ws=None):
    """Conv layer forward. t_in [B, C_in, H, W] f32, W [C_out, C_in, KH, KW]."""
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B = t_in.shape[0]
    Ho, Wo = conv_out_hw(cs)
    dev = t_in.device
    t_out = torch.empty((B, cs.C_out, Ho, Wo), dtype=torch.float32, device=dev)
    slope = torch.empty_like(t_out)
    q = torch.empty((B, cs.C_out, Ho, Wo), dtype=torch.int32, device=dev)
    need = dstd_lif_conv_forward_workspace_size(p, cs, B)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    _check("dstd_lif_conv_forward",
           dstd_lif_conv_forward(p, cs, B, _ptr(t_in), _ptr(W), _wdtype(W), _ptr(t_out),
                                 _ptr(slope), _ptr(q), _ptr(ws), ws.numel(), _stream(dev)))
    return t_out, slope, q


def conv_backward(p, cs, t_in, W, t_out, slope, q, grad_t_out, need_W=True, need_t_in=True,
                  ws=None, synfire: Optional[dstd_synfire_params] = None):
    torch = _torch()
    t_in = _cont(t_in, torch.float32)
    W = _cont(W)
    B = t_in.shape[0]
    dev = t_in.device
    gW = torch.empty(W.shape, dtype=torch.float32, device=dev) if need_W else None
    gt = torch.empty(t_in.shape, dtype=torch.float32, device=dev) if need_t_in else None
    need = dstd_lif_conv_backward_workspace_size(p, cs, B)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    args = (B, _ptr(t_in), _ptr(W), _wdtype(W), _ptr(_cont(t_out, torch.float32)),
            _ptr(_cont(slope, torch.float32)), _ptr(_cont(q, torch.int32)),
            _ptr(_cont(grad_t_out, torch.float32)), _ptr(gW), _ptr(gt), _ptr(ws), ws.numel(),
            _stream(dev))
    if synfire is None:
        _check("dstd_lif_conv_backward", dstd_lif_conv_backward(p, cs, *args))
    else:
        _check("dstd_lif_conv_backward_synfire",
               dstd_lif_conv_backward_synfire(p, synfire, cs, *args))
    return gW, gt


def synfire_penalty(sp: dstd_synfire_params, t_out, W):
    """Values (T, Q) of the synfire terms as a device tensor [2]. t_out is
    [B, N_out] (dense) or [B, C_out, H_out, W_out] (conv); W is the layer's
    weight tensor (rows = its first dimension)."""
    torch = _torch()
    t_out = _cont(t_out, torch.float32)
    W = _cont(W)
    B = t_out.shape[0]
    rows = t_out.shape[1]
    spatial = 1
    for d in t_out.shape[2:]:
        spatial *= d
    row_len = W.numel() // max(W.shape[0], 1)
    dev = t_out.device
    value = torch.empty(2, dtype=torch.float32, device=dev)
    need = dstd_synfire_penalty_workspace_size(B, rows, spatial)
    ws = workspace(need, dev)
    _check("dstd_synfire_penalty",
           dstd_synfire_penalty(sp, B, rows, spatial, row_len, _ptr(t_out), _ptr(W), _wdtype(W),
                                _ptr(value), _ptr(ws), ws.numel(), _stream(dev)))
    return value


def softmax_ce_grad(t_out, labels, tau_soft: float = 1.0, t_cap: Optional[float] = None):
    """Returns (dL/dt [B, N], loss [B + 1]): loss[0] = L, loss[1 + b] = sample b's term."""
    torch = _torch()
    t_out = _cont(t_out, torch.float32)
    labels = _cont(labels, torch.int32)
    B, N = t_out.shape
    if t_cap is None:
        raise ValueError("t_cap is required (time used for outputs that did not fire)")
    grad = torch.empty_like(t_out)
    loss = torch.empty((B + 1,), dtype=torch.float32, device=t_out.device)
    _check("dstd_softmax_ce_grad",
           dstd_softmax_ce_grad(B, N, _ptr(t_out), _ptr(labels), float(tau_soft), float(t_cap),
                                _ptr(grad), _ptr(loss), _stream(t_out.device)))
    return grad, loss


def mse_grad(t_out, target):
    """Returns (dL/dt [B, N], loss [B + 1]): loss[0] = L, loss[1 + b] = sample b's term."""
    torch = _torch()
    t_out = _cont(t_out, torch.float32)
    target = _cont(target, torch.float32)
    B, N = t_out.shape
    grad = torch.empty_like(t_out)
    loss = torch.empty((B + 1,), dtype=torch.float32, device=t_out.device)
    _check("dstd_mse_grad", dstd_mse_grad(B, N, _ptr(t_out), _ptr(target), _ptr(grad), _ptr(loss),
                                          _stream(t_out.device)))
    return grad, loss
