"""ctypes binding of the fp64 C oracle (``dstd_oracle.c``).

Test infrastructure only: the product path never imports this module.
Inputs are widened to float64 (pass the float32 arrays the GPU sees, or
float64 arrays for finite-difference pins); results are float64.
"""
from __future__ import annotations

import contextlib
import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = [os.path.join(_HERE, "dstd_oracle.c")]
_LIB_PATH = os.path.join(_HERE, "libdstd_oracle.so")
_lib = None


def build_oracle(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, fp64, no fast-math)."""
    stale = (not os.path.exists(_LIB_PATH) or
             max(os.path.getmtime(f) for f in _SRC) > os.path.getmtime(_LIB_PATH))
    if force or stale:
        compile_oracle(_SRC[0], _LIB_PATH)
    return _LIB_PATH


def compile_oracle(src: str, out: str) -> str:
    """gcc -O2 -fopenmp, fp64, no fast-math: ``src`` -> shared library ``out``."""
    cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-Wall",
           "-o", out + ".tmp", src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_D = C.c_double
_I = C.c_int
_L = C.c_int64
_P = C.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build_oracle(force=False)  # builds when missing or older than its source
    _lib = _configure(C.CDLL(_LIB_PATH))
    return _lib


@contextlib.contextmanager
def use_library(path):
    """Bind this module to another build of the oracle for the duration of
    the block (the mutation tests load copies with planted mistakes)."""
    global _lib
    saved = _load()
    _lib = _configure(C.CDLL(path))
    try:
        yield
    finally:
        _lib = saved


def _configure(lib):
    lib.oracle_kernel.restype = _D
    lib.oracle_kernel.argtypes = [_D, _D, _D]
    lib.oracle_kdstd.restype = _D
    lib.oracle_kdstd.argtypes = [_D, _D, _D, _D]
    lib.oracle_lambert_w0.restype = _D
    lib.oracle_lambert_w0.argtypes = [_D]
    lib.oracle_dstd_events.restype = None
    lib.oracle_dstd_events.argtypes = [_D, _D, _I, _D, _D, _L, _L, _P, _P, _P]
    lib.oracle_dstd_forward.restype = None
    lib.oracle_dstd_forward.argtypes = [_D, _D, _D, _I, _D, _D, _D, _L, _L, _L,
                                        _P, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_dstd_scan.restype = None
    lib.oracle_dstd_scan.argtypes = [_D, _D, _D, _I, _D, _D, _D, _L, _L, _P,
                                     _P, _P, _P, _P, _P]
    lib.oracle_dstd_backward.restype = None
    lib.oracle_dstd_backward.argtypes = [_D, _D, _D, _I, _D, _D, _D, _L, _L, _L,
                                         _P, _P, _P, _P, _P, _P, _L, _P, _P, _L, _P, _P, _P, _P,
                                         _P, _P, _P, _P]
    lib.oracle_exact_forward.restype = None
    lib.oracle_exact_forward.argtypes = [_D, _D, _D, _D, _L, _L, _L, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_exact_backward.restype = None
    lib.oracle_exact_backward.argtypes = [_D, _D, _L, _L, _L, _P, _P, _P, _P, _P, _P,
                                          _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_ms_forward.restype = None
    lib.oracle_ms_forward.argtypes = [_D, _D, _D, _I, _D, _D, _D, _L, _L, _L, _L, _L, _P, _P, _P,
                                      _P, _P, _P, _P, _P, _P]
    lib.oracle_ms_backward.restype = None
    lib.oracle_ms_backward.argtypes = [_D, _D, _D, _I, _D, _D, _D, _L, _L, _L, _L, _L, _P, _P,
                                       _P, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_conv_forward.restype = None
    lib.oracle_conv_forward.argtypes = [_D, _D, _D, _I, _D, _D, _D, _L,
                                        _I, _I, _I, _I, _I, _I, _I, _I, _I,
                                        _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_conv_backward.restype = None
    lib.oracle_conv_backward.argtypes = [_D, _D, _D, _I, _D, _D, _D, _L,
                                         _I, _I, _I, _I, _I, _I, _I, _I, _I,
                                         _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_num_threads.restype = _I
    lib.oracle_num_threads.argtypes = []
    return lib


def _f64(a):
    """Widen to float64 exactly (float32 inputs keep their bits' value)."""
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def kernel(tau_v, tau_i, t) -> float:
    """Spike kernel K(t), Table "tab:kernel" (the row follows from the pair:
    +inf constants and equal constants select the closed-form rows)."""
    return float(_load().oracle_kernel(tau_v, tau_i, t))


def kdstd(tau_v, tau_i, dt, t) -> float:
    """DSTD kernel K_DSTD(t), Table "tab:DSTD_kernels" (row as for kernel())."""
    return float(_load().oracle_kdstd(tau_v, tau_i, dt, t))


def lambert_w0(x) -> float:
    """Principal branch of the Lambert W function (used by the (tau, tau)
    candidate of Table "tab:timing_DSTD")."""
    return float(_load().oracle_lambert_w0(x))


def dstd_events(p, t_in):
    """Dense event tensor s[b, m, j] and ds/dt, Eq. (DSTD_kernel)."""
    t_in = _f64(t_in)
    B, N_in = t_in.shape
    M = int(p["M"])
    s = np.zeros((B, M + 1, N_in))
    ds = np.zeros((B, M + 1, N_in))
    tv, ti = max(p["tau_m"], p["tau_s"]), min(p["tau_m"], p["tau_s"])
    _load().oracle_dstd_events(tv, ti, M, p["t0"], p["dt"], B, N_in, _ptr(t_in), _ptr(s), _ptr(ds))
    return s, ds


def _pargs(p):
    return (float(p["tau_m"]), float(p["tau_s"]), float(p["threshold"]), int(p["M"]),
            float(p["t0"]), float(p["dt"]), float(p.get("t_max", np.inf)))


def dstd_forward(p, t_in, W, want_what=False):
    """DSTD forward of a dense layer. Returns dict of float64/int32 arrays."""
    t_in = _f64(t_in)
    W = _f64(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    assert W.shape == (N_out, N_in)
    M = int(p["M"])
    t_out = np.empty((B, N_out))
    slope = np.empty((B, N_out))
    q = np.empty((B, N_out), dtype=np.int32)
    margin = np.empty((B, N_out))
    vabs = np.empty((B, N_out))
    emass = np.empty((B, N_out))
    what = np.empty((B, M + 1, N_out)) if want_what else None
    _load().oracle_dstd_forward(*_pargs(p), B, N_in, N_out, _ptr(t_in), _ptr(W),
                                _ptr(t_out), _ptr(slope), _ptr(q), _ptr(margin), _ptr(vabs),
                                _ptr(emass), _ptr(what))
    out = dict(t_out=t_out, slope=slope, q=q, margin=margin, vabs=vabs, emass=emass)
    if want_what:
        out["what"] = what
    return out


def dstd_scan(p, what):
    """Interval scan + solve from given weighted events what[b, m, i] (float64)."""
    what = np.ascontiguousarray(np.asarray(what, dtype=np.float64))
    B, M1, N_out = what.shape
    assert M1 == int(p["M"]) + 1
    t_out = np.empty((B, N_out))
    slope = np.empty((B, N_out))
    q = np.empty((B, N_out), dtype=np.int32)
    margin = np.empty((B, N_out))
    vT = np.empty((B, M1, N_out))
    _load().oracle_dstd_scan(*_pargs(p), B, N_out, _ptr(what), _ptr(t_out), _ptr(slope), _ptr(q),
                             _ptr(margin), _ptr(vT))
    return dict(t_out=t_out, slope=slope, q=q, margin=margin, v_at_T=vT)


def dstd_backward(p, t_in, W, fwd, grad_t_out, isel=None, bsel=None, want_dW=True, want_dt=True,
                  want_abs=False, err=None):
    """DSTD backward of a dense layer (implicit-function gradients).

    ``fwd`` is a dict with t_out, slope, q (the oracle's own forward outputs).
    Returns (grad_W rows, grad_t_in rows), plus (|terms| sums of each) when
    ``want_abs``, plus (error-weighted sums of each) when ``err`` = (rho, delta)
    per neuron is given (see oracle_dstd_backward).
    """
    t_in = _f64(t_in)
    W = _f64(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    t_out = np.ascontiguousarray(fwd["t_out"], dtype=np.float64)
    slope = np.ascontiguousarray(fwd["slope"], dtype=np.float64)
    q = np.ascontiguousarray(fwd["q"], dtype=np.int32)
    g = np.ascontiguousarray(grad_t_out, dtype=np.float64)
    isel_a = None if isel is None else np.ascontiguousarray(isel, dtype=np.int64)
    bsel_a = None if bsel is None else np.ascontiguousarray(bsel, dtype=np.int64)
    ni = N_out if isel is None else len(isel_a)
    nb = B if bsel is None else len(bsel_a)
    dW = np.empty((ni, N_in)) if want_dW else None
    dt = np.empty((nb, N_in)) if want_dt else None
    dWa = np.empty((ni, N_in)) if (want_dW and want_abs) else None
    dta = np.empty((nb, N_in)) if (want_dt and want_abs) else None
    rho = delta = dWe = dte = None
    if err is not None:
        rho, delta = (np.ascontiguousarray(np.broadcast_to(a, (B, N_out)), dtype=np.float64)
                      for a in err)
        dWe = np.empty((ni, N_in)) if want_dW else None
        dte = np.empty((nb, N_in)) if want_dt else None
    _load().oracle_dstd_backward(*_pargs(p), B, N_in, N_out, _ptr(t_in), _ptr(W), _ptr(t_out),
                                 _ptr(slope), _ptr(q), _ptr(g),
                                 -1 if isel is None else ni, _ptr(isel_a), _ptr(dW),
                                 -1 if bsel is None else nb, _ptr(bsel_a), _ptr(dt),
                                 _ptr(dWa), _ptr(dta), _ptr(rho), _ptr(delta), _ptr(dWe), _ptr(dte))
    out = (dW, dt)
    if want_abs:
        out = out + (dWa, dta)
    if err is not None:
        out = out + (dWe, dte)
    return out


def exact_forward(p, t_in, W):
    """Exact continuous-time LIF spike times (Alg. 1, Eq. (timing_exact)).
    Returns t_out, slope, q (position in ascending input order of the left end
    of the crossing interval, -1 = silent), margin and vabs."""
    t_in = _f64(t_in)
    W = _f64(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    t_out = np.empty((B, N_out))
    slope = np.empty((B, N_out))
    q = np.empty((B, N_out), dtype=np.int32)
    margin = np.empty((B, N_out))
    vabs = np.empty((B, N_out))
    emass = np.empty((B, N_out))
    _load().oracle_exact_forward(float(p["tau_m"]), float(p["tau_s"]), float(p["threshold"]),
                                 float(p.get("t_max", np.inf)), B, N_in, N_out, _ptr(t_in), _ptr(W),
                                 _ptr(t_out), _ptr(slope), _ptr(q), _ptr(margin), _ptr(vabs),
                                 _ptr(emass))
    return dict(t_out=t_out, slope=slope, q=q, margin=margin, vabs=vabs, emass=emass)


def exact_backward(p, t_in, W, fwd, grad_t_out, err=None):
    """Gradients of the exact spike times (implicit function theorem over the
    causal set of the crossing interval). fwd: dict with t_out, slope, q.
    Returns grad_W [N_out, N_in], grad_t_in [B, N_in] and their |term| sums,
    and their error-weighted sums when ``err`` = (rho, delta) is given."""
    t_in = _f64(t_in)
    W = _f64(W)
    B, N_in = t_in.shape
    N_out = W.shape[0]
    t_out = _f64(fwd["t_out"])
    slope = _f64(fwd["slope"])
    q = np.ascontiguousarray(fwd["q"], dtype=np.int32)
    g = _f64(grad_t_out)
    gW = np.empty((N_out, N_in))
    gt = np.empty((B, N_in))
    gWa = np.empty((N_out, N_in))
    gta = np.empty((B, N_in))
    rho = delta = gWe = gte = None
    if err is not None:
        rho, delta = (np.ascontiguousarray(np.broadcast_to(a, (B, N_out)), dtype=np.float64)
                      for a in err)
        gWe, gte = np.empty((N_out, N_in)), np.empty((B, N_in))
    _load().oracle_exact_backward(float(p["tau_m"]), float(p["tau_s"]), B, N_in, N_out,
                                  _ptr(t_in), _ptr(W), _ptr(t_out), _ptr(slope), _ptr(q), _ptr(g),
                                  _ptr(gW), _ptr(gt), _ptr(gWa), _ptr(gta),
                                  _ptr(rho), _ptr(delta), _ptr(gWe), _ptr(gte))
    out = dict(grad_W=gW, grad_t_in=gt, grad_W_abs=gWa, grad_t_in_abs=gta)
    if err is not None:
        out.update(grad_W_err=gWe, grad_t_in_err=gte)
    return out


def ms_forward(p, t_in, W, F_out):
    """Multi-spike DSTD forward (App. "multi-spikes"): t_in [B, N_in, F_in],
    W [N_out, N_in]. Returns per output spike [B, N_out, F_out]: t_out, slope,
    q, cur (current at the spike), margin, vabs, dprev (d t_k / d t_{k-1})."""
    t_in = _f64(t_in)
    W = _f64(W)
    B, N_in, F_in = t_in.shape
    N_out = W.shape[0]
    shp = (B, N_out, F_out)
    out = {k: np.empty(shp) for k in ("t_out", "slope", "cur", "margin", "vabs", "dprev")}
    out["q"] = np.empty(shp, dtype=np.int32)
    _load().oracle_ms_forward(float(p["tau_m"]), float(p["tau_s"]), float(p["threshold"]),
                              int(p["M"]), float(p["t0"]), float(p["dt"]),
                              float(p.get("t_max", np.inf)), B, N_in, F_in, N_out, F_out,
                              _ptr(t_in), _ptr(W), _ptr(out["t_out"]), _ptr(out["slope"]),
                              _ptr(out["q"]), _ptr(out["cur"]), _ptr(out["margin"]),
                              _ptr(out["vabs"]), _ptr(out["dprev"]))
    return out


def ms_backward(p, t_in, W, fwd, grad_t_out):
    """Multi-spike DSTD backward. grad_t_out [B, N_out, F_out]; returns grad_W,
    grad_t_in [B, N_in, F_in] and their |term| sums."""
    t_in = _f64(t_in)
    W = _f64(W)
    B, N_in, F_in = t_in.shape
    N_out = W.shape[0]
    F_out = fwd["t_out"].shape[2]
    gW, gWa = np.empty((N_out, N_in)), np.empty((N_out, N_in))
    gt, gta = np.empty(t_in.shape), np.empty(t_in.shape)
    _load().oracle_ms_backward(float(p["tau_m"]), float(p["tau_s"]), float(p["threshold"]),
                               int(p["M"]), float(p["t0"]), float(p["dt"]),
                               float(p.get("t_max", np.inf)), B, N_in, F_in, N_out, F_out,
                               _ptr(t_in), _ptr(W), _ptr(_f64(fwd["t_out"])), _ptr(_f64(fwd["slope"])),
                               _ptr(np.ascontiguousarray(fwd["q"], dtype=np.int32)),
                               _ptr(_f64(fwd["cur"])), _ptr(_f64(grad_t_out)), _ptr(gW), _ptr(gt),
                               _ptr(gWa), _ptr(gta))
    return dict(grad_W=gW, grad_t_in=gt, grad_W_abs=gWa, grad_t_in_abs=gta)


def _conv_geom(cs):
    return (int(cs["C_in"]), int(cs["H"]), int(cs["W"]), int(cs["C_out"]), int(cs["KH"]),
            int(cs["KW"]), int(cs["stride"]), int(cs["pad"]), int(cs["pool_in"]))


def conv_out_hw(cs):
    C_in, H, Wd, C_out, KH, KW, st, pad, pool = _conv_geom(cs)
    if pool == 2:
        H, Wd = H // 2, Wd // 2
    elif pool == 0:
        H, Wd = 1, 1
    return (H + 2 * pad - KH) // st + 1, (Wd + 2 * pad - KW) // st + 1


def conv_forward(p, cs, t_in, W):
    """DSTD forward of a conv layer (events pooled before the convolution)."""
    t_in = _f64(t_in)
    W = _f64(W)
    B = t_in.shape[0]
    Ho, Wo = conv_out_hw(cs)
    C_out = int(cs["C_out"])
    shp = (B, C_out, Ho, Wo)
    t_out = np.empty(shp)
    slope = np.empty(shp)
    q = np.empty(shp, dtype=np.int32)
    margin = np.empty(shp)
    vabs = np.empty(shp)
    emass = np.empty(shp)
    _load().oracle_conv_forward(*_pargs(p), B, *_conv_geom(cs), _ptr(t_in), _ptr(W), _ptr(t_out),
                                _ptr(slope), _ptr(q), _ptr(margin), _ptr(vabs), _ptr(emass))
    return dict(t_out=t_out, slope=slope, q=q, margin=margin, vabs=vabs, emass=emass)


def conv_backward(p, cs, t_in, W, fwd, grad_t_out, want_abs=False, err=None):
    """DSTD backward of a conv layer. Returns (grad_W, grad_t_in), plus the
    per-element sums of |terms| of each when ``want_abs``, plus the
    error-weighted sums when ``err`` = (rho, delta) per output neuron is given."""
    t_in = _f64(t_in)
    W = _f64(W)
    t_out = np.ascontiguousarray(fwd["t_out"], dtype=np.float64)
    slope = np.ascontiguousarray(fwd["slope"], dtype=np.float64)
    q = np.ascontiguousarray(fwd["q"], dtype=np.int32)
    g = np.ascontiguousarray(grad_t_out, dtype=np.float64)
    B = t_in.shape[0]
    dW = np.empty(W.shape)
    dt = np.empty(t_in.shape)
    dWa = np.empty(W.shape) if want_abs else None
    dta = np.empty(t_in.shape) if want_abs else None
    rho = delta = dWe = dte = None
    if err is not None:
        rho, delta = (np.ascontiguousarray(np.broadcast_to(a, t_out.shape), dtype=np.float64)
                      for a in err)
        dWe, dte = np.empty(W.shape), np.empty(t_in.shape)
    _load().oracle_conv_backward(*_pargs(p), B, *_conv_geom(cs), _ptr(t_in), _ptr(W), _ptr(t_out),
                                 _ptr(slope), _ptr(q), _ptr(g), _ptr(dW), _ptr(dt), _ptr(dWa),
                                 _ptr(dta), _ptr(rho), _ptr(delta), _ptr(dWe), _ptr(dte))
    out = (dW, dt)
    if want_abs:
        out = out + (dWa, dta)
    if err is not None:
        out = out + (dWe, dte)
    return out
