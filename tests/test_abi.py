"""C-ABI contract on the CPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments before touching a device."""
import math
import os
import re

import pytest

from paper_2607_14672_amd import dstd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "dstd_lif.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(dstd_[a-z_0-9]+)\s*\(", src)
    return sorted(set(names))


def test_library_exports_every_header_symbol():
    lib = dstd._load()
    names = _header_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(dstd.exported_symbols())


def _p(**kw):
    base = dict(tau_m=1.0, tau_s=0.3, threshold=1.0, M=16, t0=0.0, dt=1 / 16, t_max=math.inf)
    base.update(kw)
    return dstd.make_params(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(tau_m=1.0, tau_s=1.0), dstd.DSTD_ERR_UNSUPPORTED),
    (dict(tau_m=1.0, tau_s=1.0005), dstd.DSTD_ERR_UNSUPPORTED),
    (dict(tau_m=-1.0), dstd.DSTD_ERR_PARAM),
    (dict(tau_s=math.inf), dstd.DSTD_ERR_PARAM),
    (dict(tau_s=math.nan), dstd.DSTD_ERR_PARAM),
    (dict(threshold=0.0), dstd.DSTD_ERR_PARAM),
    (dict(M=0), dstd.DSTD_ERR_PARAM),
    (dict(M=dstd.DSTD_MAX_M + 1), dstd.DSTD_ERR_UNSUPPORTED),
    (dict(dt=0.0), dstd.DSTD_ERR_PARAM),
    (dict(dt=math.nan), dstd.DSTD_ERR_PARAM),
    (dict(t0=math.inf), dstd.DSTD_ERR_PARAM),
    (dict(t_max=1.0), dstd.DSTD_ERR_PARAM),
    (dict(t_max=math.nan), dstd.DSTD_ERR_PARAM),
])
def test_parameter_validation(kw, status):
    p = _p(**kw)
    assert dstd.dstd_lif_forward_workspace_size(p, 4, 10, 5) == 0
    st = dstd.dstd_lif_forward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, 256, 1 << 20, None)
    assert st == status, dstd.dstd_last_error()
    st = dstd.dstd_lif_backward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, 1, 1, 1, 256, 1 << 20, None)
    assert st == status
    assert dstd.dstd_last_error()


def test_flags_must_be_zero():
    p = _p()
    p.flags = 1
    assert dstd.dstd_lif_forward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, 256, 1 << 20, None) == dstd.DSTD_ERR_PARAM


def test_shape_null_dtype_and_workspace_errors():
    p = _p()
    need = dstd.dstd_lif_forward_workspace_size(p, 4, 10, 5)
    assert need > 0
    assert dstd.dstd_lif_forward(None, 4, 10, 5, 1, 1, 0, 1, 1, 1, 256, need, None) == dstd.DSTD_ERR_NULL
    assert dstd.dstd_lif_forward(p, -1, 10, 5, 1, 1, 0, 1, 1, 1, 256, need, None) == dstd.DSTD_ERR_SHAPE
    assert dstd.dstd_lif_forward(p, 70000, 10, 5, 1, 1, 0, 1, 1, 1, 256, 1 << 40, None) == dstd.DSTD_ERR_SHAPE
    assert dstd.dstd_lif_forward(p, 4, 10, 5, None, 1, 0, 1, 1, 1, 256, need, None) == dstd.DSTD_ERR_NULL
    assert dstd.dstd_lif_forward(p, 4, 10, 5, 1, None, 0, 1, 1, 1, 256, need, None) == dstd.DSTD_ERR_NULL
    assert dstd.dstd_lif_forward(p, 4, 10, 5, 1, 1, 0, None, 1, 1, 256, need, None) == dstd.DSTD_ERR_NULL
    assert dstd.dstd_lif_forward(p, 4, 10, 5, 1, 1, 7, 1, 1, 1, 256, need, None) == dstd.DSTD_ERR_PARAM
    assert dstd.dstd_lif_forward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, None, need, None) == dstd.DSTD_ERR_NULL
    assert dstd.dstd_lif_forward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, 256, need - 1, None) == dstd.DSTD_ERR_WORKSPACE
    assert dstd.dstd_lif_forward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, 257, need, None) == dstd.DSTD_ERR_WORKSPACE
    nb = dstd.dstd_lif_backward_workspace_size(p, 4, 10, 5)
    assert nb > need
    assert dstd.dstd_lif_backward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, None, 1, 1, 256, nb, None) == dstd.DSTD_ERR_NULL
    assert dstd.dstd_lif_backward(p, 4, 10, 5, 1, 1, 0, 1, 1, 1, 1, 1, 1, 256, nb - 1, None) == dstd.DSTD_ERR_WORKSPACE


def test_workspace_grows_with_sizes():
    p = _p()
    a = dstd.dstd_lif_forward_workspace_size(p, 4, 100, 50)
    b = dstd.dstd_lif_forward_workspace_size(p, 8, 100, 50)
    c = dstd.dstd_lif_backward_workspace_size(p, 8, 100, 50)
    d = dstd.dstd_lif_backward_workspace_size(_p(M=64), 8, 100, 50)
    assert 0 < a < b < c < d
    assert dstd.dstd_lif_forward_workspace_size(p, 0, 100, 50) == 0


def test_loss_validation():
    assert dstd.dstd_softmax_ce_grad(4, 0, 1, 1, 1.0, 3.0, 1, 1, None) == dstd.DSTD_ERR_SHAPE
    assert dstd.dstd_softmax_ce_grad(4, 10, 1, 1, 0.0, 3.0, 1, 1, None) == dstd.DSTD_ERR_PARAM
    assert dstd.dstd_softmax_ce_grad(4, 10, 1, 1, 1.0, math.inf, 1, 1, None) == dstd.DSTD_ERR_PARAM
    assert dstd.dstd_softmax_ce_grad(4, 10, None, 1, 1.0, 3.0, 1, 1, None) == dstd.DSTD_ERR_NULL
    assert dstd.dstd_mse_grad(4, 2000, 1, 1, 1, 1, None) == dstd.DSTD_ERR_SHAPE
    assert dstd.dstd_mse_grad(4, 10, 1, 1, 1, None, None) == dstd.DSTD_ERR_NULL


def test_status_strings():
    for s in range(-6, 1):
        assert dstd.dstd_status_string(s)
    assert dstd.dstd_version() >= 100
