"""GPU checks of the skip-and-delay block (App. C.3, Fig. "skip_connection"):
the delayed channel concatenation and its gradient split are exact; an SD
block's third layer and the block input's gradient match the fp64 oracle
composed the same way."""
import math

import numpy as np
import pytest

import oracle
from tests.parity import check_forward, check_grad, grad_err_inputs, near_grid
from tests.test_gpu_conv import _cs, _conv_case, _gpu_backward, _gpu_forward, _window

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_14672_amd import dstd
    dstd._load()  # fail loudly if the HIP library is missing
    return torch.device("cuda:0")


def test_concat_and_split_are_exact(dev):
    import torch
    from paper_2607_14672_amd import dstd
    rng = np.random.default_rng(0)
    t1 = rng.random((3, 5, 7, 6)).astype(np.float32)
    t1[0, 1, 2, 3] = np.inf
    t2 = (2.0 + rng.random((3, 4, 7, 6))).astype(np.float32)
    t2[2, 0, 0, 0] = np.inf
    d = np.float32(2.0)
    out = dstd.skip_delay_concat(torch.from_numpy(t1).to(dev), float(d), torch.from_numpy(t2).to(dev))
    ref = np.concatenate([t1 + d, t2], axis=1)
    assert np.array_equal(out.cpu().numpy(), ref)
    g = rng.standard_normal((3, 9, 7, 6)).astype(np.float32)
    base = rng.standard_normal((3, 5, 7, 6)).astype(np.float32)
    gg = torch.from_numpy(g).to(dev)
    g1 = torch.from_numpy(base.copy()).to(dev)
    g1o, g2 = dstd.skip_delay_concat_backward(gg, 5, g1=g1)
    assert g1o is g1
    assert np.array_equal(g1.cpu().numpy(), base + g[:, :5])
    assert np.array_equal(g2.cpu().numpy(), g[:, 5:])
    g1w, _ = dstd.skip_delay_concat_backward(gg, 5, want_g2=False)
    assert np.array_equal(g1w.cpu().numpy(), g[:, :5])
    # degenerate: no skip channels, empty batch
    e = dstd.skip_delay_concat(torch.empty((3, 0, 7, 6), device=dev), 1.0, torch.from_numpy(t2).to(dev))
    assert np.array_equal(e.cpu().numpy(), t2)
    z = dstd.skip_delay_concat(torch.empty((0, 5, 7, 6), device=dev), 1.0, torch.empty((0, 4, 7, 6), device=dev))
    assert z.shape == (0, 9, 7, 6)
    torch.cuda.synchronize()


@pytest.mark.parametrize("stride,label", [(2, "SD1"), (1, "SD2")])
def test_sd_block_third_layer_and_input_gradient(dev, stride, label):
    """SD block whose input x lies in [0, 1]: layer 1 (grid [0, 1]) and layer 2
    are ordinary conv layers; layer 3 reads cat(x + delay, out2). At random
    weights the layers fire early in their windows, so layer 2's grid starts
    at 0.7 and layer 3's at 1.0 with delay 1.0, which puts both sources inside
    layer 3's window (in a trained synfire chain these are l - 1 and 2
    tau_shift). Each layer is checked against the oracle on the GPU's own
    inputs; the block input's gradient is layer 1's dt_in plus the skip
    channels of layer 3's dt_in, against the same sum from the oracle."""
    import torch
    from paper_2607_14672_amd import dstd
    B, C, H, N = 2, 6, 9, 8
    M, tm, ts = 16, 1.0, 0.3
    cs1 = _cs(C, H, H, N)
    p1, x, W1 = _conv_case(21, B, cs1, M, tm, ts, k=7.0, t0=0.0)
    cs2 = _cs(N, H, H, N)
    p2, _, W2 = _conv_case(22, B, cs2, M, tm, ts, k=14.0, t0=0.7)
    N3 = 2 * N if stride == 2 else N
    cs3 = _cs(C + N, H, H, N3, stride=stride)
    p3, _, W3 = _conv_case(23, B, cs3, M, tm, ts, k=20.0, t0=1.0)
    delay = 1.0
    o1, h1 = _gpu_forward(dev, p1, cs1, x, W1)
    o2, h2 = _gpu_forward(dev, p2, cs2, o1["t_out"], W2)
    assert (o2["q"] >= 0).mean() > 0.1
    cat = dstd.skip_delay_concat(h1[2], delay, h2[4])
    cat_np = cat.cpu().numpy()
    assert np.array_equal(cat_np, np.concatenate([x + np.float32(delay), o2["t_out"]], axis=1))
    o3, h3 = _gpu_forward(dev, p3, cs3, cat_np, W3)
    orc3 = oracle.conv_forward(p3, cs3, cat_np, W3)
    taus = (max(tm, ts), min(tm, ts))
    mask3, st3 = check_forward(o3, orc3, None, _window(p3), label=f"{label} layer 3", taus=taus)
    assert st3["fired"] > 0.1 * st3["n"]
    orc1 = oracle.conv_forward(p1, cs1, x, W1)
    mask1, st1 = check_forward(o1, orc1, None, _window(p1), label=f"{label} layer 1", taus=taus)
    rng = np.random.default_rng(5)
    g3 = np.where(mask3, 0.0, rng.standard_normal(orc3["t_out"].shape)).astype(np.float32)
    g1 = np.where(mask1, 0.0, rng.standard_normal(orc1["t_out"].shape)).astype(np.float32)
    _, gcat = _gpu_backward(dev, h3, g3, need_W=False)
    _, gx1 = _gpu_backward(dev, h1, g1, need_W=False)
    gx = torch.from_numpy(gx1).to(dev)
    _, g_o2 = dstd.skip_delay_concat_backward(torch.from_numpy(gcat).to(dev), C, g1=gx)
    torch.cuda.synchronize()
    _, ocat, _, ocat_a, _, ocat_e = oracle.conv_backward(
        p3, cs3, cat_np, W3, orc3, np.where(orc3["q"] >= 0, g3.astype(np.float64), 0.0),
        want_abs=True, err=grad_err_inputs(st3, mask3))
    _, ox1, _, ox1_a, _, ox1_e = oracle.conv_backward(
        p1, cs1, x, W1, orc1, np.where(orc1["q"] >= 0, g1.astype(np.float64), 0.0),
        want_abs=True, err=grad_err_inputs(st1, mask1))
    ox = ox1 + ocat[:, :C]
    oxa = ox1_a + ocat_a[:, :C]
    oxe = ox1_e + ocat_e[:, :C]
    n_x = 2 * (N + N3) * 9
    kink = near_grid(x, p1) | near_grid(cat_np[:, :C], p3)
    check_grad(gx.cpu().numpy()[~kink], ox[~kink], f"{label} block input dt", oxa[~kink], oxe[~kink],
               n_terms=n_x)
    kink2 = near_grid(cat_np[:, C:], p3)
    check_grad(g_o2.cpu().numpy()[~kink2], ocat[:, C:][~kink2], f"{label} layer-2 output dt",
               ocat_a[:, C:][~kink2], ocat_e[:, C:][~kink2], n_terms=2 * N3 * 9)
