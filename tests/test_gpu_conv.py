"""GPU parity of the conv DSTD-LIF layer (with event pooling) against the fp64
oracle, through the C ABI."""
import math

import numpy as np
import pytest

import oracle
from paper_2607_14672_amd import workloads as wl
from tests.parity import check_forward, check_grad, near_grid

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_14672_amd import dstd
    dstd._load()  # fail loudly if the HIP library is missing
    return torch.device("cuda:0")


def _cs(C_in, H, W, C_out, K=3, stride=1, pad=None, pool_in=1, KW=None):
    KW = K if KW is None else KW
    pad = (K // 2) if pad is None else pad
    return dict(C_in=C_in, H=H, W=W, C_out=C_out, KH=K, KW=KW, stride=stride, pad=pad,
                pool_in=pool_in)


def _prm(p):
    from paper_2607_14672_amd import dstd
    return dstd.make_params(p["tau_m"], p["tau_s"], p["threshold"], p["M"], p["t0"], p["dt"],
                            p.get("t_max", math.inf))


def _gpu_forward(dev, p, cs, t_in, W, bf16=False):
    import torch
    from paper_2607_14672_amd import dstd
    prm = _prm(p)
    c = dstd.make_conv_shape(**cs)
    tt = torch.from_numpy(np.ascontiguousarray(t_in, dtype=np.float32)).to(dev)
    Wt = torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).to(dev)
    if bf16:
        Wt = Wt.to(torch.bfloat16)
    to, sl, q = dstd.conv_forward(prm, c, tt, Wt)
    torch.cuda.synchronize()
    out = dict(t_out=to.cpu().numpy(), slope=sl.cpu().numpy(), q=q.cpu().numpy())
    return out, (prm, c, tt, Wt, to, sl, q)


def _gpu_backward(dev, handles, g, need_W=True, need_t=True):
    import torch
    from paper_2607_14672_amd import dstd
    prm, c, tt, Wt, to, sl, q = handles
    gt = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(dev)
    gW, gx = dstd.conv_backward(prm, c, tt, Wt, to, sl, q, gt, need_W=need_W, need_t_in=need_t)
    torch.cuda.synchronize()
    return (None if gW is None else gW.cpu().numpy()), (None if gx is None else gx.cpu().numpy())


def _conv_case(seed, B, cs, M, tm, ts, k=6.0, t0=0.0, spread=1.0, t_max=math.inf):
    rng = np.random.default_rng(seed)
    p = dict(tau_m=tm, tau_s=ts, threshold=1.0, M=M, t0=t0, dt=1.0 / M, t_max=t_max)
    t = (t0 + spread * rng.random((B, cs["C_in"], cs["H"], cs["W"]))).astype(np.float32)
    fan = cs["C_in"] * cs["KH"] * cs["KW"]
    z = rng.standard_normal((cs["C_out"], cs["C_in"], cs["KH"], cs["KW"]))
    W = ((k / fan) * (1 + 0.3 * math.sqrt(fan) * z)).astype(np.float32)
    return p, t, W


def _special_inputs(t, p, rng, per_sample=16):
    """Silent, NaN, -inf, out-of-grid, on-grid and grid-end inputs."""
    t = t.copy()
    B = t.shape[0]
    flat = t.reshape(B, -1)
    N = flat.shape[1]
    T = p["t0"] + p["dt"] * np.arange(p["M"] + 1)
    vals = [np.inf, np.nan, -np.inf, p["t0"] - 3 * p["dt"], T[-1] + 2 * p["dt"], T[0], T[-1],
            T[len(T) // 2], p["t0"] - 0.5 * p["dt"], T[-1] + 0.5 * p["dt"], np.inf, T[1],
            np.inf, np.inf, p["t0"] - 0.25 * p["dt"], T[-1] + 0.75 * p["dt"]]
    for b in range(B):
        idx = rng.choice(N, size=min(N, per_sample), replace=False)
        for i, v in zip(idx, vals):
            flat[b, i] = v
    return flat.reshape(t.shape).astype(np.float32)


def _window(p):
    return p["M"] * p["dt"]


def _conv_parity(dev, p, cs, t, W, label, bf16=False, need_t=True, seed=0):
    Wq = wl.bf16_round(W) if bf16 else W
    gpu, h = _gpu_forward(dev, p, cs, t, Wq, bf16=bf16)
    orc = oracle.conv_forward(p, cs, t, Wq)
    mask, stats = check_forward(gpu, orc, None, _window(p), label=label)
    g = np.random.default_rng(seed + 99).standard_normal(orc["t_out"].shape)
    g = np.where(mask, 0.0, g).astype(np.float32)
    gW, gx = _gpu_backward(dev, h, g, need_t=need_t)
    oW, ox, oWa, oxa = oracle.conv_backward(p, cs, t, Wq, orc,
                                            np.where(orc["q"] >= 0, g.astype(np.float64), 0.0),
                                            want_abs=True)
    check_grad(gW, oW, label + " dW", oWa)
    if need_t:
        kink = near_grid(t, p)
        check_grad(gx[~kink], ox[~kink], label + " dt_in", oxa[~kink])
    return gpu, orc, stats


# ------------------------------------------------------------ geometry ----
CASES = [
    # label, seed, B, conv shape, M, tau_m, tau_s, k
    ("3x3 s1 ragged, 2 channel tiles", 1, 3, _cs(5, 7, 9, 70), 8, 1.0, 0.3, 7.0),
    ("3x3 stride 2", 2, 2, _cs(6, 9, 11, 20, stride=2), 16, 1.0, 0.5, 7.0),
    ("2x2 event pool", 3, 2, _cs(7, 8, 10, 33, pool_in=2), 12, 1.0, 0.3, 7.0),
    ("global event pool 1x1", 4, 5, _cs(70, 3, 3, 10, K=1, pad=0, pool_in=0), 16, 1.5, 0.5, 6.0),
    ("wide fan-in (4 dW lane blocks)", 5, 2, _cs(100, 6, 5, 40), 32, 1.0, 0.3, 6.0),
    ("5x5 pad 2", 6, 2, _cs(3, 10, 9, 16, K=5), 8, 2.0, 0.4, 7.0),
    ("1x1 no pool", 7, 3, _cs(20, 5, 6, 12, K=1, pad=0), 10, 0.3, 1.0, 6.0),
    ("3x1 kernel, pad 0", 8, 2, _cs(9, 6, 7, 15, K=3, KW=1, pad=0), 9, 1.0, 0.3, 7.0),
    ("pool + stride 2 + M 64", 9, 2, _cs(12, 12, 8, 24, stride=2, pool_in=2), 64, 1.0, 0.3, 7.0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_conv_geometry(dev, case):
    label, seed, B, cs, M, tm, ts, k = case
    p, t, W = _conv_case(seed, B, cs, M, tm, ts, k=k)
    t = _special_inputs(t, p, np.random.default_rng(seed))
    _, orc, _ = _conv_parity(dev, p, cs, t, W, label, seed=seed)
    assert (orc["q"] >= 0).mean() > 0.1, "case should make neurons fire"


def test_conv_rows_past_64(dev):
    """M = 100 and 256: the bucket tables are walked in chunks of 64 rows."""
    for M, seed in [(100, 11), (256, 12)]:
        cs = _cs(6, 5, 6, 18)
        p, t, W = _conv_case(seed, 2, cs, M, 1.0, 0.3, k=7.0)
        _conv_parity(dev, p, cs, t, W, f"conv M={M}", seed=seed)


def test_conv_finite_t_max_and_offset_grid(dev):
    cs = _cs(8, 6, 6, 20)
    p, t, W = _conv_case(13, 2, cs, 16, 1.0, 0.3, k=5.0, t0=3.0, spread=1.1, t_max=4.3)
    _conv_parity(dev, p, cs, t, W, "conv t_max=4.3 t0=3")


def test_conv_bf16_weights(dev):
    cs = _cs(16, 6, 7, 32)
    p, t, W = _conv_case(14, 2, cs, 32, 2.0, 0.4, k=6.0)
    _conv_parity(dev, p, cs, t, W, "conv bf16 W", bf16=True)


def test_conv_silent_and_empty(dev):
    import torch
    from paper_2607_14672_amd import dstd
    cs = _cs(4, 5, 5, 6)
    prm = _prm(dict(tau_m=1.0, tau_s=0.3, threshold=1.0, M=8, t0=0.0, dt=0.125))
    c = dstd.make_conv_shape(**cs)
    # all inputs silent
    t = torch.full((2, 4, 5, 5), float("inf"), device=dev)
    W = torch.rand(6, 4, 3, 3, device=dev)
    to, sl, q = dstd.conv_forward(prm, c, t, W)
    gW, gx = dstd.conv_backward(prm, c, t, W, to, sl, q, torch.ones_like(to))
    torch.cuda.synchronize()
    assert torch.all(torch.isinf(to)) and torch.all(q == -1)
    assert torch.all(gW == 0) and torch.all(gx == 0)
    # empty batch: nothing to do, grad_W is zero
    t0 = torch.rand(0, 4, 5, 5, device=dev)
    to, sl, q = dstd.conv_forward(prm, c, t0, W)
    gW, gx = dstd.conv_backward(prm, c, t0, W, to, sl, q, torch.ones_like(to))
    torch.cuda.synchronize()
    assert to.shape == (0, 6, 5, 5) and torch.all(gW == 0)


def test_conv_deterministic(dev):
    cs = _cs(10, 8, 8, 24, pool_in=2)
    p, t, W = _conv_case(15, 3, cs, 16, 1.0, 0.3, k=7.0)
    a, h = _gpu_forward(dev, p, cs, t, W)
    b, _ = _gpu_forward(dev, p, cs, t, W)
    for key in a:
        assert np.array_equal(a[key], b[key])
    g = np.random.default_rng(0).standard_normal(a["t_out"].shape).astype(np.float32)
    r1 = _gpu_backward(dev, h, g)
    r2 = _gpu_backward(dev, h, g)
    assert np.array_equal(r1[0], r2[0]) and np.array_equal(r1[1], r2[1])


# ------------------------------------------------------- workload layers --
def _layer_inputs(lay, B, seed):
    """In-window inputs for one layer of a conv workload: t = t0 + U[0, 1)."""
    rng = np.random.default_rng(seed)
    return (lay.t0 + rng.random((B, lay.C_in, lay.H, lay.W))).astype(np.float32)


@pytest.mark.parametrize("name,l,B,k", [
    ("conv9", 1, 4, 7.0),    # 64 -> 64 at 32 x 32
    ("conv9", 2, 4, 7.0),    # 2x2 event pool, 64 -> 128 at 16 x 16
    ("conv20", 5, 8, 7.0),   # stride 2, 32 -> 32, 28 x 28 -> 14 x 14
    ("conv20", 19, 16, 6.0), # global event pool of 7 x 7 x 64, dense 64 -> 10
])
def test_workload_layer_shapes(dev, name, l, B, k):
    """Layer shapes of the conv workloads (the full channel and map sizes, a
    few samples), with in-window inputs and weights that make ~half fire."""
    w = wl.get(name)
    lay = w.layers[l]
    cs = lay.conv_shape()
    rng = np.random.default_rng(100 + l)
    fan = lay.C_in * lay.KH * lay.KW
    z = rng.standard_normal(lay.w_shape())
    W = ((k / fan) * (1 + 0.3 * math.sqrt(fan) * z)).astype(np.float32)
    t = _layer_inputs(lay, B, 200 + l)
    _conv_parity(dev, lay.params(), cs, t, W, f"{name} layer {l + 1}", seed=l)


def test_conv9_layer2_full_batch_sampled(dev):
    """conv9 layer 2 (64 -> 64, 32 x 32) at the full batch of 64 on the GPU;
    the oracle checks all outputs and dt_in of 3 sampled images, and dW on
    the gradient of those images alone (other images get zero upstream
    gradient on both sides)."""
    w = wl.get("conv9")
    lay = w.layers[1]
    cs = lay.conv_shape()
    rng = np.random.default_rng(7)
    fan = lay.C_in * lay.KH * lay.KW
    W = ((7.0 / fan) * (1 + 0.3 * math.sqrt(fan) * rng.standard_normal(lay.w_shape()))).astype(np.float32)
    t = _layer_inputs(lay, w.batch, 8)
    gpu, h = _gpu_forward(dev, lay.params(), cs, t, W)
    bsel = np.array([0, 31, 63])
    orc = oracle.conv_forward(lay.params(), cs, t[bsel], W)
    mask, _ = check_forward({k: v[bsel] for k, v in gpu.items()}, orc, None, 1.0,
                            label="conv9 layer 2 sampled images")
    g = np.zeros(gpu["t_out"].shape, dtype=np.float32)
    g[bsel] = np.where(mask, 0.0, rng.standard_normal(orc["t_out"].shape)).astype(np.float32)
    gW, gx = _gpu_backward(dev, h, g)
    oW, ox, oWa, oxa = oracle.conv_backward(lay.params(), cs, t[bsel], W, orc,
                                            np.where(orc["q"] >= 0, g[bsel].astype(np.float64), 0.0),
                                            want_abs=True)
    check_grad(gW, oW, "conv9 layer 2 dW (sampled images)", oWa)
    kink = near_grid(t[bsel], lay.params())
    check_grad(gx[bsel][~kink], ox[~kink], "conv9 layer 2 dt_in", oxa[~kink])
    others = np.setdiff1d(np.arange(w.batch), bsel)
    assert np.all(gx[others] == 0.0)
