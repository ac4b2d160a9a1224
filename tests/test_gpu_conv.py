"""GPU parity of the conv DSTD-LIF layer (with event pooling) against the fp64
oracle, through the C ABI."""
import math

import numpy as np
import pytest

import oracle
from paper_2607_14672_amd import workloads as wl
from tests.parity import check_forward, check_grad, grad_err_inputs, near_grid

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


def _taus(p):
    return (max(p["tau_m"], p["tau_s"]), min(p["tau_m"], p["tau_s"]))


def _n_terms(cs, B):
    """Upper bounds of the number of terms of a dW and of a dt_in element."""
    Ho, Wo = oracle.conv_out_hw(cs)
    P = {1: 1, 2: 4, 0: cs["H"] * cs["W"]}[cs["pool_in"]]
    return 2 * B * Ho * Wo * P, 2 * cs["C_out"] * cs["KH"] * cs["KW"]


def _conv_grad_check(p, cs, t, W, orc, mask, st, g_sel, gW, gx_sel, label):
    """Oracle backward on the (sampled) images t with upstream gradient
    g_sel, error-weighted sums from the forward's error model, and the
    per-element checks of dW and dt_in."""
    oW, ox, oWa, oxa, oWe, oxe = oracle.conv_backward(
        p, cs, t, W, orc, np.where(orc["q"] >= 0, g_sel.astype(np.float64), 0.0), want_abs=True,
        err=grad_err_inputs(st, mask))
    nW, nx = _n_terms(cs, t.shape[0])
    check_grad(gW, oW, label + " dW", oWa, oWe, n_terms=nW)
    if gx_sel is not None:
        kink = near_grid(t, p)
        check_grad(gx_sel[~kink], ox[~kink], label + " dt_in", oxa[~kink], oxe[~kink], n_terms=nx)


def _conv_parity(dev, p, cs, t, W, label, bf16=False, need_t=True, seed=0):
    Wq = wl.bf16_round(W) if bf16 else W
    gpu, h = _gpu_forward(dev, p, cs, t, Wq, bf16=bf16)
    orc = oracle.conv_forward(p, cs, t, Wq)
    mask, stats = check_forward(gpu, orc, None, _window(p), label=label, taus=_taus(p))
    g = np.random.default_rng(seed + 99).standard_normal(orc["t_out"].shape)
    g = np.where(mask, 0.0, g).astype(np.float32)
    gW, gx = _gpu_backward(dev, h, g, need_t=need_t)
    _conv_grad_check(p, cs, t, Wq, orc, mask, stats, g, gW, gx if need_t else None, label)
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
    # channel counts of the deep conv layers: 129-256 and > 256 output channels
    ("256 channels", 16, 2, _cs(24, 5, 6, 256), 32, 1.0, 0.3, 7.0),
    ("200 channels (ragged tile)", 17, 2, _cs(20, 6, 8, 200, pool_in=2), 16, 1.0, 0.3, 7.0),
    ("300 channels", 18, 2, _cs(16, 4, 5, 300), 16, 1.5, 0.5, 7.0),
    ("3 input channels, 64 out", 19, 2, _cs(3, 12, 10, 64), 32, 1.0, 0.3, 7.0),
    # two positions per wave (<= 32 channels, <= 32 event rows, <= 320 raw
    # inputs per receptive field): pooled input at the row limit M = 30 with
    # an odd number of positions (the last wave's second half is empty), and
    # a 5x5 kernel with 31 channels; M = 31 is one row past the limit
    ("paired: 2x2 pool, M 30, odd positions", 20, 1, _cs(8, 10, 14, 32, pool_in=2), 30, 1.0, 0.3, 7.0),
    ("paired: 5x5, 31 channels", 21, 3, _cs(4, 7, 9, 31, K=5), 24, 1.5, 0.5, 7.0),
    ("one position per wave at M 31", 22, 2, _cs(8, 6, 7, 32), 31, 1.0, 0.3, 7.0),
    # receptive fields small enough that the forward bins its inputs itself
    # (at most 32 raw inputs with two positions per wave, 64 with one), on
    # pooled input
    ("direct, paired: 1x1 on 2x2 pool", 23, 3, _cs(6, 8, 10, 20, K=1, pad=0, pool_in=2), 16, 1.0, 0.3, 6.0),
    ("direct: 3x3 on 2x2 pool, 1 input channel", 24, 3, _cs(1, 12, 10, 40, pool_in=2), 20, 1.0, 0.3, 14.0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_conv_geometry(dev, case):
    label, seed, B, cs, M, tm, ts, k = case
    p, t, W = _conv_case(seed, B, cs, M, tm, ts, k=k)
    t = _special_inputs(t, p, np.random.default_rng(seed))
    _, orc, _ = _conv_parity(dev, p, cs, t, W, label, seed=seed)
    assert (orc["q"] >= 0).mean() > 0.1, "case should make neurons fire"


_REUSE_CASES = [c for c in CASES if c[0] in (
    "3x3 s1 ragged, 2 channel tiles", "3x3 stride 2", "2x2 event pool", "global event pool 1x1",
    "256 channels", "paired: 2x2 pool, M 30, odd positions", "direct, paired: 1x1 on 2x2 pool",
    "direct: 3x3 on 2x2 pool, 1 input channel", "pool + stride 2 + M 64")]


@pytest.mark.parametrize("case", _REUSE_CASES, ids=[c[0] for c in _REUSE_CASES])
def test_conv_backward_reuses_kept_forward_sort(dev, case):
    """A forward with DSTD_FLAG_CONV_KEEP and a backward with
    DSTD_FLAG_CONV_REUSE on the same workspace give the plain calls' results
    bit for bit: forward outputs, dW and dt_in (the chunked, list and direct
    forwards, pooled and strided geometry, several channel tiles)."""
    import torch
    from paper_2607_14672_amd import dstd
    label, seed, B, cs, M, tm, ts, k = case
    p, t, W = _conv_case(seed, B, cs, M, tm, ts, k=k)
    t = _special_inputs(t, p, np.random.default_rng(seed))
    plain, (prm, c, tt, Wt, to, sl, q) = _gpu_forward(dev, p, cs, t, W)
    g = np.random.default_rng(seed + 5).standard_normal(plain["t_out"].shape).astype(np.float32)
    gW0, gx0 = _gpu_backward(dev, (prm, c, tt, Wt, to, sl, q), g)
    keep, reuse = _prm(p), _prm(p)
    keep.flags = dstd.DSTD_FLAG_CONV_KEEP
    reuse.flags = dstd.DSTD_FLAG_CONV_REUSE
    ws = dstd.workspace(dstd.dstd_lif_conv_backward_workspace_size(reuse, c, B), dev)
    ws.fill_(0x7f)  # stale contents must not matter
    to2, sl2, q2 = dstd.conv_forward(keep, c, tt, Wt, ws=ws)
    gt = torch.from_numpy(g).to(dev)
    gW, gx = dstd.conv_backward(reuse, c, tt, Wt, to2, sl2, q2, gt, ws=ws)
    torch.cuda.synchronize()
    assert np.array_equal(to2.cpu().numpy(), plain["t_out"])
    assert np.array_equal(sl2.cpu().numpy(), plain["slope"])
    assert np.array_equal(q2.cpu().numpy(), plain["q"])
    assert np.array_equal(gW.cpu().numpy(), gW0), label
    assert np.array_equal(gx.cpu().numpy(), gx0), label


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
    ("conv9", 0, 4, 7.0),    # 3 -> 64 at 32 x 32 (fan-in 27)
    ("conv9", 1, 4, 7.0),    # 64 -> 64 at 32 x 32
    ("conv9", 2, 4, 7.0),    # 2x2 event pool, 64 -> 128 at 16 x 16
    ("conv9", 3, 4, 7.0),    # 128 -> 128 at 16 x 16
    ("conv9", 4, 4, 7.0),    # 2x2 event pool, 128 -> 256 at 8 x 8
    ("conv9", 5, 4, 7.0),    # 256 -> 256 at 8 x 8 (fan-in 2304)
    ("conv9", 6, 6, 7.0),    # 2x2 event pool, 256 -> 256 at 4 x 4
    ("conv9", 7, 6, 7.0),    # 256 -> 256 at 4 x 4
    ("conv20", 0, 4, 7.0),   # 1 -> 32 at 28 x 28 (fan-in 9)
    ("conv20", 5, 8, 7.0),   # stride 2, 32 -> 32, 28 x 28 -> 14 x 14
    ("conv20", 10, 8, 7.0),  # 32 -> 64 at 14 x 14
    ("conv20", 12, 8, 7.0),  # stride 2, 64 -> 64, 14 x 14 -> 7 x 7
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
    p = lay.params()
    orc = oracle.conv_forward(p, cs, t[bsel], W)
    mask, st = check_forward({k: v[bsel] for k, v in gpu.items()}, orc, None, 1.0,
                             label="conv9 layer 2 sampled images", taus=_taus(p))
    g = np.zeros(gpu["t_out"].shape, dtype=np.float32)
    g[bsel] = np.where(mask, 0.0, rng.standard_normal(orc["t_out"].shape)).astype(np.float32)
    gW, gx = _gpu_backward(dev, h, g)
    _conv_grad_check(p, cs, t[bsel], W, orc, mask, st, g[bsel], gW, gx[bsel],
                     "conv9 layer 2 (sampled images)")
    others = np.setdiff1d(np.arange(w.batch), bsel)
    assert np.all(gx[others] == 0.0)


@pytest.mark.parametrize("l,bsel", [(4, (0, 40, 63)), (6, (5, 62))])
def test_conv9_deep_layer_full_batch_sampled(dev, l, bsel):
    """conv9 layers 5 (pool, 128 -> 256 at 8 x 8) and 7 (pool, 256 -> 256 at
    4 x 4) at the full batch of 64 on the GPU, the launch configuration of
    the timed step; the oracle checks the sampled images."""
    w = wl.get("conv9")
    lay = w.layers[l]
    cs = lay.conv_shape()
    rng = np.random.default_rng(70 + l)
    fan = lay.C_in * lay.KH * lay.KW
    W = ((7.0 / fan) * (1 + 0.3 * math.sqrt(fan) * rng.standard_normal(lay.w_shape()))).astype(np.float32)
    t = _layer_inputs(lay, w.batch, 80 + l)
    gpu, h = _gpu_forward(dev, lay.params(), cs, t, W)
    bsel = np.array(bsel)
    p = lay.params()
    orc = oracle.conv_forward(p, cs, t[bsel], W)
    mask, st = check_forward({k: v[bsel] for k, v in gpu.items()}, orc, None, 1.0,
                             label=f"conv9 layer {l + 1} sampled images", taus=_taus(p))
    g = np.zeros(gpu["t_out"].shape, dtype=np.float32)
    g[bsel] = np.where(mask, 0.0, rng.standard_normal(orc["t_out"].shape)).astype(np.float32)
    gW, gx = _gpu_backward(dev, h, g)
    _conv_grad_check(p, cs, t[bsel], W, orc, mask, st, g[bsel], gW, gx[bsel],
                     f"conv9 layer {l + 1} (sampled images)")
