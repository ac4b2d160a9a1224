"""GPU parity of the dense DSTD-LIF layer against the fp64 oracle (through the C ABI)."""
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


def _gpu_forward(dev, p, t_in, W, bf16=False):
    import torch
    from paper_2607_14672_amd import dstd
    prm = dstd.make_params(p["tau_m"], p["tau_s"], p["threshold"], p["M"], p["t0"], p["dt"],
                           p.get("t_max", math.inf), p.get("flags", 0))
    tt = torch.from_numpy(np.ascontiguousarray(t_in, dtype=np.float32)).to(dev)
    Wt = torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).to(dev)
    if bf16:
        Wt = Wt.to(torch.bfloat16)
    to, sl, q = dstd.forward(prm, tt, Wt)
    torch.cuda.synchronize()
    return dict(t_out=to.cpu().numpy(), slope=sl.cpu().numpy(), q=q.cpu().numpy()), (prm, tt, Wt,
                                                                                      to, sl, q)


def _gpu_backward(dev, handles, g, need_W=True, need_t=True):
    import torch
    from paper_2607_14672_amd import dstd
    prm, tt, Wt, to, sl, q = handles
    gt = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(dev)
    gW, gx = dstd.backward(prm, tt, Wt, to, sl, q, gt, need_W=need_W, need_t_in=need_t)
    torch.cuda.synchronize()
    return (None if gW is None else gW.cpu().numpy()), (None if gx is None else gx.cpu().numpy())


def _window(p):
    return p["M"] * p["dt"]


def _taus(p):
    return (max(p["tau_m"], p["tau_s"]), min(p["tau_m"], p["tau_s"]))


def _layer_case(seed, B, N_in, N_out, M, tm, ts, k=6.0, t0=0.0, t_max=math.inf, spread=1.0):
    rng = np.random.default_rng(seed)
    p = dict(tau_m=tm, tau_s=ts, threshold=1.0, M=M, t0=t0, dt=1.0 / M, t_max=t_max)
    t = (t0 + spread * rng.random((B, N_in))).astype(np.float32)
    W = ((k / N_in) * (1 + 0.3 * math.sqrt(N_in) * rng.standard_normal((N_out, N_in)))).astype(np.float32)
    return p, t, W


def _special_inputs(t, p, rng):
    """Silent, NaN, -inf, out-of-grid, exactly-on-grid and grid-end inputs."""
    t = t.copy()
    B, N = t.shape
    T = p["t0"] + p["dt"] * np.arange(p["M"] + 1)
    for b in range(B):
        idx = rng.choice(N, size=min(N, 12), replace=False)
        vals = [np.inf, np.nan, -np.inf, p["t0"] - 3 * p["dt"], T[-1] + 2 * p["dt"],
                T[0], T[-1], T[len(T) // 2], p["t0"] - 0.5 * p["dt"], T[-1] + 0.5 * p["dt"],
                np.inf, T[1]]
        for i, v in zip(idx, vals):
            t[b, i] = v
    return t.astype(np.float32)


def _fwd_bwd_parity(dev, p, t, W, label, bf16=False, need_t=True, seed=0):
    Wq = wl.bf16_round(W) if bf16 else W
    gpu, h = _gpu_forward(dev, p, t, Wq, bf16=bf16)
    orc = oracle.dstd_forward(p, t, Wq)
    mask, st = check_forward(gpu, orc, t.shape[1], _window(p), label=label, taus=_taus(p))
    g = np.random.default_rng(seed + 99).standard_normal(orc["t_out"].shape)
    g = np.where(mask, 0.0, g).astype(np.float32)
    gW, gx = _gpu_backward(dev, h, g, need_t=need_t)
    g64 = g.astype(np.float64)
    oW, ox, oWa, oxa, oWe, oxe = oracle.dstd_backward(
        p, t, Wq, orc, np.where(orc["q"] >= 0, g64, 0.0), want_dt=need_t, want_abs=True,
        err=grad_err_inputs(st, mask))
    B, N_out = orc["q"].shape
    check_grad(gW, oW, label + " dW", oWa, oWe, n_terms=2 * B)
    if need_t:
        kink = near_grid(t, p)
        check_grad(gx[~kink], ox[~kink], label + " dt_in", oxa[~kink], oxe[~kink], n_terms=2 * N_out)
    return gpu, orc


# ------------------------------------------------------------- forward ----
@pytest.mark.parametrize("M,tm,ts", [(8, 1.0, 0.3), (16, 1.0, 0.5), (13, 2.0, 0.4), (32, 1.5, 0.5),
                                     (5, 0.3, 1.0)])
def test_small_ragged_layer(dev, M, tm, ts):
    p, t, W = _layer_case(M, 5, 37, 70, M, tm, ts, k=8.0)
    t = _special_inputs(t, p, np.random.default_rng(M))
    _fwd_bwd_parity(dev, p, t, W, f"ragged M={M} tau=({tm},{ts})", seed=M)


def test_multi_tile_ragged(dev):
    p, t, W = _layer_case(3, 9, 530, 200, 24, 1.0, 0.3, k=7.0, t0=2.0, spread=1.2)
    _fwd_bwd_parity(dev, p, t, W, "multi-tile B=9 530->200 M=24")


def test_finite_t_max(dev):
    p, t, W = _layer_case(4, 6, 100, 130, 16, 1.0, 0.3, k=5.0, t_max=1.4)
    _fwd_bwd_parity(dev, p, t, W, "t_max=1.4")


def test_max_M(dev):
    p, t, W = _layer_case(5, 4, 300, 65, 256, 1.0, 0.3, k=7.0)
    _fwd_bwd_parity(dev, p, t, W, "M=256")


def test_bf16_weights(dev):
    p, t, W = _layer_case(6, 6, 256, 96, 32, 2.0, 0.4, k=6.0)
    _fwd_bwd_parity(dev, p, t, W, "bf16 W", bf16=True)


def test_single_input_and_silent_layer(dev):
    p = dict(tau_m=1.0, tau_s=0.3, threshold=1.0, M=8, t0=0.0, dt=0.125)
    t = np.array([[0.25], [np.inf], [0.3]], dtype=np.float32)
    kmax = 0.3 * (0.3 / 1.0) ** (0.3 / 0.7)
    W = np.array([[1.2 / kmax], [0.8 / kmax]], dtype=np.float32)
    gpu, _ = _gpu_forward(dev, p, t, W)
    orc = oracle.dstd_forward(p, t, W)
    check_forward(gpu, orc, 1, 1.0, label="single input", taus=_taus(p))
    assert gpu["q"][1, 0] == -1 and gpu["q"][1, 1] == -1
    assert gpu["q"][0, 1] == -1 and gpu["q"][0, 0] >= 0


def test_empty_shapes(dev):
    import torch
    from paper_2607_14672_amd import dstd
    prm = dstd.make_params(1.0, 0.3, 1.0, 8, 0.0, 0.125)
    for B, N_in, N_out in [(0, 10, 5), (3, 0, 5), (3, 10, 0)]:
        t = torch.rand(B, N_in, device=dev)
        W = torch.rand(N_out, N_in, device=dev)
        to, sl, q = dstd.forward(prm, t, W)
        g = torch.ones_like(to)
        gW, gx = dstd.backward(prm, t, W, to, sl, q, g)
        torch.cuda.synchronize()
        if B * N_out:
            assert torch.all(torch.isinf(to)) and torch.all(q == -1)
        assert torch.all(gW == 0)
        assert torch.all(gx == 0)


def test_deterministic(dev):
    p, t, W = _layer_case(7, 8, 400, 300, 16, 1.0, 0.3, k=7.0)
    a, h = _gpu_forward(dev, p, t, W)
    b, _ = _gpu_forward(dev, p, t, W)
    for k in a:
        assert np.array_equal(a[k], b[k])
    g = np.random.default_rng(0).standard_normal(a["t_out"].shape).astype(np.float32)
    r1 = _gpu_backward(dev, h, g)
    r2 = _gpu_backward(dev, h, g)
    assert np.array_equal(r1[0], r2[0]) and np.array_equal(r1[1], r2[1])


# ------------------------------------------------------- workload layers --
def test_dense1_as_stated_is_silent(dev):
    w = wl.get("dense1")
    d = wl.Draws(w)
    lay = w.layers[0]
    W = d.weights(0)
    gpu, _ = _gpu_forward(dev, lay.params(), d.t_in, W)
    orc = oracle.dstd_forward(lay.params(), d.t_in, W)
    check_forward(gpu, orc, lay.n_in, 1.0, label="dense1 as stated", taus=_taus(lay.params()))
    assert (orc["q"] < 0).all() and (gpu["q"] < 0).all()


def test_dense1_calibrated(dev):
    w = wl.get("dense1-cal")
    d = wl.Draws(w)
    lay = w.layers[0]
    _fwd_bwd_parity(dev, lay.params(), d.t_in, d.weights(0), "dense1-cal", need_t=True)


def test_mlp3_layers_teacher_forced(dev):
    """Each layer receives the oracle's fp32-rounded spike times of the layer
    below, so one ambiguous neuron cannot cascade across layers."""
    w = wl.get("mlp3")
    d = wl.Draws(w)
    t = d.t_in
    for l, lay in enumerate(w.layers):
        W = d.weights(l)
        _, orc = _fwd_bwd_parity(dev, lay.params(), t, W, f"mlp3 layer {l + 1}", need_t=l > 0,
                                 seed=l)
        t = orc["t_out"].astype(np.float32)


def test_conv9_dense_head(dev):
    """The dense output layer of the 9-layer conv workload at its full batch
    (4096 -> 10, B 64, M 32), with in-window inputs. (The 20-layer workload's
    head is a conv layer with global event pooling, tested with the conv
    layers.)"""
    name, l = "conv9", 8
    w = wl.get(name)
    lay = w.layers[l]
    p = lay.params()
    rng = np.random.default_rng(300 + l)
    t = (lay.t0 + rng.random((w.batch, lay.n_in))).astype(np.float32)
    W = ((6.0 / lay.n_in) * (1 + 0.3 * math.sqrt(lay.n_in) *
                              rng.standard_normal((lay.n_out, lay.n_in)))).astype(np.float32)
    _fwd_bwd_parity(dev, p, t, W, f"{name} dense head {lay.n_in}->{lay.n_out}", seed=l)


@pytest.mark.parametrize("M,flags", [(8, 0), (32, 0), (64, 0), (128, 0), (8, 0x2), (32, 0x4)],
                         ids=["M8-auto", "M32-auto", "M64-auto", "M128-auto", "M8-sparse", "M32-mfma"])
def test_wide_layer_full_size_sampled(dev, M, flags):
    """Full 256 x 4096 -> 4096 layer on the GPU; oracle on sampled rows: all
    neurons of 4 samples (forward, dt_in) and 8 neurons over the whole batch
    (forward, dW). The automatic contraction choice takes the MFMA product at
    M = 8; the forced cases run the other path at M = 8 and the MFMA product
    at M = 32."""
    w = wl.get(f"wide-M{M}")
    d = wl.Draws(w)
    lay = w.layers[0]
    p = dict(lay.params(), flags=flags)
    W = d.weights(0)
    import torch
    gpu, h = _gpu_forward(dev, p, d.t_in, W, bf16=True)
    rng = np.random.default_rng(M)
    g = rng.standard_normal(gpu["t_out"].shape)
    bsel = np.array([0, 77, 128, 255])
    isel = np.array([0, 1, 999, 2048, 3071, 4000, 4094, 4095])
    # sampled forward + masks from the oracle
    orc_b = oracle.dstd_forward(p, d.t_in[bsel], W)
    mask_b, st_b = check_forward({k: v[bsel] for k, v in gpu.items()}, orc_b, lay.n_in, 1.0,
                                 label=f"wide M={M} rows", taus=_taus(p))
    orc_i = oracle.dstd_forward(p, d.t_in, W[isel])
    mask_i, st_i = check_forward({k: v[:, isel] for k, v in gpu.items()}, orc_i, lay.n_in, 1.0,
                                 label=f"wide M={M} cols", taus=_taus(p))
    # full-batch mask for the GPU side: zero g wherever either sample found an
    # excluded neuron; neurons never sampled keep their g (they only enter the
    # sampled dt_in rows through their own sample, whose full row is checked)
    gm = g.copy()
    gm[bsel] = np.where(mask_b, 0.0, gm[bsel])
    gm[:, isel] = np.where(mask_i, 0.0, gm[:, isel])
    gm = gm.astype(np.float32)
    gW, gx = _gpu_backward(dev, h, gm)
    oW, _, oWa, _, oWe, _ = oracle.dstd_backward(
        p, d.t_in, W[isel], orc_i, np.where(orc_i["q"] >= 0, gm[:, isel].astype(np.float64), 0.0),
        want_dt=False, want_abs=True, err=grad_err_inputs(st_i, mask_i))
    B = d.t_in.shape[0]
    check_grad(gW[isel], oW, f"wide M={M} dW rows", oWa, oWe, n_terms=2 * B)
    _, ox, _, oxa, _, oxe = oracle.dstd_backward(
        p, d.t_in[bsel], W, orc_b, np.where(orc_b["q"] >= 0, gm[bsel].astype(np.float64), 0.0),
        want_dW=False, want_abs=True, err=grad_err_inputs(st_b, mask_b))
    kink = near_grid(d.t_in[bsel], p)
    check_grad(gx[bsel][~kink], ox[~kink], f"wide M={M} dt_in rows", oxa[~kink], oxe[~kink],
               n_terms=2 * W.shape[0])
    del torch


# ---------------------------------------------------------------- losses --
@pytest.mark.parametrize("B,N", [(37, 10), (300, 64), (50, 65), (1024, 64), (1025, 64)])
def test_softmax_ce_grad(dev, B, N):
    import torch
    from paper_2607_14672_amd import dstd
    rng = np.random.default_rng(1 + B + N)
    t = rng.random((B, N)).astype(np.float32) * 2 + 1
    t[rng.random((B, N)) < 0.2] = np.inf
    lab = rng.integers(0, N, B).astype(np.int32)
    tau, cap = 0.7, 4.0
    g, loss = dstd.softmax_ce_grad(torch.from_numpy(t).to(dev), torch.from_numpy(lab).to(dev),
                                   tau, cap)
    tt = np.where(np.isfinite(t), t, cap).astype(np.float64)
    z = -tt / tau
    s = np.exp(z - z.max(1, keepdims=True))
    s /= s.sum(1, keepdims=True)
    ref_loss = -np.mean(np.log(s[np.arange(B), lab]))
    onehot = np.eye(N)[lab]
    ref_g = np.where(np.isfinite(t), -(s - onehot) / tau / B, 0.0)
    np.testing.assert_allclose(g.cpu().numpy(), ref_g, rtol=1e-5, atol=1e-7)
    loss = loss.cpu().numpy()
    assert float(loss[0]) == pytest.approx(ref_loss, rel=1e-5)
    per = -np.log(s[np.arange(B), lab]) / B
    np.testing.assert_allclose(loss[1:], per, rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("B,N", [(21, 100), (21, 64), (1024, 64), (7, 3)])
def test_mse_grad(dev, B, N):
    import torch
    from paper_2607_14672_amd import dstd
    rng = np.random.default_rng(2 + B + N)
    t = (rng.random((B, N)) * 2).astype(np.float32)
    t[rng.random((B, N)) < 0.3] = np.inf
    y = (1 + rng.random((B, N))).astype(np.float32)
    g, loss = dstd.mse_grad(torch.from_numpy(t).to(dev), torch.from_numpy(y).to(dev))
    f = np.isfinite(t)
    d = np.where(f, t.astype(np.float64) - y, 0.0)
    np.testing.assert_allclose(g.cpu().numpy(), d / B, rtol=1e-6, atol=1e-8)
    loss = loss.cpu().numpy()
    assert float(loss[0]) == pytest.approx(0.5 * np.sum(d * d) / B, rel=1e-5)
    np.testing.assert_allclose(loss[1:], 0.5 * np.sum(d * d, axis=1) / B, rtol=1e-5, atol=1e-8)


@pytest.mark.parametrize("B,N", [(3, 4096), (256, 4096), (1, 1)])
def test_loss_kernels_wide(dev, B, N):
    """Many outputs per sample (the 4096-wide layer) and tiny shapes."""
    import torch
    from paper_2607_14672_amd import dstd
    rng = np.random.default_rng(B + N)
    t = (rng.random((B, N)) * 2).astype(np.float32)
    t[rng.random((B, N)) < 0.3] = np.inf
    y = (1 + rng.random((B, N))).astype(np.float32)
    g, loss = dstd.mse_grad(torch.from_numpy(t).to(dev), torch.from_numpy(y).to(dev))
    d = np.where(np.isfinite(t), t.astype(np.float64) - y, 0.0)
    np.testing.assert_allclose(g.cpu().numpy(), d / B, rtol=1e-6, atol=1e-9)
    assert float(loss[0].cpu()) == pytest.approx(0.5 * np.sum(d * d) / B, rel=1e-5)
    lab = rng.integers(0, N, B).astype(np.int32)
    g2, loss2 = dstd.softmax_ce_grad(torch.from_numpy(t).to(dev), torch.from_numpy(lab).to(dev),
                                     0.5, 5.0)
    tt = np.where(np.isfinite(t), t, 5.0).astype(np.float64)
    z = -tt / 0.5
    sm = np.exp(z - z.max(1, keepdims=True))
    sm /= sm.sum(1, keepdims=True)
    ref_g = np.where(np.isfinite(t), -(sm - np.eye(N)[lab]) / 0.5 / B, 0.0)
    np.testing.assert_allclose(g2.cpu().numpy(), ref_g, rtol=1e-4, atol=1e-9)
    assert float(loss2[0].cpu()) == pytest.approx(-np.mean(np.log(sm[np.arange(B), lab])), rel=1e-5)
