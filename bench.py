"""DSTD-LIF training-step benchmark on one MI355X.

A step is one forward + backward pass of the whole workload: every layer's
spike binning, event contraction, interval scan and root solve, the loss
gradient on the output spike times, and every layer's backward (dL/dW for
all layers, dL/dt_in for all but the first). All of it runs in the HIP
library through its C ABI; inputs, weights, outputs and workspaces are
allocated before the timed region.

Prints ONE JSON line (rank 0) with the throughput in samples/s, the roofline
of the dominant kernel (timed with the library's hipEvent timer on the stream
the kernels run on) and the fp64 CPU oracle timed on the host as a baseline.

  python bench.py [--steps K] [--warmup W] [--workload conv9] [--no-configs]
"""
from __future__ import annotations

import argparse
import hashlib
import glob
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "DSTD LIF fwd+bwd samples/s; % MFMA peak (GEMM) and % HBM peak (scan)"
# MI355X published peaks (dense, per GPU)
PEAK_FP32_VECTOR_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
PEAK_BF16_MFMA_TFLOPS = 2500.0
# algorithmic flops per (sample, input with events, neuron) update: the two
# halves of an event are multiplied by the weight and added to two bins
FLOPS_PER_UPDATE = 4
# algorithmic flops of the interval scan per (neuron, grid point): the state
# recurrences V <- alpha V + K(dt) I (a multiply and an FMA) and I <- beta I + w
# (an add and a multiply), and the interval bound max(V,0) + max(I,0) K_max
# (an FMA); the forward kernels fuse it with the contraction
FLOPS_PER_SCAN_STEP = 7


def kernel_source_sha():
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2607_14672_amd", "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


class Net:
    """Preallocated buffers and raw C-ABI calls for one workload."""

    def __init__(self, wl, dev, contract="auto"):
        import torch
        from paper_2607_14672_amd import dstd, workloads
        self.torch, self.dstd, self.wl, self.dev = torch, dstd, wl, dev
        d = workloads.Draws(wl)
        self.draws = d
        B = wl.batch
        self.B = B
        self.stream = torch.cuda.current_stream(dev).cuda_stream
        self.t0 = torch.from_numpy(d.t_in).to(dev)
        self.L = []
        t_prev = self.t0
        for l, lay in enumerate(wl.layers):
            W = torch.from_numpy(d.weights(l)).to(dev)
            if lay.w_dtype == "bf16":
                W = W.to(torch.bfloat16)
            flags = 0
            if lay.kind != "conv":
                flags = {"auto": 0, "sparse": dstd.DSTD_FLAG_CONTRACT_SPARSE,
                         "mfma": dstd.DSTD_FLAG_CONTRACT_MFMA}[contract]
            p = dstd.make_params(lay.tau_m, lay.tau_s, lay.threshold, lay.M, lay.t0, lay.dt,
                                 lay.t_max, flags)
            p_b = p
            if lay.kind == "conv" and l > 0:
                # the forward keeps its binned, sorted inputs in the backward's
                # workspace, and the backward reuses them (the first layer's
                # backward computes no dt_in, so it needs no sort)
                p = dstd.make_params(lay.tau_m, lay.tau_s, lay.threshold, lay.M, lay.t0, lay.dt,
                                     lay.t_max, dstd.DSTD_FLAG_CONV_KEEP)
                p_b = dstd.make_params(lay.tau_m, lay.tau_s, lay.threshold, lay.M, lay.t0, lay.dt,
                                       lay.t_max, dstd.DSTD_FLAG_CONV_REUSE)
            skip = None
            if lay.skip_back:
                # SD block's third layer: t_in = cat(block input + delay, t_prev)
                src = l - lay.skip_back
                blk_in = self.t0 if src < 0 else self.L[src]["t_out"]
                C1 = lay.C_in - t_prev.shape[1]
                cat = torch.empty((B, lay.C_in, lay.H, lay.W), dtype=torch.float32, device=dev)
                skip = dict(src=src, t1=blk_in, C1=C1, C2=t_prev.shape[1], HW=lay.H * lay.W,
                            t2=t_prev, cat=cat, g_cat=torch.empty_like(cat))
                t_prev = cat
            if lay.kind == "conv":
                cs = dstd.make_conv_shape(**lay.conv_shape())
                out_shape = (B, lay.C_out) + dstd.conv_out_hw(cs)
                t_in = t_prev.reshape(B, lay.C_in, lay.H, lay.W)
                ws_f = dstd.dstd_lif_conv_forward_workspace_size(p, cs, B)
                ws_b = dstd.dstd_lif_conv_backward_workspace_size(p_b, cs, B)
            else:
                cs = None
                out_shape = (B, lay.n_out)
                t_in = t_prev.reshape(B, lay.n_in)
                ws_f = dstd.dstd_lif_forward_workspace_size(p, B, lay.n_in, lay.n_out)
                ws_b = dstd.dstd_lif_backward_workspace_size(p, B, lay.n_in, lay.n_out)
            e = dict(lay=lay, p=p, p_b=p_b, cs=cs, W=W,
                     wdt=dstd.DSTD_BF16 if lay.w_dtype == "bf16" else dstd.DSTD_F32,
                     t_in=t_in,
                     t_out=torch.empty(out_shape, dtype=torch.float32, device=dev),
                     slope=torch.empty(out_shape, dtype=torch.float32, device=dev),
                     q=torch.empty(out_shape, dtype=torch.int32, device=dev),
                     g_out=torch.empty(out_shape, dtype=torch.float32, device=dev),
                     gW=torch.empty(tuple(W.shape), dtype=torch.float32, device=dev))
            e["ws_b"] = dstd.workspace(ws_b, dev)
            # a keeping forward writes into the backward's workspace
            keeps = cs is not None and (p.flags & dstd.DSTD_FLAG_CONV_KEEP) != 0
            e["ws_f"] = e["ws_b"] if keeps else dstd.workspace(ws_f, dev)
            e["skip"] = skip
            self.L.append(e)
            t_prev = e["t_out"]
        # the skip channels' gradient joins the block input's gradient once the
        # block's first layer has written its dt_in there
        self.skip_adds = {}
        for l in range(1, len(self.L)):
            sk = self.L[l]["skip"]
            self.L[l]["g_in_buf"] = sk["g_cat"] if sk else self.L[l - 1]["g_out"]
            if sk and sk["src"] >= 0:
                self.skip_adds.setdefault(sk["src"] + 1, []).append(l)
        last = wl.layers[-1]
        self.t_cap = float(last.t0 + last.M * last.dt + 2.0)
        if wl.loss == "ce":
            self.labels = torch.from_numpy(d.labels).to(dev)
        else:
            self.targets = torch.from_numpy(d.targets).to(dev)
        self.loss = torch.empty((B + 1,), dtype=torch.float32, device=dev)  # total, per sample

    def _ck(self, name, st):
        if st != 0:
            raise self.dstd.DSTDError(name, st)

    def forward(self):
        for l in range(len(self.L)):
            self.forward_layer(l)

    def forward_layer(self, l):
        ds = self.dstd
        e = self.L[l]
        lay = e["lay"]
        sk = e["skip"]
        if sk is not None:
            self._ck("dstd_skip_delay_concat", ds.dstd_skip_delay_concat(
                self.B, sk["C1"], sk["C2"], sk["HW"], sk["t1"].data_ptr(), lay.skip_delay,
                sk["t2"].data_ptr(), sk["cat"].data_ptr(), self.stream))
        if e["cs"] is not None:
            self._ck("dstd_lif_conv_forward", ds.dstd_lif_conv_forward(
                e["p"], e["cs"], self.B, e["t_in"].data_ptr(), e["W"].data_ptr(), e["wdt"],
                e["t_out"].data_ptr(), e["slope"].data_ptr(), e["q"].data_ptr(),
                e["ws_f"].data_ptr(), e["ws_f"].numel(), self.stream))
            return
        self._ck("dstd_lif_forward", ds.dstd_lif_forward(
            e["p"], self.B, lay.n_in, lay.n_out, e["t_in"].data_ptr(), e["W"].data_ptr(), e["wdt"],
            e["t_out"].data_ptr(), e["slope"].data_ptr(), e["q"].data_ptr(),
            e["ws_f"].data_ptr(), e["ws_f"].numel(), self.stream))

    def loss_grad(self):
        ds = self.dstd
        e = self.L[-1]
        if self.wl.loss == "ce":
            self._ck("dstd_softmax_ce_grad", ds.dstd_softmax_ce_grad(
                self.B, e["lay"].n_out, e["t_out"].data_ptr(), self.labels.data_ptr(), 1.0, self.t_cap,
                e["g_out"].data_ptr(), self.loss.data_ptr(), self.stream))
        else:
            self._ck("dstd_mse_grad", ds.dstd_mse_grad(
                self.B, e["lay"].n_out, e["t_out"].data_ptr(), self.targets.data_ptr(),
                e["g_out"].data_ptr(), self.loss.data_ptr(), self.stream))

    def backward(self):
        ds = self.dstd
        for l in reversed(range(len(self.L))):
            self.backward_layer(l)
            sk = self.L[l]["skip"]
            if sk is not None:  # the second layer's share of the concatenated input's gradient
                self._ck("dstd_skip_delay_concat_backward", ds.dstd_skip_delay_concat_backward(
                    self.B, sk["C1"], sk["C2"], sk["HW"], sk["g_cat"].data_ptr(), None, 0,
                    self.L[l - 1]["g_out"].data_ptr(), self.stream))
            for m in self.skip_adds.get(l, ()):  # the block input's share, added
                sm = self.L[m]["skip"]
                self._ck("dstd_skip_delay_concat_backward", ds.dstd_skip_delay_concat_backward(
                    self.B, sm["C1"], sm["C2"], sm["HW"], sm["g_cat"].data_ptr(),
                    self.L[sm["src"]]["g_out"].data_ptr(), 1, None, self.stream))

    def backward_layer(self, l):
        ds = self.dstd
        e = self.L[l]
        lay = e["lay"]
        g_in = e["g_in_buf"].data_ptr() if l > 0 else None
        if e["cs"] is not None:
            self._ck("dstd_lif_conv_backward", ds.dstd_lif_conv_backward(
                e["p_b"], e["cs"], self.B, e["t_in"].data_ptr(), e["W"].data_ptr(), e["wdt"],
                e["t_out"].data_ptr(), e["slope"].data_ptr(), e["q"].data_ptr(),
                e["g_out"].data_ptr(), e["gW"].data_ptr(), g_in, e["ws_b"].data_ptr(),
                e["ws_b"].numel(), self.stream))
            return
        self._ck("dstd_lif_backward", ds.dstd_lif_backward(
            e["p"], self.B, lay.n_in, lay.n_out, e["t_in"].data_ptr(), e["W"].data_ptr(), e["wdt"],
            e["t_out"].data_ptr(), e["slope"].data_ptr(), e["q"].data_ptr(), e["g_out"].data_ptr(),
            e["gW"].data_ptr(), g_in, e["ws_b"].data_ptr(), e["ws_b"].numel(), self.stream))

    def step(self):
        self.forward()
        self.loss_grad()
        self.backward()

    def capture(self, warmup=3):
        """Record one whole step into a HIP graph (the library's calls are
        asynchronous, allocate nothing and use no memset, so they capture)."""
        torch = self.torch
        eager = self.stream
        side = torch.cuda.Stream(self.dev)
        side.wait_stream(torch.cuda.current_stream(self.dev))
        with torch.cuda.stream(side):
            self.stream = side.cuda_stream
            for _ in range(warmup):
                self.step()
        torch.cuda.current_stream(self.dev).wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        try:
            with torch.cuda.graph(graph):
                self.stream = torch.cuda.current_stream(self.dev).cuda_stream
                self.step()
        finally:
            self.stream = eager
        return graph

    def activity(self):
        """Per layer: inputs with events (in-grid), fraction of neurons firing."""
        out = []
        for e in self.L:
            lay = e["lay"]
            t = e["t_in"].float().cpu().numpy()
            lo, hi = lay.t0 - lay.dt, lay.t0 + (lay.M + 1) * lay.dt
            ing = np.isfinite(t) & (t >= lo) & (t < hi)
            q = e["q"].cpu().numpy()
            out.append(dict(in_grid_inputs=int(ing.sum()), in_grid_frac=float(ing.mean()),
                            fire_frac=float((q >= 0).mean()),
                            updates=int(event_updates(lay, ing))))
        return out


def layer_profile(net, dstd, torch, reps=5):
    """Per layer: milliseconds of each library kernel in its forward and its
    backward (hipEvent timer, mean over reps full steps)."""
    out = [dict(fwd={}, bwd={}) for _ in net.L]

    def timed(fn, into):
        dstd.dstd_profile_reset()
        dstd.dstd_profile_enable(True)
        fn()
        torch.cuda.synchronize()
        dstd.dstd_profile_enable(False)
        for k, v in dstd.profile_table().items():
            into[k] = into.get(k, 0.0) + v[1] / reps

    for _ in range(reps):
        for l in range(len(net.L)):
            timed(lambda: net.forward_layer(l), out[l]["fwd"])
        net.loss_grad()
        for l in reversed(range(len(net.L))):
            timed(lambda: net.backward_layer(l), out[l]["bwd"])
    return [{d: {k: round(v, 4) for k, v in sorted(x[d].items())} for d in x} for x in out]


def event_updates(lay, ing):
    """(input with events, output neuron) connections of one layer over the
    batch: each such pair costs one weighted-event update in the forward, dW
    and dt_in contractions. `ing` is the in-grid indicator of the inputs."""
    B = ing.shape[0]
    if lay.kind == "dense":
        return ing.reshape(B, -1).sum() * lay.n_out
    x = ing.reshape(B, lay.C_in, lay.H, lay.W).sum(axis=1).astype(np.int64)  # per pixel
    if lay.pool_in == 2:
        x = x.reshape(B, lay.H // 2, 2, lay.W // 2, 2).sum(axis=(2, 4))
    elif lay.pool_in == 0:
        x = x.sum(axis=(1, 2)).reshape(B, 1, 1)
    Hp, Wp = x.shape[1], x.shape[2]
    xp = np.zeros((B, Hp + 2 * lay.pad, Wp + 2 * lay.pad), dtype=np.int64)
    xp[:, lay.pad:lay.pad + Hp, lay.pad:lay.pad + Wp] = x
    Ho = (Hp + 2 * lay.pad - lay.KH) // lay.stride + 1
    Wo = (Wp + 2 * lay.pad - lay.KW) // lay.stride + 1
    tot = 0
    for ky in range(lay.KH):
        for kx in range(lay.KW):
            tot += xp[:, ky:ky + lay.stride * (Ho - 1) + 1:lay.stride,
                      kx:kx + lay.stride * (Wo - 1) + 1:lay.stride].sum()
    return tot * lay.C_out


def layer_desc(lay):
    if lay.kind == "conv":
        pool = {0: " global-pool", 1: "", 2: " pool2"}[lay.pool_in]
        return (f"conv{lay.KH}x{lay.KW}/s{lay.stride}{pool} {lay.C_in}x{lay.H}x{lay.W}"
                f"->{lay.C_out} M={lay.M}")
    return f"{lay.n_in}->{lay.n_out} M={lay.M}"


def kernel_algorithmic_flops(net, act, with_scan=True, fused_dwdt=False):
    """Algorithmic flops of one step, per kernel name (2-sparse events:
    FLOPS_PER_UPDATE per (sample, input with events, neuron)); the forward
    kernels, which run the interval scan of their neurons too, also count
    FLOPS_PER_SCAN_STEP per (neuron, grid point) when with_scan. With
    fused_dwdt, the conv layers that compute dt_in ran dW and the dt_in
    partials in one launch (conv_dwdt)."""
    fl = {k: 0.0 for k in ("fwd_dense", "dw_dense", "dtin_rows", "conv_fwd", "conv_dw",
                           "conv_dtp", "conv_dwdt", "fwd_mfma")}
    for l, (e, a) in enumerate(zip(net.L, act)):
        upd = a["updates"]
        conv = e["cs"] is not None
        fwd, dw, dt = (("conv_fwd", "conv_dw", "conv_dtp") if conv else
                       ("fwd_dense", "dw_dense", "dtin_rows"))
        if conv and fused_dwdt and l > 0:
            dw = dt = "conv_dwdt"
        fl[fwd] += FLOPS_PER_UPDATE * upd
        if with_scan:
            fl[fwd] += FLOPS_PER_SCAN_STEP * e["t_out"].numel() * (e["lay"].M + 1)
        fl[dw] += FLOPS_PER_UPDATE * upd
        if l > 0:
            fl[dt] += FLOPS_PER_UPDATE * upd
    return fl


def traffic_for(kernel, workload, sha):
    """HBM bytes (FETCH + WRITE, copy-calibrated) per launch of `kernel` from
    the committed rocprofv3 counter summary, or None if none exists or the
    kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_source_sha") != sha:
        return None
    return round(d["hbm_bytes_per_step"] / d["dispatches_per_step"])


def cpu_baseline(wl, min_seconds=10.0):
    """The fp64 oracle (as it stands) on the host: fwd + bwd of the whole
    workload, repeated until min_seconds of CPU work. Dense workloads run the
    full batch per repetition; conv workloads a 2-image sub-batch (a full
    conv batch takes minutes in the oracle)."""
    import oracle
    from paper_2607_14672_amd import workloads
    d = workloads.Draws(wl)
    Ws = [d.weights(l) for l in range(len(wl.layers))]
    conv = any(lay.kind == "conv" for lay in wl.layers)
    nb = 2 if conv else wl.batch
    t_first = d.t_in[:nb]
    labels = None if d.labels is None else d.labels[:nb]
    targets = None if d.targets is None else d.targets[:nb]

    def fwd(lay, t, W):
        if lay.kind == "conv":
            return oracle.conv_forward(lay.params(), lay.conv_shape(),
                                       t.reshape(t.shape[0], lay.C_in, lay.H, lay.W), W)
        return oracle.dstd_forward(lay.params(), t.reshape(t.shape[0], -1), W)

    def bwd(lay, t, W, r, g, need_dt):
        g = np.where(r["q"] >= 0, g.reshape(r["q"].shape), 0.0)
        if lay.kind == "conv":
            _, gx = oracle.conv_backward(lay.params(), lay.conv_shape(),
                                         t.reshape(t.shape[0], lay.C_in, lay.H, lay.W), W, r, g)
            return gx
        _, gx = oracle.dstd_backward(lay.params(), t.reshape(t.shape[0], -1), W, r, g,
                                     want_dt=need_dt)
        return gx

    reps, n, t_start = 0, 0, time.perf_counter()
    while True:
        t = t_first
        fw = []
        for l, lay in enumerate(wl.layers):
            if lay.skip_back:  # SD block: cat(block input + delay, previous output)
                blk = fw[l - lay.skip_back][1]["t_out"].astype(np.float32)
                t = np.concatenate([blk + np.float32(lay.skip_delay), t.reshape(blk.shape[0], -1,
                                    *blk.shape[2:])], axis=1)
            r = fwd(lay, t, Ws[l])
            fw.append((t, r))
            t = r["t_out"].astype(np.float32)
        to = fw[-1][1]["t_out"].reshape(nb, -1)
        last = wl.layers[-1]
        if wl.loss == "ce":
            cap = last.t0 + last.M * last.dt + 2.0
            tt = np.where(np.isfinite(to), to, cap)
            z = -tt
            s = np.exp(z - z.max(1, keepdims=True))
            s /= s.sum(1, keepdims=True)
            g = np.where(np.isfinite(to), -(s - np.eye(to.shape[1])[labels]) / nb, 0.0)
        else:
            g = np.where(np.isfinite(to), (to - targets) / nb, 0.0)
        pend = {}  # block input's share of a skip gradient, keyed by the block's first layer
        for l in reversed(range(len(wl.layers))):
            tin, r = fw[l]
            gx = bwd(wl.layers[l], tin, Ws[l], r, g, l > 0)
            lay = wl.layers[l]
            if lay.skip_back and l > 0:
                c1 = fw[l - lay.skip_back][1]["t_out"].shape[1]
                pend[l - lay.skip_back + 1] = gx[:, :c1]
                gx = gx[:, c1:]
            if l in pend and l > 0:
                gx = gx.reshape(pend[l].shape) + pend.pop(l)
            if l > 0:
                g = gx
        reps += 1
        n += nb
        el = time.perf_counter() - t_start
        if el >= min_seconds:
            break
    return dict(value=n / el, unit="samples/s", cores=oracle.num_threads(), kind="oracle",
                sample=f"{reps} x {'sub-batch' if conv else 'full batch'} of {nb} samples "
                       f"(fwd+bwd of all layers, fp64), {el:.1f} s")


def exact_sweep(torch, dstd, workloads, dev, n_ins, models, Ms, reps=20, warmup=3):
    """The paper's single-layer timing comparison (App. D.1, Fig. "DSTD_exp" (b)):
    forward + backward (dL/dW and dL/dt_in) of one dense layer of 1000 neurons,
    batch 100, inputs U[0, 1), by the exact sorted-input method and by DSTD
    with M intervals on [0, 1], on the same inputs, weights and upstream
    gradient. Times are wall-clock per pass over `reps` back-to-back passes
    (eager launches on one stream); the library's workspace bytes of each
    method are reported beside them."""
    st = torch.cuda.current_stream(dev).cuda_stream
    rows = []

    def ck(name, s):
        if s != 0:
            raise RuntimeError(f"{name}: {dstd.dstd_last_error().decode()}")

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        return 1e3 * (time.perf_counter() - t0) / reps

    def kernels(fn, n=5):
        """per-kernel ms per pass (library hipEvent timer, separate passes)"""
        dstd.dstd_profile_reset()
        dstd.dstd_profile_enable(True)
        for _ in range(n):
            fn()
        torch.cuda.synchronize()
        dstd.dstd_profile_enable(False)
        return {k: round(v[1] / n, 4) for k, v in sorted(dstd.profile_table().items())}

    for model in models:
        for n_in in n_ins:
            cfg = workloads.exact_config(model, n_in=n_in)
            t_np, W_np = workloads.exact_inputs(cfg)
            B, N_out = cfg["batch"], cfg["n_out"]
            tt = torch.from_numpy(t_np).to(dev)
            Wt = torch.from_numpy(W_np).to(dev)
            g = torch.from_numpy(np.random.default_rng(1).standard_normal((B, N_out)).astype(np.float32)).to(dev)
            to = torch.empty((B, N_out), device=dev)
            sl = torch.empty_like(to)
            ix = torch.empty((B, N_out), dtype=torch.int32, device=dev)
            gW = torch.empty_like(Wt)
            gx = torch.empty_like(tt)
            pe = dstd.make_params(cfg["tau_m"], cfg["tau_s"], cfg["threshold"], 1, 0.0, 1.0)
            nf = dstd.dstd_exact_forward_workspace_size(pe, B, n_in, N_out)
            nb = dstd.dstd_exact_backward_workspace_size(pe, B, n_in, N_out)
            wf = dstd.workspace(nf, dev)
            wb = dstd.workspace(nb, dev)

            def run_exact():
                ck("dstd_exact_forward", dstd.dstd_exact_forward(
                    pe, B, n_in, N_out, tt.data_ptr(), Wt.data_ptr(), dstd.DSTD_F32, to.data_ptr(),
                    sl.data_ptr(), ix.data_ptr(), wf.data_ptr(), wf.numel(), st))
                ck("dstd_exact_backward", dstd.dstd_exact_backward(
                    pe, B, n_in, N_out, tt.data_ptr(), Wt.data_ptr(), dstd.DSTD_F32, to.data_ptr(),
                    sl.data_ptr(), ix.data_ptr(), g.data_ptr(), gW.data_ptr(), gx.data_ptr(),
                    wb.data_ptr(), wb.numel(), st))

            ms_exact = timed(run_exact)
            fired = float((ix >= 0).float().mean())
            walked = float((ix.float() + 1).clamp(min=0).mean())
            row = dict(model=model, n_in=n_in, exact_ms=round(ms_exact, 4),
                       exact_ws_bytes=int(nf + nb), exact_fired=round(fired, 4),
                       exact_mean_causal_inputs=round(walked, 1),
                       exact_kernel_ms=kernels(run_exact), dstd={})
            for M in Ms:
                pd = dstd.make_params(cfg["tau_m"], cfg["tau_s"], cfg["threshold"], M, 0.0, 1.0 / M)
                mf = dstd.dstd_lif_forward_workspace_size(pd, B, n_in, N_out)
                mb = dstd.dstd_lif_backward_workspace_size(pd, B, n_in, N_out)
                vf = dstd.workspace(mf, dev)
                vb = dstd.workspace(mb, dev)

                def run_dstd():
                    ck("dstd_lif_forward", dstd.dstd_lif_forward(
                        pd, B, n_in, N_out, tt.data_ptr(), Wt.data_ptr(), dstd.DSTD_F32,
                        to.data_ptr(), sl.data_ptr(), ix.data_ptr(), vf.data_ptr(), vf.numel(), st))
                    ck("dstd_lif_backward", dstd.dstd_lif_backward(
                        pd, B, n_in, N_out, tt.data_ptr(), Wt.data_ptr(), dstd.DSTD_F32,
                        to.data_ptr(), sl.data_ptr(), ix.data_ptr(), g.data_ptr(), gW.data_ptr(),
                        gx.data_ptr(), vb.data_ptr(), vb.numel(), st))

                ms = timed(run_dstd)
                row["dstd"][str(M)] = dict(ms=round(ms, 4), ws_bytes=int(mf + mb),
                                           fired=round(float((ix >= 0).float().mean()), 4),
                                           speedup_vs_exact=round(ms_exact / ms, 3),
                                           kernel_ms=kernels(run_dstd))
                del vf, vb
            rows.append(row)
            print(json.dumps(row), file=sys.stderr, flush=True)
            del wf, wb
    return rows


def multispike_bench(torch, dstd, dev, reps=20, warmup=3):
    """One multi-spike dense layer (App. "multi-spikes") fwd + bwd at the mlp3
    first layer's size (B 128, 784 inputs, 1000 neurons, M 32 on [0, 1],
    tau (1.0, 0.5)) for several input / output spike counts, against the TTFS
    layer on the same first input spikes. Inputs U[0, 1) per spike; weights
    (k / (N_in F_in)) (1 + 0.3 sqrt(N_in F_in) z) with k = 24 (most neurons
    fire F_out times). Eager launches; ms per pass and per kernel."""
    st = torch.cuda.current_stream(dev).cuda_stream
    B, N_in, N_out, M = 128, 784, 1000, 32
    p = dstd.make_params(1.0, 0.5, 1.0, M, 0.0, 1.0 / M)
    rows = []

    def ck(name, s):
        if s != 0:
            raise RuntimeError(f"{name}: {dstd.dstd_last_error().decode()}")

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        ms = 1e3 * (time.perf_counter() - t0) / reps
        dstd.dstd_profile_reset()
        dstd.dstd_profile_enable(True)
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        dstd.dstd_profile_enable(False)
        return ms, {k: round(v[1] / 5, 4) for k, v in sorted(dstd.profile_table().items())}

    for F_in, F_out in [(1, 1), (2, 4), (4, 8)]:
        rng = np.random.Generator(np.random.PCG64(12))
        t = rng.random((B, N_in, F_in)).astype(np.float32)
        n = N_in * F_in
        W = ((24.0 / n) * (1 + 0.3 * math.sqrt(n) * rng.standard_normal((N_out, N_in)))).astype(np.float32)
        tt, Wt = torch.from_numpy(t).to(dev), torch.from_numpy(W).to(dev)
        shp = (B, N_out, F_out)
        to = torch.empty(shp, device=dev)
        sl, cur = torch.empty_like(to), torch.empty_like(to)
        q = torch.empty(shp, dtype=torch.int32, device=dev)
        g = torch.from_numpy(rng.standard_normal(shp).astype(np.float32)).to(dev)
        gW = torch.empty_like(Wt)
        gx = torch.empty_like(tt)
        wf = dstd.workspace(dstd.dstd_lif_multispike_forward_workspace_size(p, B, N_in, F_in, N_out, F_out), dev)
        wb = dstd.workspace(dstd.dstd_lif_multispike_backward_workspace_size(p, B, N_in, F_in, N_out, F_out), dev)

        def run():
            ck("ms fwd", dstd.dstd_lif_multispike_forward(
                p, B, N_in, F_in, N_out, F_out, tt.data_ptr(), Wt.data_ptr(), dstd.DSTD_F32,
                to.data_ptr(), sl.data_ptr(), q.data_ptr(), cur.data_ptr(), wf.data_ptr(),
                wf.numel(), st))
            ck("ms bwd", dstd.dstd_lif_multispike_backward(
                p, B, N_in, F_in, N_out, F_out, tt.data_ptr(), Wt.data_ptr(), dstd.DSTD_F32,
                to.data_ptr(), sl.data_ptr(), q.data_ptr(), cur.data_ptr(), g.data_ptr(),
                gW.data_ptr(), gx.data_ptr(), wb.data_ptr(), wb.numel(), st))

        ms, kern = timed(run)
        spikes = (q >= 0).float().sum(dim=2)
        row = dict(F_in=F_in, F_out=F_out, multispike_ms=round(ms, 4), kernel_ms=kern,
                   mean_spikes_per_neuron=round(float(spikes.mean()), 3))
        # the TTFS layer on the first input spikes
        t1 = tt[:, :, 0].contiguous()
        o1, s1 = torch.empty((B, N_out), device=dev), torch.empty((B, N_out), device=dev)
        q1 = torch.empty((B, N_out), dtype=torch.int32, device=dev)
        g1, gx1 = g[:, :, 0].contiguous(), torch.empty_like(t1)
        vf = dstd.workspace(dstd.dstd_lif_forward_workspace_size(p, B, N_in, N_out), dev)
        vb = dstd.workspace(dstd.dstd_lif_backward_workspace_size(p, B, N_in, N_out), dev)

        def run1():
            ck("fwd", dstd.dstd_lif_forward(p, B, N_in, N_out, t1.data_ptr(), Wt.data_ptr(),
                                            dstd.DSTD_F32, o1.data_ptr(), s1.data_ptr(),
                                            q1.data_ptr(), vf.data_ptr(), vf.numel(), st))
            ck("bwd", dstd.dstd_lif_backward(p, B, N_in, N_out, t1.data_ptr(), Wt.data_ptr(),
                                             dstd.DSTD_F32, o1.data_ptr(), s1.data_ptr(),
                                             q1.data_ptr(), g1.data_ptr(), gW.data_ptr(),
                                             gx1.data_ptr(), vb.data_ptr(), vb.numel(), st))

        row["ttfs_ms"] = round(timed(run1)[0], 4)
        rows.append(row)
        print(json.dumps(row), file=sys.stderr, flush=True)
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="conv9",
                    help="the timed headline workload (default: the 9-layer conv net, the "
                         "largest single-GPU configuration)")
    ap.add_argument("--configs", default="dense1,dense1-cal,mlp3,wide-M8,wide-M32,wide-M64,"
                                         "wide-M128,conv20",
                    help="further workloads timed after the headline, reported in detail.configs")
    ap.add_argument("--config-steps", type=int, default=50)
    ap.add_argument("--contract", default="auto", choices=["auto", "sparse", "mfma"],
                    help="dense layers' forward contraction: the library's choice by shape, the "
                         "event-sparse kernels, or the bf16 MFMA product (bf16 weights only)")
    ap.add_argument("--no-configs", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="launch every kernel from Python each step instead of replaying a "
                         "HIP graph of the step")
    ap.add_argument("--layer-profile", action="store_true",
                    help="add per-layer kernel times to the detail section")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a 256 MiB device copy (HBM counter calibration)")
    ap.add_argument("--exact-sweep", action="store_true",
                    help="instead of the training step: time the exact sorted-input method "
                         "against DSTD on the paper's single-layer timing workload")
    ap.add_argument("--multispike", action="store_true",
                    help="instead of the training step: time the multi-spike dense layer")
    ap.add_argument("--exact-n-in", default="1000,2000,4000,6000")
    ap.add_argument("--exact-models", default="0.4-0.2,inf-0.2,inf-inf")
    ap.add_argument("--exact-M", default="10,20")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the data-parallel design is described, not built).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_14672_amd import dstd, workloads
    dstd._load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.exact_sweep:
        rows = exact_sweep(torch, dstd, workloads, dev,
                           [int(x) for x in args.exact_n_in.split(",")],
                           args.exact_models.split(","), [int(x) for x in args.exact_M.split(",")])
        print(json.dumps({"report": "exact vs DSTD, single dense layer fwd+bwd",
                          "config": {"batch": 100, "n_out": 1000, "inputs": "U[0,1) per input",
                                     "grid": "[0,1] with M intervals"},
                          "rows": rows}), flush=True)
        return
    if args.multispike:
        print(json.dumps({"report": "multi-spike dense layer fwd+bwd (B 128, 784 -> 1000, M 32)",
                          "rows": multispike_bench(torch, dstd, dev)}), flush=True)
        return
    wl = workloads.get(args.workload)
    head = measure(torch, dstd, wl, dev, args.steps, args.warmup, args.profile_steps, args.eager,
                   args.contract)
    net = head.pop("net")

    if args.copy_probe:
        a = torch.empty(64 << 20, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    per_layer = layer_profile(net, dstd, torch) if args.layer_profile else None
    loss = float(net.loss[0].cpu())
    del net
    others = []
    if not args.no_configs:
        for name in [x for x in args.configs.split(",") if x and x != args.workload]:
            r = measure(torch, dstd, workloads.get(name), dev, args.config_steps,
                        max(3, args.config_steps // 5), 5, args.eager, args.contract)
            r.pop("net")
            others.append(dict(workload=name, description=workloads.get(name).description,
                               batch=workloads.get(name).batch, value=r["value"], unit="samples/s",
                               ms_per_step=r["ms_per_step"], roofline=r["roofline"],
                               roofline_mfma=r["roofline_mfma"],
                               hbm_kernels=r["hbm_kernels"],
                               kernel_ms_per_step=r["kernel_ms_per_step"]))
            print(json.dumps(dict(config=name, value=r["value"], ms_per_step=r["ms_per_step"])),
                  file=sys.stderr, flush=True)
            torch.cuda.empty_cache()
    cpu = None if args.no_cpu_baseline else cpu_baseline(wl)
    out = {
        "metric": METRIC, "value": head["value"], "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded uniform spike times; calibrated random weights)",
        "config": {"workload": wl.description, "name": wl.name, "global_batch": wl.batch,
                   "layers": [layer_desc(lay) for lay in wl.layers],
                   "parallelism": "single GPU",
                   "execution": "eager launches" if args.eager else "HIP graph of the step"},
        "roofline": head["roofline"],
        "roofline_mfma": head["roofline_mfma"],
        "cpu_baseline": cpu,
        "detail": {"kernel_ms_per_step": head["kernel_ms_per_step"],
                   "launches_per_step": head["launches_per_step"], "activity": head["activity"],
                   "hbm_kernels": head["hbm_kernels"],
                   "kernel_source_sha": head["kernel_source_sha"],
                   "loss": loss, "per_layer_ms": per_layer, "configs": others},
    }
    print(json.dumps(out), flush=True)


def measure(torch, dstd, wl, dev, steps, warmup, profile_steps, eager, contract="auto"):
    """Time `steps` whole training steps of workload `wl` (HIP graph replays
    unless eager), then one profiling pass with the library's hipEvent timer:
    samples/s, per-kernel ms per step, the dominant kernel's roofline and the
    HBM rate of the bandwidth-bound kernels that have committed counters."""
    net = Net(wl, dev, contract)
    run = net.step
    if not eager:
        graph = net.capture()
        run = graph.replay
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = 1e3 * elapsed / max(steps, 1)
    value = wl.batch * steps / elapsed

    # per-kernel durations with the library's hipEvent timer (separate pass)
    act = net.activity()
    dstd.dstd_profile_reset()
    dstd.dstd_profile_enable(True)
    for _ in range(profile_steps):
        net.step()
    torch.cuda.synchronize()
    dstd.dstd_profile_enable(False)
    prof = dstd.profile_table()
    per_step = {k: v[1] / profile_steps for k, v in prof.items()}
    launches = {k: v[0] / profile_steps for k, v in prof.items()}
    # the library runs a conv layer's dW and dt_in partials in one launch
    # where it has that launch for the layer's shapes (every bench layer)
    fused = "conv_dwdt" in per_step
    if fused and "conv_dtp" in per_step:
        raise RuntimeError("conv layers ran both fused and separate dW / dt_in launches; "
                           "the per-kernel flop attribution assumes one form")
    flops = kernel_algorithmic_flops(net, act, fused_dwdt=fused)
    contraction = kernel_algorithmic_flops(net, act, with_scan=False, fused_dwdt=fused)
    if "fwd_mfma" in per_step and "fwd_dense" not in per_step:
        # the MFMA kernel only contracts; its scan runs in mfma_scan
        flops["fwd_mfma"] = contraction.pop("fwd_dense")
        flops.pop("fwd_dense")
        contraction["fwd_mfma"] = flops["fwd_mfma"]
    sha = kernel_source_sha()
    # the dominant contraction kernel (the step's largest kernel is one of them)
    cand = {k: v for k, v in per_step.items() if k in flops and flops[k] > 0}
    dom = max(cand, key=cand.get) if cand else None
    roof = None
    if dom is not None:
        achieved = flops[dom] / (per_step[dom] * 1e-3) / 1e12
        n_launch = launches[dom]
        roof = dict(bound="alu", achieved=round(achieved, 3), peak=PEAK_FP32_VECTOR_TFLOPS,
                    unit="TFLOP/s", frac=round(achieved / PEAK_FP32_VECTOR_TFLOPS, 4),
                    traffic=traffic_for(dom, wl.name, sha), traffic_unit="bytes per launch",
                    kernel=dom, launches_per_step=n_launch,
                    avg_launch_ms=round(per_step[dom] / n_launch, 4),
                    algorithmic_flops_per_launch=round(flops[dom] / n_launch),
                    kernel_ms_per_step=round(per_step[dom], 4),
                    largest_kernel=max(per_step, key=per_step.get),
                    contraction_only_TFLOPs=round(contraction[dom] / (per_step[dom] * 1e-3) / 1e12, 3),
                    flops_counted="contraction (4 per update) + interval scan (7 per neuron "
                                  "and grid point) for forward kernels; contraction for dW, dt_in")
    mfma = None
    if "fwd_mfma" in per_step:
        # the dense product: 2 flops per (row (b, m), input, neuron) and event plane
        ex = sum(2 * 3 * wl.batch * (e["lay"].M + 1) * e["lay"].n_in * e["lay"].n_out
                 for e in net.L if e["cs"] is None)
        t = per_step["fwd_mfma"] * 1e-3
        mfma = dict(bound="mfma", kernel="fwd_mfma", executed_flops_per_step=ex,
                    achieved=round(ex / t / 1e12, 2), peak=PEAK_BF16_MFMA_TFLOPS, unit="TFLOP/s",
                    frac=round(ex / t / 1e12 / PEAK_BF16_MFMA_TFLOPS, 4),
                    algorithmic_TFLOPs=round(flops["fwd_mfma"] / t / 1e12, 3),
                    kernel_ms_per_step=round(per_step["fwd_mfma"], 4))
    hbm = {}
    for k, v in per_step.items():
        if k in flops:
            continue
        b = traffic_for(k, wl.name, sha)
        if b is None:
            continue
        gbs = b * launches[k] / (v * 1e-3) / 1e9
        hbm[k] = dict(bytes_per_launch=b, ms_per_step=round(v, 4), achieved_GBs=round(gbs, 1),
                      frac=round(gbs / PEAK_HBM_GBS, 4))
    return dict(net=net, value=round(value, 1), ms_per_step=round(ms, 4), roofline=roof,
                roofline_mfma=mfma,
                kernel_ms_per_step={k: round(v, 4) for k, v in sorted(per_step.items())},
                launches_per_step=launches, activity=act, hbm_kernels=hbm,
                kernel_source_sha=sha)


if __name__ == "__main__":
    main()
