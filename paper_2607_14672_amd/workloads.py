"""Seeded synthetic workloads shaped like the paper's experiments.

This module only draws random numbers and describes shapes; it holds none of
the method's arithmetic, so both the HIP path and the fp64 oracle can use it.
Input spike times stand in for pixel intensities encoded as t = tau_in (1 - x)
with tau_in = 1 (App. C.2); no dataset item is reproduced. Grids follow the
synfire windowing of App. C.1 read as "layer l (1-based) discretizes its input
window [l-1, l] with M intervals".

Weights: the paper leaves the initial distribution open (it searches a
positive and a negative scale, Table "tab:search_space"). Workloads other
than the as-stated single layer use W = (k / N_in) (1 + 0.3 sqrt(N_in) z),
z ~ N(0, 1), with k chosen per layer so that ~70 % of the layer's neurons fire
on the first 8 samples; the constants are produced by
``oracle/calibrate.py`` and stored in ``calibration.json`` next to this file.
"""
from __future__ import annotations

import json
import math
import os
from dataclasses import dataclass, field, replace
from typing import List, Optional

import numpy as np

_CAL_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "calibration.json")


@dataclass
class LayerSpec:
    kind: str                 # "dense" or "conv"
    n_in: int                 # flattened input size
    n_out: int                # flattened output size
    M: int
    t0: float
    dt: float
    tau_m: float
    tau_s: float
    threshold: float = 1.0
    t_max: float = math.inf
    w_dtype: str = "f32"      # "f32" or "bf16"
    # conv geometry (kind == "conv")
    C_in: int = 0
    H: int = 0
    W: int = 0
    C_out: int = 0
    KH: int = 3
    KW: int = 3
    stride: int = 1
    pad: int = 1
    pool_in: int = 1          # 1 none, 2 = 2x2 average of input events, 0 = global average
    # skip-and-delay (third layer of an SD block): the input is the channel
    # concatenation of the output of the layer skip_back positions earlier
    # (the block input) delayed by skip_delay, then the previous layer's output
    skip_back: int = 0
    skip_delay: float = 0.0

    def params(self) -> dict:
        return dict(tau_m=self.tau_m, tau_s=self.tau_s, threshold=self.threshold, M=self.M,
                    t0=self.t0, dt=self.dt, t_max=self.t_max)

    def conv_shape(self) -> dict:
        return dict(C_in=self.C_in, H=self.H, W=self.W, C_out=self.C_out, KH=self.KH, KW=self.KW,
                    stride=self.stride, pad=self.pad, pool_in=self.pool_in)

    def w_shape(self):
        if self.kind == "dense":
            return (self.n_out, self.n_in)
        return (self.C_out, self.C_in, self.KH, self.KW)

    def fan_in(self) -> int:
        if self.kind == "dense":
            return self.n_in
        return self.C_in * self.KH * self.KW


@dataclass
class Workload:
    name: str
    batch: int
    layers: List[LayerSpec]
    input_rule: str            # "one_minus_u" or "u"
    silent_frac: float = 0.0
    w_rule: str = "calibrated" # "as_stated" or "calibrated"
    loss: str = "ce"           # "ce" (softmax on -t) or "mse" (targets U[1,2])
    n_classes: int = 10
    seed: int = 0
    description: str = ""
    extra: dict = field(default_factory=dict)


def _conv_out(H, W, KH, KW, stride, pad, pool):
    if pool == 2:
        H, W = H // 2, W // 2
    elif pool == 0:
        H, W = 1, 1
    return (H + 2 * pad - KH) // stride + 1, (W + 2 * pad - KW) // stride + 1


def _conv_layer(l, C_in, H, W, C_out, M, tau_m, tau_s, stride=1, pool_in=1, K=3, pad=1):
    Ho, Wo = _conv_out(H, W, K, K, stride, pad, pool_in)
    return LayerSpec(kind="conv", n_in=C_in * H * W, n_out=C_out * Ho * Wo, M=M,
                     t0=float(l - 1), dt=1.0 / M, tau_m=tau_m, tau_s=tau_s,
                     C_in=C_in, H=H, W=W, C_out=C_out, KH=K, KW=K, stride=stride, pad=pad,
                     pool_in=pool_in)


def dense1(calibrated: bool = False) -> Workload:
    """Single dense layer 784 -> 100, B 8, M 16 on [0, 1], tau (1.0, 0.3)."""
    L = [LayerSpec("dense", 784, 100, 16, 0.0, 1.0 / 16, 1.0, 0.3)]
    return Workload("dense1-cal" if calibrated else "dense1", 8, L, "one_minus_u",
                    w_rule="calibrated" if calibrated else "as_stated", loss="mse", seed=1,
                    description="single dense DSTD-LIF layer 784->100, batch 8, M=16")


def mlp3() -> Workload:
    """Dense 3-layer TTFS MLP 784-1000-1000-10, B 128, M 32 per layer, tau (1.0, 0.5)."""
    sizes = [784, 1000, 1000, 10]
    L = [LayerSpec("dense", sizes[l - 1], sizes[l], 32, float(l - 1), 1.0 / 32, 1.0, 0.5)
         for l in range(1, 4)]
    return Workload("mlp3", 128, L, "one_minus_u", loss="ce", seed=2,
                    description="dense 3-layer TTFS MLP 784-1000-1000-10, batch 128, M=32/layer")


def wide(M: int = 64) -> Workload:
    """Wide dense layer 4096 -> 4096, B 256, bf16 W, tau (2.0, 0.4), 20 % silent inputs."""
    L = [LayerSpec("dense", 4096, 4096, M, 0.0, 1.0 / M, 2.0, 0.4, w_dtype="bf16")]
    return Workload(f"wide-M{M}", 256, L, "u", silent_frac=0.2, loss="mse", seed=3,
                    description=f"wide dense DSTD-LIF layer 4096->4096, batch 256, M={M}, bf16 W")


def conv9() -> Workload:
    """9-layer conv net on 32x32x3, B 64, M 32, tau (1.0, 0.3)."""
    M, tm, ts = 32, 1.0, 0.3
    chans = [3, 64, 64, 128, 128, 256, 256, 256, 256]
    L, H = [], 32
    for l in range(1, 9):
        pool = 2 if l in (3, 5, 7) else 1  # average pooling after layers 2, 4, 6
        if pool == 2:
            lay = _conv_layer(l, chans[l - 1], H, H, chans[l], M, tm, ts, pool_in=2)
            H //= 2
        else:
            lay = _conv_layer(l, chans[l - 1], H, H, chans[l], M, tm, ts)
        L.append(lay)
    L.append(LayerSpec("dense", 256 * H * H, 10, M, 8.0, 1.0 / M, tm, ts))
    return Workload("conv9", 64, L, "one_minus_u", loss="ce", seed=4,
                    description="9-layer conv DSTD-LIF net on 32x32x3, batch 64, M=32")


def conv20() -> Workload:
    """20-layer conv net on 28x28x1, B 128, M 16, tau (1.5, 0.5)."""
    M, tm, ts = 16, 1.5, 0.5
    L, H, C = [], 28, 1
    for l in range(1, 20):
        co = 32 if l <= 10 else 64
        st = 2 if l in (6, 13) else 1
        lay = _conv_layer(l, C, H, H, co, M, tm, ts, stride=st)
        L.append(lay)
        H = (H + 2 - 3) // st + 1
        C = co
    # global average pooling of the input events, then dense 64 -> 10
    L.append(LayerSpec("conv", C * H * H, 10, M, 19.0, 1.0 / M, tm, ts, C_in=C, H=H, W=H,
                       C_out=10, KH=1, KW=1, stride=1, pad=0, pool_in=0))
    return Workload("conv20", 128, L, "u", loss="ce", seed=5,
                    description="20-layer conv DSTD-LIF net on 28x28x1, batch 128, M=16")


def synsnn20_sd(n_ch: int = 32) -> Workload:
    """Syn-SNN-20 of Table "tab:architectures": C(N,3,1)-SD2(N)-SD1(N)-SD2(2N)-
    SD1(2N)-SD2(4N)-SD1(4N)-10 on 28x28x1, B 128, M 16, tau (1.5, 0.5). An SD
    block is three 3x3 convs; its third reads cat(block input delayed by
    2 tau_shift, second layer's output) (App. C.3, Fig. "skip_connection"),
    with stride 2 and doubled channels in SD1, stride 1 in SD2. Layer l
    (1-based) discretizes [l-1, l] (tau_shift = 1), so the delay is 2. The
    classifier is a global pool of events and a dense 4N -> 10 layer, as for
    conv20. Weights: a fixed k = 7 for every layer (no calibration; deep
    layers mostly stay silent at random init, as in the conv workloads)."""
    M, tm, ts = 16, 1.5, 0.5
    L, H, C, l = [], 28, 1, 1
    L.append(_conv_layer(l, C, H, H, n_ch, M, tm, ts))
    C = n_ch
    for kind, mult in (("SD2", 1), ("SD1", 1), ("SD2", 2), ("SD1", 2), ("SD2", 4), ("SD1", 4)):
        N = n_ch * mult
        Cb = C  # block input channels (= N)
        L.append(_conv_layer(l + 1, Cb, H, H, N, M, tm, ts))
        L.append(_conv_layer(l + 2, N, H, H, N, M, tm, ts))
        st = 2 if kind == "SD1" else 1
        N3 = 2 * N if kind == "SD1" else N
        lay = _conv_layer(l + 3, Cb + N, H, H, N3, M, tm, ts, stride=st)
        lay.skip_back, lay.skip_delay = 3, 2.0
        L.append(lay)
        H = (H + 2 - 3) // st + 1
        C = N3
        l += 3
    L.append(LayerSpec("conv", C * H * H, 10, M, float(l), 1.0 / M, tm, ts, C_in=C, H=H, W=H,
                       C_out=10, KH=1, KW=1, stride=1, pad=0, pool_in=0))
    return Workload("synsnn20-sd", 128, L, "u", loss="ce", seed=6,
                    description="Syn-SNN-20 with skip-and-delay blocks on 28x28x1, batch 128, M=16",
                    extra={"k": [7.0] * len(L)})


WORKLOADS = {
    "dense1": lambda: dense1(False),
    "dense1-cal": lambda: dense1(True),
    "mlp3": mlp3,
    "wide-M8": lambda: wide(8),
    "wide-M32": lambda: wide(32),
    "wide-M64": lambda: wide(64),
    "wide-M128": lambda: wide(128),
    "conv9": conv9,
    "conv20": conv20,
    "synsnn20-sd": synsnn20_sd,
}


def get(name: str) -> Workload:
    return WORKLOADS[name]()


def load_calibration() -> dict:
    if os.path.exists(_CAL_PATH):
        with open(_CAL_PATH) as f:
            return json.load(f)
    return {}


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even), returned as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


class Draws:
    """All random draws of one workload, in a fixed order: inputs, then the
    standard-normal weight templates layer by layer, then targets/labels."""

    def __init__(self, wl: Workload, batch: Optional[int] = None):
        self.wl = wl
        B = wl.batch if batch is None else batch
        rng = np.random.Generator(np.random.PCG64(wl.seed))
        n0 = wl.layers[0].n_in
        x = rng.random((wl.batch, n0))
        if wl.input_rule == "one_minus_u":
            t = 1.0 - x
        else:
            t = x
        if wl.silent_frac > 0:
            silent = rng.random((wl.batch, n0)) < wl.silent_frac
            t = np.where(silent, np.inf, t)
        self.t_in = t.astype(np.float32)[:B]
        self.z = []
        for lay in wl.layers:
            self.z.append(rng.standard_normal(lay.w_shape()))
        if wl.loss == "mse":
            self.targets = (1.0 + rng.random((wl.batch, wl.layers[-1].n_out))).astype(np.float32)[:B]
            self.labels = None
        else:
            self.labels = rng.integers(0, wl.n_classes, size=wl.batch).astype(np.int32)[:B]
            self.targets = None

    def weights(self, l: int, k: Optional[float] = None) -> np.ndarray:
        """Weights of layer l (0-based) as float32 (bf16-rounded when the layer says so)."""
        lay = self.wl.layers[l]
        z = self.z[l]
        if self.wl.w_rule == "as_stated":
            n = lay.fan_in()
            w = z * (2.0 / n) + 0.5 / n
        else:
            if k is None and "k" in self.wl.extra:
                k = self.wl.extra["k"][l]
            if k is None:
                k = load_calibration().get(self.wl.name, {}).get("k", [None] * len(self.wl.layers))[l]
                if k is None:
                    raise KeyError(f"no calibration constant for {self.wl.name} layer {l}")
            n = lay.fan_in()
            w = (k / n) * (1.0 + 0.3 * math.sqrt(n) * z)
        w = w.astype(np.float32)
        if lay.w_dtype == "bf16":
            w = bf16_round(w)
        return w


def with_batch(wl: Workload, batch: int) -> Workload:
    return replace(wl, batch=batch)


# --------------------------------------------------- exact vs DSTD timing --
# The paper's single-layer timing experiment (App. D.1, Fig. "DSTD_exp" (b)):
# 1000 neurons, batch 100, input spikes uniform on [0, 1], the number of
# inputs swept up to 6000, three neuron models, M in {10, 20}. The paper does
# not give the weights; here W = (k / N_in) (1 + 0.3 sqrt(N_in) z), z ~ N(0, 1),
# where k sets the mean summed weight per model (k = 2.5 V_th divided by the
# peak of that model's kernel; for (inf, inf) the kernel has no peak and
# k = 2.5), so most neurons fire within or shortly after the input window.
EXACT_MODELS = {
    "0.4-0.2": dict(tau_m=0.4, tau_s=0.2, k=25.0),
    "inf-0.2": dict(tau_m=math.inf, tau_s=0.2, k=12.5),
    "inf-inf": dict(tau_m=math.inf, tau_s=math.inf, k=2.5),
}


def exact_config(model: str = "0.4-0.2", n_in: int = 6000, M: int = 20, batch: int = 100,
                 n_out: int = 1000, seed: int = 11) -> dict:
    m = EXACT_MODELS[model]
    return dict(model=model, batch=batch, n_in=n_in, n_out=n_out, M=M, t0=0.0, dt=1.0 / M,
                tau_m=m["tau_m"], tau_s=m["tau_s"], threshold=1.0, k=m["k"], seed=seed)


def exact_inputs(cfg: dict):
    """(t_in [B, N_in], W [N_out, N_in]) float32 for an exact_config."""
    rng = np.random.Generator(np.random.PCG64(cfg["seed"]))
    t = rng.random((cfg["batch"], cfg["n_in"])).astype(np.float32)
    n = cfg["n_in"]
    z = rng.standard_normal((cfg["n_out"], n))
    W = ((cfg["k"] / n) * (1.0 + 0.3 * math.sqrt(n) * z)).astype(np.float32)
    return t, W
