"""fp64 oracle of the synfire-chain training terms (App. C.1).

Test infrastructure only: the product path never imports this module. Plain
numpy in float64, written from the paper's definitions:

- temporal penalty, Eq. (temporal_penalty): for every neuron of layer l,
  gamma_head (t - t_head^(l))^2 when t < t_head^(l) plus
  gamma_tail (t - t_tail^(l))^2 when t > t_tail^(l), with the layer's window
  ends t_head^(l) = l tau_shift + t_head and
  t_tail^(l) = l tau_shift + tau_width - t_tail;
- dead-neuron penalty, Eq. (dead_neuron_penalty): Q = -sum over silent
  neurons (t = inf) of the sum of their incoming weights;
- the cost adds gamma_Q Q; both terms are averaged over the mini-batch, and
  for conv layers also divided by the spatial size.

Reading (stated in the design notes): a silent neuron has t = inf, for which
the temporal penalty's tail term would be infinite; the paper introduces Q
because the temporal penalty gives silent neurons no gradient, so silent
neurons are left out of the temporal penalty here. ``scale`` carries the
batch mean and the conv division (1/B, or 1/(B*H_out*W_out)).
"""
from __future__ import annotations

import numpy as np


def window(layer: int, tau_shift: float, tau_width: float, t_head: float, t_tail: float):
    """Layer l's window ends (t_head^(l), t_tail^(l))."""
    return layer * tau_shift + t_head, layer * tau_shift + tau_width - t_tail


def temporal_penalty(t, gamma_head, gamma_tail, t_head_l, t_tail_l, scale):
    """Value and gradient dT/dt of the temporal penalty over all entries of
    t (any shape); silent entries (non-finite) contribute nothing."""
    t = np.asarray(t, dtype=np.float64)
    fire = np.isfinite(t)
    tf = np.where(fire, t, 0.0)
    below = fire & (tf < t_head_l)
    above = fire & (tf > t_tail_l)
    val = np.sum(np.where(below, gamma_head * (tf - t_head_l) ** 2, 0.0))
    val += np.sum(np.where(above, gamma_tail * (tf - t_tail_l) ** 2, 0.0))
    grad = np.where(below, 2.0 * gamma_head * (tf - t_head_l), 0.0)
    grad += np.where(above, 2.0 * gamma_tail * (tf - t_tail_l), 0.0)
    return scale * val, scale * grad


def dead_neuron_penalty(t, W, gamma_q, scale):
    """Value gamma_q * scale * Q and its gradient with respect to W.

    t: [B, rows, *spatial] layer outputs; W: [rows, ...] weights, row i
    feeding every output of channel/neuron i. Returns (value, dW) with dW of
    W's shape."""
    t = np.asarray(t, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    B, rows = t.shape[0], t.shape[1]
    silent = ~np.isfinite(t.reshape(B, rows, -1))
    count = silent.sum(axis=(0, 2)).astype(np.float64)  # silent outputs per row
    row_sum = W.reshape(rows, -1).sum(axis=1)
    val = -gamma_q * scale * float(np.dot(count, row_sum))
    dW = -gamma_q * scale * np.broadcast_to(count.reshape((rows,) + (1,) * (W.ndim - 1)), W.shape)
    return val, np.array(dW)
