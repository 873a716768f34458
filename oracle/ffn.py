"""SwiGLU expert FFN and weighted combine (oracle; test infrastructure only).

The paper names the gate, up and down tensors of each expert (its Native
Serving Path section) but gives no formula; this uses the textbook SwiGLU
form, without biases:

    f_e(x) = W_down,e ( silu(W_gate,e x) * (W_up,e x) ),   silu(s) = s / (1 + exp(-s))
    y      = sum over routed e of  w_e * f_e(x)
"""
import numpy as np


def silu(s):
    s = np.asarray(s, dtype=np.float64)
    with np.errstate(over="ignore"):
        return s / (1.0 + np.exp(-s))


def expert_ffn(x, wg, wu, wd):
    """f_e(x) for x [H] or [T, H] (fp64)."""
    x = np.asarray(x, dtype=np.float64)
    g = x @ wg.T
    u = x @ wu.T
    return (silu(g) * u) @ wd.T


def combine(x, experts, weights):
    """sum_i weights[i] * f_{experts[i]}(x) for one token x [H]."""
    y = np.zeros(experts[0][2].shape[0], np.float64)
    for (wg, wu, wd), w in zip(experts, weights):
        y += w * expert_ffn(x, wg, wu, wd)
    return y
