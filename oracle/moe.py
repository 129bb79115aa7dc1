"""Oracle: the MoE layer forward in float64.  TEST INFRASTRUCTURE ONLY.

The layer is the DeepSeek MoE block of Fig. 1 (middle): a router, ``n_shared``
always-on shared experts and ``E`` routed experts, each a SwiGLU feed-forward
network.  With ``(idx, w)`` from the router:

    y_t = sum_{j<k} w[t, j] * FFN_{idx[t, j]}(x_t) + sum_s FFN^shared_s(x_t)
    FFN(x) = W_down @ (silu(W_gate @ x) * (W_up @ x)),   silu(g) = g / (1 + e^-g)

The compute estimate of Section 3.2 (about ``2 * sum_i k_i P_i`` FLOPs per
token) counts exactly these expert products.  Shared experts are not scaled
by the routed weights.  Everything here is float64 with numpy's matrix
product as the only library step.
"""
import numpy as np

from . import quant


def bf16_bits_to_f64(bits):
    """bfloat16 bit patterns (uint16) -> float64, exactly."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def silu(g):
    with np.errstate(over="ignore"):
        return g / (1.0 + np.exp(-g))


def expert_ffn(x, w_gate, w_up, w_down):
    """x float64 ``[m, H]``; gate/up ``[I, H]``; down ``[H, I]`` -> ``[m, H]``."""
    g = x @ w_gate.T
    u = x @ w_up.T
    return (silu(g) * u) @ w_down.T


def dequant_tensor(t, K):
    """A packed tensor dict ``{bits, codes, scales}`` -> float64 ``[R, K]``."""
    codes = quant.unpack(t["codes"], t["bits"], K)
    return quant.dequantize(codes, t["scales"], t["bits"])


def moe_forward(x_bits, idx, w, routed, shared):
    """The layer output, float64 ``[n, H]``.

    x_bits  bfloat16 bit patterns ``[n, H]``
    idx, w  router output ``[n, k]``
    routed  callable ``e -> (W_gate, W_up, W_down)`` in float64 (only experts
            that some token chose are requested, each once)
    shared  list of ``(W_gate, W_up, W_down)`` float64 tuples
    """
    x = bf16_bits_to_f64(x_bits)
    n, H = x.shape
    y = np.zeros((n, H), np.float64)
    idx = np.asarray(idx)
    for e in np.unique(idx):
        rows, slots = np.nonzero(idx == e)
        wg, wu, wd = routed(int(e))
        y[rows] += np.asarray(w)[rows, slots][:, None] * expert_ffn(x[rows], wg, wu, wd)
    for wg, wu, wd in shared:
        y += expert_ffn(x, wg, wu, wd)
    return y


def token_errors(y, ref):
    """Per-token normwise error ``max_i |y - ref| / max_i |ref|`` (absolute if ref is all 0)."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(y - ref).max(axis=1)
    scale = np.abs(ref).max(axis=1)
    return np.where(scale > 0, err / np.where(scale > 0, scale, 1.0), err)
