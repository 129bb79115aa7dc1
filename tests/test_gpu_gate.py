"""The router gate (logits = x W_r^T) on the GPU, and forwards that compute
their own logits, against the CPU oracle.

* grid inputs (integers times 2^-12) make every float32 logit exact in any
  summation order: the gate must match the float64 oracle bit for bit, and a
  forward with computed logits must equal, bit for bit, the forward given the
  oracle's logits;
* Gaussian inputs: each logit within the first-order float32 error bound of
  a sum of H products, H * 2^-24 * sum |x_h w_h| (any summation order);
* both kernels: n <= 8 (streaming) and n > 8 (tiled, ragged in tokens and in
  experts on the tiny layer's 16 experts)."""
import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import moe, router

pytestmark = pytest.mark.gpu

TOL = 2e-3


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.view(dtype)


def _xdev(bits):
    return _dev(bits.view(np.int16), torch.bfloat16)


def _route_oracle(shape, mask, logits):
    return router.route(logits, mask, n_group=shape.n_group, topk_group=shape.topk_group,
                        top_k=shape.top_k, group_topn=shape.group_topn,
                        norm_topk=shape.norm_topk, routed_scale=shape.routed_scale,
                        regroup=bool(shape.regroup))


@pytest.fixture(scope="module")
def tiny_gate(gpu_lib):
    data = layers.quantized_layer(synth.TINY, "all4", "gate-tiny")
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=200)
    yield data, L
    L.close()


@pytest.fixture(scope="module")
def v3_gate(gpu_lib):
    data = layers.random_packed_layer(synth.V3, "gu3_d4_sh4", "gate-v3")
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=300)
    yield data, L
    L.close()


@pytest.mark.parametrize("which", ["tiny_gate", "v3_gate"])
@pytest.mark.parametrize("n", [1, 3, 8, 9, 70, 130])
def test_gate_exact_on_grid(request, which, n):
    data, L = request.getfixturevalue(which)
    E, H = data.shape.n_experts, data.shape.hidden
    w = synth.grid_router_weight(E, H, "gate-grid", which)
    L.set_router_weight(w)
    x_bits = synth.grid_activations(n, H, "gate-grid", which, n)
    got = L.router_logits(_xdev(x_bits))
    torch.cuda.synchronize()
    ref = router.gate_logits(x_bits, w)
    assert np.array_equal(got.cpu().numpy().astype(np.float64), ref)


@pytest.mark.parametrize("n", [1, 5, 8, 9, 64, 257])
def test_gate_within_float32_bound(v3_gate, n):
    data, L = v3_gate
    E, H = data.shape.n_experts, data.shape.hidden
    w = synth.router_weight(E, H, "gate-normal")
    L.set_router_weight(torch.from_numpy(w).cuda())   # device-resident copy path
    x_bits = synth.activations(n, H, "gate-normal", n)
    got = L.router_logits(_xdev(x_bits)).cpu().numpy().astype(np.float64)
    ref = router.gate_logits(x_bits, w)
    xa = np.abs((x_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    bound = H * 2.0 ** -24 * (xa @ np.abs(w.astype(np.float64)).T)
    assert np.all(np.abs(got - ref) <= bound)
    # the bound is loose: the error seen is far smaller
    assert np.max(np.abs(got - ref)) < 1e-4


def test_gate_deterministic(v3_gate):
    data, L = v3_gate
    E, H = data.shape.n_experts, data.shape.hidden
    L.set_router_weight(synth.router_weight(E, H, "gate-det"))
    for n in (4, 100):
        x = _xdev(synth.activations(n, H, "gate-det", n))
        a = L.router_logits(x)
        b = L.router_logits(x)
        torch.cuda.synchronize()
        assert torch.equal(a, b)


@pytest.mark.parametrize("which", ["tiny_gate", "v3_gate"])
@pytest.mark.parametrize("n", [1, 8, 40])
def test_forward_computes_logits(gpu_lib, request, which, n):
    """forward(x) with the gate set == forward(x, oracle logits), bit for bit, and
    both match the oracle layer within the usual tolerance."""
    data, L = request.getfixturevalue(which)
    shape = data.shape
    w = synth.grid_router_weight(shape.n_experts, shape.hidden, "gate-fwd", which)
    L.set_router_weight(w)
    x_bits = synth.grid_activations(n, shape.hidden, "gate-fwd", which, n)
    x = _xdev(x_bits)
    logits = router.gate_logits(x_bits, w).astype(np.float32)
    for path in (gpu_lib.MOEQ_PATH_DECODE, gpu_lib.MOEQ_PATH_PREFILL):
        L.set_path(path)
        y_self = L.forward(x)
        y_given = L.forward(x, _dev(logits))
        torch.cuda.synchronize()
        assert torch.equal(y_self, y_given)
        rows = np.arange(n) if n <= 8 else np.array([0, n // 2, n - 1])
        idx, wts = _route_oracle(shape, data.mask, logits[rows])
        ref = layers.oracle_forward(data, x_bits[rows], idx, wts)
        err = moe.token_errors(y_self.cpu().numpy()[rows], ref)
        assert err.max() <= TOL, err.max()
    L.set_path(gpu_lib.MOEQ_PATH_AUTO)


def test_gate_errors(gpu_lib, tiny_gate):
    data, L = tiny_gate
    H, E = data.shape.hidden, data.shape.n_experts
    x = _xdev(synth.activations(2, H, "gate-err"))
    L.set_router_weight(None)
    with pytest.raises(gpu_lib.MoeqError) as ei:
        L.forward(x)
    assert ei.value.status == gpu_lib.MOEQ_ERR_INVALID_ARG
    with pytest.raises(gpu_lib.MoeqError) as ei:
        L.router_logits(x)
    assert ei.value.status == gpu_lib.MOEQ_ERR_INVALID_ARG
    bad = synth.router_weight(E, H, "gate-err")
    bad[3, 5] = np.nan
    with pytest.raises(gpu_lib.MoeqError) as ei:
        L.set_router_weight(bad)
    assert ei.value.status == gpu_lib.MOEQ_ERR_INVALID_ARG
    with pytest.raises(gpu_lib.MoeqError) as ei:
        gpu_lib.moeq_set_router_weight(L.handle, 0, 7)
    assert ei.value.status == gpu_lib.MOEQ_ERR_INVALID_ARG
    # a rejected set leaves no weight behind; a good one works after it
    L.set_router_weight(synth.router_weight(E, H, "gate-err"))
    y = L.forward(x)
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()
    L.set_router_weight(None)
