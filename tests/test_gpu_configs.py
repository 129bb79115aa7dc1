"""Layer configurations beyond the benchmark's, against the oracle (small
hidden and intermediate sizes so that each case runs in a moment): no shared
expert and several shared experts, unnormalised weights, group scores from
one or three experts, top-1 and wide top-k, a single group, a score-correction
bias, and routers over 512 and 1024 experts (their own kernel
instantiations).  Routing is compared bit for bit, outputs within the usual
per-token normwise 2e-3 on both forward paths."""
import dataclasses

import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import moe, router

pytestmark = pytest.mark.gpu

TOL = 2e-3
BASE = synth.LayerShape(hidden=256, inter=128, n_experts=32, n_kept=24, n_shared=1, n_group=4, topk_group=2,
                        top_k=4)

CASES = {
    "no_shared": dict(n_shared=0),
    "two_shared": dict(n_shared=2),
    "four_shared": dict(n_shared=4),
    "unnormalised": dict(norm_topk=0, routed_scale=1.0),
    "group_top1": dict(group_topn=1),
    "group_top3": dict(group_topn=3),
    "top1": dict(top_k=1, topk_group=1),
    "top12": dict(top_k=12, topk_group=4),
    "one_group": dict(n_group=1, topk_group=1),
    "biased": dict(),
    # expert counts per router lane of 2 and 4 (the one-token forward routes
    # inside the gate/up kernel up to 256 experts), 200 with groups of 25
    "experts128": dict(n_experts=128, n_kept=96, n_group=8, topk_group=4, top_k=8),
    "experts200": dict(n_experts=200, n_kept=150, n_group=8, topk_group=4, top_k=8),
    "experts512": dict(n_experts=512, n_kept=384, n_group=8, topk_group=4, top_k=8),
    "experts1024": dict(n_experts=1024, n_kept=768, n_group=8, topk_group=4, top_k=8),
}


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.view(dtype)


def _bias(name, shape):
    if name != "biased":
        return None
    return (synth.rng("cfg-bias", name).standard_normal(shape.n_experts) * 0.05).astype(np.float32)


@pytest.fixture(scope="module", params=sorted(CASES))
def case(gpu_lib, request):
    name = request.param
    shape = dataclasses.replace(BASE, **CASES[name])
    data = layers.quantized_layer(shape, "p234_602020", f"cfg-{name}")
    bias = _bias(name, shape)
    L = gpu_lib.Layer(shape, data.mask, data.routed(), data.shared(), max_tokens=128, bias=bias)
    yield name, data, bias, L
    L.close()


def _route_oracle(shape, mask, bias, logits):
    return router.route(logits, mask, bias, n_group=shape.n_group, topk_group=shape.topk_group, top_k=shape.top_k,
                        group_topn=shape.group_topn, norm_topk=shape.norm_topk, routed_scale=shape.routed_scale)


@pytest.mark.parametrize("n", [1, 7, 70])
def test_route_config(case, n):
    name, data, bias, L = case
    shape = data.shape
    logits = synth.normal_logits(n, shape.n_experts, "cfg-route", name, n)
    idx, w = L.route(_dev(logits))
    torch.cuda.synchronize()
    ridx, rw = _route_oracle(shape, data.mask, bias, logits)
    assert np.array_equal(idx.cpu().numpy(), ridx)
    assert np.allclose(w.cpu().numpy().astype(np.float64), rw, rtol=0, atol=1e-6 * max(1.0, shape.routed_scale))


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("n", [1, 7, 70])
def test_forward_config(gpu_lib, case, n, path):
    name, data, bias, L = case
    shape = data.shape
    x_bits = synth.activations(n, shape.hidden, "cfg-x", name, n)
    logits = synth.normal_logits(n, shape.n_experts, "cfg-fwd", name, n)
    L.set_path(path)
    y = L.forward(_dev(x_bits.view(np.int16), torch.bfloat16), _dev(logits))
    torch.cuda.synchronize()
    L.set_path(gpu_lib.MOEQ_PATH_AUTO)
    rows = np.arange(n) if n <= 7 else np.array([0, 33, n - 1])
    idx, w = _route_oracle(shape, data.mask, bias, logits[rows])
    ref = layers.oracle_forward(data, x_bits[rows], idx, w)
    err = moe.token_errors(y.cpu().numpy()[rows], ref)
    assert err.max() <= TOL, err.max()
