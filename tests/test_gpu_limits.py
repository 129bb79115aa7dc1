"""Layers at the size limits of this library (hidden or intermediate 8192),
against the oracle: the decode kernels for 2-64 tokens then stage more than
64 KiB of activations in LDS (gate/up at hidden 8192, down at intermediate
8192), which takes the larger-LDS launch path.  Widths drawn from
{2,3,4,5,6,8}, so the 5/6/8-bit kernels run at these sizes too."""
import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import moe, router

pytestmark = pytest.mark.gpu

TOL = 2e-3

WIDE_H = synth.LayerShape(hidden=8192, inter=256, n_experts=8, n_kept=6, n_shared=1, n_group=2, topk_group=1,
                          top_k=2)
WIDE_I = synth.LayerShape(hidden=256, inter=8192, n_experts=8, n_kept=6, n_shared=1, n_group=2, topk_group=1,
                          top_k=2)


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.view(dtype)


@pytest.fixture(scope="module", params=["hidden8192", "inter8192"])
def big(gpu_lib, request):
    shape = WIDE_H if request.param == "hidden8192" else WIDE_I
    data = layers.quantized_layer(shape, "wide_all", f"limits-{request.param}")
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=128)
    yield data, L
    L.close()


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("n", [1, 16, 100])
def test_forward_at_size_limits(gpu_lib, big, n, path):
    data, L = big
    shape = data.shape
    x_bits = synth.activations(n, shape.hidden, "limits-x", shape.hidden, n)
    logits = synth.normal_logits(n, shape.n_experts, "limits-l", shape.hidden, n)
    L.set_path(path)
    y = L.forward(_dev(x_bits.view(np.int16), torch.bfloat16), _dev(logits))
    torch.cuda.synchronize()
    L.set_path(gpu_lib.MOEQ_PATH_AUTO)
    rows = np.arange(n)
    idx, w = router.route(logits[rows], data.mask, n_group=shape.n_group, topk_group=shape.topk_group,
                          top_k=shape.top_k, group_topn=shape.group_topn, norm_topk=shape.norm_topk,
                          routed_scale=shape.routed_scale)
    ref = layers.oracle_forward(data, x_bits[rows], idx, w)
    err = moe.token_errors(y.cpu().numpy()[rows], ref)
    assert err.max() <= TOL, err.max()
