"""Corner points of the pruning/precision sweep at full V3 shape: 256 and 128
kept experts (Section 3.1's retention at r = 1 and r = 0.5), every routed and
shared tensor 2-bit or every one 4-bit (Section 3.3's extremes), 64 tokens with
Zipf(1.1)-skewed routing over the kept experts, on the automatic path (the
decode matrix-vector kernels at 64 tokens).  Every token against the oracle;
routing bit-exact."""
import dataclasses

import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import moe, router

pytestmark = pytest.mark.gpu

TOL = 2e-3


@pytest.mark.parametrize("plan", ["all2", "all4"])
@pytest.mark.parametrize("kept", [256, 128])
def test_sweep_corner(gpu_lib, kept, plan):
    shape = dataclasses.replace(synth.V3, n_kept=kept)
    key = f"sweep-corner-{kept}-{plan}"
    data = layers.DeviceLayerData(shape, plan, key)
    L = data.make_layer(gpu_lib, max_tokens=64)
    try:
        n = 64
        x_bits = synth.activations(n, shape.hidden, key, "x")
        logits = synth.zipf_logits(n, data.mask, key, "l")
        x = torch.from_numpy(x_bits.view(np.int16)).cuda().view(torch.bfloat16)
        lg = torch.from_numpy(logits).cuda()
        idx_g, _ = L.route(lg)
        y = L.forward(x, lg)
        torch.cuda.synchronize()
        idx, w = router.route(logits, data.mask, n_group=shape.n_group, topk_group=shape.topk_group,
                              top_k=shape.top_k, group_topn=shape.group_topn, norm_topk=shape.norm_topk,
                              routed_scale=shape.routed_scale)
        assert np.array_equal(idx_g.cpu().numpy(), idx)
        ref = layers.oracle_forward(data, x_bits, idx, w)
        err = moe.token_errors(y.cpu().numpy(), ref)
        print(f"sweep corner kept {kept} {plan}: {len(np.unique(idx))} experts, worst {err.max():.2e}")
        assert err.max() <= TOL, err.max()
    finally:
        L.close()
