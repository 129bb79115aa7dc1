"""The 58-layer stack of the deployment (Section 4: batch-1 decode through
every MoE layer of the pruned model; 58 MoE layers, the count Section 3.3's
back-off order is printed for): 58 independent V3-shape layers, 192 of 256
experts kept in each, per-tensor widths from {2,3,4} with p = (0.7, 0.1,
0.2), about 185 GB resident -- built as the benchmark builds them (random
packed tensors drawn on the GPU, keyed per tensor).

Per layer, with its own x and logits: routing and bucketing bit-exact
against the oracle on all 58 layers, and the layer outputs of the 58
forwards run back to back on one stream against the oracle on three seeded
layers (first, middle, last)."""
import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import bucket as obucket
from oracle import moe, router

pytestmark = pytest.mark.gpu

N_LAYERS = 58
CHECK_Y = (0, 29, 57)


def _route(shape, mask, logits):
    return router.route(logits, mask, n_group=shape.n_group, topk_group=shape.topk_group, top_k=shape.top_k,
                        group_topn=shape.group_topn, norm_topk=shape.norm_topk, routed_scale=shape.routed_scale)


def test_stack_58_layers(gpu_lib):
    shape = synth.V3
    datas, Ls = [], []
    try:
        for li in range(N_LAYERS):
            d = layers.DeviceLayerData(shape, "p234_701020", f"stack-{li}")
            datas.append(d)
            Ls.append(d.make_layer(gpu_lib, max_tokens=1))
        resident = sum(L.bytes()[0] for L in Ls)
        print(f"stack: {N_LAYERS} layers, {resident / 1e9:.1f} GB resident", flush=True)
        xs = [synth.activations(1, shape.hidden, "stack-x", li) for li in range(N_LAYERS)]
        lgs = [synth.normal_logits(1, shape.n_experts, "stack-l", li) for li in range(N_LAYERS)]
        x_dev = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in xs]
        lg_dev = [torch.from_numpy(lg).cuda() for lg in lgs]

        # routing and bucketing of every layer
        for li, (d, L) in enumerate(zip(datas, Ls)):
            idx, w = L.route(lg_dev[li])
            offsets, perm = L.bucket(idx)
            torch.cuda.synchronize()
            ridx, rw = _route(shape, d.mask, lgs[li])
            assert np.array_equal(idx.cpu().numpy(), ridx), li
            np.testing.assert_allclose(w.cpu().numpy(), rw, rtol=1e-6, atol=1e-7)
            roff, rperm, _ = obucket.bucket(ridx, shape.n_experts)
            assert np.array_equal(offsets.cpu().numpy(), roff), li
            assert np.array_equal(perm.cpu().numpy(), rperm), li
            assert not np.any(d.mask[ridx[0]] == 0)

        # the 58 forwards back to back on one stream, as one decode step
        ys = [torch.empty((1, shape.hidden), device="cuda") for _ in range(N_LAYERS)]
        for li, L in enumerate(Ls):
            L.forward(x_dev[li], lg_dev[li], y=ys[li])
        torch.cuda.synchronize()
        for li in CHECK_Y:
            d = datas[li]
            idx, w = _route(shape, d.mask, lgs[li])
            ref = layers.oracle_forward(d, xs[li], idx, w)
            err = moe.token_errors(ys[li].cpu().numpy(), ref)
            print(f"stack layer {li}: per-token error {err.max():.2e}", flush=True)
            assert err.max() < 1e-3, (li, err.max())
        for y in ys:
            assert torch.isfinite(y).all()
    finally:
        for L in Ls:
            L.close()
