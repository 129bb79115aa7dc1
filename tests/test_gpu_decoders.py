"""Every decoder of the weight format the products run, bit for bit against
the format's definition (Section 3.3's per-tensor widths in this library's
block format: weight = d * (c - 2^(b-1))).

* the bfloat16-form unpacking (matrix-vector kernels for 5/6/8-bit
  tensors): float32 d * (c - z), exact;
* the binary16-subnormal code pairs (the 2-4-bit gate/up and down
  matrix-vector kernels): each code rebuilt from its pair value, float32
  d * (c - z), exact;
* the grouped GEMMs' weight decoder: binary16(d * (c - z)), one rounding to
  nearest even -- the oracle's dequantize_half, which is pinned by closed
  forms and an exhaustive binary16 search on the CPU.

Tensors: every tensor of tiny layers with 2/3/4-bit and with every width of
{2,3,4,5,6,8}, and sampled tensors of the V3-shape layers at each width."""
import dataclasses

import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import quant

pytestmark = pytest.mark.gpu


def _codes_scales(t, K):
    return quant.unpack(t["codes"], t["bits"], K), t["scales"]


def _check_tensor(moeq, data, L, kind, e, p):
    t = data.tensor(kind, e, p)
    K = data.shape.rows_cols(p)[1]
    codes, scales = _codes_scales(t, K)
    exact = quant.dequantize(codes, scales, t["bits"])
    half = quant.dequantize_half(codes, scales, t["bits"])
    eid = e if kind == "r" else -1 - e
    got_x = L.dequant_as(eid, p, moeq.MOEQ_DECODER_EXACT)
    got_h = L.dequant_as(eid, p, moeq.MOEQ_DECODER_GEMM_F16)
    got_s = L.dequant_as(eid, p, moeq.MOEQ_DECODER_GEMV_SUBNORMAL) if t["bits"] <= 4 else None
    torch.cuda.synchronize()
    assert np.array_equal(got_x.cpu().numpy().astype(np.float64), exact), (kind, e, p, t["bits"], "exact")
    assert np.array_equal(got_h.cpu().numpy().view(np.uint16), half), (kind, e, p, t["bits"], "gemm f16")
    if got_s is not None:
        assert np.array_equal(got_s.cpu().numpy().astype(np.float64), exact), (kind, e, p, t["bits"], "subnormal")
    return t["bits"]


@pytest.mark.parametrize("plan", ["p234_602020", "wide_all"])
def test_every_decoder_every_tensor_tiny(gpu_lib, plan):
    data = layers.quantized_layer(synth.TINY, plan, f"decoders-{plan}")
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=8)
    try:
        seen = set()
        for e in np.nonzero(data.mask)[0]:
            for p in range(3):
                seen.add(_check_tensor(gpu_lib, data, L, "r", int(e), p))
        for p in range(3):
            seen.add(_check_tensor(gpu_lib, data, L, "s", 0, p))
        assert seen == ({2, 3, 4} if plan == "p234_602020" else {2, 3, 4, 5, 6, 8})
    finally:
        L.close()


def test_every_decoder_v3_samples(gpu_lib):
    """V3-shape tensors of every width (32 kept experts, widths drawn from
    {2,3,4,5,6,8}): the first tensor of each width found, in each projection."""
    shape = dataclasses.replace(synth.V3, n_kept=32)
    data = layers.DeviceLayerData(shape, "wide_all", "decoders-v3")
    L = data.make_layer(gpu_lib, max_tokens=8)
    try:
        todo = {(b, p) for b in quant.SUPPORTED_BITS for p in range(3)}
        for e in np.nonzero(data.mask)[0]:
            for p in range(3):
                key = (int(data.bits_r[e, p]), p)
                if key in todo:
                    _check_tensor(gpu_lib, data, L, "r", int(e), p)
                    todo.discard(key)
        # the draw leaves no (width, projection) pair out
        assert not todo, todo
    finally:
        L.close()


def test_subnormal_decoder_rejects_wide(gpu_lib):
    data = layers.quantized_layer(synth.TINY, "all6", "decoders-reject")
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=8)
    try:
        with pytest.raises(gpu_lib.MoeqError) as ei:
            L.dequant_as(-1, 0, gpu_lib.MOEQ_DECODER_GEMV_SUBNORMAL)
        assert ei.value.status == gpu_lib.MOEQ_ERR_UNSUPPORTED
        with pytest.raises(gpu_lib.MoeqError) as ei:
            gpu_lib.moeq_dequant_as(L.handle, -1, 0, 7, 0)
        assert ei.value.status == gpu_lib.MOEQ_ERR_INVALID_ARG
    finally:
        L.close()
