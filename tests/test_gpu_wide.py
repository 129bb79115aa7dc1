"""Wide widths (5, 6 and 8-bit blocks: Section 3.3's Q6/Q8 upgrades of small
and medium tensors, here in this library's block format) against the oracle.

Bit-exact: quantizer codes and scales, every dequantized tensor of a tiny
layer whose tensors draw their widths from {2,3,4,5,6,8}, sampled tensors of
the V3-shape layers.  Layer outputs: per-token normwise error <= 2e-3 on both
forward paths for
* the tiny layer with every width mixed in (gate and up of one expert often
  differ, narrow and wide),
* V3 shape with the shared expert upgraded to 6 or 8 bits (routed gate/up
  3-bit, down 4-bit), decode batch 1 and 16 and 2048-token prefill,
* V3 shape with 32 kept routed experts whose tensors take every width."""
import dataclasses

import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import moe, quant, router

pytestmark = pytest.mark.gpu

TOL = 2e-3
WIDE = (5, 6, 8)


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.view(dtype)


def _x(n, H, *key):
    bits = synth.activations(n, H, *key)
    return bits, _dev(bits.view(np.int16), torch.bfloat16)


def _forward_check(moeq, data, L, n, key, path, logits=None, sample=None):
    shape = data.shape
    x_bits, x = _x(n, shape.hidden, key, n)
    if logits is None:
        logits = synth.normal_logits(n, shape.n_experts, key, n)
    L.set_path(path)
    y = L.forward(x, _dev(logits))
    torch.cuda.synchronize()
    L.set_path(moeq.MOEQ_PATH_AUTO)
    rows = np.arange(n) if sample is None else np.asarray(sample)
    idx, w = router.route(logits[rows], data.mask, n_group=shape.n_group, topk_group=shape.topk_group,
                          top_k=shape.top_k, group_topn=shape.group_topn, norm_topk=shape.norm_topk,
                          routed_scale=shape.routed_scale)
    ref = layers.oracle_forward(data, x_bits[rows], idx, w)
    err = moe.token_errors(y.cpu().numpy()[rows], ref)
    assert err.max() <= TOL, (err.max(), np.median(err))
    return err


def _layer(moeq, data, max_tokens):
    return moeq.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=max_tokens)


@pytest.fixture(scope="module")
def tiny_wide(gpu_lib):
    data = layers.quantized_layer(synth.TINY, "wide_all", "tiny-wide")
    L = _layer(gpu_lib, data, 200)
    yield data, L
    L.close()


@pytest.fixture(scope="module", params=[6, 8])
def v3_shared_wide(gpu_lib, request):
    data = layers.DeviceLayerData(synth.V3, f"gu3_d4_sh{request.param}", f"v3-sh{request.param}")
    L = data.make_layer(gpu_lib, max_tokens=2048)
    yield data, L
    L.close()


@pytest.fixture(scope="module")
def v3_routed_wide(gpu_lib):
    shape = dataclasses.replace(synth.V3, n_kept=32)
    data = layers.DeviceLayerData(shape, "wide_all", "v3-routed-wide")
    L = data.make_layer(gpu_lib, max_tokens=512)
    yield data, L
    L.close()


@pytest.mark.parametrize("bits", WIDE)
def test_quantize_bit_exact_wide(gpu_lib, bits):
    w = synth.normal_weights(48, 256, "q-wide", bits)
    codes_ref, scales_ref = quant.quantize(w, bits)
    codes, scales = gpu_lib.quantize(torch.from_numpy(w).cuda(), bits)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), quant.pack(codes_ref, bits))
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), scales_ref)


def test_tiny_plan_covers_every_width():
    data = layers.quantized_layer(synth.TINY, "wide_all", "tiny-wide")
    used = set(data.bits_r[data.mask.astype(bool)].ravel()) | set(data.bits_s.ravel())
    assert used == {2, 3, 4, 5, 6, 8}


def test_dequant_bit_exact_every_tensor(tiny_wide):
    data, L = tiny_wide
    for e in list(np.nonzero(data.mask)[0]) + [-1]:
        ref = data.dequant("r", e) if e >= 0 else data.dequant("s", 0)
        for p in range(3):
            got = L.dequant(int(e), p)
            torch.cuda.synchronize()
            assert np.array_equal(got.cpu().numpy().astype(np.float64), ref[p]), (e, p)


def test_dequant_bit_exact_v3_samples(v3_shared_wide, v3_routed_wide):
    for data, L in (v3_shared_wide, v3_routed_wide):
        ref = data.dequant("s", 0)
        for p in range(3):
            got = L.dequant(-1, p)
            torch.cuda.synchronize()
            assert np.array_equal(got.cpu().numpy().astype(np.float64), ref[p])
    data, L = v3_routed_wide
    for e in np.nonzero(data.mask)[0][:6]:
        ref = data.dequant("r", int(e))
        for p in range(3):
            got = L.dequant(int(e), p)
            torch.cuda.synchronize()
            assert np.array_equal(got.cpu().numpy().astype(np.float64), ref[p]), (e, p)


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("n", [1, 3, 8, 40, 200])
def test_forward_tiny_wide(gpu_lib, tiny_wide, n, path):
    data, L = tiny_wide
    _forward_check(gpu_lib, data, L, n, "fwd-tiny-wide", path)


def test_forward_v3_shared_wide_decode(gpu_lib, v3_shared_wide):
    data, L = v3_shared_wide
    err = _forward_check(gpu_lib, data, L, 1, "fwd-v3-shw-b1", gpu_lib.MOEQ_PATH_AUTO)
    assert err.max() < 1e-3     # h in binary16 in the 2-4-bit down GEMV: about 2e-4
    _forward_check(gpu_lib, data, L, 16, "fwd-v3-shw-b16", gpu_lib.MOEQ_PATH_AUTO)


def test_forward_v3_shared_wide_prefill(gpu_lib, v3_shared_wide):
    data, L = v3_shared_wide
    n = 2048
    logits = synth.zipf_logits(n, data.mask, "fwd-v3-shw-prefill")
    _forward_check(gpu_lib, data, L, n, "fwd-v3-shw-prefill", gpu_lib.MOEQ_PATH_AUTO, logits=logits)


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("n", [1, 16, 300])
def test_forward_v3_routed_wide(gpu_lib, v3_routed_wide, n, path):
    data, L = v3_routed_wide
    _forward_check(gpu_lib, data, L, n, "fwd-v3-rw", path)


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("s", [-20, 12])
def test_forward_wide_activation_magnitudes(gpu_lib, tiny_wide, path, s):
    """x scaled by 2^s on the layer with every width of {2,3,4,5,6,8}: the
    5/6/8-bit kernels (bfloat16 activations, h as hi + lo parts on the decode
    path; the same binary16 prescales as the 2-4-bit GEMMs on the grouped-GEMM
    path) stay within the tolerance far from N(0, 1) activations."""
    data, L = tiny_wide
    shape = data.shape
    n = 3 if path == 1 else 40
    bits = layers.scaled_bits(synth.activations(n, shape.hidden, "fwd-wide-mag", f"s{s}", path), s)
    logits = synth.normal_logits(n, shape.n_experts, "fwd-wide-mag", f"s{s}", path)
    L.set_path(path)
    try:
        y = L.forward(_dev(bits.view(np.int16), torch.bfloat16), _dev(logits))
        torch.cuda.synchronize()
    finally:
        L.set_path(gpu_lib.MOEQ_PATH_AUTO)
    idx, w = router.route(logits, data.mask, n_group=shape.n_group, topk_group=shape.topk_group,
                          top_k=shape.top_k, group_topn=shape.group_topn, norm_topk=shape.norm_topk,
                          routed_scale=shape.routed_scale)
    ref = layers.oracle_forward(data, bits, idx, w)
    assert np.all(np.isfinite(y.cpu().numpy()))
    err = moe.token_errors(y.cpu().numpy(), ref)
    assert err.max() <= TOL, (s, path, err.max())
