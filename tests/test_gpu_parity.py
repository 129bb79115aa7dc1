"""Parity of the HIP path with the CPU oracle, through the C interface.

Bit-exact: quantizer codes and scales, dequantized weights, router indices,
bucketing offsets and permutation.  Floating point: routing weights within
1e-6 relative; layer outputs within a per-token normwise error of 2e-3
(max |y - ref| / max |ref|, float64 reference), on both forward paths.

Sizes: the tiny layer (several tiles, ragged buckets) and the
DeepSeek-V3-shape layer at the sizes the benchmark runs (batch 1 and 16
decode, 2048-token Zipf-routed prefill), every token compared."""
import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import bucket as obucket
from oracle import moe, quant, router

pytestmark = pytest.mark.gpu

TOL = 2e-3


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.view(dtype)


def _x(n, H, *key):
    bits = synth.activations(n, H, *key)
    return bits, _dev(bits.view(np.int16), torch.bfloat16)


def _route_oracle(shape, mask, logits):
    return router.route(logits, mask, n_group=shape.n_group, topk_group=shape.topk_group,
                        top_k=shape.top_k, group_topn=shape.group_topn,
                        norm_topk=shape.norm_topk, routed_scale=shape.routed_scale,
                        regroup=bool(shape.regroup))


def _make_layer(moeq, data, max_tokens, **kw):
    return moeq.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=max_tokens, **kw)


@pytest.fixture(scope="module")
def tiny(gpu_lib):
    data = layers.quantized_layer(synth.TINY, "all4", "tiny")
    L = _make_layer(gpu_lib, data, max_tokens=200)
    yield data, L
    L.close()


@pytest.fixture(scope="module")
def tiny_mixed(gpu_lib):
    data = layers.quantized_layer(synth.TINY, "p234_602020", "tiny-mixed")
    L = _make_layer(gpu_lib, data, max_tokens=200)
    yield data, L
    L.close()


@pytest.fixture(scope="module")
def v3_decode(gpu_lib):
    data = layers.DeviceLayerData(synth.V3, "gu3_d4_sh4", "v3_decode")
    L = data.make_layer(gpu_lib, max_tokens=64)
    yield data, L
    L.close()


@pytest.fixture(scope="module")
def v3_prefill(gpu_lib):
    data = layers.DeviceLayerData(synth.V3, "p234_602020", "v3_prefill")
    L = data.make_layer(gpu_lib, max_tokens=2048)
    yield data, L
    L.close()


# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bits", [2, 3, 4])
def test_quantize_bit_exact(gpu_lib, bits):
    w = synth.normal_weights(96, 7168, "quantize", bits)
    w[0, :32] = 0.0                                          # a zero block
    w[1, :32] = np.float32(0.01) * np.arange(32, dtype=np.float32)
    w[2, :32] = np.float32(0.5) * np.arange(-16, 16, dtype=np.float32)  # ties at half codes
    codes, scales = gpu_lib.quantize(_dev(w), bits)
    torch.cuda.synchronize()
    ref_c, ref_s = quant.quantize(w, bits)
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), ref_s)
    assert np.array_equal(codes.cpu().numpy(), quant.pack(ref_c, bits))


@pytest.mark.parametrize("which", ["tiny", "tiny_mixed"])
def test_dequant_bit_exact_every_tensor(request, which):
    data, L = request.getfixturevalue(which)
    slots = [("r", int(e)) for e in np.nonzero(data.mask)[0]] + [("s", s) for s in range(data.shape.n_shared)]
    for kind, e in slots:
        ref = data.dequant(kind, e)
        for p in range(3):
            got = L.dequant(e if kind == "r" else -1 - e, p).cpu().numpy()
            assert np.array_equal(got.astype(np.float64), ref[p]), (kind, e, p)


def test_dequant_bit_exact_v3_sample(v3_prefill):
    data, L = v3_prefill
    kept = np.nonzero(data.mask)[0]
    for e in [int(kept[0]), int(kept[77]), int(kept[-1])]:
        ref = data.dequant("r", e)
        for p in range(3):
            got = L.dequant(e, p).cpu().numpy()
            assert np.array_equal(got.astype(np.float64), ref[p]), (e, p, data.bits_r[e, p])


# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n", [1, 5, 8, 64, 65, 200])
def test_route_tiny(tiny, n):
    data, L = tiny
    logits = synth.normal_logits(n, data.shape.n_experts, "route", n)
    idx, w = L.route(_dev(logits))
    torch.cuda.synchronize()
    ridx, rw = _route_oracle(data.shape, data.mask, logits)
    assert np.array_equal(idx.cpu().numpy(), ridx)
    assert np.allclose(w.cpu().numpy(), rw, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("n,kind", [(1, "normal"), (16, "normal"), (64, "normal"), (65, "zipf"),
                                    (2048, "zipf")])
def test_route_v3(v3_prefill, n, kind):
    data, L = v3_prefill
    E = data.shape.n_experts
    logits = (synth.normal_logits(n, E, "route-v3", n) if kind == "normal"
              else synth.zipf_logits(n, data.mask, "route-v3", n))
    idx, w = L.route(_dev(logits))
    torch.cuda.synchronize()
    ridx, rw = _route_oracle(data.shape, data.mask, logits)
    assert np.array_equal(idx.cpu().numpy(), ridx)
    assert np.allclose(w.cpu().numpy(), rw, rtol=1e-6, atol=1e-7)


def test_route_ties(tiny):
    """Logits from four values: exact score ties everywhere; lower ids must win."""
    data, L = tiny
    r = np.random.default_rng(7)
    logits = r.choice(np.array([-1.0, 0.0, 0.5, 1.0], np.float32), (64, data.shape.n_experts))
    idx, _ = L.route(_dev(logits))
    torch.cuda.synchronize()
    ridx, _ = _route_oracle(data.shape, data.mask, logits)
    assert np.array_equal(idx.cpu().numpy(), ridx)


@pytest.mark.parametrize("n", [1, 2, 16, 63, 64, 65, 130, 2048])
def test_bucket_bit_exact(v3_prefill, n):
    data, L = v3_prefill
    logits = synth.zipf_logits(n, data.mask, "bucket", n)
    ridx, _ = _route_oracle(data.shape, data.mask, logits)
    offsets, perm = L.bucket(_dev(ridx.astype(np.int32)))
    torch.cuda.synchronize()
    roff, rperm, _ = obucket.bucket(ridx, data.shape.n_experts)
    assert np.array_equal(offsets.cpu().numpy(), roff)
    assert np.array_equal(perm.cpu().numpy(), rperm)


# ---------------------------------------------------------------------------
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
    idx, w = _route_oracle(shape, data.mask, logits[rows])
    ref = layers.oracle_forward(data, x_bits[rows], idx, w)
    err = moe.token_errors(y.cpu().numpy()[rows], ref)
    assert err.max() <= TOL, (err.max(), np.median(err))
    return err


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("n", [1, 3, 8, 40, 200])
def test_forward_tiny(gpu_lib, tiny, n, path):
    data, L = tiny
    _forward_check(gpu_lib, data, L, n, "fwd-tiny", path)


@pytest.mark.parametrize("n", [64, 65, 128, 129, 192, 193])
@pytest.mark.parametrize("which", ["tiny", "tiny_mixed"])
def test_prefill_tile_edges(request, gpu_lib, which, n):
    """Every token routed to the same two kept experts, so those buckets and
    the shared expert's hold n rows each: one 64-row tile (n = 64), one
    128-row tile of 65 or 128 rows, a 128-row tile plus a 64-row tile of 1
    or 64 rows (129, 192), two 128-row tiles (193); grouped-GEMM path."""
    data, L = request.getfixturevalue(which)
    shape = data.shape
    kept = np.nonzero(data.mask)[0]
    per = shape.n_experts // shape.n_group
    pair = [int(e) for e in kept if e // per == kept[0] // per][:2]
    logits = (0.1 * synth.normal_logits(n, shape.n_experts, "tile-edges", n)).astype(np.float32)
    logits[:, pair] += 8.0
    ridx, _ = _route_oracle(shape, data.mask, logits)
    assert (np.sort(ridx, axis=1) == np.array(sorted(pair))).all()
    _forward_check(gpu_lib, data, L, n, "tile-edges", gpu_lib.MOEQ_PATH_PREFILL, logits=logits)


@pytest.mark.parametrize("n", [23, 24, 25])
@pytest.mark.parametrize("which", ["tiny", "tiny_mixed"])
def test_decode_hybrid_cutover(request, gpu_lib, which, n):
    """The decode path around its hybrid cutover: from 24 tokens, buckets of
    more than 2 rows take the grouped GEMMs and the smaller ones the
    dequant-GEMV kernels, both summed by one combine (below 24 tokens every
    bucket takes the GEMVs).  The inputs give buckets on both sides of that
    size, which the oracle's routing confirms here; every token compared."""
    data, L = request.getfixturevalue(which)
    shape = data.shape
    logits = synth.normal_logits(n, shape.n_experts, "hybrid-cutover", n)
    idx, _ = _route_oracle(shape, data.mask, logits)
    sizes = np.bincount(idx.ravel())
    sizes = sizes[sizes > 0]
    assert (sizes <= 2).any() and (sizes > 2).any(), sizes
    _forward_check(gpu_lib, data, L, n, "hybrid-cutover", gpu_lib.MOEQ_PATH_DECODE, logits=logits)


@pytest.mark.parametrize("path", [1, 2])
def test_forward_tiny_mixed_bits(gpu_lib, tiny_mixed, path):
    data, L = tiny_mixed
    _forward_check(gpu_lib, data, L, 33, "fwd-tiny-mixed", path)


def test_forward_v3_decode_batch1(gpu_lib, v3_decode):
    data, L = v3_decode
    for i in range(3):
        err = _forward_check(gpu_lib, data, L, 1, f"fwd-v3-b1-{i}", gpu_lib.MOEQ_PATH_AUTO)
        # h enters the down products in binary16 (relative rounding 2^-11 per
        # element after a power-of-two prescale per block), everything else
        # is exact products with float32 accumulation: about 2e-4
        assert err.max() < 1e-3


def test_forward_v3_decode_batch16(gpu_lib, v3_decode):
    data, L = v3_decode
    _forward_check(gpu_lib, data, L, 16, "fwd-v3-b16", gpu_lib.MOEQ_PATH_AUTO)


@pytest.mark.parametrize("n,kind", [(23, "zipf"), (24, "zipf"), (48, "normal"), (64, "zipf")])
def test_forward_v3_auto_gemv(gpu_lib, v3_prefill, n, kind):
    """23-64 tokens on the automatic path (the decode path by default):
    buckets of one token through the one-token gate/up kernel, those of 2
    through the 2-64-token GEMVs, and from 24 tokens the larger ones through
    the grouped GEMMs (below 24 through the 2-64-token GEMVs too); mixed
    2/3/4-bit widths."""
    data, L = v3_prefill
    E = data.shape.n_experts
    logits = (synth.normal_logits(n, E, "fwd-v3-auto", n) if kind == "normal"
              else synth.zipf_logits(n, data.mask, "fwd-v3-auto", n))
    _forward_check(gpu_lib, data, L, n, "fwd-v3-auto", gpu_lib.MOEQ_PATH_AUTO, logits=logits)


def test_forward_v3_prefill(gpu_lib, v3_prefill):
    """The 2048-token Zipf-routed prefill, every token: buckets from 1598 rows
    (13 tiles of 128) down to a few rows, the shared expert's 16 full tiles,
    mixed 2/3/4-bit tensors."""
    data, L = v3_prefill
    n = 2048
    logits = synth.zipf_logits(n, data.mask, "fwd-v3-prefill")
    err = _forward_check(gpu_lib, data, L, n, "fwd-v3-prefill", gpu_lib.MOEQ_PATH_AUTO, logits=logits)
    print(f"prefill 2048 tokens: worst per-token error {err.max():.2e}, median {np.median(err):.2e}")


# ---------------------------------------------------------------------------
def test_deterministic(tiny):
    data, L = tiny
    _, x = _x(40, data.shape.hidden, "det")
    lg = _dev(synth.normal_logits(40, data.shape.n_experts, "det"))
    y1 = L.forward(x, lg).clone()
    y2 = L.forward(x, lg)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


def test_zero_tokens_is_noop(gpu_lib, tiny):
    data, L = tiny
    y = torch.full((1, data.shape.hidden), 7.0, device="cuda")
    x = torch.zeros((1, data.shape.hidden), dtype=torch.bfloat16, device="cuda")
    lg = torch.zeros((1, data.shape.n_experts), device="cuda")
    gpu_lib.moeq_forward(L.handle, x.data_ptr(), lg.data_ptr(), 0, y.data_ptr(),
                         torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.all(y == 7.0)


def test_capacity_and_alignment_errors(gpu_lib, tiny):
    data, L = tiny
    x = torch.zeros((201, data.shape.hidden), dtype=torch.bfloat16, device="cuda")
    lg = torch.zeros((201, data.shape.n_experts), device="cuda")
    y = torch.empty((201, data.shape.hidden), device="cuda")
    with pytest.raises(gpu_lib.MoeqError) as ei:
        gpu_lib.moeq_forward(L.handle, x.data_ptr(), lg.data_ptr(), 201, y.data_ptr(), 0)
    assert ei.value.status == gpu_lib.MOEQ_ERR_CAPACITY
    with pytest.raises(gpu_lib.MoeqError) as ei:
        gpu_lib.moeq_forward(L.handle, x.data_ptr() + 2, lg.data_ptr(), 1, y.data_ptr(), 0)
    assert ei.value.status == gpu_lib.MOEQ_ERR_INVALID_ARG
    with pytest.raises(gpu_lib.MoeqError):
        L.dequant(int(np.nonzero(data.mask == 0)[0][0]), 0)       # a pruned expert
    wb, wsb = L.bytes()
    n_kept = int(data.mask.sum())
    assert wb == (n_kept + 1) * sum(quant.tensor_bytes(*data.shape.rows_cols(p), 4) for p in range(3))
    assert wsb > 0


def test_device_resident_weights(gpu_lib):
    """Weights handed over as device pointers give the same layer."""
    data = layers.quantized_layer(synth.TINY, "p234_602020", "device-weights")
    routed = {e: tuple(dict(bits=t["bits"], codes=_dev(t["codes"]), scales=_dev(t["scales"].view(np.int16)))
                       for t in tr) for e, tr in data.routed().items()}
    shared = [tuple(dict(bits=t["bits"], codes=_dev(t["codes"]), scales=_dev(t["scales"].view(np.int16)))
                    for t in tr) for tr in data.shared()]
    L = gpu_lib.Layer(data.shape, data.mask, routed, shared, max_tokens=16, device_weights=True)
    _forward_check(gpu_lib, data, L, 16, "device-weights", gpu_lib.MOEQ_PATH_AUTO)
    L.close()


# ---------------------------------------------------------------------------
# Section 3.2's activation adjustment: after keeping r = 0.75 of the experts,
# each token activates ceil(r * 8) = 6 of them instead of 8.
@pytest.fixture(scope="module")
def v3_k6(gpu_lib):
    import dataclasses
    shape = dataclasses.replace(synth.V3, top_k=6)
    data = layers.DeviceLayerData(shape, "gu3_d4_sh4", "v3_k6")
    L = data.make_layer(gpu_lib, max_tokens=300)
    yield data, L
    L.close()


@pytest.mark.parametrize("n", [1, 16, 100])
def test_route_v3_k6(v3_k6, n):
    data, L = v3_k6
    logits = synth.normal_logits(n, data.shape.n_experts, "route-k6", n)
    idx, w = L.route(_dev(logits))
    ref_idx, ref_w = _route_oracle(data.shape, data.mask, logits)
    assert idx.shape[1] == 6
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_allclose(w.cpu().numpy(), ref_w, atol=1e-6 * data.shape.routed_scale)


def test_forward_v3_k6_decode(gpu_lib, v3_k6):
    data, L = v3_k6
    err = _forward_check(gpu_lib, data, L, 1, "fwd-k6-b1", gpu_lib.MOEQ_PATH_AUTO)
    assert err.max() < 1e-3     # h in binary16 in the 2-4-bit down GEMV: about 2e-4
    _forward_check(gpu_lib, data, L, 16, "fwd-k6-b16", gpu_lib.MOEQ_PATH_AUTO)


def test_forward_v3_k6_prefill(gpu_lib, v3_k6):
    data, L = v3_k6
    _forward_check(gpu_lib, data, L, 300, "fwd-k6-prefill", gpu_lib.MOEQ_PATH_PREFILL)


# ---------------------------------------------------------------------------
# Section 3.2 read literally: the kept experts are partitioned into groups of
# their own (regroup = 1) instead of masking the original groups.
@pytest.fixture(scope="module", params=["tiny", "v3"])
def regrouped(gpu_lib, request):
    import dataclasses
    base = synth.TINY if request.param == "tiny" else synth.V3
    shape = dataclasses.replace(base, regroup=1)
    data = layers.random_packed_layer(shape, "all4" if request.param == "tiny" else "gu3_d4_sh4",
                                      f"regroup-{request.param}")
    L = _make_layer(gpu_lib, data, max_tokens=128)
    yield data, L
    L.close()


@pytest.mark.parametrize("n", [1, 16, 100])
def test_route_regrouped(regrouped, n):
    data, L = regrouped
    logits = synth.normal_logits(n, data.shape.n_experts, "route-regroup", n)
    idx, w = L.route(_dev(logits))
    ref_idx, ref_w = _route_oracle(data.shape, data.mask, logits)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_allclose(w.cpu().numpy(), ref_w, atol=1e-6 * data.shape.routed_scale)
    # the seeded masks leave the original groups uneven, so the two readings differ
    masked, _ = router.route(logits, data.mask, n_group=data.shape.n_group, topk_group=data.shape.topk_group,
                             top_k=data.shape.top_k, group_topn=data.shape.group_topn)
    if n >= 16:
        assert not np.array_equal(masked, ref_idx)


@pytest.mark.parametrize("path", [1, 2])
def test_forward_regrouped(gpu_lib, regrouped, path):
    data, L = regrouped
    _forward_check(gpu_lib, data, L, 24, "fwd-regroup", path)



@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("s", [-20, -8, 6, 12])
def test_forward_activation_magnitudes(gpu_lib, tiny_mixed, path, s):
    """x scaled by 2^s, far from N(0, 1): the activations enter the GEMVs and
    GEMMs in binary16 after power-of-two prescales (per block of 32 on the
    decode path, per token / per h row on the grouped-GEMM path), and h
    reaches about 2^(2s) times its usual size.  The layer must stay within
    the tolerance at every scale, on both paths and all 2/3/4-bit widths."""
    data, L = tiny_mixed
    shape = data.shape
    n = 3 if path == 1 else 40
    bits = layers.scaled_bits(synth.activations(n, shape.hidden, "fwd-mag", f"s{s}", path), s)
    logits = synth.normal_logits(n, shape.n_experts, "fwd-mag", f"s{s}", path)
    L.set_path(path)
    try:
        y = L.forward(_dev(bits.view(np.int16), torch.bfloat16), _dev(logits))
        torch.cuda.synchronize()
    finally:
        L.set_path(gpu_lib.MOEQ_PATH_AUTO)
    idx, w = _route_oracle(shape, data.mask, logits)
    ref = layers.oracle_forward(data, bits, idx, w)
    assert np.all(np.isfinite(y.cpu().numpy()))
    err = moe.token_errors(y.cpu().numpy(), ref)
    assert err.max() <= TOL, (s, path, err.max())


def test_binding_rejects_mismatched_tensors(gpu_lib, tiny):
    """The Python layer checks dtype, shape, layout and device before it
    hands pointers to the kernels, which trust them."""
    data, L = tiny
    H, E = data.shape.hidden, data.shape.n_experts
    x = torch.zeros((4, H), dtype=torch.bfloat16, device="cuda")
    lg = torch.zeros((4, E), device="cuda")
    bad = [
        (x.float(), lg),                                              # dtype
        (x, lg[:, : E - 1].contiguous()),                             # logits too narrow
        (torch.zeros((4, 2 * H), dtype=torch.bfloat16, device="cuda")[:, ::2], lg),  # not contiguous
        (x.cpu(), lg),                                                # host tensor
    ]
    for xb, lb in bad:
        with pytest.raises((ValueError, TypeError)):
            L.forward(xb, lb)
    with pytest.raises(ValueError):
        L.forward(x, lg, y=torch.empty((3, H), device="cuda"))       # y too small
    with pytest.raises(ValueError):
        L.route(lg.double())
    with pytest.raises(ValueError):
        L.bucket(torch.zeros((4, data.shape.top_k), dtype=torch.int64, device="cuda"))
