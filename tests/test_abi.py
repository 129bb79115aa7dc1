"""The C interface on a machine without a GPU: the library loads, exports every
function its header declares, and rejects invalid arguments on the host
before any HIP runtime call."""
import ctypes

import numpy as np
import pytest

from inputs import synth

moeq = pytest.importorskip("paper_2509_25689_amd.moeq")


def test_exports_every_header_function():
    names = moeq.header_functions()
    assert "moeq_layer_create" in names and "moeq_forward" in names and "moeq_destroy" in names
    for name in names:
        assert hasattr(moeq.lib, name), name


def _cfg(**kw):
    shape = synth.TINY
    c = moeq.make_config(shape, max_tokens=8)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def _tensors(E, S, bits=4, codes=1, scales=1):
    r = (moeq.moeq_qtensor * (3 * E))(*[moeq.moeq_qtensor(bits, codes, scales)] * (3 * E))
    s = (moeq.moeq_qtensor * max(1, 3 * S))(*[moeq.moeq_qtensor(bits, codes, scales)] * max(1, 3 * S))
    return r, s


def _create(cfg, mask=None, bias=None, bits=4, codes=1, scales=1, loc=0, out=True):
    E = cfg.n_experts
    if mask is None:
        mask = np.ones(max(E, 1), np.uint8)
    r, s = _tensors(max(E, 1), max(cfg.n_shared, 0), bits, codes, scales)
    handle = ctypes.c_void_p()
    st = moeq.lib.moeq_layer_create(ctypes.byref(cfg), mask.ctypes.data,
                                    None if bias is None else bias.ctypes.data, r, s, loc,
                                    ctypes.byref(handle) if out else None)
    return st, handle


def test_peaks_library_exports_every_header_function():
    """The benchmark's roofline probes: a library of their own, every function
    of include/moeq_peaks.h exported."""
    from paper_2509_25689_amd import peaks
    lib = peaks.load()
    names = peaks.header_functions()
    assert set(names) == {"moeq_peaks_stream_read", "moeq_peaks_read_workgroups", "moeq_peaks_mfma",
                          "moeq_peaks_mfma_flops"}
    for name in names:
        assert hasattr(lib, name), name
    # host-only figures and argument checks (no GPU call is made)
    assert lib.moeq_peaks_read_workgroups(1 << 30) == (1 << 30) // (256 * 8 * 16)
    assert lib.moeq_peaks_mfma_flops(2, 3) == 2 * 4 * 3 * 8 * 2 * 16 * 16 * 32
    assert lib.moeq_peaks_stream_read(None, 16, None, None) != 0
    assert lib.moeq_peaks_mfma(0, 1, None, None) != 0


@pytest.mark.parametrize("field,value,status", [
    ("hidden", 0, moeq.MOEQ_ERR_INVALID_ARG),
    ("hidden", 500, moeq.MOEQ_ERR_INVALID_ARG),          # not a multiple of 32
    ("hidden", 544, moeq.MOEQ_ERR_UNSUPPORTED),          # multiple of 32, not of 128
    ("inter", 96, moeq.MOEQ_ERR_UNSUPPORTED),
    ("hidden", 16384, moeq.MOEQ_ERR_UNSUPPORTED),
    ("n_experts", 0, moeq.MOEQ_ERR_INVALID_ARG),
    ("n_experts", 2048, moeq.MOEQ_ERR_INVALID_ARG),
    ("n_group", 3, moeq.MOEQ_ERR_INVALID_ARG),           # 16 % 3 != 0
    ("topk_group", 0, moeq.MOEQ_ERR_INVALID_ARG),
    ("topk_group", 3, moeq.MOEQ_ERR_INVALID_ARG),        # > n_group
    ("top_k", 0, moeq.MOEQ_ERR_INVALID_ARG),
    ("top_k", 33, moeq.MOEQ_ERR_INVALID_ARG),
    ("group_topn", 0, moeq.MOEQ_ERR_INVALID_ARG),
    ("group_topn", 9, moeq.MOEQ_ERR_INVALID_ARG),        # > experts per group
    ("norm_topk", 2, moeq.MOEQ_ERR_INVALID_ARG),
    ("routed_scale", float("nan"), moeq.MOEQ_ERR_INVALID_ARG),
    ("routed_scale", float("inf"), moeq.MOEQ_ERR_INVALID_ARG),
    ("n_shared", -1, moeq.MOEQ_ERR_INVALID_ARG),
    ("n_shared", 5, moeq.MOEQ_ERR_INVALID_ARG),
    ("max_tokens", 0, moeq.MOEQ_ERR_INVALID_ARG),
    ("decode_max_tokens", 65, moeq.MOEQ_ERR_INVALID_ARG),
    ("decode_max_tokens", -1, moeq.MOEQ_ERR_INVALID_ARG),
])
def test_config_validation(field, value, status):
    st, h = _create(_cfg(**{field: value}))
    assert st == status, moeq.moeq_last_error()
    assert h.value is None
    assert moeq.moeq_last_error()


@pytest.mark.parametrize("bits", [0, 1, 7, 9, 16])
def test_bit_width_validation(bits):
    st, _ = _create(_cfg(), bits=bits)
    assert st == moeq.MOEQ_ERR_INVALID_ARG
    assert moeq.lib.moeq_quantize(1, 1, 32, bits, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG


@pytest.mark.parametrize("bits", [2, 3, 4, 5, 6, 8])
def test_every_supported_width_passes_validation(bits):
    """Validation accepts the width; without a device the call then stops at the device step."""
    st, _ = _create(_cfg(), bits=bits)
    assert st not in (moeq.MOEQ_ERR_INVALID_ARG, moeq.MOEQ_ERR_UNSUPPORTED), moeq.moeq_last_error()


def test_null_pointers():
    cfg = _cfg()
    assert _create(cfg, codes=0)[0] == moeq.MOEQ_ERR_INVALID_ARG
    assert _create(cfg, scales=0)[0] == moeq.MOEQ_ERR_INVALID_ARG
    assert _create(cfg, out=False)[0] == moeq.MOEQ_ERR_INVALID_ARG
    assert moeq.lib.moeq_layer_create(None, None, None, None, None, 0, None) == moeq.MOEQ_ERR_INVALID_ARG
    h = ctypes.c_void_p()
    assert moeq.lib.moeq_layer_create(ctypes.byref(cfg), None, None, None, None, 0,
                                      ctypes.byref(h)) == moeq.MOEQ_ERR_INVALID_ARG
    assert _create(cfg, loc=7)[0] == moeq.MOEQ_ERR_INVALID_ARG


def test_pruned_expert_tensors_are_not_read():
    """NULL tensors of a pruned expert are fine; a kept expert with NULL tensors is not.

    Real host buffers back every kept tensor, so on a GPU machine the create
    succeeds (and the layer is destroyed again)."""
    shape = synth.TINY
    cfg = _cfg()
    bufs = []
    def qt(p):
        rows, K = shape.rows_cols(p)
        c = np.zeros(rows * K // 2, np.uint8)
        s_ = np.zeros(rows * K // 32, np.uint16)
        bufs.extend([c, s_])
        return moeq.moeq_qtensor(4, c.ctypes.data, s_.ctypes.data)
    r = (moeq.moeq_qtensor * 48)(*[qt(i % 3) for i in range(48)])
    s = (moeq.moeq_qtensor * 3)(*[qt(i) for i in range(3)])
    mask = np.ones(16, np.uint8)
    mask[3] = 0
    for p in range(3):
        r[9 + p] = moeq.moeq_qtensor(4, 0, 0)
    h = ctypes.c_void_p()
    st = moeq.lib.moeq_layer_create(ctypes.byref(cfg), mask.ctypes.data, None, r, s, 0, ctypes.byref(h))
    assert st in (moeq.MOEQ_OK, moeq.MOEQ_ERR_DEVICE, moeq.MOEQ_ERR_OUT_OF_MEMORY), moeq.moeq_last_error()
    if h.value:
        moeq.lib.moeq_destroy(h)
    mask[3] = 1
    st = moeq.lib.moeq_layer_create(ctypes.byref(cfg), mask.ctypes.data, None, r, s, 0, ctypes.byref(h))
    assert st == moeq.MOEQ_ERR_INVALID_ARG


def test_infeasible_routing_rejected():
    cfg = _cfg(top_k=5)                              # 2 groups of 8, one group per token
    mask = np.ones(16, np.uint8)
    mask[:4] = 0                                     # group 0 keeps 4 < top_k
    assert _create(cfg, mask=mask)[0] == moeq.MOEQ_ERR_INVALID_ARG
    mask = np.zeros(16, np.uint8)
    mask[8:] = 1                                     # one non-empty group, topk_group 2
    assert _create(_cfg(topk_group=2), mask=mask)[0] == moeq.MOEQ_ERR_INVALID_ARG


def test_bias_validation():
    bias = np.zeros(16, np.float32)
    bias[2] = np.nan
    assert _create(_cfg(), bias=bias)[0] == moeq.MOEQ_ERR_INVALID_ARG
    bias[2] = 1e31
    assert _create(_cfg(), bias=bias)[0] == moeq.MOEQ_ERR_INVALID_ARG


def test_entry_points_reject_null_layer():
    L = moeq.lib
    assert L.moeq_forward(None, 1, 1, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_route(None, 1, 1, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_bucket(None, 1, 1, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_dequant(None, 0, 0, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_dequant_as(None, 0, 0, moeq.MOEQ_DECODER_GEMM_F16, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_set_path(None, 0) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_layer_bytes(None, None, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_set_router_weight(None, 1, moeq.MOEQ_WEIGHTS_HOST) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_router_logits(None, 1, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    L.moeq_destroy(None)                             # NULL-safe


def test_quantize_validation():
    L = moeq.lib
    assert L.moeq_quantize(None, 1, 32, 4, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_quantize(1, 1, 33, 4, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_quantize(1, -1, 32, 4, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_quantize(1, 1, 32, 7, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_quantize(1, 1, 32, 1, 1, 1, None) == moeq.MOEQ_ERR_INVALID_ARG
    assert L.moeq_quantize(1, 0, 32, 4, 1, 1, None) == moeq.MOEQ_OK   # empty: nothing to do


def test_error_text_is_per_call():
    _create(_cfg(top_k=0))
    assert "top_k" in moeq.moeq_last_error()
    with pytest.raises(moeq.MoeqError) as ei:
        moeq.moeq_set_path(None, 0)
    assert ei.value.status == moeq.MOEQ_ERR_INVALID_ARG


def test_expert_importance_validation():
    """Every argument check of moeq_expert_importance runs before any HIP call."""
    lib = moeq.lib
    cfg = _cfg()
    E = cfg.n_experts
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first

    def call(c=cfg, bias=None, logits=fake, n=8, alpha=0.5, retain=0.75, imp=fake, mask=fake):
        return lib.moeq_expert_importance(ctypes.byref(c) if c is not None else None, bias, logits, n,
                                          alpha, retain, imp, mask, None, None)

    assert call(c=None) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(n=0) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(logits=None) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(imp=None) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(mask=None) == moeq.MOEQ_ERR_INVALID_ARG
    for a in (-0.1, 1.5, float("nan")):
        assert call(alpha=a) == moeq.MOEQ_ERR_INVALID_ARG
    for r in (0.0, -1.0, 1.01, float("nan")):
        assert call(retain=r) == moeq.MOEQ_ERR_INVALID_ARG
    bad = np.zeros(E, np.float32)
    bad[3] = np.inf
    assert call(bias=bad.ctypes.data) == moeq.MOEQ_ERR_INVALID_ARG
    assert "score_bias" in moeq.moeq_last_error()
    # top_k larger than what topk_group groups can hold even with every expert kept
    c2 = _cfg(topk_group=1, top_k=12)
    assert call(c=c2) == moeq.MOEQ_ERR_INVALID_ARG


def test_expert_importance_noalloc_validation():
    """The entry point without allocation checks what the allocating one checks,
    and the size of its static scratch, all before any HIP call."""
    lib = moeq.lib
    cfg = _cfg()
    fake = ctypes.c_void_p(16)

    def call(c=cfg, logits=fake, n=8, alpha=0.5, retain=0.75, imp=fake, mask=fake):
        return lib.moeq_expert_importance_noalloc(ctypes.byref(c) if c is not None else None, None, logits, n,
                                                  alpha, retain, imp, mask, None, None)

    assert call(c=None) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(n=0) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(logits=None) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(alpha=2.0) == moeq.MOEQ_ERR_INVALID_ARG
    assert call(retain=0.0) == moeq.MOEQ_ERR_INVALID_ARG
    # 16 bytes per (token, slot) of ids, weights, ranks and permutation alone:
    # 2^20 tokens at top_k 2 need 32 MiB, more than the 16 MiB static scratch
    assert call(n=1 << 20) == moeq.MOEQ_ERR_CAPACITY
    assert "static scratch" in moeq.moeq_last_error()


def test_regroup_validation():
    """regroup must be 0 or 1 and needs a kept count divisible by n_group."""
    assert _create(_cfg(regroup=2))[0] == moeq.MOEQ_ERR_INVALID_ARG
    E = synth.TINY.n_experts
    mask = np.ones(E, np.uint8)
    mask[:3] = 0                      # 13 kept, not a multiple of 2 groups
    assert _create(_cfg(regroup=1), mask=mask)[0] == moeq.MOEQ_ERR_INVALID_ARG
    assert "multiple of n_group" in moeq.moeq_last_error()
