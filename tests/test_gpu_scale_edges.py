"""Block scales at the edges of the grouped GEMMs' register decoder.

That decoder forms binary16(d * (c - z)) with one fused multiply-add from
d * 2^(14 + b), so it takes a tensor only if every scale is a positive finite
binary16 no larger than the largest d for which that product stays finite; a
scan at layer creation sends every other 2-4-bit tensor to the LDS-decoded
GEMMs, whose decoder has no such bound.  Both must produce the format's
binary16 weights bit for bit (the oracle's dequantize_half: Section 3.3's
weight = d * (c - 2^(b-1)), rounded once) and a prefill forward within the
output tolerance of the fp64 oracle.

Edits on the tiny layer (one per tensor, the rest of the tensor unchanged):
* shared gate: every scale times 64 (far above the bound at any width);
* a routed down tensor: one block scale zero;
* a routed up tensor: one block scale negated;
* a routed gate tensor: one block scale the smallest positive subnormal
  (still on the register decoder);
* another routed down tensor: one block scale exactly at the bound (still on
  the register decoder; d * 2^(14 + b) is the largest finite binary16)."""
import numpy as np
import pytest
import torch

import layers
from inputs import synth
from oracle import moe, quant, router

pytestmark = pytest.mark.gpu

TOL = 2e-3


def rd_scale_limit(bits):
    """The largest scale bit pattern the register decoder takes (binary16 d
    with d * 2^(14 + bits) at most 65504)."""
    return 0x7BFF - ((14 + bits) << 10)


class EditedLayer(layers.LayerData):
    def __init__(self, base, edits):
        super().__init__(base.shape, base.mask, base.bits_r, base.bits_s, base._make)
        self._edits = edits

    def tensor(self, kind, e, p):
        t = dict(super().tensor(kind, e, p))
        f = self._edits.get((kind, int(e), p))
        if f is not None:
            t["scales"] = f(np.array(t["scales"], dtype=np.uint16), t["bits"])
        return t


def _times64(s, bits):
    return (s.view(np.float16).astype(np.float32) * 64.0).astype(np.float16).view(np.uint16)


def _set_block(value):
    def f(s, bits):
        s = s.copy()
        s[1, 2] = value(s[1, 2], bits)
        return s
    return f


@pytest.fixture(scope="module")
def edited(gpu_lib):
    base = layers.quantized_layer(synth.TINY, "p234_602020", "scale-edges")
    kept = [int(e) for e in np.nonzero(base.mask)[0]]
    edits = {
        ("s", 0, 0): _times64,
        ("r", kept[0], 2): _set_block(lambda v, b: 0),
        ("r", kept[1], 1): _set_block(lambda v, b: int(v) | 0x8000),
        ("r", kept[2], 0): _set_block(lambda v, b: 1),
        ("r", kept[3], 2): _set_block(lambda v, b: rd_scale_limit(b)),
    }
    data = EditedLayer(base, edits)
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=256)
    yield data, L, edits
    L.close()


def test_gemm_decoder_bit_exact_at_scale_edges(gpu_lib, edited):
    data, L, edits = edited
    for kind, e, p in list(edits) + [("r", int(np.nonzero(data.mask)[0][5]), 1)]:
        t = data.tensor(kind, e, p)
        K = data.shape.rows_cols(p)[1]
        codes = quant.unpack(t["codes"], t["bits"], K)
        want = quant.dequantize_half(codes, t["scales"], t["bits"])
        eid = e if kind == "r" else -1 - e
        got = L.dequant_as(eid, p, gpu_lib.MOEQ_DECODER_GEMM_F16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, want), (kind, e, p, t["bits"])


def test_scale_edges_reach_both_decoders(edited):
    """The edits hit both sides of the bound, so both GEMM families run."""
    data, _, edits = edited
    lim_over, lim_under = 0, 0
    for kind, e, p in edits:
        t = data.tensor(kind, e, p)
        s = np.asarray(t["scales"], dtype=np.uint16)
        bad = ((s & 0x8000) != 0) | ((s & 0x7FFF) == 0) | ((s & 0x7FFF) > rd_scale_limit(t["bits"]))
        lim_over += bool(bad.any())
        lim_under += bool(not bad.any())
    assert lim_over == 3 and lim_under == 2


@pytest.mark.parametrize("path", [1, 2])
def test_forward_at_scale_edges(gpu_lib, edited, path):
    data, L, _ = edited
    shape = data.shape
    n = 200
    x_bits = synth.activations(n, shape.hidden, "scale-edges-x", path)
    logits = synth.normal_logits(n, shape.n_experts, "scale-edges-l", path)
    x = torch.from_numpy(x_bits.view(np.int16)).cuda().view(torch.bfloat16)
    L.set_path(path)
    y = L.forward(x, torch.from_numpy(logits).cuda())
    torch.cuda.synchronize()
    L.set_path(gpu_lib.MOEQ_PATH_AUTO)
    idx, w = router.route(logits, data.mask, n_group=shape.n_group, topk_group=shape.topk_group,
                          top_k=shape.top_k, group_topn=shape.group_topn, norm_topk=shape.norm_topk,
                          routed_scale=shape.routed_scale, regroup=bool(shape.regroup))
    ref = layers.oracle_forward(data, x_bits, idx, w)
    err = moe.token_errors(y.cpu().numpy(), ref)
    assert err.max() <= TOL, (err.max(), np.median(err))
