"""Layer fixtures shared by the GPU tests: seeded weights in the canonical
packing, built either by the oracle's quantizer from N(0, 0.02) weights or as
uniformly random packed codes (any byte string is a valid packing)."""
import numpy as np

from inputs import synth
from oracle import moe, quant


class LayerData:
    """Canonical tensors of one layer plus what the oracle needs to rebuild them."""

    def __init__(self, shape, mask, bits_r, bits_s, make):
        self.shape, self.mask, self.bits_r, self.bits_s, self._make = shape, mask, bits_r, bits_s, make

    def tensor(self, kind, e, p):
        bits = int(self.bits_r[e, p] if kind == "r" else self.bits_s[e, p])
        return self._make(kind, e, p, bits)

    def routed(self):
        return {int(e): tuple(self.tensor("r", e, p) for p in range(3)) for e in np.nonzero(self.mask)[0]}

    def shared(self):
        return [tuple(self.tensor("s", s, p) for p in range(3)) for s in range(self.shape.n_shared)]

    def dequant(self, kind, e):
        """float64 (gate, up, down) of one expert, regenerated from its seed."""
        return tuple(moe.dequant_tensor(self.tensor(kind, e, p), self.shape.rows_cols(p)[1])
                     for p in range(3))


def quantized_layer(shape, plan, key):
    """N(0, 0.02) weights quantized by the oracle's quantizer."""
    mask = synth.expert_mask(shape, key)
    bits_r, bits_s = synth.bit_plan(shape, plan, key)

    def make(kind, e, p, bits):
        rows, K = shape.rows_cols(p)
        w = synth.normal_weights(rows, K, key, kind, e, p)
        codes, scales = quant.quantize(w, bits)
        return dict(bits=bits, codes=quant.pack(codes, bits), scales=scales)
    return LayerData(shape, mask, bits_r, bits_s, make)


def random_packed_layer(shape, plan, key, mask=None):
    """Uniformly random codes, scales spread around the typical N(0, 0.02) scale."""
    if mask is None:
        mask = synth.expert_mask(shape, key)
    bits_r, bits_s = synth.bit_plan(shape, plan, key)

    def make(kind, e, p, bits):
        rows, K = shape.rows_cols(p)
        codes, scales = synth.random_packed(rows, K, bits, key, kind, e, p)
        return dict(bits=bits, codes=codes, scales=scales)
    return LayerData(shape, mask, bits_r, bits_s, make)


class DeviceLayerData(LayerData):
    """Random packed tensors drawn on the GPU per tensor key
    (synth.device_random_packed): the layer is built from the device tensors,
    and the oracle regenerates any tensor it needs and copies it to the host."""

    def __init__(self, shape, plan, key, mask=None):
        import torch
        self._torch = torch
        if mask is None:
            mask = synth.expert_mask(shape, key)
        bits_r, bits_s = synth.bit_plan(shape, plan, key)
        self.key = key

        def make(kind, e, p, bits):
            dev = self.device_tensor(kind, e, p)
            return dict(bits=bits, codes=dev["codes"].cpu().numpy(),
                        scales=dev["scales"].cpu().numpy().view(np.uint16))
        super().__init__(shape, mask, bits_r, bits_s, make)

    def device_tensor(self, kind, e, p):
        bits = int(self.bits_r[e, p] if kind == "r" else self.bits_s[e, p])
        rows, K = self.shape.rows_cols(p)
        codes, scales = synth.device_random_packed(self._torch, rows, K, bits, self.key, kind, e, p)
        return dict(bits=bits, codes=codes, scales=scales)

    def make_layer(self, moeq, max_tokens, **kw):
        routed = {int(e): tuple(self.device_tensor("r", e, p) for p in range(3)) for e in np.nonzero(self.mask)[0]}
        shared = [tuple(self.device_tensor("s", s, p) for p in range(3)) for s in range(self.shape.n_shared)]
        self._torch.cuda.synchronize()
        return moeq.Layer(self.shape, self.mask, routed, shared, max_tokens=max_tokens, device_weights=True, **kw)


def oracle_forward(data, x_bits, idx, w):
    """The oracle's layer output for the given routing.  Every expert is
    dequantized once, when the oracle asks for it, and not kept."""
    shared = [data.dequant("s", s) for s in range(data.shape.n_shared)]
    return moe.moe_forward(x_bits, idx, w, lambda e: data.dequant("r", e), shared)


def scaled_bits(bits, s):
    """bfloat16 bit patterns times 2^s, exactly (the exponent field moves;
    the draws stay far from the bfloat16 range limits)."""
    f = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64) * 2.0 ** s
    out = (f.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal((out.astype(np.uint32) << 16).view(np.float32).astype(np.float64), f)
    return out
