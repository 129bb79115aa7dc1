"""Pins for the oracle's bucketing and expert/combine arithmetic.

* bucketing against a brute-force per-expert scan and its invariants;
* the identity-weight fixture, in which the layer output reproduces the
  dense combine-weight matrix;
* zero routed weights leave the shared expert alone;
* the float64 forward against explicit per-token, per-slot Python loops;
* silu's closed forms."""
import numpy as np
import pytest

from oracle import bucket, moe, quant, router
from inputs import synth


def test_bucket_matches_bruteforce_scan():
    r = np.random.default_rng(0)
    for n, k, E in [(1, 8, 256), (5, 3, 16), (64, 8, 256), (0, 2, 16)]:
        idx = np.stack([r.choice(E, k, replace=False) for _ in range(n)]) if n else \
            np.zeros((0, k), np.int32)
        offsets, perm, active = bucket.bucket(idx, E)
        expect = []
        for e in range(E):
            for t in range(n):
                for j in range(k):
                    if idx[t, j] == e:
                        expect.append(t * k + j)
        assert perm.tolist() == expect
        assert offsets[E] == n * k and offsets[0] == 0
        assert np.all(np.diff(offsets) >= 0)
        assert sorted(perm.tolist()) == list(range(n * k))
        for e in range(E):
            seg = perm[offsets[e]:offsets[e + 1]]
            assert np.all(idx.ravel()[seg] == e)
        assert active.tolist() == [e for e in range(E) if offsets[e + 1] > offsets[e]]


def test_bucket_of_routed_tokens_skips_pruned():
    shape = synth.V3
    mask = synth.expert_mask(shape, "pin")
    logits = synth.normal_logits(16, shape.n_experts, "pin")
    idx, _ = router.route(logits, mask, n_group=8, topk_group=4, top_k=8, routed_scale=2.5)
    offsets, _, active = bucket.bucket(idx, shape.n_experts)
    counts = np.diff(offsets)
    assert np.all(counts[mask == 0] == 0)
    assert np.all(mask[active] == 1)


def test_silu_closed_forms():
    assert moe.silu(np.array([0.0]))[0] == 0.0
    assert moe.silu(np.array([40.0]))[0] == pytest.approx(40.0, rel=1e-15)
    assert moe.silu(np.array([-800.0]))[0] == 0.0
    assert moe.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + np.exp(-1.0)), rel=1e-15)


def _identity_fixture(E, H, I, kept, bits=4):
    """Every kept expert: W_gate[0,0] = W_up[0,0] = c, W_down[e,0] = v, all else 0.

    With x[:, 0] = 1 every expert has h_0 = silu(c) * c and h_i = 0 otherwise,
    so y[t, e] = w(t, e) * v * h_0 on the first E coordinates and 0 elsewhere."""
    c, v = 7.0 / 16.0, 7.0 / 32.0        # amax / 7 is a power of two: both on the 4-bit grid
    def tensor(rows, K, entries):
        w = np.zeros((rows, K), np.float32)
        for (i, j), val in entries.items():
            w[i, j] = val
        codes, scales = quant.quantize(w, bits)
        return dict(bits=bits, codes=quant.pack(codes, bits), scales=scales)
    routed = {}
    for e in np.nonzero(kept)[0]:
        routed[int(e)] = (tensor(I, H, {(0, 0): c}), tensor(I, H, {(0, 0): c}),
                          tensor(H, I, {(int(e), 0): v}))
    shared = (tensor(I, H, {}), tensor(I, H, {}), tensor(H, I, {}))
    return routed, shared, c, v


def test_identity_weight_fixture_reproduces_combine_weights():
    shape = synth.TINY
    E, H, I = shape.n_experts, shape.hidden, shape.inter
    mask = synth.expert_mask(shape, "pin")
    routed_t, shared_t, c, v = _identity_fixture(E, H, I, mask)
    # the grid value survives quantization exactly
    e0 = int(np.nonzero(mask)[0][0])
    assert moe.dequant_tensor(routed_t[e0][0], H)[0, 0] == c
    assert moe.dequant_tensor(routed_t[e0][2], I)[e0, 0] == v
    n = 8
    x = synth.activations(n, H, "pin")
    x[:, 0] = synth.bf16_from_f32(np.ones(n, np.float32))
    logits = synth.normal_logits(n, E, "pin")
    idx, w = router.route(logits, mask, n_group=2, topk_group=1, top_k=2, routed_scale=2.5)
    deq = lambda e: tuple(moe.dequant_tensor(t, K) for t, K in zip(routed_t[e], (H, H, I)))
    shared = [tuple(moe.dequant_tensor(t, K) for t, K in zip(shared_t, (H, H, I)))]
    y = moe.moe_forward(x, idx, w, deq, shared)
    h0 = moe.silu(np.array([c]))[0] * c
    dense = np.zeros((n, E))
    for t in range(n):
        for j in range(2):
            dense[t, idx[t, j]] = w[t, j]
    assert np.allclose(y[:, :E], dense * v * h0, rtol=1e-14, atol=0)
    assert np.all(y[:, E:] == 0)


def test_zero_routed_weights_leave_shared_only():
    r = np.random.default_rng(2)
    n, H, I = 3, 64, 32
    x = synth.bf16_from_f32(r.standard_normal((n, H)).astype(np.float32))
    zeros = (np.zeros((I, H)), np.zeros((I, H)), np.zeros((H, I)))
    sh = (r.standard_normal((I, H)), r.standard_normal((I, H)), r.standard_normal((H, I)))
    idx = np.array([[0, 1], [1, 2], [2, 0]])
    w = r.random((n, 2))
    y = moe.moe_forward(x, idx, w, lambda e: zeros, [sh])
    assert np.allclose(y, moe.expert_ffn(moe.bf16_bits_to_f64(x), *sh), rtol=1e-14, atol=0)


def test_forward_matches_explicit_loops():
    r = np.random.default_rng(4)
    n, H, I, E, k = 3, 16, 8, 4, 2
    x = synth.bf16_from_f32(r.standard_normal((n, H)).astype(np.float32))
    W = {e: (r.standard_normal((I, H)) * 0.3, r.standard_normal((I, H)) * 0.3,
             r.standard_normal((H, I)) * 0.3) for e in range(E)}
    sh = (r.standard_normal((I, H)) * 0.3, r.standard_normal((I, H)) * 0.3,
          r.standard_normal((H, I)) * 0.3)
    idx = np.array([[3, 0], [1, 2], [0, 1]])
    w = r.random((n, k))
    y = moe.moe_forward(x, idx, w, lambda e: W[e], [sh])
    xf = moe.bf16_bits_to_f64(x)
    for t in range(n):
        out = [0.0] * H
        experts = [(W[int(idx[t, j])], w[t, j]) for j in range(k)] + [(sh, 1.0)]
        for (wg, wu, wd), scale in experts:
            h = []
            for i in range(I):
                g = sum(wg[i, q] * xf[t, q] for q in range(H))
                u = sum(wu[i, q] * xf[t, q] for q in range(H))
                h.append(g / (1.0 + np.exp(-g)) * u)
            for o in range(H):
                out[o] += scale * sum(wd[o, i] * h[i] for i in range(I))
        assert np.allclose(y[t], out, rtol=1e-12, atol=1e-12)


def test_bf16_decoding():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x3F81], np.uint16)
    assert moe.bf16_bits_to_f64(bits).tolist() == [1.0, -2.0, 0.0, 1.0 + 2 ** -7]
    assert synth.bf16_from_f32(np.array([1.0 + 2 ** -8], np.float32))[0] == 0x3F80   # tie -> even
    assert synth.bf16_from_f32(np.array([1.0 + 3 * 2 ** -8], np.float32))[0] == 0x3F82


def test_token_errors():
    ref = np.array([[1.0, -2.0], [0.0, 0.0]])
    y = np.array([[1.0, -2.002], [0.0, 1e-3]])
    e = moe.token_errors(y, ref)
    assert e[0] == pytest.approx(1e-3) and e[1] == pytest.approx(1e-3)
