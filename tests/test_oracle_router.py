"""Pins for the oracle router.

* special cases that reduce to plain top-k of the logits (the sigmoid is
  monotone), checked with ``numpy.argsort`` and no exponential at all;
* an independent selection algorithm (repeated arg-max with masking instead of
  full sorts) on tiny inputs with many forced ties;
* invariants: pruned experts are never chosen, weights sum to the scale;
* a hand-worked example (``tests/golden/router_tiny.json``)."""
import json
import os

import numpy as np
import pytest

from oracle import router
from inputs import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_sigmoid_closed_forms():
    s = router.sigmoid_f32(np.array([0.0, 50.0, -200.0, np.inf, -np.inf], np.float32))
    assert s.dtype == np.float32
    assert s[0] == np.float32(0.5) and s[1] == np.float32(1.0)
    assert s[2] == 0.0 and s[3] == 1.0 and s[4] == 0.0
    # sigmoid(-x) = 1 - sigmoid(x) exactly where both are representable
    x = np.linspace(-3, 3, 101).astype(np.float32)
    assert np.allclose(router.sigmoid_f32(-x).astype(np.float64),
                       1 - router.sigmoid_f32(x).astype(np.float64), atol=1.2e-7)


def _grid_logits(r, n, E):
    """Distinct logits on a 1/1024 grid in [-4, 4]: their float32 sigmoids stay distinct."""
    vals = (np.arange(-4096, 4097) / 1024.0).astype(np.float32)
    return np.stack([r.choice(vals, E, replace=False) for _ in range(n)])


@pytest.mark.parametrize("n_group,topk_group", [(1, 1), (4, 4)])
def test_reduces_to_plain_topk(n_group, topk_group):
    """One group (or every group selected) and no bias: top-k of the logits."""
    r = np.random.default_rng(3)
    E, k = 32, 5
    mask = np.ones(E, np.uint8)
    mask[r.choice(E, 7, replace=False)] = 0
    logits = _grid_logits(r, 20, E)
    idx, w = router.route(logits, mask, n_group=n_group, topk_group=topk_group,
                          top_k=k, norm_topk=False, routed_scale=1.0)
    for t in range(20):
        order = [e for e in np.argsort(-logits[t], kind="stable") if mask[e]]
        assert list(idx[t]) == order[:k]
        assert np.all(np.diff(w[t]) <= 0)


def _route_by_argmax(logits, mask, bias, G, TG, k, topn, lam):
    """Independent router: repeated arg-max over masked arrays, first index on ties."""
    E = len(logits)
    s = router.sigmoid_f32(logits)
    b = (s + (np.zeros(E, np.float32) if bias is None else bias)).astype(np.float32)
    b = np.where(mask.astype(bool), b, -np.inf).astype(np.float32)
    per = E // G
    gs = np.full(G, -np.inf)
    for g in range(G):
        seg = b[g * per:(g + 1) * per].astype(np.float64).copy()
        acc, taken = np.float32(0), 0
        for _ in range(topn):
            j = int(np.argmax(seg))
            if seg[j] == -np.inf:
                break
            acc = np.float32(acc + np.float32(seg[j]))
            seg[j] = -np.inf
            taken += 1
        gs[g] = float(acc) if taken else -np.inf
    allowed = np.zeros(E, bool)
    picked = []
    for _ in range(TG):
        best = None
        for g in range(G):
            if g not in picked and (best is None or gs[g] > gs[best]):
                best = g
        picked.append(best)
        allowed[best * per:(best + 1) * per] = True
    cand = np.where(allowed, b.astype(np.float64), -np.inf)
    idx = []
    for _ in range(k):
        e = int(np.argmax(cand))
        idx.append(e)
        cand[e] = -np.inf
    sel = s[idx].astype(np.float64)
    return np.array(idx), sel / sel.sum() * lam


def test_matches_argmax_router_with_ties():
    r = np.random.default_rng(5)
    E, G, TG, k = 16, 4, 2, 3
    for trial in range(300):
        mask = np.ones(E, np.uint8)
        mask[r.choice(E, 3, replace=False)] = 0
        if not router.routing_is_feasible(mask, G, TG, k):
            continue
        # few distinct values: exact ties in scores and in group sums
        logits = r.choice(np.array([-1.0, 0.0, 0.5, 1.0], np.float32), E)
        idx, w = router.route(logits[None], mask, n_group=G, topk_group=TG, top_k=k,
                              routed_scale=2.5)
        i2, w2 = _route_by_argmax(logits, mask, None, G, TG, k, 2, 2.5)
        assert list(idx[0]) == list(i2), (trial, logits, mask)
        assert np.allclose(w[0], w2, rtol=0, atol=1e-15)


def test_pruned_never_chosen_even_with_largest_logits():
    shape = synth.TINY
    mask = synth.expert_mask(shape, "pin")
    logits = synth.normal_logits(64, shape.n_experts, "pin")
    logits[:, mask == 0] = 30.0
    idx, _ = router.route(logits, mask, n_group=shape.n_group, topk_group=shape.topk_group,
                          top_k=shape.top_k, routed_scale=2.5)
    assert np.all(mask[idx] == 1)


def test_weights_sum_to_scale_and_follow_scores():
    shape = synth.V3
    mask = synth.expert_mask(shape, "pin")
    logits = synth.normal_logits(8, shape.n_experts, "pin")
    idx, w = router.route(logits, mask, n_group=8, topk_group=4, top_k=8, routed_scale=2.5)
    assert np.allclose(w.sum(axis=1), 2.5, rtol=0, atol=1e-12)
    s = router.sigmoid_f32(logits)
    for t in range(8):
        assert len(set(idx[t])) == 8
        assert np.all(np.diff(s[t, idx[t]].astype(np.float64)) <= 0)
        groups = set(int(e) // 32 for e in idx[t])
        assert len(groups) <= 4


def test_unnormalised_weights_are_scaled_scores():
    mask = np.ones(8, np.uint8)
    logits = np.array([[0, 1, 2, 3, -1, -2, -3, 0.5]], np.float32)
    idx, w = router.route(logits, mask, n_group=2, topk_group=2, top_k=2, norm_topk=False,
                          routed_scale=3.0)
    s = router.sigmoid_f32(logits[0]).astype(np.float64)
    assert list(idx[0]) == [3, 2]
    assert np.array_equal(w[0], s[[3, 2]] * 3.0)


def test_golden_worked_example():
    with open(os.path.join(GOLDEN, "router_tiny.json")) as f:
        g = json.load(f)
    idx, w = router.route(np.array(g["logits"], np.float32), np.array(g["mask"], np.uint8),
                          n_group=g["n_group"], topk_group=g["topk_group"], top_k=g["top_k"],
                          group_topn=g["group_topn"], routed_scale=g["routed_scale"])
    assert idx.tolist() == g["expected_idx"]
    assert np.allclose(w, np.array(g["expected_w"]), rtol=0, atol=1e-12)


def test_feasibility_rule():
    m = np.array([1, 1, 0, 0, 1, 0, 0, 0], np.uint8)          # groups of 4: counts 2, 1
    assert router.routing_is_feasible(m, 2, 1, 1)
    assert not router.routing_is_feasible(m, 2, 1, 2)          # the 1-expert group may win
    assert router.routing_is_feasible(m, 2, 2, 3)
    assert not router.routing_is_feasible(np.array([1, 1, 0, 0], np.uint8), 2, 2, 1)


def test_regroup_equals_masking_when_groups_are_untouched():
    """No pruning, or pruning that leaves every original group the same number
    of survivors at the same positions, gives the same groups either way."""
    r = np.random.default_rng(11)
    E, G = 16, 4
    lg = _grid_logits(r, 30, E)
    full = np.ones(E, np.uint8)
    kw = dict(n_group=G, topk_group=2, top_k=3, routed_scale=2.5)
    a = router.route(lg, full, **kw)
    b = router.route(lg, full, regroup=True, **kw)
    assert np.array_equal(a[0], b[0]) and np.allclose(a[1], b[1])
    even = np.array([1, 1, 1, 0] * 4, np.uint8)      # three survivors in every group
    a = router.route(lg, even, **kw)
    b = router.route(lg, even, regroup=True, **kw)
    assert np.array_equal(a[0], b[0])


def test_regroup_hand_example():
    """E = 8, two groups, kept {0, 1, 2, 4}, one group per token, k = 2.
    Masking keeps the original groups {0, 1, 2} and {4}: group 0 scores
    s(1.0) + s(0.95), group 1 only s(0.99), so experts 0 and 2 are chosen.
    Regrouping makes {0, 1} and {2, 4}: s(0.99) + s(0.95) beats s(1.0) + s(0.9),
    so experts 4 and 2 are chosen (the sigmoid keeps the logits' order)."""
    mask = np.array([1, 1, 1, 0, 1, 0, 0, 0], np.uint8)
    lg = np.array([[1.0, 0.9, 0.95, 5.0, 0.99, 5.0, 5.0, 5.0]], np.float32)
    kw = dict(n_group=2, topk_group=1, top_k=2, group_topn=2, routed_scale=1.0)
    idx_m, _ = router.route(lg, mask, **kw)
    idx_r, _ = router.route(lg, mask, regroup=True, **kw)
    assert idx_m[0].tolist() == [0, 2]
    assert idx_r[0].tolist() == [4, 2]


# ---------------------------------------------------------------------------
# The router gate l = x W_r^T.
def _bf16_value(bits):
    """bfloat16 bits -> float, by sign, exponent and mantissa fields (normals and zero)."""
    b = int(bits)
    sign = -1.0 if b >> 15 else 1.0
    exp, man = (b >> 7) & 0xFF, b & 0x7F
    if exp == 0:
        return sign * man * 2.0 ** -133
    return sign * (1.0 + man / 128.0) * 2.0 ** (exp - 127)


def test_gate_logits_brute_force():
    """Triple loop over tokens, experts and the hidden index, with x decoded field by field."""
    x_bits = synth.activations(3, 32, "gate-brute")
    w = synth.router_weight(5, 32, "gate-brute")
    got = router.gate_logits(x_bits, w)
    assert got.shape == (3, 5)
    for t in range(3):
        for e in range(5):
            ref = sum(_bf16_value(x_bits[t, h]) * float(w[e, h]) for h in range(32))
            assert abs(got[t, e] - ref) <= 1e-12 * (1 + abs(ref))


def test_gate_logits_one_hot_picks_a_column():
    """x = unit vector e_h gives logits W_r[:, h]: catches a transposed gate."""
    E, H = 6, 40
    w = synth.router_weight(E, H, "gate-onehot")
    for h in (0, 17, 39):
        x = np.zeros(H, np.float32)
        x[h] = 1.0
        l = router.gate_logits(synth.bf16_from_f32(x)[None, :], w)
        assert np.array_equal(l[0], w[:, h].astype(np.float64))


def test_gate_grid_inputs_are_exact_in_float32():
    """The grid generators' logits are integers times 2^-12 within float32's exact range."""
    x_bits = synth.grid_activations(4, 7168, "gate-grid")
    w = synth.grid_router_weight(8, 7168, "gate-grid")
    l = router.gate_logits(x_bits, w)
    units = l * 4096.0
    assert np.array_equal(units, np.round(units))
    assert np.abs(units).max() < 2 ** 24
    # every partial sum is bounded by the sum of magnitudes
    xa = np.abs((x_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    assert (xa @ np.abs(w.astype(np.float64)).T * 4096.0).max() < 2 ** 24
    assert np.array_equal(l.astype(np.float32).astype(np.float64), l)
