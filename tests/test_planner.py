"""The library's bit-allocation planner (host code behind the C interface)
against the oracle planner: identical levels and budget figures.

Cases: the hand-worked plans, seeded random tensor sets with many
sensitivity ties, and the 722 quantizable matrices of a DeepSeek-V3-shape
model pruned to 192 experts with llama.cpp-like widths (IQ1_S 1.5625, IQ1_M
1.75, Q4 4.5, Q5 5.5, Q6 6.5625, Q8 8.5 bits per weight) under memory limits
from infeasible (95 GB) to ample (128 GB), so that every back-off rule runs.
Sensitivities come from seeded synthetic perplexities (no model is run)."""
import json
import os

import numpy as np
import pytest

from inputs import synth
from oracle import planner as P
from paper_2509_25689_amd import moeq

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
LLAMA_LADDER = dict(ladder=[100, 112, 288, 352, 420, 544], low_prime=0, low=1, floor=2, small_level=5,
                    medium_level=4)


def _compare(params, sens, kind, layer, m_limit_bytes, kw):
    lv_o, rep_o = P.plan_bits(params, sens, kind, layer, m_limit_bytes=m_limit_bytes, **kw)
    p = moeq.plan_params(m_limit_bytes=m_limit_bytes, **kw)
    lv_n, rep_n = moeq.moeq_plan_bits(p, params, sens, kind, layer)
    assert list(lv_n) == lv_o
    assert rep_n.s_low_gb == P.gb(rep_o["S_low"])
    assert rep_n.b_base_gb == P.gb(rep_o["B_base"])
    assert rep_n.b_delta_gb == P.gb(rep_o["B_delta"])
    assert rep_n.b_total_gb == P.gb(rep_o["B_total"])
    assert rep_n.upgrade_gb == P.gb(rep_o["used"])
    assert rep_n.total_gb == P.gb(rep_o["total"])
    assert (rep_n.n_upgraded, rep_n.n_rule2, rep_n.n_rule3, bool(rep_n.feasible)) == \
        (rep_o["n_upgraded"], rep_o["n_rule2"], rep_o["n_rule3"], rep_o["feasible"])
    return lv_o, rep_o


def test_hand_worked_plans():
    with open(os.path.join(GOLDEN, "planner_hand.json")) as f:
        g = json.load(f)
    t = g["tensors"]
    for c in g["cases"]:
        lv, _ = _compare(t["params"], t["sens"], t["kind"], t["layer"], c["m_limit_bytes"], g["params"])
        assert lv == c["levels"]


@pytest.mark.parametrize("seed", range(60))
def test_random_tensor_sets(seed):
    r = np.random.default_rng(1000 + seed)
    n_layers = int(r.integers(1, 12))
    n = int(r.integers(1, 60))
    kind = r.choice([0, 0, 0, 1, 2, 3], size=n)
    layer = np.where(kind > 0, r.integers(0, n_layers, size=n), -1)
    params = np.where(kind == 0, r.choice([2, 9, 10, 11, 49, 50, 51, 300], size=n), r.integers(30, 200, size=n))
    sens = np.round(r.standard_normal(n), 1)
    kw = dict(ladder=[96, 112, 256, 320, 384, 512], low_prime=0, low=1, floor=2, small_level=5,
              medium_level=4, n_moe_layers=n_layers, small_params=10, medium_params=50)
    s_low_bytes = int(params.sum()) * 112 // 512
    for m in sorted({max(0, s_low_bytes + d) for d in (-60, -15, -3, 0, 4, 20, 90, 400)}):
        _compare([int(x) for x in params], [float(x) for x in sens], [int(x) for x in kind],
                 [int(x) for x in layer], m, kw)


def test_short_ladder_without_intermediate_levels():
    """Three widths only (2-, 3-, 4-bit blocks of this library: 2.5, 3.5, 4.5 bits):
    every tier target is the floor, rule 1 has a single try."""
    r = np.random.default_rng(5)
    n = 40
    kind = r.choice([0, 1, 2, 3], size=n)
    layer = np.where(kind > 0, r.integers(0, 6, size=n), -1)
    params = r.integers(1, 80, size=n)
    sens = r.standard_normal(n)
    kw = dict(ladder=[160, 224, 288], low_prime=0, low=1, floor=2, small_level=2, medium_level=2,
              n_moe_layers=6, small_params=10, medium_params=50)
    s_low_bytes = int(params.sum()) * 224 // 512
    for d in (-10, -2, 0, 3, 30):
        _compare([int(x) for x in params], [float(x) for x in sens], [int(x) for x in kind],
                 [int(x) for x in layer], s_low_bytes + d, kw)


@pytest.fixture(scope="module")
def v3_model():
    names, params, kind, layer, layer_params = synth.v3_tensor_inventory(192)
    ppl_low, ppl_high = synth.synthetic_perplexities(params, layer_params, "planner-v3")
    sens = P.sensitivity(ppl_low, ppl_high, params, layer_params)
    return names, params, kind, layer, layer_params, ppl_low, ppl_high, sens


def test_sensitivity_matches_oracle(v3_model):
    _, params, _, _, layer_params, ppl_low, ppl_high, sens = v3_model
    got = moeq.moeq_sensitivity(ppl_low, ppl_high, params, layer_params)
    assert list(got) == sens


@pytest.mark.parametrize("gb", [95, 100, 103, 106, 110, 112, 116, 128])
def test_v3_model_plans(v3_model, gb):
    names, params, kind, layer, _, _, _, sens = v3_model
    lv, rep = _compare(params, sens, kind, layer, gb * 10 ** 9, dict(LLAMA_LADDER, n_moe_layers=58))
    if rep["feasible"]:
        assert P.gb(rep["total"]) <= gb
    else:
        assert rep["n_rule3"] == 58 * 3


def test_layer_order_matches_oracle():
    for L in list(range(1, 70)) + [127, 128, 129, 1000]:
        assert list(moeq.moeq_layer_order(L)) == P.binary_partition_order(L)


def test_planner_validation():
    ok = moeq.plan_params(m_limit_bytes=10 ** 6, n_moe_layers=2, small_params=10, medium_params=50,
                          ladder=[96, 112, 256, 320, 384, 512], low_prime=0, low=1, floor=2, small_level=5,
                          medium_level=4)
    args = ([10, 20], [1.0, 0.5], [0, 1], [0, 1])
    moeq.moeq_plan_bits(ok, *args)

    def bad(**over):
        kw = dict(m_limit_bytes=10 ** 6, n_moe_layers=2, small_params=10, medium_params=50,
                  ladder=[96, 112, 256, 320, 384, 512], low_prime=0, low=1, floor=2, small_level=5,
                  medium_level=4)
        kw.update(over)
        return moeq.plan_params(**kw)
    for p in (bad(ladder=[96, 112]), bad(ladder=[96, 112, 112, 320]), bad(low=0), bad(floor=1),
              bad(medium_level=1), bad(small_level=6), bad(small_params=0), bad(medium_params=5),
              bad(m_limit_bytes=1 << 51)):
        with pytest.raises(moeq.MoeqError) as ei:
            moeq.moeq_plan_bits(p, *args)
        assert ei.value.status == moeq.MOEQ_ERR_INVALID_ARG
    for a in (([0, 20], [1.0, 0.5], [0, 1], [0, 1]),          # non-positive size
              ([10, 20], [float("nan"), 0.5], [0, 1], [0, 1]),  # non-finite sensitivity
              ([10, 20], [1.0, 0.5], [0, 4], [0, 1]),         # unknown kind
              ([10, 20], [1.0, 0.5], [0, 1], [0, 2]),         # routed layer out of range
              ([10, 20], [1.0, 0.5], [0, 1], None)):          # routed tensors without layers
        with pytest.raises(moeq.MoeqError) as ei:
            moeq.moeq_plan_bits(ok, *a)
        assert ei.value.status == moeq.MOEQ_ERR_INVALID_ARG
    with pytest.raises(moeq.MoeqError):
        moeq.moeq_layer_order(0)
    with pytest.raises(moeq.MoeqError):
        moeq.moeq_sensitivity(1.0, [0.5], [10], [5])           # tensor larger than its layer
    with pytest.raises(moeq.MoeqError):
        moeq.moeq_sensitivity(float("inf"), [0.5], [1], [5])
