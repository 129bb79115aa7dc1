"""Pins for the oracle bit-allocation planner (Section 3.3).

* hand-worked plans (``tests/golden/planner_hand.json``) that exercise the
  upgrade tiers, every back-off rule, a base that does not fit and an
  infeasible budget;
* the binary-partition layer order against the prefix the paper prints for
  58 MoE layers (29, 15, 44, 8);
* the sensitivity on a hand example, and S_low against the paper's
  single-width formula P_pruned * b(Q_low) / (8 * 10^9);
* invariants on seeded random tensor sets: the memory limit holds when the
  plan is feasible, routed experts never rise above Q_low and are lowered in
  queue order, upgrades stay between the floor and their tier's target."""
import json
import os

import numpy as np
import pytest

from oracle import planner as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    with open(os.path.join(GOLDEN, "planner_hand.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("case", range(4))
def test_hand_worked_plans(case):
    g = _golden()
    c = g["cases"][case]
    levels, rep = P.plan_bits(**g["tensors"], m_limit_bytes=c["m_limit_bytes"], **g["params"])
    assert levels == c["levels"]
    for k, v in rep.items():
        assert v == c[k], k


def test_binary_partition_prefix_printed_in_the_paper():
    order = P.binary_partition_order(58)
    assert order[:4] == [29, 15, 44, 8]
    assert sorted(order) == list(range(58))


@pytest.mark.parametrize("L", [1, 2, 3, 7, 8, 58, 61, 100])
def test_binary_partition_is_a_balanced_permutation(L):
    order = P.binary_partition_order(L)
    assert sorted(order) == list(range(L))
    # after the first 2^j - 1 picks, every run of unpicked positions is at most ceil(L / 2^j) long
    j = 1
    while (1 << j) - 1 <= L:
        picked = sorted(order[:(1 << j) - 1])
        edges = [-1] + picked + [L]
        longest = max(b - a - 1 for a, b in zip(edges, edges[1:]))
        assert longest <= -(-L // (1 << j)), (L, j, longest)
        j += 1


def test_sensitivity_hand_example():
    # a tensor holding a quarter of its layer that lowers PPL by 0.5 -> 2.0 per unit share
    assert P.sensitivity(10.0, [9.5, 10.0, 10.25], [1_000_000, 5, 3], [4_000_000, 10, 3]) == [2.0, 0.0, -0.25]


def test_s_low_matches_single_width_formula():
    params = [7168 * 2048] * 3 + [1536 * 7168, 129280 * 7168]
    levels, rep = P.plan_bits(params, [0.0] * 5, [0] * 5, [0] * 5, ladder=[100, 112, 288, 352, 420, 544],
                              low_prime=0, low=1, floor=2, small_level=5, medium_level=4,
                              m_limit_bytes=10 ** 12, n_moe_layers=1)
    assert P.gb(rep["S_low"]) == pytest.approx(sum(params) * 1.75 / (8 * 10 ** 9), rel=1e-15)


def _random_case(seed):
    r = np.random.default_rng(seed)
    n_layers = int(r.integers(1, 9))
    n = int(r.integers(4, 40))
    kind = r.choice([0, 0, 1, 2, 3], size=n)
    layer = r.integers(0, n_layers, size=n)
    params = np.where(kind == 0, r.choice([3, 9, 10, 30, 50, 51, 80], size=n), r.integers(40, 120, size=n))
    sens = np.round(r.standard_normal(n), 1)        # many ties
    kw = dict(ladder=[96, 112, 256, 320, 384, 512], low_prime=0, low=1, floor=2, small_level=5, medium_level=4,
              n_moe_layers=n_layers, small_params=10, medium_params=50)
    s_low = int(params.sum()) * 112
    m = int(r.integers(s_low // 512 - 20, s_low // 512 + 120))
    return [int(p) for p in params], [float(s) for s in sens], [int(k) for k in kind], [int(l) for l in layer], m, kw


@pytest.mark.parametrize("seed", range(40))
def test_plan_invariants(seed):
    params, sens, kind, layer, m, kw = _random_case(seed)
    levels, rep = P.plan_bits(params, sens, kind, layer, m_limit_bytes=m, **kw)
    ladder, low, floor = kw["ladder"], kw["low"], kw["floor"]
    total = sum(p * ladder[lv] for p, lv in zip(params, levels))
    assert total == rep["total"]
    assert rep["B_total"] == rep["B_base"] + rep["B_delta"]
    if rep["feasible"]:
        assert total <= m * 8 * 64
    # routed tensors: only Q_low or Q_low', lowered ones form a prefix of the queue
    order = P.binary_partition_order(kw["n_moe_layers"])
    pos = {L: i for i, L in enumerate(order)}
    routed = [t for t in range(len(params)) if kind[t] != 0]
    queue = sorted(routed, key=lambda t: (kind[t] == 3, pos[layer[t]], kind[t], t))
    lowered = [levels[t] == kw["low_prime"] for t in queue]
    assert all(levels[t] in (low, kw["low_prime"]) for t in routed)
    assert lowered == sorted(lowered, reverse=True)
    assert sum(lowered) == rep["n_rule3"]
    for t in range(len(params)):
        if kind[t] != 0 or params[t] > kw["medium_params"]:
            assert levels[t] in (low, kw["low_prime"])
        elif levels[t] != low:
            target = kw["small_level"] if params[t] < kw["small_params"] else kw["medium_level"]
            assert floor <= levels[t] <= target


def test_ample_budget_gives_every_target_and_lowers_nothing():
    params, sens, kind, layer, _, kw = _random_case(7)
    levels, rep = P.plan_bits(params, sens, kind, layer, m_limit_bytes=10 ** 9, **kw)
    for t in range(len(params)):
        if kind[t] == 0 and params[t] < 10:
            assert levels[t] == kw["small_level"]
        elif kind[t] == 0 and params[t] <= 50:
            assert levels[t] == kw["medium_level"]
        else:
            assert levels[t] == kw["low"]
    assert rep["n_rule2"] == rep["n_rule3"] == 0


def test_gate_and_up_are_lowered_before_any_down_projection():
    """58 MoE layers of (gate, up, down) routed tensors and nothing to upgrade:
    a budget short by 70 releases lowers 70 tensors, all gate/up, starting
    with layer 29's gate."""
    L = 58
    kind = [k for _ in range(L) for k in (1, 2, 3)]
    layer = [l for l in range(L) for _ in range(3)]
    params = [64] * (3 * L)
    s_low = sum(params) * 112
    release = 64 * 16
    m_bytes = (s_low - 70 * release) // 512
    assert m_bytes * 512 == s_low - 70 * release
    levels, rep = P.plan_bits(params, [0.0] * (3 * L), kind, layer, ladder=[96, 112, 256, 320, 384, 512],
                              low_prime=0, low=1, floor=2, small_level=5, medium_level=4,
                              m_limit_bytes=m_bytes, n_moe_layers=L)
    assert rep["n_rule3"] == 70 and rep["feasible"]
    lowered = [t for t in range(3 * L) if levels[t] == 0]
    assert all(kind[t] in (1, 2) for t in lowered)
    first35 = P.binary_partition_order(L)[:35]
    assert sorted({layer[t] for t in lowered}) == sorted(first35)
