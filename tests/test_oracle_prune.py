"""Pins for the expert-importance oracle (Section 3.1).

* one group and no bias reduce the router to plain top-k of the logits, so the
  counts are a histogram of ``argsort`` picks and the score sums are sums of
  independently evaluated sigmoids;
* alpha = 1 ranks by frequency alone, alpha = 0 by mean score alone, and the
  score is linear in alpha in between (a sign or weight error in the mix
  breaks it);
* invariants: counts add up to n * k, exactly ceil(rE) experts are kept and
  every kept expert ranks above every dropped one;
* a hand-worked example (``tests/golden/prune_tiny.json``)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import prune

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _distinct_logits(seed, n, E):
    r = np.random.default_rng(seed)
    vals = (np.arange(-4096, 4097) / 1024.0).astype(np.float32)
    return np.stack([r.choice(vals, E, replace=False) for _ in range(n)])


def test_kept_count():
    assert prune.kept_count(0.75, 256) == 192
    assert prune.kept_count(0.7, 10) == 7      # 0.7 * 10 rounds to 7.000000000000001
    assert prune.kept_count(0.71, 10) == 8
    assert prune.kept_count(1.0, 16) == 16
    assert prune.kept_count(0.01, 16) == 1


def test_plain_topk_special_case():
    """G = 1, no bias: counts and score sums from argsort and a float64 sigmoid."""
    n, E, k = 40, 16, 3
    lg = _distinct_logits(1, n, E)
    counts, sums = prune.router_stats(lg, None, n_group=1, topk_group=1, top_k=k)
    ref_counts = np.zeros(E, np.int64)
    ref_sums = np.zeros(E, np.float64)
    for t in range(n):
        top = np.argsort(-lg[t].astype(np.float64), kind="stable")[:k]
        for e in top:
            ref_counts[e] += 1
            ref_sums[e] += 1.0 / (1.0 + math.exp(-float(lg[t, e])))
    assert np.array_equal(counts, ref_counts)
    assert counts.sum() == n * k
    np.testing.assert_allclose(sums.astype(np.float64), ref_sums, rtol=2e-6, atol=1e-7)


@pytest.mark.parametrize("alpha", [0.0, 0.3, 0.5, 1.0])
def test_brute_force_importance(alpha):
    n, E, k = 24, 8, 2
    lg = _distinct_logits(2, n, E)
    imp, mask, counts, sums = prune.expert_importance(lg, n_group=1, topk_group=1, top_k=k,
                                                      alpha=alpha, retain=0.5)
    for e in range(E):
        f = counts[e] / n
        sbar = sums[e] / counts[e] if counts[e] else 0.0
        assert imp[e] == pytest.approx(alpha * f + (1 - alpha) * sbar, rel=1e-6, abs=1e-9)
    assert mask.sum() == 4


def test_alpha_extremes_and_linearity():
    n, E, k = 64, 16, 4
    lg = _distinct_logits(3, n, E)
    kw = dict(n_group=4, topk_group=2, top_k=k, retain=0.5)
    i1, m1, counts, _ = prune.expert_importance(lg, alpha=1.0, **kw)
    i0, m0, _, sums = prune.expert_importance(lg, alpha=0.0, **kw)
    ih, _, _, _ = prune.expert_importance(lg, alpha=0.25, **kw)
    np.testing.assert_array_equal(i1, counts / n)
    # by frequency: the kept set is the 8 most frequent (ties to lower id)
    order = sorted(range(E), key=lambda e: (-counts[e], e))
    assert set(np.nonzero(m1)[0]) == set(order[:8])
    sbar = np.where(counts > 0, sums / np.maximum(counts, 1), 0.0)
    np.testing.assert_allclose(i0, sbar, rtol=1e-6)
    np.testing.assert_allclose(ih, 0.25 * i1 + 0.75 * i0, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("retain", [0.25, 0.5, 0.75, 1.0])
def test_invariants(retain):
    n, E, k = 50, 32, 4
    lg = _distinct_logits(4, n, E)
    imp, mask, counts, _ = prune.expert_importance(lg, n_group=4, topk_group=2, top_k=k, alpha=0.5,
                                                   retain=retain)
    assert counts.sum() == n * k
    keep = prune.kept_count(retain, E)
    assert mask.sum() == keep
    kept, dropped = np.nonzero(mask)[0], np.nonzero(mask == 0)[0]
    if len(dropped):
        worst_kept = min((imp[e], -e) for e in kept)
        best_dropped = max((imp[e], -e) for e in dropped)
        assert worst_kept > best_dropped
    assert np.all(imp[counts == 0] == 0.0)


def test_bias_steers_selection():
    """A large bias on one expert makes every token select it."""
    n, E, k = 20, 8, 2
    lg = _distinct_logits(5, n, E)
    bias = np.zeros(E, np.float32)
    bias[6] = 10.0
    counts, _ = prune.router_stats(lg, bias, n_group=1, topk_group=1, top_k=k)
    assert counts[6] == n


def test_golden_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "prune_tiny.json")))
    lg = np.array(g["logits"], np.float32)
    for r, want in g["masks"].items():
        imp, mask, counts, _ = prune.expert_importance(lg, n_group=1, topk_group=1, top_k=2, alpha=0.5,
                                                       retain=float(r))
        assert mask.tolist() == want
        assert counts.tolist() == g["counts"]
        np.testing.assert_allclose(imp, g["importance"], atol=g["tolerance"])
