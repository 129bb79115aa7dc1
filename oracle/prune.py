"""Oracle: performance-aware expert pruning.  TEST INFRASTRUCTURE ONLY.

Section 3.1 ranks the experts of one MoE layer by an importance score built
from router statistics over a calibration set and keeps the best ``ceil(rE)``:

    I_e = alpha * f_e + (1 - alpha) * sbar_e

with ``f_e`` the activation frequency of expert ``e`` and ``sbar_e`` the
average routing score ``e`` receives when it is selected.

Readings where the paper is silent (listed with the design notes):

* the statistics come from the unpruned router (every expert kept), with the
  layer's grouped top-k routing and score-correction bias;
* ``f_e`` = (tokens that selected ``e``) / (calibration tokens), a fraction in
  [0, 1]; ``sbar_e`` = mean of the sigmoid score ``s_e`` over those tokens
  (0 for an expert never selected).  Both lie in [0, 1], so ``alpha`` mixes
  quantities of the same scale;
* arithmetic: the score sum is float32, accumulated in token order; ``f_e``
  and ``sbar_e`` are float32 quotients; ``I_e`` is evaluated in float64 from
  them as ``alpha * f_e + (1 - alpha) * sbar_e`` (two products, one sum);
* ranking: ``I_e`` descending, lower expert id first on ties;
* ``ceil(rE)`` is taken with a tolerance of 1e-9 so that products such as
  0.7 * 10 that land a rounding error above an integer keep that integer.
"""
import math

import numpy as np

from . import router


def kept_count(retain, n_experts):
    """ceil(r * E), with a 1e-9 tolerance against rounding just above an integer."""
    return int(math.ceil(float(retain) * n_experts - 1e-9))


def router_stats(logits, bias, *, n_group, topk_group, top_k, group_topn=2):
    """Counts (int64 ``[E]``) and float32 score sums (``[E]``, token order) of
    the unpruned router over the calibration logits ``[n, E]``."""
    logits = np.asarray(logits, dtype=np.float32)
    n, E = logits.shape
    mask = np.ones(E, np.uint8)
    idx, w = router.route(logits, mask, bias, n_group=n_group, topk_group=topk_group, top_k=top_k,
                          group_topn=group_topn, norm_topk=False, routed_scale=1.0)
    # without renormalisation and with scale 1 the weights are the sigmoid scores
    scores = w.astype(np.float32)
    counts = np.zeros(E, np.int64)
    sums = np.zeros(E, np.float32)
    for t in range(n):
        for j in range(top_k):
            e = int(idx[t, j])
            counts[e] += 1
            sums[e] = np.float32(sums[e] + scores[t, j])
    return counts, sums


def expert_importance(logits, bias=None, *, n_group, topk_group, top_k, group_topn=2, alpha, retain):
    """-> (importance float64 ``[E]``, mask uint8 ``[E]``, counts, sums)."""
    logits = np.asarray(logits, dtype=np.float32)
    n, E = logits.shape
    counts, sums = router_stats(logits, bias, n_group=n_group, topk_group=topk_group, top_k=top_k,
                                group_topn=group_topn)
    f = (counts.astype(np.float32) / np.float32(n)).astype(np.float32)
    with np.errstate(invalid="ignore", divide="ignore"):
        sbar = np.where(counts > 0, sums / counts.astype(np.float32), np.float32(0)).astype(np.float32)
    a = float(alpha)
    imp = a * f.astype(np.float64) + (1.0 - a) * sbar.astype(np.float64)
    keep = kept_count(retain, E)
    order = sorted(range(E), key=lambda e: (-imp[e], e))
    mask = np.zeros(E, np.uint8)
    mask[order[:keep]] = 1
    return imp, mask, counts, sums
