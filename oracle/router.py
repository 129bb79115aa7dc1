"""Oracle: the router over the experts that survive pruning.  TEST INFRASTRUCTURE ONLY.

What it follows:

* Section 3.1: pruning keeps the top ``ceil(rE)`` experts of each MoE layer;
  the rest are gone and can never be chosen again.  The kept set arrives here
  as a boolean mask over the original expert ids.
* Section 3.2: after pruning, each token activates ``num_experts_per_tok``
  (``k``) experts chosen by grouped top-k routing governed by ``topk_group``.
* The routing function itself is the DeepSeek-V3 one used by the paper's
  model (Section 4.1): sigmoid affinities, groups scored by the sum of their
  best scores, the best ``topk_group`` groups kept, the best ``k`` experts
  inside them, weights renormalised over the chosen experts and multiplied by
  a routed scaling factor.

Readings where the paper is silent (all listed with the design notes):

* groups are the original contiguous id ranges ``[g*E/G, (g+1)*E/G)``; pruned
  experts are masked inside them, not regrouped;
* a group's score is the float32 sum of its ``group_topn`` best kept biased
  scores, added in descending order; a group with fewer kept experts sums what
  it has; a group with none scores -inf;
* ties go to the lower group id, then to the lower expert id;
* the sigmoid is evaluated in float64 and rounded once to float32;
* the optional per-expert bias enters selection only; weights use the
  unbiased score;
* if the chosen scores sum to zero, all weights are zero;
* with ``regroup`` (the literal reading of Section 3.2, "topk_group
  partitions the pruned expert pool into groups"), the kept experts in
  ascending id order are cut into ``n_group`` contiguous groups of equal size
  and routing runs over them alone.
"""
import numpy as np


def gate_logits(x_bits, w_r):
    """Router affinities ``l = x W_r^T``: bfloat16 bit patterns ``[n, H]`` and a
    float32 gate ``[E, H]`` -> float64 ``[n, E]`` (Section 3.2 routes on these;
    the paper's model computes them in float32 from the hidden state)."""
    x = (np.asarray(x_bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x @ np.asarray(w_r, dtype=np.float32).astype(np.float64).T


def sigmoid_f32(logits):
    """float32(1 / (1 + exp(-l))) with the expression evaluated in float64."""
    l64 = np.asarray(logits, dtype=np.float32).astype(np.float64)
    with np.errstate(over="ignore"):
        s = 1.0 / (1.0 + np.exp(-l64))
    return s.astype(np.float32)


def route_token(logits, mask, bias, n_group, topk_group, top_k, group_topn,
                norm_topk, routed_scale):
    """Route one token.  Returns (idx int32 [k], w float64 [k]).

    A direct transcription of the selection rules with full sorts; no partial
    selection, no blocking."""
    E = logits.shape[0]
    s = sigmoid_f32(logits)                                   # float32 [E]
    beta = np.zeros(E, np.float32) if bias is None else np.asarray(bias, np.float32)
    biased = (s + beta).astype(np.float32)                    # float32 add
    per = E // n_group

    group_score = []
    for g in range(n_group):
        members = [e for e in range(g * per, (g + 1) * per) if mask[e]]
        if not members:
            group_score.append(-np.inf)
            continue
        best = sorted(members, key=lambda e: (-float(biased[e]), e))[:group_topn]
        acc = np.float32(0.0)
        for e in best:
            acc = np.float32(acc + biased[e])
        group_score.append(float(acc))

    groups = sorted(range(n_group), key=lambda g: (-group_score[g], g))[:topk_group]
    candidates = [e for g in groups for e in range(g * per, (g + 1) * per) if mask[e]]
    chosen = sorted(candidates, key=lambda e: (-float(biased[e]), e))[:top_k]
    if len(chosen) < top_k:
        raise ValueError("fewer than top_k kept experts in the selected groups")

    idx = np.array(chosen, dtype=np.int32)
    sel = s[idx].astype(np.float64)
    if norm_topk:
        total = sel.sum()
        w = np.zeros_like(sel) if total == 0.0 else sel / total * routed_scale
    else:
        w = sel * routed_scale
    return idx, w


def route(logits, mask, bias=None, *, n_group, topk_group, top_k, group_topn=2,
          norm_topk=True, routed_scale=1.0, regroup=False):
    """Route every token: logits float32 ``[n, E]`` -> (idx int32 ``[n, k]``, w float64 ``[n, k]``).

    Slot order is selection order (score descending, lower id first on ties).
    With ``regroup`` the groups are formed over the kept experts only."""
    logits = np.asarray(logits, dtype=np.float32)
    mask = np.asarray(mask).astype(bool)
    if regroup:
        kept = np.nonzero(mask)[0]
        if len(kept) % n_group:
            raise ValueError("regrouping needs a kept count divisible by n_group")
        sub_bias = None if bias is None else np.asarray(bias, np.float32)[kept]
        idx, w = route(logits[:, kept], np.ones(len(kept), np.uint8), sub_bias, n_group=n_group,
                       topk_group=topk_group, top_k=top_k, group_topn=group_topn, norm_topk=norm_topk,
                       routed_scale=routed_scale)
        return kept[idx].astype(np.int32), w
    n = logits.shape[0]
    idx = np.zeros((n, top_k), np.int32)
    w = np.zeros((n, top_k), np.float64)
    for t in range(n):
        idx[t], w[t] = route_token(logits[t], mask, bias, n_group, topk_group,
                                   top_k, group_topn, norm_topk, routed_scale)
    return idx, w


def routing_is_feasible(mask, n_group, topk_group, top_k):
    """True if every possible group choice leaves at least ``top_k`` candidates.

    The worst case picks the ``topk_group`` groups with the fewest kept experts
    among the non-empty ones; empty groups score -inf and are picked last."""
    mask = np.asarray(mask).astype(bool)
    per = mask.shape[0] // n_group
    counts = sorted(int(mask[g * per:(g + 1) * per].sum()) for g in range(n_group))
    nonempty = [c for c in counts if c > 0]
    if topk_group > len(nonempty):
        return False
    return sum(nonempty[:topk_group]) >= top_k
