"""Expert importance and pruning mask on the GPU against the oracle (Section
3.1): counts and masks bit-exact, importance bit-exact (the kernel mirrors the
oracle's float32 sums in token order and float64 mix), on the tiny and the
DeepSeek-V3 shapes, with and without a score-correction bias, for several
alpha and retention ratios."""
import dataclasses

import numpy as np
import pytest

from inputs import synth
from oracle import prune

pytestmark = pytest.mark.gpu


def _run(gpu_lib, shape, logits, alpha, retain, bias=None):
    import torch
    moeq = gpu_lib
    lg = torch.from_numpy(logits).cuda()
    imp, mask, counts = moeq.expert_importance(shape, lg, alpha=alpha, retain=retain, bias=bias)
    torch.cuda.synchronize()
    return imp.cpu().numpy(), mask.cpu().numpy(), counts.cpu().numpy()


def _oracle(shape, logits, alpha, retain, bias=None):
    return prune.expert_importance(logits, bias, n_group=shape.n_group, topk_group=shape.topk_group,
                                   top_k=shape.top_k, group_topn=shape.group_topn, alpha=alpha, retain=retain)


@pytest.mark.parametrize("alpha,retain", [(0.5, 0.75), (1.0, 0.5), (0.0, 0.25), (0.3, 1.0)])
def test_importance_tiny(gpu_lib, alpha, retain):
    shape = synth.TINY
    lg = synth.normal_logits(300, shape.n_experts, "prune-tiny", alpha, retain)
    imp, mask, counts = _run(gpu_lib, shape, lg, alpha, retain)
    ref_imp, ref_mask, ref_counts, _ = _oracle(shape, lg, alpha, retain)
    assert np.array_equal(counts, ref_counts)
    assert np.array_equal(imp, ref_imp)
    assert np.array_equal(mask, ref_mask)


def test_importance_with_bias_and_zipf(gpu_lib):
    shape = synth.TINY
    full = np.ones(shape.n_experts, np.uint8)
    lg = synth.zipf_logits(257, full, "prune-zipf")
    bias = synth.rng("prune-bias").normal(0, 0.05, shape.n_experts).astype(np.float32)
    imp, mask, counts = _run(gpu_lib, shape, lg, 0.5, 0.75, bias)
    ref_imp, ref_mask, ref_counts, _ = _oracle(shape, lg, 0.5, 0.75, bias)
    assert np.array_equal(counts, ref_counts)
    assert np.array_equal(imp, ref_imp)
    assert np.array_equal(mask, ref_mask)


def test_importance_v3_shape(gpu_lib):
    """DeepSeek-V3 router shape (256 experts, 8 groups, top-4 groups, top-8),
    r = 0.75 keeps 192: the mask the rest of the layer is built with."""
    shape = dataclasses.replace(synth.V3, n_kept=256)
    full = np.ones(shape.n_experts, np.uint8)
    lg = synth.zipf_logits(1500, full, "prune-v3")
    imp, mask, counts = _run(gpu_lib, shape, lg, 0.5, 0.75)
    ref_imp, ref_mask, ref_counts, _ = _oracle(shape, lg, 0.5, 0.75)
    assert counts.sum() == 1500 * shape.top_k
    assert np.array_equal(counts, ref_counts)
    assert np.array_equal(imp, ref_imp)
    assert np.array_equal(mask, ref_mask)
    assert mask.sum() == 192


def test_importance_mask_builds_a_layer(gpu_lib):
    """The mask it emits is accepted by layer creation as the pruned set."""
    from layers import random_packed_layer
    shape = synth.TINY
    lg = synth.normal_logits(128, shape.n_experts, "prune-build")
    _, mask, _ = _run(gpu_lib, shape, lg, 0.5, 0.75)
    assert mask.sum() == 12
    data = random_packed_layer(shape, "all4", "prune-build", mask=mask)
    layer = gpu_lib.Layer(shape, mask, data.routed(), data.shared(), max_tokens=8)
    idx, _ = layer.route(__import__("torch").from_numpy(synth.normal_logits(8, shape.n_experts, "pb")).cuda())
    assert set(idx.cpu().numpy().ravel().tolist()) <= set(np.nonzero(mask)[0].tolist())
    layer.close()
