"""moeq_expert_importance_noalloc (the router-statistics pass of Section 3.1
with its scratch in the library's static device array) against
moeq_expert_importance on the same inputs, through the C interface: two calls
in a row on one device, the second with fewer tokens (the static scratch then
holds the first call's data), and the capacity check."""
import ctypes

import numpy as np
import pytest
import torch

from inputs import synth

pytestmark = pytest.mark.gpu


def _importance(moeq, fn, shape, logits, bias, alpha, retain):
    n, E = logits.shape
    cfg = moeq.make_config(shape, max_tokens=1)
    imp = torch.full((E,), -1.0, dtype=torch.float64, device="cuda")
    mask = torch.full((E,), 7, dtype=torch.uint8, device="cuda")
    counts = torch.full((E,), -1, dtype=torch.int32, device="cuda")
    st = fn(ctypes.byref(cfg), bias.ctypes.data, ctypes.c_void_p(logits.data_ptr()), n, alpha, retain,
            ctypes.c_void_p(imp.data_ptr()), ctypes.c_void_p(mask.data_ptr()), ctypes.c_void_p(counts.data_ptr()),
            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == moeq.MOEQ_OK, moeq.moeq_last_error()
    torch.cuda.synchronize()
    return imp.cpu().numpy(), mask.cpu().numpy(), counts.cpu().numpy()


def test_noalloc_matches_allocating_entry_point(gpu_lib):
    moeq = gpu_lib
    shape = synth.V3
    E = shape.n_experts
    results = []
    for i, n in enumerate((20000, 700)):
        logits = torch.from_numpy(synth.normal_logits(n, E, "noalloc", n)).cuda()
        bias = (0.01 * synth.normal_logits(1, E, "noalloc-bias", i)[0]).astype(np.float32)
        alpha, retain = (0.5, 0.75) if i == 0 else (0.3, 0.5)
        got = _importance(moeq, moeq.lib.moeq_expert_importance_noalloc, shape, logits, bias, alpha, retain)
        ref = _importance(moeq, moeq.lib.moeq_expert_importance, shape, logits, bias, alpha, retain)
        for g, r, what in zip(got, ref, ("importance", "mask", "counts")):
            assert np.array_equal(g, r), (n, what)
        assert got[1].sum() == int(np.ceil(retain * E - 1e-9))
        assert got[2].sum() == n * shape.top_k
        results.append(got)
    assert not np.array_equal(results[0][2], results[1][2])


def test_noalloc_rejects_scratch_beyond_its_size(gpu_lib):
    moeq = gpu_lib
    shape = synth.V3
    cfg = moeq.make_config(shape, max_tokens=1)
    fake = ctypes.c_void_p(256)   # never dereferenced: the size check fails first
    n = 200000                    # 16 * n * 8 bytes of ids, weights, ranks and permutation alone exceed 16 MiB
    st = moeq.lib.moeq_expert_importance_noalloc(ctypes.byref(cfg), None, fake, n, 0.5, 0.75, fake, fake, None,
                                                 None)
    assert st == moeq.MOEQ_ERR_CAPACITY
    assert "static scratch" in moeq.moeq_last_error()
