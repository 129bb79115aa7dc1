"""Graph capture: a captured forward replays to the eager result.

The forward allocates nothing and waits on nothing, so it can be captured
into a HIP graph (the benchmark replays one).  Each case captures one
forward, then replays the graph several times.  Before each replay it zeroes
the output, runs an eager forward of other inputs on the same layer (which
rewrites the shared workspace) and synchronizes.  Every replay must equal
the eager output of the captured inputs bit for bit: the forward is
deterministic.
"""
import numpy as np
import pytest
import torch

import layers
from inputs import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny_layer(gpu_lib):
    data = layers.quantized_layer(synth.TINY, "p234_602020", "graph-tiny")
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=200)
    yield data, L
    L.close()


@pytest.fixture(scope="module")
def v3_layer(gpu_lib):
    data = layers.random_packed_layer(synth.V3, "gu3_d4_sh4", "graph-v3")
    L = gpu_lib.Layer(data.shape, data.mask, data.routed(), data.shared(), max_tokens=64)
    yield data, L
    L.close()


def _inputs(shape, n, key):
    bits = synth.activations(n, shape.hidden, key)
    x = torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)
    lg = torch.from_numpy(synth.normal_logits(n, shape.n_experts, key)).cuda()
    return x, lg


def _check_replays(moeq, L, shape, n, path, key, replays=3):
    L.set_path(path)
    try:
        x, lg = _inputs(shape, n, key)
        xo, lgo = _inputs(shape, n, key + "-other")
        y_ref = L.forward(x, lg)
        y_other = torch.empty_like(y_ref)
        y = torch.empty_like(y_ref)
        torch.cuda.synchronize()
        # one forward on a side stream before capture, as the benchmark does
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            L.forward(x, lg, y=y)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            L.forward(x, lg, y=y)
        for r in range(replays):
            y.zero_()
            L.forward(xo, lgo, y=y_other)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(y, y_ref), (n, path, r)
    finally:
        L.set_path(moeq.MOEQ_PATH_AUTO)


@pytest.mark.parametrize("n,path", [(1, 1), (3, 1), (40, 1), (40, 2), (200, 2)])
def test_graph_replay_tiny(gpu_lib, tiny_layer, n, path):
    """Decode path (one-token and batched kernels) and grouped-GEMM path,
    mixed 2/3/4-bit widths."""
    data, L = tiny_layer
    _check_replays(gpu_lib, L, data.shape, n, path, f"graph-tiny-{n}-{path}")


@pytest.mark.parametrize("n", [1, 16, 48])
def test_graph_replay_v3(gpu_lib, v3_layer, n):
    """The V3 decode layer on the automatic path: the benchmark's batch-1
    forward, 16 tokens, and 48 tokens (8-wave gate/up workgroups)."""
    data, L = v3_layer
    _check_replays(gpu_lib, L, data.shape, n, gpu_lib.MOEQ_PATH_AUTO, f"graph-v3-{n}")


@pytest.mark.parametrize("n", [1, 8, 40])
def test_graph_replay_router_gate(gpu_lib, n):
    """Forwards that compute their logits from the layer's router weight
    (no logits given): the gate kernel for few and for many tokens, then
    routing, in one captured graph."""
    data = layers.quantized_layer(synth.TINY, "all4", "graph-gate")
    shape = data.shape
    L = gpu_lib.Layer(shape, data.mask, data.routed(), data.shared(), max_tokens=64)
    try:
        L.set_router_weight(synth.router_weight(shape.n_experts, shape.hidden, "graph-gate-wr"))
        x, _ = _inputs(shape, n, f"graph-gate-{n}")
        xo, _ = _inputs(shape, n, f"graph-gate-{n}-other")
        y_ref = L.forward(x)
        y, y_other = torch.empty_like(y_ref), torch.empty_like(y_ref)
        torch.cuda.synchronize()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            L.forward(x, y=y)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            L.forward(x, y=y)
        for r in range(3):
            y.zero_()
            L.forward(xo, y=y_other)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(y, y_ref), (n, r)
    finally:
        L.close()
