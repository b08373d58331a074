"""The enqueue-only entry points under HIP graph capture.

A caller that replays a captured decode step needs the forward, the stack,
the top-k and the unfused forward to record nothing but kernel launches (and
device-to-device copies): no allocation, no memset, no host synchronisation.
Each case captures one call into a graph, then replays it several times on
new inputs written into the captured input buffer, with ordinary eager work
and synchronisations between the replays, and compares every replay bit for
bit with an eager call on the same input.
"""
import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import workloads as W

from gpu_util import device_layer, say

pytestmark = pytest.mark.gpu

REPLAYS = 3


@pytest.fixture(scope="module")
def layers():
    assert torch.cuda.is_available(), "GPU tests need a device"
    out = []
    for l in range(2):
        wg, wu, wd = W.weights(1024, 700, torch.bfloat16, layer=20 + l)
        out.append(device_layer(wg, wu, wd))
    return out


def _inputs(B, d, n, seed):
    g = torch.Generator().manual_seed(seed)
    return [torch.randn((B, d), generator=g).cuda() for _ in range(n)]


def _replay_check(label, call, x_static, y_static, eager, xs):
    """Capture call() once, replay on each x in xs, compare with eager(x)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()  # warm-up off the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for r, x in enumerate(xs):
        say("graph replay", label, r)
        x_static.copy_(x)
        g.replay()
        torch.cuda.synchronize()
        got = y_static.clone()
        _ = (x * 2.0).sum()  # eager work between replays
        ref = eager(x.clone())
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int32), ref.view(torch.int32)), f"{label}: replay {r}"


@pytest.mark.parametrize("B", [1, 3, 8])
def test_forward_graph(layers, B):
    """B = 8 at d = 1024 takes the matrix-core path (three kernels)."""
    layer = layers[0]
    t = 0.15
    x_static = torch.zeros((B, 1024), device="cuda")
    y_static = torch.empty_like(x_static)
    ws = P.workspace(1024, 700, B)
    ws_e = P.workspace(1024, 700, B)
    _replay_check(f"forward B{B}", lambda: P.mlp_forward(layer, x_static, t, out=y_static, ws=ws),
                  x_static, y_static, lambda x: P.mlp_forward(layer, x, t, ws=ws_e),
                  _inputs(B, 1024, REPLAYS, 40 + B))


def test_stack_graph(layers):
    st = P.Stack(layers, [0.1, 0.2])
    B = 2
    x_static = torch.zeros((B, 1024), device="cuda")
    ws = P.workspace(1024, 700, B)
    ws_e = P.workspace(1024, 700, B)
    y_static = torch.empty_like(x_static)

    def call():
        P.stack_forward(st, x_static, eps=1e-5, out=y_static, ws=ws)

    def eager(x):
        return P.stack_forward(st, x, eps=1e-5, ws=ws_e)

    _replay_check("stack", call, x_static, y_static, eager, _inputs(B, 1024, REPLAYS, 50))


@pytest.mark.parametrize("B", [1, 2])
def test_topk_graph(layers, B):
    """One row selects inside the gate kernel (its ticket word: a replay
    repeats the captured epoch and takes the compare-and-swap path), two
    rows use the select kernel."""
    layer = layers[1]
    x_static = torch.zeros((B, 1024), device="cuda")
    y_static = torch.empty_like(x_static)
    nb = int(P.raw().cats_topk_workspace_bytes(1024, 700, B))
    ws = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    ws_e = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    _replay_check("topk", lambda: P.mlp_forward_topk(layer, x_static, 0.7, out=y_static, ws=ws),
                  x_static, y_static, lambda x: P.mlp_forward_topk(layer, x, 0.7, ws=ws_e)[0],
                  _inputs(B, 1024, REPLAYS, 60))


@pytest.mark.parametrize("mode", ["mask", "index"])
def test_unfused_graph(layers, mode):
    layer = layers[1]
    B = 1
    x_static = torch.zeros((B, 1024), device="cuda")
    y_static = torch.empty_like(x_static)
    nb = int(P.raw().cats_unfused_workspace_bytes(1024, 700, B))
    ws = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    ws_e = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    _replay_check(f"unfused {mode}",
                  lambda: P.mlp_forward_unfused(layer, x_static, 0.15, mode=mode, out=y_static, ws=ws),
                  x_static, y_static, lambda x: P.mlp_forward_unfused(layer, x, 0.15, mode=mode, ws=ws_e),
                  _inputs(B, 1024, REPLAYS, 70))


@pytest.mark.parametrize("B,shared", [(1, False), (3, False), (3, True)])
def test_sparse_input_graph(B, shared):
    """The sparse-input product at n = 1024 (8 column tiles of 32 channel
    groups: the cross-block sum with tickets).  With shared=True the eager
    calls between replays use the captured call's own workspace, so replays
    meet tickets left by calls with other tags."""
    d, n = 2048, 1024
    g = torch.Generator().manual_seed(80 + B)
    w = (torch.randn((d, n), generator=g) * 0.02).to(torch.bfloat16).cuda()
    x_static = torch.zeros((B, d), device="cuda")
    y_static = torch.empty((B, n), device="cuda")
    ws = P.sparse_input_workspace(d, n, B)
    ws_e = ws if shared else P.sparse_input_workspace(d, n, B)
    t = 0.6
    _replay_check(f"sparse input B{B} shared={shared}",
                  lambda: P.sparse_input_gemv(w, x_static, t, out=y_static, ws=ws),
                  x_static, y_static, lambda x: P.sparse_input_gemv(w, x, t, ws=ws_e),
                  _inputs(B, d, REPLAYS, 90 + B))
