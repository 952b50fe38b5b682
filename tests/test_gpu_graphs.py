"""HIP-graph capture of the library's launches: a captured attention step and
a captured convolution backward are replayed several times, with eager work
and synchronizations between the replays, and every replay must reproduce
the eager results bit for bit (the library records no memset and allocates
nothing, so its launches are safe to capture).
"""
import numpy as np
import pytest

from gpu_util import say
from workloads import make_inputs
from workloads.conv import make_conv_inputs

pytestmark = pytest.mark.gpu


def _replay_and_check(graph, outputs, expected, eager_work):
    import torch
    for rep in range(3):
        for t in outputs:
            t.fill_(float("nan"))
        eager_work()                  # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("out%d" % i for i in range(len(outputs))), outputs,
                                   expected):
            assert torch.equal(got, want), (rep, name)


@pytest.mark.parametrize("contract,causal", [("strict_f32", True), ("fast_bf16", True),
                                             ("accelerated", False)])
def test_attention_step_in_a_graph(gpu_lib, contract, causal):
    import torch
    mg = gpu_lib
    say("graph replay: attention %s causal=%s" % (contract, causal))
    x = make_inputs(2, 4, 300, 64, causal=causal, contract=contract, seed=21, Lk=260)
    if contract == "fast_bf16":
        dev = lambda n: torch.from_numpy(x.bits[n].view(np.int16).copy()).cuda().view(
            torch.bfloat16)
    else:
        dev = lambda n: torch.from_numpy(getattr(x, n).copy()).cuda()
    Q, K, V, dO = (dev(n) for n in ("Q", "K", "V", "dO"))
    O, LSE = torch.empty_like(Q), torch.empty(Q.shape[:3], device="cuda")
    dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    ws = torch.empty(max(1, mg.mg_attn_bwd_cross_workspace_bytes(2, 4, 300, 260, 64, causal,
                                                                 contract)),
                     dtype=torch.uint8, device="cuda")

    def step():
        mg.mg_attn_fwd_cross(Q, K, V, O, LSE, causal=causal, scale=x.scale, contract=contract)
        mg.mg_attn_bwd_cross(Q, K, V, O, LSE, dO, dQ, dK, dV, causal=causal, scale=x.scale,
                             contract=contract, workspace=ws)

    step()
    torch.cuda.synchronize()
    expected = [t.clone() for t in (O, LSE, dQ, dK, dV)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, capture_error_mode="relaxed"):
        step()
    scratch = torch.randn(1 << 20, device="cuda")
    _replay_and_check(graph, [O, LSE, dQ, dK, dV], expected,
                      lambda: scratch.mul_(1.0001).add_(0.5))


def test_convolution_backward_in_a_graph(gpu_lib):
    import torch
    mg = gpu_lib
    say("graph replay: convolution backward")
    layers = [(4, 14, 14, 64, 128, 3, 3, 2, 1), (4, 7, 7, 128, 128, 3, 3, 1, 1),
              (2, 28, 28, 32, 64, 1, 1, 1, 0)]
    bufs = []
    for i, (N, H, W, C, K, R, S, st, pd) in enumerate(layers):
        x = make_conv_inputs(N, H, W, C, K, R, S, st, pd, seed=40 + i)
        X, Wt, dY = (torch.from_numpy(a.copy()).cuda() for a in (x.X, x.W, x.dY))
        need = mg.mg_conv2d_bwd_workspace_bytes(X.shape, Wt.shape, x.stride, x.pad)
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
        bufs.append((x, X, Wt, dY, torch.empty_like(X), torch.empty_like(Wt), ws))

    def step():
        for x, X, Wt, dY, dX, dW, ws in bufs:
            mg.mg_conv2d_bwd(X, Wt, dY, dX, dW, stride=x.stride, pad=x.pad, workspace=ws)

    step()
    torch.cuda.synchronize()
    outs = [t for b in bufs for t in (b[4], b[5])]
    expected = [t.clone() for t in outs]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, capture_error_mode="relaxed"):
        step()
    scratch = torch.randn(1 << 20, device="cuda")
    _replay_and_check(graph, outs, expected, lambda: scratch.sin_())
