"""Reentrancy of the C ABI: the library keeps no per-call state, so problems
enqueued on several streams at once, from one host thread or from several,
must give bit-identical results to the same problems run one after another
on one stream (the kernels are deterministic: no atomics, fixed reduction
orders).  Every buffer is allocated before the concurrent phase; the threads
only launch and synchronize their own stream.
"""
import threading

import numpy as np
import pytest

from gpu_util import say
from workloads import make_inputs

pytestmark = pytest.mark.gpu

# (B, H, Lq, Lk, d, causal, contract, key-length range, seed): a mix of
# contracts, masks, head dimensions and split / unsplit backward grids
CASES = [
    (2, 4, 300, 300, 64, True, "strict_f32", None, 71),
    (2, 3, 257, 200, 128, False, "fast_bf16", (1, 200), 72),
    (1, 4, 190, 77, 64, False, "accelerated", None, 73),
    (2, 2, 129, 129, 32, True, "strict_f32", (60, 129), 74),
]


class _Problem:
    def __init__(self, mg, case):
        import torch
        B, H, Lq, Lk, d, causal, contract, klr, seed = case
        x = make_inputs(B, H, Lq, d, causal=causal, contract=contract, seed=seed, Lk=Lk,
                        key_len_range=klr)
        if contract == "fast_bf16":
            dev = lambda n: torch.from_numpy(x.bits[n].view(np.int16).copy()).cuda().view(
                torch.bfloat16)
        else:
            dev = lambda n: torch.from_numpy(getattr(x, n).copy()).cuda()
        self.mg, self.x, self.contract, self.causal = mg, x, contract, causal
        self.Q, self.K, self.V, self.dO = (dev(n) for n in ("Q", "K", "V", "dO"))
        self.kl = None if x.key_len is None else torch.from_numpy(
            np.asarray(x.key_len, dtype=np.int32).copy()).cuda()
        self.O, self.LSE = torch.empty_like(self.Q), torch.empty(self.Q.shape[:3], device="cuda")
        self.dQ, self.dK, self.dV = (torch.empty_like(self.Q), torch.empty_like(self.K),
                                     torch.empty_like(self.V))
        self.ws = torch.empty(max(256, mg.mg_attn_bwd_cross_workspace_bytes(
            B, H, Lq, Lk, d, causal, contract)), dtype=torch.uint8, device="cuda")

    def outputs(self):
        return (self.O, self.LSE, self.dQ, self.dK, self.dV)

    def poison(self):
        for t in self.outputs():
            t.fill_(float("nan"))

    def step(self, stream):
        mg, x = self.mg, self.x
        mg.mg_attn_fwd_cross(self.Q, self.K, self.V, self.O, self.LSE, self.kl,
                             causal=self.causal, scale=x.scale, contract=self.contract,
                             stream=stream)
        mg.mg_attn_bwd_cross(self.Q, self.K, self.V, self.O, self.LSE, self.dO, self.dQ,
                             self.dK, self.dV, self.kl, causal=self.causal, scale=x.scale,
                             contract=self.contract, workspace=self.ws, stream=stream)


def _serial_reference(problems):
    import torch
    stream = torch.cuda.current_stream()
    expected = []
    for p in problems:
        p.step(stream)
        torch.cuda.synchronize()
        expected.append([t.clone() for t in p.outputs()])
    return expected


def _check(problems, expected, tag):
    import torch
    for i, (p, want) in enumerate(zip(problems, expected)):
        for name, got, ref in zip(("O", "LSE", "dQ", "dK", "dV"), p.outputs(), want):
            assert torch.equal(got, ref), (tag, i, name)


def test_streams_from_one_thread_match_serial(gpu_lib):
    import torch
    say("streams: %d problems on %d streams, one host thread" % (len(CASES), len(CASES)))
    problems = [_Problem(gpu_lib, c) for c in CASES]
    expected = _serial_reference(problems)
    streams = [torch.cuda.Stream() for _ in problems]   # default priority
    for rep in range(3):
        for p in problems:
            p.poison()
        torch.cuda.synchronize()
        for p, s in zip(problems, streams):   # interleaved launches
            p.step(s)
        torch.cuda.synchronize()
        _check(problems, expected, "rep %d" % rep)


def test_threads_each_with_a_stream_match_serial(gpu_lib):
    import torch
    say("streams: %d host threads, one stream each" % len(CASES))
    problems = [_Problem(gpu_lib, c) for c in CASES]
    expected = _serial_reference(problems)
    streams = [torch.cuda.Stream() for _ in problems]
    for p in problems:
        p.poison()
    torch.cuda.synchronize()
    errors = []
    start = threading.Barrier(len(problems))

    def worker(p, s):
        try:
            torch.cuda.set_device(0)
            start.wait(timeout=60)
            for _ in range(4):
                p.step(s)
            s.synchronize()
        except Exception as e:   # reported by the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(p, s)) for p, s in zip(problems, streams)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a launching thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    _check(problems, expected, "threads")


def test_binding_temporaries_on_side_streams(gpu_lib):
    """Workspaces and outputs that the binding allocates itself (no
    workspace given) belong to the stream the kernels run on: freeing them
    on return while those kernels still run, then allocating and filling
    memory on the current stream, must leave every result intact."""
    import torch
    from workloads.conv import make_conv_inputs
    mg = gpu_lib
    say("streams: binding-allocated workspaces on side streams")
    problems = [_Problem(gpu_lib, c) for c in CASES]
    expected = _serial_reference(problems)
    cx = make_conv_inputs(2, 20, 20, 64, 96, 3, 3, 1, 1, seed=75)
    X, W, dY = (torch.from_numpy(a.copy()).cuda() for a in (cx.X, cx.W, cx.dY))
    cref = mg.conv2d_backward(X, W, dY, stride=cx.stride, pad=cx.pad)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in problems]   # default priority
    conv_stream = torch.cuda.Stream()
    for rep in range(3):
        results = []
        for p, s in zip(problems, streams):
            O, LSE = mg.attention_forward(p.Q, p.K, p.V, causal=p.causal, scale=p.x.scale,
                                          key_len=p.kl, contract=p.contract, stream=s)
            g = mg.attention_backward(p.Q, p.K, p.V, O, LSE, p.dO, causal=p.causal,
                                      scale=p.x.scale, key_len=p.kl, contract=p.contract,
                                      stream=s)
            results.append((O, LSE) + tuple(g))
            # the backward's workspace is already freed: memory taken and
            # written on the current stream must not be that block
            torch.full((1 << 22,), float("nan"), device="cuda")
        cout = mg.conv2d_backward(X, W, dY, stride=cx.stride, pad=cx.pad, stream=conv_stream)
        torch.full((1 << 22,), float("nan"), device="cuda")
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(results, expected)):
            for name, a, b in zip(("O", "LSE", "dQ", "dK", "dV"), got, want):
                assert torch.equal(a, b), ("rep %d" % rep, i, name)
        assert torch.equal(cout[0], cref[0]) and torch.equal(cout[1], cref[1]), rep
