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
