"""mg_attn_bwd_noalloc (the backward whose workspace is the library's static
scratch array) against mg_attn_bwd_cross (caller workspace) through the C
ABI: two calls in a row per case, the second on a smaller problem, so the
second call reuses the array the first one left behind.

Where the caller-workspace layout fits in the array, the same kernels run
on the same data and the outputs must be bitwise equal.  Where it does not
(the strict B8 H8 L1024 workload needs 128 MiB of dQ partials), the call
keeps only D in the array and runs the separate dK/dV and dQ passes, whose
sums run in another order: every output must then agree with the
caller-workspace call within the contract's tolerance (normwise 1e-4 for
strict f32).
"""
import ctypes

import pytest

from gpu_util import TOL, key_len_device, normwise_error, say, to_device
from workloads import make_inputs, workload_inputs

pytestmark = pytest.mark.gpu

SCRATCH = 64 << 20


def _problem(mg, x):
    import torch
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    kl = key_len_device(x)
    O, LSE = mg.attention_forward(Q, K, V, causal=x.causal, scale=x.scale, key_len=kl,
                                  contract=x.contract)
    torch.cuda.synchronize()
    return Q, K, V, O, LSE, dO, kl


def _both(mg, x):
    """(reference outputs from mg_attn_bwd_cross, outputs of the no-alloc call)."""
    import torch
    Q, K, V, O, LSE, dO, kl = _problem(mg, x)
    ref = [torch.full_like(t, float("nan")) for t in (Q, K, V)]
    got = [torch.full_like(t, float("nan")) for t in (Q, K, V)]
    mg.mg_attn_bwd_cross(Q, K, V, O, LSE, dO, *ref, kl, causal=x.causal, scale=x.scale,
                         contract=x.contract)
    torch.cuda.synchronize()
    mg.mg_attn_bwd_noalloc(Q, K, V, O, LSE, dO, *got, kl, causal=x.causal, scale=x.scale,
                           contract=x.contract)
    torch.cuda.synchronize()
    return ref, got


def _fits(mg, x):
    B, H, Lq, d = x.Q.shape
    Lk = x.K.shape[2]
    return mg.mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, x.causal,
                                                x.contract) <= SCRATCH


def _check(mg, x, tag):
    import torch
    ref, got = _both(mg, x)
    for name, a, b in zip(("dQ", "dK", "dV"), got, ref):
        assert not torch.isnan(a).any(), (tag, name)
        if _fits(mg, x):
            assert torch.equal(a, b), (tag, name)
        else:
            e = normwise_error(a.double().cpu().numpy(), b.double().cpu().numpy())
            assert e <= TOL[x.contract], (tag, name, e)


CASES = [
    # (first call, second smaller call)
    ("strict, fits: B4 H4 L256 causal, then B2 H3 L100 padded",
     lambda: workload_inputs(2),
     lambda: make_inputs(2, 3, 100, 64, causal=False, seed=41, key_len=[37, 100])),
    ("strict, D only: B8 H8 L1024 causal, then B1 H2 L129 cross Lk 77",
     lambda: workload_inputs(3),
     lambda: make_inputs(1, 2, 129, 32, causal=True, seed=42, Lk=77)),
    ("bf16: B2 H4 L1000 d128 causal, then B1 H1 L65 d64",
     lambda: make_inputs(2, 4, 1000, 128, causal=True, contract="fast_bf16", seed=43),
     lambda: make_inputs(1, 1, 65, 64, causal=False, contract="fast_bf16", seed=44)),
    ("accelerated: B2 H2 L300 causal, then B1 H1 L17 d32",
     lambda: make_inputs(2, 2, 300, 64, causal=True, contract="accelerated", seed=45),
     lambda: make_inputs(1, 1, 17, 32, causal=True, contract="accelerated", seed=46)),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0].split(":")[0])
def test_noalloc_matches_workspace_backward(gpu_lib, case):
    tag, first, second = case
    say("no-alloc backward: %s" % tag)
    _check(gpu_lib, first(), tag + " (first call)")
    _check(gpu_lib, second(), tag + " (second, smaller call)")


def test_noalloc_refuses_rows_beyond_the_scratch(gpu_lib):
    """B*H*Lq f32 of D above the array: MG_ERR_WORKSPACE, nothing enqueued."""
    import torch
    mg = gpu_lib
    say("no-alloc backward: size beyond the scratch")
    x = make_inputs(1, 1, 64, 32, causal=True, seed=47)
    Q, K, V, O, LSE, dO, _ = _problem(mg, x)
    dQ = torch.full_like(Q, 7.0)
    lib = mg.load_library()
    rows = SCRATCH // 4 + 1            # one query row more than D can hold
    st = lib.mg_attn_bwd_noalloc(*(ctypes.c_void_p(t.data_ptr()) for t in
                                   (Q, K, V, O, LSE, dO, dQ, dQ, dQ)), None, 1, 1, rows, 64,
                                 32, 1, ctypes.c_float(x.scale), 0, None)
    assert st == 4 and "scratch" in mg.mg_last_error_detail()
    torch.cuda.synchronize()
    assert torch.all(dQ == 7.0)
