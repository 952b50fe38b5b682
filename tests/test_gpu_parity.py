"""GPU parity: the HIP path (through the C ABI) against the f64 oracle on the
same seeded inputs, plus bitwise pins that need no oracle.

Tolerance (normwise, per output tensor): max|gpu - oracle| / max|oracle|
<= 1e-4 for strict_f32 and <= 2e-2 for fast_bf16.  The end-to-end cases feed
the GPU's own O and LSE into the GPU backward; the isolation case feeds the
oracle's O and LSE instead.
"""
import math

import numpy as np
import pytest

from gpu_util import (TOL, TOL_ACCEL_ROUNDED, compare, key_len_device, normwise_error,
                      oracle_reference, run_gpu, say, to_device)
from workloads import WORKLOADS, AttnInputs, make_inputs, workload_inputs

pytestmark = pytest.mark.gpu

SMALL = [(L, d, mode) for L in (1, 17, 64, 65, 200) for d in (32, 64, 128)
         for mode in ("causal", "full", "padded")]


def small_inputs(L, d, mode, contract="strict_f32", B=2, H=3, seed=0):
    kl = None
    if mode == "padded":
        kl = [max(1, L // 2), L][:B] + [L] * max(0, B - 2)
    return make_inputs(B, H, L, d, causal=(mode == "causal"), contract=contract,
                       seed=seed + 1000 * L + d, key_len=kl)


@pytest.mark.parametrize("L,d,mode", SMALL)
def test_small_shapes_strict(gpu_lib, L, d, mode):
    say("small strict L=%d d=%d %s" % (L, d, mode))
    x = small_inputs(L, d, mode)
    errs = compare(run_gpu(x), oracle_reference(x), "strict_f32")
    assert max(errs.values()) <= TOL["strict_f32"], errs


@pytest.mark.parametrize("B,H,Lq,Lk,d,causal,kl", [
    (4, 4, 256, 256, 64, True, None),      # workload 2's shape: four key groups
    (1, 2, 300, 257, 32, True, None),      # nine 32-key tiles: the last group is empty
    (2, 2, 513, 513, 64, False, [513, 40]),   # padded: one batch's groups mostly idle
    (1, 3, 100, 300, 64, True, None),      # cross, bottom-right causal
])
def test_strict_four_group_forward(gpu_lib, B, H, Lq, Lk, d, causal, kl):
    """Small grids with long key sides split their key tiles over four groups
    of waves, merged in group order; against the oracle."""
    say("strict four-group forward B%d H%d Lq%d Lk%d d%d causal=%s" % (B, H, Lq, Lk, d, causal))
    assert B * H * -(-Lq // 32) <= 256 and Lk >= 256
    x = make_inputs(B, H, Lq, d, causal=causal, seed=41 + Lq + Lk, key_len=kl, Lk=Lk)
    errs = compare(run_gpu(x), oracle_reference(x), "strict_f32")
    assert max(errs.values()) <= TOL["strict_f32"], errs


@pytest.mark.parametrize("wid", [1, 2, 3, 5])
def test_workload_full_compare_strict(gpu_lib, wid):
    w = WORKLOADS[wid]
    say("workload %d %s" % (wid, w.name))
    x = workload_inputs(wid)
    errs = compare(run_gpu(x), oracle_reference(x), w.contract)
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL[w.contract], errs


def test_backward_isolated_with_oracle_forward(gpu_lib):
    say("backward isolation, workload 2")
    x = workload_inputs(2)
    ref = oracle_reference(x)
    got = run_gpu(x, O_in=ref["O"], LSE_in=ref["LSE"])
    errs = compare(got, ref, "strict_f32", names=("dQ", "dK", "dV"))
    assert max(errs.values()) <= TOL["strict_f32"], errs


def test_bitwise_pins(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    say("bitwise pins")
    x = make_inputs(2, 8, 192, 64, causal=True, seed=7)
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    s = x.scale
    O, LSE = mg.attention_forward(Q, K, V, causal=True, scale=s)
    # causal row 0 attends only to key 0 with probability exp(0) = 1
    assert torch.equal(O[:, :, 0, :], V[:, :, 0, :])
    # O is linear in V with the same P; doubling is exact in binary floating point
    O2, LSE2 = mg.attention_forward(Q, K, 2 * V, causal=True, scale=s)
    assert torch.equal(O2, 2 * O) and torch.equal(LSE2, LSE)
    g1 = mg.attention_backward(Q, K, V, O, LSE, dO, causal=True, scale=s)
    g2 = mg.attention_backward(Q, K, V, O, LSE, 2 * dO, causal=True, scale=s)
    for a, b in zip(g1, g2):
        assert torch.equal(2 * a, b)
    # run-to-run determinism (no atomics anywhere)
    g3 = mg.attention_backward(Q, K, V, O, LSE, dO, causal=True, scale=s)
    for a, b in zip(g1, g3):
        assert torch.equal(a, b)
    Oa, LSEa = mg.attention_forward(Q, K, V, causal=True, scale=s)
    assert torch.equal(Oa, O) and torch.equal(LSEa, LSE)
    # a head computed alone equals the same head computed in the batch
    b, h = 1, 5
    sl = lambda t: t[b:b + 1, h:h + 1].contiguous()
    O1, L1 = mg.attention_forward(sl(Q), sl(K), sl(V), causal=True, scale=s)
    assert torch.equal(O1, sl(O)) and torch.equal(L1, sl(LSE))
    gs = mg.attention_backward(sl(Q), sl(K), sl(V), O1, L1, sl(dO), causal=True, scale=s)
    for a, full in zip(gs, g1):
        assert torch.equal(a, sl(full))
    # rows of P sum to one: sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i, up to
    # rounding bounded by the sums of magnitudes
    dQ, dK, dV = (t.double() for t in g1)
    go = dO.double()
    assert torch.all(torch.abs(dK.sum(2)) <= 1e-4 * torch.abs(dK).sum(2))
    assert torch.all(torch.abs(dV.sum(2) - go.sum(2)) <= 1e-4 * torch.abs(go).sum(2))


def test_padded_keys_get_exact_zero_gradients(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    say("padded zero gradients")
    x = make_inputs(3, 2, 160, 64, causal=False, seed=11, key_len=[37, 160, 64])
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    kl = key_len_device(x)
    O, LSE = mg.attention_forward(Q, K, V, causal=False, scale=x.scale, key_len=kl)
    dQ, dK, dV = mg.attention_backward(Q, K, V, O, LSE, dO, causal=False, scale=x.scale,
                                       key_len=kl)
    for b, n in enumerate(x.key_len):
        assert torch.count_nonzero(dK[b, :, n:]) == 0
        assert torch.count_nonzero(dV[b, :, n:]) == 0


def test_fully_masked_batch_and_out_of_range_key_len(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    say("fully masked batch")
    L = 70
    x = make_inputs(3, 2, L, 32, causal=True, seed=3, key_len=[0, L, 1000])
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    kl = key_len_device(x)
    O, LSE = mg.attention_forward(Q, K, V, causal=True, scale=x.scale, key_len=kl)
    g = mg.attention_backward(Q, K, V, O, LSE, dO, causal=True, scale=x.scale, key_len=kl)
    assert torch.count_nonzero(O[0]) == 0
    assert torch.all(torch.isinf(LSE[0])) and torch.all(LSE[0] < 0)
    for t in g:
        assert torch.count_nonzero(t[0]) == 0
    # key_len beyond L behaves as L
    O_nopad, L_nopad = mg.attention_forward(Q, K, V, causal=True, scale=x.scale)
    assert torch.equal(O[1], O_nopad[1]) and torch.equal(O[2], O_nopad[2])
    assert torch.equal(LSE[2], L_nopad[2])


def test_every_output_element_is_written(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    say("NaN poison")
    for L, d, causal in ((65, 64, True), (200, 32, False), (17, 128, True)):
        x = make_inputs(1, 3, L, d, causal=causal, seed=5)
        Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
        O = torch.full_like(Q, float("nan"))
        LSE = torch.full(Q.shape[:3], float("nan"), device=Q.device)
        mg.mg_attn_fwd(Q, K, V, O, LSE, causal=causal, scale=x.scale)
        dQ, dK, dV = (torch.full_like(Q, float("nan")) for _ in range(3))
        mg.mg_attn_bwd(Q, K, V, O, LSE, dO, dQ, dK, dV, causal=causal, scale=x.scale)
        torch.cuda.synchronize()
        for t in (O, LSE, dQ, dK, dV):
            assert not torch.isnan(t).any()


def test_argument_errors_enqueue_nothing(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    say("argument errors")
    x = make_inputs(1, 2, 64, 64, causal=True, seed=9)
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    O, LSE = mg.attention_forward(Q, K, V, causal=True, scale=x.scale)
    dQ = torch.full_like(Q, 7.0)
    small = torch.empty(16, dtype=torch.uint8, device=Q.device)
    with pytest.raises(mg.MgError) as e:
        mg.mg_attn_bwd(Q, K, V, O, LSE, dO, dQ, dQ.clone(), dQ.clone(), causal=True,
                       scale=x.scale, workspace=small)
    assert e.value.status == 4
    torch.cuda.synchronize()
    assert torch.all(dQ == 7.0)
    with pytest.raises(mg.MgError) as e:
        mg.mg_attn_fwd(Q, K, V, O, LSE, causal=True, scale=math.inf)
    assert e.value.status == 1


# ------------------------------------------------------------ fast_bf16 --

@pytest.mark.parametrize("L,d,mode", SMALL)
def test_small_shapes_bf16(gpu_lib, L, d, mode):
    say("small bf16 L=%d d=%d %s" % (L, d, mode))
    x = small_inputs(L, d, mode, contract="fast_bf16")
    errs = compare(run_gpu(x), oracle_reference(x), "fast_bf16")
    assert max(errs.values()) <= TOL["fast_bf16"], errs


@pytest.fixture(scope="module")
def workload4():
    """Workload 4's inputs and the oracle on every one of its 32 heads
    (computed once for the end-to-end and the backward-isolation test)."""
    w = WORKLOADS[4]
    say("workload 4 %s: oracle on all %d heads" % (w.name, w.B * w.H))
    x = workload_inputs(4)
    return w, x, oracle_reference(x)


def test_workload4_all_heads_bf16(gpu_lib, workload4):
    w, x, ref = workload4
    say("workload 4 %s end to end" % w.name)
    got = run_gpu(x)
    errs = compare(got, ref, w.contract)
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL[w.contract], errs
    # the same gate head by head, so that one bad head cannot hide behind
    # the others' larger maxima
    for b in range(w.B):
        for h in range(w.H):
            e = compare(got, ref, w.contract, heads=[(b, h)])
            assert max(e.values()) <= TOL[w.contract], (b, h, e)


def test_workload4_backward_isolated_bf16(gpu_lib, workload4):
    """The fast_bf16 backward alone: the oracle's O (rounded to bf16, nearest
    even, as the contract stores it) and f32 LSE go into the GPU backward."""
    w, x, ref = workload4
    say("workload 4 backward isolation")
    got = run_gpu(x, O_in=ref["O"], LSE_in=ref["LSE"])
    errs = compare(got, ref, w.contract, names=("dQ", "dK", "dV"))
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL[w.contract], errs


@pytest.mark.parametrize("L,d,mode", [(200, 128, "padded"), (65, 64, "causal"),
                                       (17, 32, "full")])
def test_backward_isolated_bf16_ragged(gpu_lib, L, d, mode):
    """fast_bf16 backward isolation on ragged tails and key padding."""
    say("bf16 backward isolation L=%d d=%d %s" % (L, d, mode))
    x = small_inputs(L, d, mode, contract="fast_bf16", seed=5)
    ref = oracle_reference(x)
    got = run_gpu(x, O_in=ref["O"], LSE_in=ref["LSE"])
    errs = compare(got, ref, "fast_bf16", names=("dQ", "dK", "dV"))
    assert max(errs.values()) <= TOL["fast_bf16"], errs


def test_bitwise_pins_bf16(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    say("bitwise pins bf16")
    x = make_inputs(2, 8, 192, 128, causal=True, contract="fast_bf16", seed=17)
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    s = x.scale
    O, LSE = mg.attention_forward(Q, K, V, causal=True, scale=s)
    assert torch.equal(O[:, :, 0, :], V[:, :, 0, :])
    O2, LSE2 = mg.attention_forward(Q, K, 2 * V, causal=True, scale=s)
    assert torch.equal(O2, 2 * O) and torch.equal(LSE2, LSE)
    g1 = mg.attention_backward(Q, K, V, O, LSE, dO, causal=True, scale=s)
    g2 = mg.attention_backward(Q, K, V, O, LSE, dO, causal=True, scale=s)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)
    b, h = 0, 3
    sl = lambda t: t[b:b + 1, h:h + 1].contiguous()
    O1, L1 = mg.attention_forward(sl(Q), sl(K), sl(V), causal=True, scale=s)
    assert torch.equal(O1, sl(O)) and torch.equal(L1, sl(LSE))
    gs = mg.attention_backward(sl(Q), sl(K), sl(V), O1, L1, sl(dO), causal=True, scale=s)
    for a, full in zip(gs, g1):
        assert torch.equal(a, sl(full))


def test_padded_keys_exact_zero_bf16(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    say("padded zero gradients bf16")
    x = make_inputs(2, 2, 130, 64, causal=False, contract="fast_bf16", seed=19,
                    key_len=[45, 0])
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    kl = key_len_device(x)
    O, LSE = mg.attention_forward(Q, K, V, causal=False, scale=x.scale, key_len=kl)
    dQ, dK, dV = mg.attention_backward(Q, K, V, O, LSE, dO, causal=False, scale=x.scale,
                                       key_len=kl)
    assert torch.count_nonzero(dK[0, :, 45:]) == 0 and torch.count_nonzero(dV[0, :, 45:]) == 0
    assert torch.count_nonzero(O[1]) == 0 and torch.all(torch.isinf(LSE[1]))
    for t in (dQ, dK, dV):
        assert torch.count_nonzero(t[1]) == 0


# One head below the element limit B*H*max(Lq, Lk)*d <= 2^31 - 1 that the
# C ABI accepts: every tensor spans about 2^31 elements, so each byte offset
# past 2^32 and each element index past 2^31 - 1 would show here.
MAX_SIZE_CASES = [("strict_f32", 64, True, 524287, 1), ("fast_bf16", 128, False, 87381, 3)]


@pytest.mark.parametrize("contract,d,causal,B,H", MAX_SIZE_CASES,
                         ids=["strict_d64_causal", "bf16_d128_full"])
def test_maximum_size_sampled_heads(gpu_lib, contract, d, causal, B, H):
    """Inputs drawn on the device from a seeded generator; the first, a middle
    and the last head (the one whose rows end just below 2^31 elements) are
    copied back and compared with the oracle on exactly those values."""
    import torch
    import paper_2608_01563_amd as mg
    L = 64
    assert B * H * L * d <= 2 ** 31 - 1 < (B * H + 1) * L * d
    say("maximum size %s B%d H%d L%d d%d (%.2f G elements per tensor)"
        % (contract, B, H, L, d, B * H * L * d / 2 ** 30))
    dt = torch.bfloat16 if contract == "fast_bf16" else torch.float32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(97)
    Q, K, V, dO = (torch.randn(B, H, L, d, device="cuda", generator=gen).to(dt) for _ in range(4))
    scale = d ** -0.5
    O, LSE = mg.attention_forward(Q, K, V, causal=causal, scale=scale, contract=contract)
    dQ, dK, dV = mg.attention_backward(Q, K, V, O, LSE, dO, causal=causal, scale=scale,
                                       contract=contract)
    torch.cuda.synchronize()
    heads = [(0, 0), (B // 2, H // 2), (B - 1, H - 1)]

    def sub(t):   # the sampled heads as one batch of len(heads) heads, f32 on the host
        return np.ascontiguousarray(np.stack([t[b, h].float().cpu().numpy() for b, h in heads])[None])

    x = AttnInputs(Q=sub(Q), K=sub(K), V=sub(V), dO=sub(dO), key_len=None, contract=contract,
                   causal=causal, scale=scale)
    got = {n: sub(t) for n, t in zip(("O", "LSE", "dQ", "dK", "dV"), (O, LSE, dQ, dK, dV))}
    del Q, K, V, dO, O, LSE, dQ, dK, dV
    torch.cuda.empty_cache()
    errs = compare(got, oracle_reference(x), contract)
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL[contract], errs


def test_strict_separate_dq_fallback_sampled_heads(gpu_lib):
    """Non-causal B32 H16 L1024 d64 needs 2 GiB of dQ partials, above the
    1 GiB cap, so dQ comes from the separate query-stationary kernel."""
    import paper_2608_01563_amd as mg
    B, H, L, d = 32, 16, 1024, 64
    need = mg.mg_attn_bwd_workspace_bytes(B, H, L, d, 0, "strict_f32")
    assert need == B * H * L * 4       # D only: the fallback path
    say("separate dQ fallback B%d H%d L%d d%d" % (B, H, L, d))
    x = make_inputs(B, H, L, d, causal=False, seed=23, key_len_range=(1, L))
    heads = [(0, 0), (7, 3), (19, 15), (31, 8)]
    errs = compare(run_gpu(x), oracle_reference(x, heads=heads), "strict_f32", heads=heads)
    assert max(errs.values()) <= TOL["strict_f32"], errs


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("padded", [False, True])
def test_wide_key_tiles_ragged(gpu_lib, d, padded):
    """Causal problems with ceil(L/128)*B*H >= 512 take the 128-key fused
    backward (8 waves); a ragged L exercises its tail tiles, key padding its
    masked waves."""
    B, H, L = 4, 16, 1000
    kl = [1000, 517, 128, 1] if padded else None
    say("wide key tiles B%d H%d L%d d%d padded=%s" % (B, H, L, d, padded))
    x = make_inputs(B, H, L, d, causal=True, seed=77 + d, key_len=kl)
    errs = compare(run_gpu(x), oracle_reference(x), "strict_f32")
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL["strict_f32"], errs


@pytest.mark.parametrize("d,padded,neg", [(32, False, False), (64, True, False),
                                           (64, False, True)])
def test_unsplit_forward_cross_ragged(gpu_lib, d, padded, neg):
    """Strict forward grids of 512 or more 64-row workgroups keep the unsplit
    kernel (smaller grids split their key tiles); B*H = 64 heads of Lq = 520
    queries over Lk = 333 keys give 576 workgroups with ragged query and key
    tails, a negative scale in one case."""
    B, H, Lq, Lk = 8, 8, 520, 333
    kl = [333, 300, 65, 64, 1, 0, 200, 333] if padded else None
    scale = (-1.0 if neg else 1.0) / d ** 0.5
    say("unsplit forward B%d H%d Lq%d Lk%d d%d padded=%s scale=%.3f" % (B, H, Lq, Lk, d,
                                                                         padded, scale))
    x = make_inputs(B, H, Lq, d, causal=False, seed=131 + d, key_len=kl, scale=scale, Lk=Lk)
    errs = compare(run_gpu(x), oracle_reference(x), "strict_f32")
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL["strict_f32"], errs


@pytest.mark.parametrize("contract,d", [("fast_bf16", 128), ("fast_bf16", 64),
                                        ("accelerated", 64)])
def test_resident_causal_grid_ragged(gpu_lib, contract, d):
    """B*H = 64 heads of a ragged causal L = 1000: the forward grids (and the
    bf16 dQ grid) fit on the chip at once, so their tiles are dealt in
    alternating-direction layers of 256 / (B*H) ranks; every tile must still
    be computed once."""
    B, H, L = 4, 16, 1000
    say("resident causal grid %s B%d H%d L%d d%d" % (contract, B, H, L, d))
    x = make_inputs(B, H, L, d, causal=True, contract=contract, seed=91 + d)
    if contract == "accelerated":
        accel_check(x)
        return
    errs = compare(run_gpu(x), oracle_reference(x), contract)
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL[contract], errs


# ---- accelerated contract: f32 tensors, f16 forward matrix inputs, strict backward

ACCEL_SMALL = [(L, d, mode) for L in (1, 17, 65, 200) for d in (32, 64, 128)
               for mode in ("causal", "full", "padded")]


def accel_check(x):
    from oracle import oracle_forward, round_to_f16
    got = run_gpu(x)
    Or, Lr = oracle_forward(round_to_f16(x.Q), round_to_f16(x.K), round_to_f16(x.V), x.causal,
                            x.scale, key_len=x.key_len)
    e_o, e_l = normwise_error(got["O"], Or), normwise_error(got["LSE"], Lr)
    assert e_o <= TOL_ACCEL_ROUNDED["O"] and e_l <= TOL_ACCEL_ROUNDED["LSE"], (e_o, e_l)
    errs = compare(got, oracle_reference(x), "accelerated")
    assert max(errs.values()) <= TOL["accelerated"], errs
    return e_o, e_l, errs


@pytest.mark.parametrize("L,d,mode", ACCEL_SMALL)
def test_small_shapes_accelerated(gpu_lib, L, d, mode):
    say("small accelerated L=%d d=%d %s" % (L, d, mode))
    accel_check(small_inputs(L, d, mode, contract="accelerated"))


def test_workload6_accelerated(gpu_lib):
    w = WORKLOADS[6]
    say("workload 6 %s" % w.name)
    e_o, e_l, errs = accel_check(workload_inputs(6))
    say("  rounded-input O %.2e LSE %.2e; exact %s" % (e_o, e_l,
                                                        {k: "%.2e" % v for k, v in errs.items()}))


@pytest.mark.parametrize("B,H,L,d,scale_sign", [(2, 8, 1024, 64, 1), (1, 4, 1000, 32, 1),
                                                 (2, 3, 777, 64, -1)])
def test_accelerated_key_split_forward(gpu_lib, B, H, L, d, scale_sign):
    """Causal grids of at most 256 query tiles take the key-split forward
    (two key groups per workgroup, merged through LDS): long key chains, an
    odd key-tile count (777 keys: 13 tiles, the second group idles through
    one iteration) and a negative scale, against the oracle."""
    say("accelerated key-split forward B%d H%d L%d d%d scale sign %d" % (B, H, L, d, scale_sign))
    x = make_inputs(B, H, L, d, causal=True, contract="accelerated", seed=31 + L,
                    scale=scale_sign / math.sqrt(d))
    assert B * H * -(-L // 128) <= 256
    accel_check(x)


def test_accelerated_backward_is_the_strict_backward(gpu_lib):
    """Given the same O and LSE, the accelerated backward is the strict one:
    bitwise equal outputs, and the oracle's O/LSE in gives strict parity."""
    import torch
    import paper_2608_01563_amd as mg
    say("accelerated backward vs strict backward")
    x = workload_inputs(2)
    ref = oracle_reference(x)
    got = run_gpu(x, O_in=ref["O"], LSE_in=ref["LSE"])
    errs = compare(got, ref, "strict_f32", names=("dQ", "dK", "dV"))
    assert max(errs.values()) <= TOL["strict_f32"], errs
    Q, K, V, dO = (to_device(x, n) for n in ("Q", "K", "V", "dO"))
    O = torch.from_numpy(ref["O"].astype(np.float32)).cuda()
    LSE = torch.from_numpy(ref["LSE"].astype(np.float32)).cuda()
    ga = mg.attention_backward(Q, K, V, O, LSE, dO, causal=True, scale=x.scale,
                               contract="accelerated")
    gs = mg.attention_backward(Q, K, V, O, LSE, dO, causal=True, scale=x.scale,
                               contract="strict_f32")
    for a, b in zip(ga, gs):
        assert torch.equal(a, b)


def test_bitwise_pins_accelerated(gpu_lib):
    import torch
    import paper_2608_01563_amd as mg
    from oracle import round_to_f16
    say("bitwise pins accelerated")
    x = make_inputs(2, 4, 130, 64, causal=True, contract="accelerated", seed=21)
    Q, K, V = (to_device(x, n) for n in ("Q", "K", "V"))
    O, LSE = mg.attention_forward(Q, K, V, causal=True, scale=x.scale, contract="accelerated")
    # causal row 0 attends only to key 0 with probability exactly 1, so O is
    # the f16-rounded V row, exactly
    v0 = torch.from_numpy(round_to_f16(x.V[:, :, 0, :]).astype(np.float32)).cuda()
    assert torch.equal(O[:, :, 0, :], v0)
    # run-to-run determinism
    O2, LSE2 = mg.attention_forward(Q, K, V, causal=True, scale=x.scale, contract="accelerated")
    assert torch.equal(O, O2) and torch.equal(LSE, LSE2)
