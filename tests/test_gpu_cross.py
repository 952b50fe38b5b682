"""GPU parity for cross-attention: queries and keys of different lengths
(Sec. 10 workloads: the U-Net's 77-token context, the action expert's 50
action tokens over 16 context tokens plus themselves, Whisper's 1,500
positions), in every arithmetic contract, against the f64 oracle.

The causal mask is bottom-right aligned: row i sees keys j <= i + Lk - Lq.
With Lk < Lq the first Lq - Lk rows see no key at all; the oracle gives them
O = 0, LSE = -inf and zero gradients, and `compare` demands those exactly.
"""
import numpy as np
import pytest

from gpu_util import TOL, TOL_ACCEL_BWD, TOL_ACCEL_ROUNDED, accel_backward_reference, \
    compare, normwise_error, oracle_reference, run_gpu, say
from workloads import WORKLOADS, make_inputs, workload_inputs

pytestmark = pytest.mark.gpu

CONTRACTS = ("strict_f32", "fast_bf16", "accelerated")

# (Lq, Lk, mode): longer and shorter key sides, single rows and single keys,
# lengths off every tile size
SHAPES = [
    (50, 66, "causal"), (66, 50, "causal"),
    (17, 130, "causal"), (130, 17, "causal"),
    (1, 65, "causal"), (65, 1, "causal"),
    (200, 77, "full"), (77, 200, "full"),
    (100, 77, "padded"), (50, 66, "causal_padded"), (140, 70, "causal_padded"),
]


def cross_inputs(Lq, Lk, d, mode, contract, B=2, H=3, seed=0):
    kl = None
    if mode.endswith("padded"):
        kl = [max(1, Lk // 2), Lk]
    return make_inputs(B, H, Lq, d, causal=mode.startswith("causal"), contract=contract,
                       seed=seed + 7919 * Lq + 31 * Lk + d, key_len=kl, Lk=Lk)


def check(x, contract):
    got = run_gpu(x)
    ref = oracle_reference(x)
    errs = compare(got, ref, contract)
    assert max(errs.values()) <= TOL[contract], errs
    if contract == "accelerated":
        from oracle import oracle_forward, round_to_f16
        Or, Lr = oracle_forward(round_to_f16(x.Q), round_to_f16(x.K), round_to_f16(x.V),
                                x.causal, x.scale, key_len=x.key_len)
        e_o, e_l = normwise_error(got["O"], Or), normwise_error(got["LSE"], Lr)
        assert e_o <= TOL_ACCEL_ROUNDED["O"] and e_l <= TOL_ACCEL_ROUNDED["LSE"], (e_o, e_l)
        # the backward against the backward equations at the rounded-input forward
        eb = compare(got, accel_backward_reference(x), "accelerated", names=("dQ", "dK", "dV"))
        assert max(eb.values()) <= TOL_ACCEL_BWD, eb
    return got, ref, errs


@pytest.mark.parametrize("contract", CONTRACTS)
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("Lq,Lk,mode", SHAPES)
def test_cross_small_shapes(gpu_lib, Lq, Lk, mode, d, contract):
    say("cross %s Lq=%d Lk=%d d=%d %s" % (contract, Lq, Lk, d, mode))
    check(cross_inputs(Lq, Lk, d, mode, contract), contract)


@pytest.mark.parametrize("contract", CONTRACTS)
def test_rows_that_see_no_key(gpu_lib, contract):
    """Causal with Lk < Lq: rows i < Lq - Lk are empty; their outputs are
    exactly O = 0, LSE = -inf, dQ = 0, on every contract."""
    Lq, Lk = 90, 20
    say("empty rows %s Lq=%d Lk=%d" % (contract, Lq, Lk))
    got, _, _ = check(cross_inputs(Lq, Lk, 64, "causal", contract), contract)
    empty = Lq - Lk
    assert np.all(got["O"][:, :, :empty] == 0.0)
    assert np.all(got["LSE"][:, :, :empty] == -np.inf)
    assert np.all(got["dQ"][:, :, :empty] == 0.0)
    assert np.all(np.isfinite(got["LSE"][:, :, empty:]))
    for n in ("dK", "dV"):
        assert np.all(np.isfinite(got[n]))


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("Lq,Lk", [(300, 1000), (1000, 520)])
def test_cross_wide_key_tiles(gpu_lib, Lq, Lk, d):
    """Causal problems with ceil(Lk/128)*B*H >= 512 take the 128-key fused
    backward; both signs of Lk - Lq and ragged tails on both sides."""
    B, H = 8, (8 if Lk >= 1000 else 16)   # 512 and 640 tiles of 128 keys
    kl = [Lk, Lk // 3, 128, 1, Lk, Lk - 1, 64, 2][:B]
    say("cross wide key tiles B%d H%d Lq%d Lk%d d%d" % (B, H, Lq, Lk, d))
    x = make_inputs(B, H, Lq, d, causal=True, seed=91 + d + Lq, key_len=kl, Lk=Lk)
    errs = compare(run_gpu(x), oracle_reference(x), "strict_f32")
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL["strict_f32"], errs


@pytest.mark.parametrize("wid", [7, 8])
def test_cross_and_ragged_workloads(gpu_lib, wid):
    w = WORKLOADS[wid]
    say("workload %d %s" % (wid, w.name))
    x = workload_inputs(wid)
    errs = compare(run_gpu(x), oracle_reference(x), w.contract)
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL[w.contract], errs


@pytest.mark.parametrize("contract", ("fast_bf16", "accelerated"))
def test_unet_cross_shape_low_precision(gpu_lib, contract):
    w = WORKLOADS[7]
    say("workload 7 shape, %s" % contract)
    x = make_inputs(w.B, w.H, w.L, w.d, causal=False, contract=contract, seed=w.seed,
                    Lk=w.key_length)
    _, _, errs = check(x, contract)
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})


def test_square_entry_points_are_the_cross_ones(gpu_lib):
    """mg_attn_fwd/bwd with L equal mg_attn_fwd_cross/bwd_cross with Lq = Lk = L
    bit for bit."""
    import torch
    mg = gpu_lib
    x = make_inputs(2, 3, 100, 64, causal=True, seed=5)
    Q, K, V, dO = (torch.from_numpy(getattr(x, n).copy()).cuda() for n in ("Q", "K", "V", "dO"))
    outs = []
    for cross in (False, True):
        O, LSE = torch.empty_like(Q), torch.empty(Q.shape[:3], device=Q.device)
        dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
        fwd = mg.mg_attn_fwd_cross if cross else mg.mg_attn_fwd
        bwd = mg.mg_attn_bwd_cross if cross else mg.mg_attn_bwd
        fwd(Q, K, V, O, LSE, causal=True, scale=x.scale)
        bwd(Q, K, V, O, LSE, dO, dQ, dK, dV, causal=True, scale=x.scale)
        torch.cuda.synchronize()
        outs.append([t.cpu() for t in (O, LSE, dQ, dK, dV)])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("B,H,Lq,Lk,causal,kl", [
    (2, 4, 1000, 300, True, [300, 129]),     # 40 key-tile workgroups -> 8 splits
    (1, 2, 300, 1000, True, [997]),          # 32 -> 2 splits, Lk > Lq
    (2, 3, 777, 77, False, [77, 1]),         # 12 -> 6 splits, one key left
])
def test_split_query_tiles(gpu_lib, B, H, Lq, Lk, causal, kl, d):
    """Few key tiles: the fused backward splits each key tile's query tiles
    over several workgroups and adds their dK/dV partials in a fixed order;
    results match the oracle and repeat bit for bit."""
    import torch
    say("split query tiles B%d H%d Lq%d Lk%d causal=%s d%d" % (B, H, Lq, Lk, causal, d))
    x = make_inputs(B, H, Lq, d, causal=causal, seed=123 + Lq + d, key_len=kl, Lk=Lk)
    got = run_gpu(x)
    errs = compare(got, oracle_reference(x), "strict_f32")
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL["strict_f32"], errs
    again = run_gpu(x)
    for n in ("dQ", "dK", "dV"):
        assert np.array_equal(got[n], again[n]), n
    torch.cuda.synchronize()


# Small fused grids compute D inside the fused kernel; with a single key tile
# and no query split the fused kernel writes dQ itself, including zero rows
# for queries that see no key.  The outputs start as NaN, so a row that no
# kernel writes fails the comparison.
SMALL_GRID_CASES = [
    # B, H, Lq, Lk, d, causal, key_len
    (2, 3, 200, 40, 64, True, None),        # one key tile; rows below 160 see no key
    (1, 1, 1, 1, 32, True, None),
    (3, 2, 70, 64, 32, False, [0, 17, 64]),  # one key tile; batch 0 has no keys at all
    (2, 2, 300, 250, 64, True, None),       # four key tiles, query split, local D
    (2, 2, 64, 64, 64, True, [64, 5]),      # one key tile, padded
]


@pytest.mark.parametrize("B,H,Lq,Lk,d,causal,kl", SMALL_GRID_CASES)
def test_small_grid_backward_writes_every_row(gpu_lib, B, H, Lq, Lk, d, causal, kl):
    import torch
    import paper_2608_01563_amd as mg
    say("small-grid backward B%d H%d Lq%d Lk%d d%d causal=%s key_len=%s"
        % (B, H, Lq, Lk, d, causal, kl))
    x = make_inputs(B, H, Lq, d, causal=causal, seed=500 + Lq + Lk + d, key_len=kl, Lk=Lk)
    Q, K, V, dO = (torch.from_numpy(getattr(x, n).copy()).cuda() for n in ("Q", "K", "V", "dO"))
    key_len = None if kl is None else torch.tensor(kl, dtype=torch.int32).cuda()
    O = torch.full((B, H, Lq, d), float("nan"), device="cuda")
    LSE = torch.full((B, H, Lq), float("nan"), device="cuda")
    dQ, dK, dV = (torch.full(t.shape, float("nan"), device="cuda") for t in (Q, K, V))
    ws = torch.full((max(mg.mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, causal,
                                                             "strict_f32"), 16),),
                    0xFF, dtype=torch.uint8, device="cuda")   # NaN patterns throughout
    mg.mg_attn_fwd_cross(Q, K, V, O, LSE, key_len, causal=causal, scale=x.scale,
                         contract="strict_f32")
    mg.mg_attn_bwd_cross(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len, causal=causal,
                         scale=x.scale, contract="strict_f32", workspace=ws)
    torch.cuda.synchronize()
    got = {n: t.cpu().numpy() for n, t in (("O", O), ("LSE", LSE), ("dQ", dQ), ("dK", dK),
                                          ("dV", dV))}
    errs = compare(got, oracle_reference(x), "strict_f32")
    say("  errors %s" % {k: "%.2e" % v for k, v in errs.items()})
    assert max(errs.values()) <= TOL["strict_f32"], errs
