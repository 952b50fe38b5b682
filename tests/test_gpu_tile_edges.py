"""GPU parity at tile edges, every contract.

The bf16 dK/dV kernel streams 64 query rows against 64 stationary keys (16
per wave), the bf16 dQ kernel 64-key tiles against 128 query rows, and the
bf16 and accelerated forwards 64-key tiles against 128 query rows (software-
pipelined for d <= 64, K and V double-buffered).  The strict forward takes
64 query rows (32 in its key-split form) against 64-key tiles, and the
strict fused backward 64 or 128 stationary keys against 32-row query steps,
split over several workgroups when the grid is small.  Each kernel masks
only the tiles that cross the causal diagonal or the key length, and decides
that per tile (per wave in the bf16 dK/dV kernel).  These cases put the query and key
lengths, the causal diagonal (bottom-right aligned when Lq != Lk) and the
key lengths on, just below and just above those tile edges, so that a tile
taken for full one row or key too early, a pipelined tile one step off, or a
last partial tile shows up against the f64 oracle.
"""
import pytest

from gpu_util import TOL, TOL_ACCEL_BWD, TOL_ACCEL_ROUNDED, accel_backward_reference, \
    compare, oracle_reference, run_gpu, say
from workloads import make_inputs

pytestmark = pytest.mark.gpu

CONTRACTS = ("strict_f32", "fast_bf16", "accelerated")

SQUARE = [31, 33, 63, 64, 65, 127, 128, 129, 191, 192, 193, 257]
CROSS = [(64, 127), (127, 64), (129, 192), (192, 129), (65, 256), (256, 65), (1, 129), (129, 1)]
# (Lk, key lengths of the two batches): on, below and above 64-key edges
PADDED = [(192, [64, 65]), (192, [63, 128]), (129, [1, 129]), (256, [191, 193])]


def check(x, contract):
    """strict_f32, fast_bf16: every output against the oracle.  accelerated: the forward
    against the oracle and against the oracle on f16-rounded inputs, the
    backward against the backward equations at that rounded-input forward
    (a batch whose rows each see one key has exact gradients of zero and
    contract gradients of the rounding residual of V; see
    accel_backward_reference)."""
    got = run_gpu(x)
    ref = oracle_reference(x)
    if contract != "accelerated":
        errs = compare(got, ref, contract)
        assert max(errs.values()) <= TOL[contract], errs
        return
    errs = compare(got, ref, contract, names=("O", "LSE"))
    assert max(errs.values()) <= TOL[contract], errs
    acc = accel_backward_reference(x)
    e_o, e_l = (compare(got, acc, contract, names=(n,))[n] for n in ("O", "LSE"))
    assert e_o <= TOL_ACCEL_ROUNDED["O"] and e_l <= TOL_ACCEL_ROUNDED["LSE"], (e_o, e_l)
    errs = compare(got, acc, contract, names=("dQ", "dK", "dV"))
    say("  accelerated backward vs its reference: %s" % errs)
    assert max(errs.values()) <= TOL_ACCEL_BWD, errs


@pytest.mark.parametrize("contract", CONTRACTS)
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("L", SQUARE)
def test_square_tile_edges(gpu_lib, L, causal, d, contract):
    say("tile edges %s L=%d d=%d causal=%s" % (contract, L, d, causal))
    x = make_inputs(1, 2, L, d, causal=causal, contract=contract, seed=97 * L + d + causal)
    check(x, contract)


@pytest.mark.parametrize("contract", CONTRACTS)
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("Lq,Lk", CROSS)
def test_cross_causal_tile_edges(gpu_lib, Lq, Lk, d, contract):
    say("tile edges %s Lq=%d Lk=%d d=%d causal" % (contract, Lq, Lk, d))
    x = make_inputs(1, 2, Lq, d, causal=True, contract=contract, seed=31 * Lq + 7 * Lk + d,
                    Lk=Lk)
    check(x, contract)


@pytest.mark.parametrize("contract", CONTRACTS)
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("Lk,key_len", PADDED)
def test_key_length_tile_edges(gpu_lib, Lk, key_len, causal, d, contract):
    say("tile edges %s Lk=%d key_len=%s d=%d causal=%s" % (contract, Lk, key_len, d, causal))
    x = make_inputs(2, 2, Lk, d, causal=causal, contract=contract, seed=13 * Lk + d + causal,
                    key_len=key_len)
    check(x, contract)
