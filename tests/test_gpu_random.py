"""Randomised GPU parity sweep against the f64 oracle.

Seeded draws over batch and head counts, query and key lengths (1..600,
equal or not), head size, causal masking, key padding (key lengths from 0 to
Lk, per batch), contract, and the sign and size of `scale` (negative and
zero scales take the forward's non-positive-scale path; magnitudes stay at
or below 1/sqrt(d) so that the bf16 and f16 tolerances keep their meaning).
A quarter of the draws have B*H a multiple of 8, so that key-padded
non-causal grids take the XCD-grouped tile orders.  The case list is fixed
by the seed; each case prints its parameters before it runs.
"""
import math

import numpy as np
import pytest

from gpu_util import TOL, TOL_ACCEL_BWD, TOL_ACCEL_ROUNDED, accel_backward_reference, \
    compare, normwise_error, oracle_reference, run_gpu, say
from workloads import make_inputs

pytestmark = pytest.mark.gpu

CONTRACTS = ("strict_f32", "fast_bf16", "accelerated")
N_CASES = 96


def _draw_cases(n, seed=20261202):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        contract = CONTRACTS[i % 3]
        d = int((32, 64, 128)[rng.integers(3)])
        if i % 4 == 1:
            B, H = [(1, 8), (2, 4), (4, 2), (2, 8)][rng.integers(4)]
        else:
            B, H = int(rng.integers(1, 4)), int(rng.integers(1, 6))
        Lq = int(rng.integers(1, 601))
        Lk = Lq if rng.random() < 0.5 else int(rng.integers(1, 601))
        causal = bool(rng.random() < 0.5)
        key_len = None
        if rng.random() < 0.5:
            key_len = [int(v) for v in rng.integers(0, Lk + 1, size=B)]
            if rng.random() < 0.3:
                key_len[int(rng.integers(B))] = Lk
        scale = float((1.0, 0.5, -1.0, 0.0)[rng.integers(4)]) / math.sqrt(d)
        cases.append(dict(contract=contract, d=d, B=B, H=H, Lq=Lq, Lk=Lk, causal=causal,
                          key_len=key_len, scale=scale, seed=1000 + i))
    return cases


CASES = _draw_cases(N_CASES)


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_case(gpu_lib, i):
    c = CASES[i]
    say("random case %d: %s" % (i, c))
    x = make_inputs(c["B"], c["H"], c["Lq"], c["d"], causal=c["causal"], contract=c["contract"],
                    seed=c["seed"], key_len=c["key_len"], scale=c["scale"], Lk=c["Lk"])
    got = run_gpu(x)
    ref = oracle_reference(x)
    errs = compare(got, ref, c["contract"])
    assert max(errs.values()) <= TOL[c["contract"]], errs
    if c["contract"] == "accelerated":
        from oracle import oracle_forward, round_to_f16
        Or, Lr = oracle_forward(round_to_f16(x.Q), round_to_f16(x.K), round_to_f16(x.V),
                                x.causal, x.scale, key_len=x.key_len)
        e_o, e_l = normwise_error(got["O"], Or), normwise_error(got["LSE"], Lr)
        assert e_o <= TOL_ACCEL_ROUNDED["O"] and e_l <= TOL_ACCEL_ROUNDED["LSE"], (e_o, e_l)
        # the backward against the backward equations at the rounded-input forward
        eb = compare(got, accel_backward_reference(x), "accelerated", names=("dQ", "dK", "dV"))
        assert max(eb.values()) <= TOL_ACCEL_BWD, eb
