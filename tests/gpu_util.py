"""Helpers shared by the GPU tests: move seeded inputs to the device, run the
library through its C ABI, and compare against the oracle."""
import sys

import numpy as np

TOL = {"strict_f32": 1e-4, "fast_bf16": 2e-2,
       # accelerated: f16 forward matrix inputs (unit roundoff u = 2^-11);
       # against the oracle on the unrounded inputs, about 10u
       "accelerated": 5e-3}
# accelerated forward against the oracle on f16-rounded Q, K, V: only the
# f16 rounding of P as the operand of P V remains (about 2u for O), and LSE
# differs by f32 accumulation order only
TOL_ACCEL_ROUNDED = {"O": 1e-3, "LSE": 1e-5}
# accelerated backward against the backward equations evaluated at the
# oracle's rounded-input forward (oracle_backward_from): what is left is the
# f16 rounding of P inside the GPU forward's O (reaching dS through D) and f32
# arithmetic
TOL_ACCEL_BWD = 2e-3


def say(msg):
    """Name the case about to run on the GPU (flushed, so it survives a crash)."""
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(inputs, name):
    import torch
    if inputs.contract == "fast_bf16":
        bits = inputs.bits[name]
        return torch.from_numpy(bits.view(np.int16).copy()).cuda().view(torch.bfloat16)
    return torch.from_numpy(getattr(inputs, name).copy()).cuda()


def key_len_device(inputs):
    import torch
    if inputs.key_len is None:
        return None
    return torch.from_numpy(np.asarray(inputs.key_len, dtype=np.int32).copy()).cuda()


def to_host(t):
    import torch
    return t.detach().float().cpu().numpy().astype(np.float64) if t.dtype != torch.float32 \
        else t.detach().cpu().numpy().astype(np.float64)


def run_gpu(inputs, O_in=None, LSE_in=None):
    """Forward then backward on the GPU.  The backward consumes the GPU's own
    O and LSE unless O_in/LSE_in (host arrays) are given."""
    import torch
    import paper_2608_01563_amd as mg
    Q, K, V, dO = (to_device(inputs, n) for n in ("Q", "K", "V", "dO"))
    kl = key_len_device(inputs)
    O, LSE = mg.attention_forward(Q, K, V, causal=inputs.causal, scale=inputs.scale,
                                  key_len=kl, contract=inputs.contract)
    Ob, LSEb = O, LSE
    if O_in is not None:
        Ob = torch.from_numpy(O_in.astype(np.float32)).cuda().to(Q.dtype).contiguous()
        LSEb = torch.from_numpy(LSE_in.astype(np.float32)).cuda().contiguous()
    dQ, dK, dV = mg.attention_backward(Q, K, V, Ob, LSEb, dO, causal=inputs.causal,
                                       scale=inputs.scale, key_len=kl,
                                       contract=inputs.contract)
    torch.cuda.synchronize()
    return {"O": to_host(O), "LSE": to_host(LSE), "dQ": to_host(dQ), "dK": to_host(dK),
            "dV": to_host(dV)}


def normwise_error(got, ref):
    """max |got - ref| / max |ref| over entries where ref is finite; entries
    where ref is infinite must match exactly."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    fin = np.isfinite(ref)
    if not np.array_equal(got[~fin], ref[~fin]):
        return np.inf
    if not fin.any():
        return 0.0
    den = np.max(np.abs(ref[fin]))
    num = np.max(np.abs(got[fin] - ref[fin])) if np.all(np.isfinite(got[fin])) else np.inf
    return num / den if den > 0 else num


def oracle_reference(inputs, heads=None):
    from oracle import oracle_forward, oracle_backward
    O, LSE = oracle_forward(inputs.Q, inputs.K, inputs.V, inputs.causal, inputs.scale,
                            key_len=inputs.key_len, heads=heads)
    dQ, dK, dV, D = oracle_backward(inputs.Q, inputs.K, inputs.V, inputs.dO, inputs.causal,
                                    inputs.scale, key_len=inputs.key_len, heads=heads)
    return {"O": O, "LSE": LSE, "dQ": dQ, "dK": dK, "dV": dV, "D": D}


def accel_backward_reference(inputs):
    """The accelerated contract's backward from the oracle alone: the strict
    backward equations on the unrounded Q, K, V and dO, evaluated at the O and
    LSE of the oracle's forward on f16-rounded Q, K, V (the saved outputs that
    backward consumes).  Where a row sees a single key the exact gradient is
    zero but this one is the f16 rounding residual of V, which the end-to-end
    comparison cannot follow."""
    from oracle import oracle_forward, oracle_backward_from, round_to_f16
    O, LSE = oracle_forward(round_to_f16(inputs.Q), round_to_f16(inputs.K),
                            round_to_f16(inputs.V), inputs.causal, inputs.scale,
                            key_len=inputs.key_len)
    dQ, dK, dV, _ = oracle_backward_from(inputs.Q, inputs.K, inputs.V, O, LSE, inputs.dO,
                                         inputs.causal, inputs.scale, key_len=inputs.key_len)
    return {"O": O, "LSE": LSE, "dQ": dQ, "dK": dK, "dV": dV}


def compare(got, ref, contract, heads=None, names=("O", "LSE", "dQ", "dK", "dV")):
    """Per-tensor normwise errors (restricted to `heads` if given)."""
    errs = {}
    for n in names:
        g, r = got[n], ref[n]
        if heads is not None:
            g = np.stack([g[b, h] for b, h in heads])
            r = np.stack([r[b, h] for b, h in heads])
        errs[n] = normwise_error(g, r)
    return errs
