"""Canary guards: every tensor the library reads or writes (inputs, outputs,
LSE, key lengths and the backward workspace) is a view into a larger buffer
whose guard regions before and after it hold a known value.  After the
forward and the backward every guard must be unchanged, so no kernel wrote
out of bounds, including the tail tiles of ragged lengths, the 128-key fused
backward, the split fused backward of short key sides and the separate dQ
kernels.  Inputs are also checked for being untouched."""
import numpy as np
import pytest

from gpu_util import say
from workloads import make_inputs

pytestmark = pytest.mark.gpu

GUARD = 4096          # guard elements on each side (a multiple of 16 bytes for every dtype)

CASES = [
    # contract, B, H, Lq, Lk, d, mode
    ("strict_f32", 2, 3, 65, 65, 32, "causal"),
    ("strict_f32", 2, 3, 65, 65, 64, "padded"),
    ("strict_f32", 2, 3, 200, 200, 128, "causal"),      # separate dQ kernel (d = 128)
    ("strict_f32", 2, 3, 17, 17, 64, "full"),
    ("strict_f32", 4, 16, 1000, 1000, 64, "causal"),    # 128-key fused backward, serpentine
    ("strict_f32", 1, 4, 1024, 77, 64, "full"),         # split fused backward (few key tiles)
    ("strict_f32", 1, 4, 300, 260, 32, "causal"),       # cross-attention, bottom-right causal
    ("fast_bf16", 2, 3, 200, 200, 128, "causal"),
    ("fast_bf16", 2, 3, 65, 65, 64, "padded"),
    ("accelerated", 2, 3, 200, 200, 64, "causal"),
]


class Guarded:
    """A tensor view with `GUARD` canary elements on each side."""

    def __init__(self, shape, dtype, fill):
        import torch
        n = int(np.prod(shape))
        self.n, self.fill = n, fill
        self.buf = torch.full((n + 2 * GUARD,), fill, dtype=dtype, device="cuda")
        self.view = self.buf[GUARD:GUARD + n].view(shape)

    def guards_intact(self):
        import torch
        head, tail = self.buf[:GUARD], self.buf[GUARD + self.n:]
        return bool(torch.all(head == self.fill)) and bool(torch.all(tail == self.fill))


@pytest.mark.parametrize("contract,B,H,Lq,Lk,d,mode", CASES)
def test_no_write_outside_any_buffer(gpu_lib, contract, B, H, Lq, Lk, d, mode):
    import torch
    import paper_2608_01563_amd as mg
    say("canary %s B%d H%d Lq%d Lk%d d%d %s" % (contract, B, H, Lq, Lk, d, mode))
    causal = mode == "causal"
    kl = None
    if mode == "padded":
        kl = [max(1, Lk // 3), Lk][:B] + [Lk] * max(0, B - 2)
    x = make_inputs(B, H, Lq, d, causal=causal, contract=contract, seed=300 + Lq + d,
                    key_len=kl, Lk=Lk)
    dt = torch.bfloat16 if contract == "fast_bf16" else torch.float32
    fill = 1234.5 if dt == torch.float32 else 1232.0   # exact in bf16
    qs, ks = (B, H, Lq, d), (B, H, Lk, d)
    t = {n: Guarded(s, dt, fill) for n, s in (("Q", qs), ("K", ks), ("V", ks), ("dO", qs),
                                            ("O", qs), ("dQ", qs), ("dK", ks), ("dV", ks))}
    t["LSE"] = Guarded((B, H, Lq), torch.float32, 1234.5)
    for n in ("Q", "K", "V", "dO"):
        src = (torch.from_numpy(x.bits[n].view(np.int16).copy()).view(torch.bfloat16)
               if contract == "fast_bf16" else torch.from_numpy(getattr(x, n).copy()))
        t[n].view.copy_(src.cuda())
    inputs_before = {n: t[n].view.clone() for n in ("Q", "K", "V", "dO")}
    key_len = None
    if kl is not None:
        t["key_len"] = Guarded((B,), torch.int32, -7)
        t["key_len"].view.copy_(torch.tensor(kl, dtype=torch.int32).cuda())
        key_len = t["key_len"].view
    need = mg.mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, causal, contract)
    t["workspace"] = Guarded((max(need, 16),), torch.uint8, 0xA5)

    mg.mg_attn_fwd_cross(t["Q"].view, t["K"].view, t["V"].view, t["O"].view, t["LSE"].view,
                         key_len, causal=causal, scale=x.scale, contract=contract)
    mg.mg_attn_bwd_cross(t["Q"].view, t["K"].view, t["V"].view, t["O"].view, t["LSE"].view,
                         t["dO"].view, t["dQ"].view, t["dK"].view, t["dV"].view, key_len,
                         causal=causal, scale=x.scale, contract=contract,
                         workspace=t["workspace"].view)
    torch.cuda.synchronize()
    for name, g in t.items():
        assert g.guards_intact(), "guard of %s overwritten" % name
    for n, before in inputs_before.items():
        assert torch.equal(t[n].view, before), "input %s modified" % n
    for n in ("O", "dQ", "dK", "dV"):
        assert bool(torch.all(torch.isfinite(t[n].view.float()))), n
