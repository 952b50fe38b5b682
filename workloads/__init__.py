"""Seeded synthetic attention workloads shared by the tests, the benchmark and
the smoke check.

This module holds no attention arithmetic: it only draws random tensors,
applies the per-workload value scaling and rounds them to the stored element
type (f32, or bf16 by round-to-nearest-even on the bit pattern).  Both the
oracle and the HIP path consume exactly the values it returns.

The paper times its workloads on synthetic deterministic inputs (Sec. 10) and
runs attention in two arithmetic contracts (Sec. 4.2): strict f32, and a
reduced-input mode with f32 accumulation.  Workloads 1-5 are the attention
shapes this library is measured and parity-tested on; workload 6 is the
headline shape under the paper's own practical default ("accelerated":
f32 tensors, f16 forward matrix inputs, strict backward).  Workloads 7 and 8
take the attention shapes of two of the paper's model workloads (Sec. 10):
the U-Net's cross-attention of 32x32 latent positions onto a 77-token
context, and the Whisper-tiny encoder's non-causal self-attention over 1,500
positions (6 heads of 64), a length that is no multiple of any tile.

Draw recipe (fixed so that every run sees identical values):
  rng = numpy.random.default_rng(seed)
  if padded: key_len = rng.integers(key_len_lo, key_len_hi + 1, size=B)
  Q, K, V, dO = four successive rng.standard_normal draws (f64) of shapes
    (B, H, L, d), (B, H, Lk, d), (B, H, Lk, d), (B, H, L, d); Lk = L unless
    the workload is a cross-attention one
  Q, K, V *= qkv_std;  dO *= do_std
  cast to float32 (round to nearest even); for bf16, round the f32 bits to
  bf16 (round to nearest even).
"""
import math
from dataclasses import dataclass, asdict

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    L: int
    d: int
    causal: bool
    contract: str          # "strict_f32", "fast_bf16" or "accelerated"
    qkv_std: float = 1.0
    do_std: float = 1.0
    padded: bool = False
    key_len_lo: int = 0
    key_len_hi: int = 0
    seed: int = 0
    Lk: int = 0            # key/value length; 0 means L (self-attention)

    @property
    def key_length(self):
        return self.Lk or self.L

    @property
    def scale(self):
        return 1.0 / math.sqrt(self.d)

    def as_dict(self):
        out = asdict(self)
        out["scale"] = self.scale
        return out


WORKLOADS = {
    1: Workload("causal_1x1x64_d32_f32", 1, 1, 64, 32, True, "strict_f32", seed=1),
    2: Workload("causal_4x4x256_d64_f32", 4, 4, 256, 64, True, "strict_f32",
                do_std=0.1, seed=2),
    3: Workload("causal_8x8x1024_d64_f32", 8, 8, 1024, 64, True, "strict_f32",
                qkv_std=0.5, seed=3),
    4: Workload("causal_2x16x4096_d128_bf16", 2, 16, 4096, 128, True, "fast_bf16",
                seed=4),
    5: Workload("padded_16x12x512_d64_f32", 16, 12, 512, 64, False, "strict_f32",
                padded=True, key_len_lo=128, key_len_hi=512, seed=5),
    6: Workload("causal_8x8x1024_d64_accel", 8, 8, 1024, 64, True, "accelerated",
                qkv_std=0.5, seed=6),
    7: Workload("cross_4x8x1024x77_d64_f32", 4, 8, 1024, 64, False, "strict_f32",
                seed=7, Lk=77),
    8: Workload("full_2x6x1500_d64_f32", 2, 6, 1500, 64, False, "strict_f32",
                seed=8),
}


def f32_to_bf16_bits(x):
    """Round float32 values to bfloat16 (nearest even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounding = ((u >> 16) & 1) + 0x7FFF
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits):
    """Widen bfloat16 bit patterns to float32 exactly."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


@dataclass
class AttnInputs:
    """Stored input values.  `Q` etc. are float32 arrays holding the exact
    values (already bf16-representable for the bf16 contract); `bits` holds
    the uint16 bf16 patterns for that contract, else None."""
    Q: np.ndarray
    K: np.ndarray
    V: np.ndarray
    dO: np.ndarray
    key_len: object        # np.ndarray[int32] of shape [B], or None
    contract: str
    causal: bool
    scale: float
    bits: object = None    # dict name -> uint16 array, bf16 contract only


def make_inputs(B, H, L, d, *, causal, contract="strict_f32", seed=0,
                qkv_std=1.0, do_std=1.0, key_len=None, key_len_range=None,
                scale=None, Lk=None):
    """Draw one seeded input set following the recipe in the module doc.

    L is the query length; Lk the key/value length (None: L).
    key_len: explicit per-batch key lengths (sequence of B ints), or
    key_len_range=(lo, hi) to draw them (inclusive) first from the stream.
    """
    if contract not in ("strict_f32", "fast_bf16", "accelerated"):
        raise ValueError("unknown contract %r" % (contract,))
    rng = np.random.default_rng(seed)
    kl = None
    if key_len_range is not None:
        lo, hi = key_len_range
        kl = rng.integers(lo, hi + 1, size=B).astype(np.int32)
    elif key_len is not None:
        kl = np.asarray(key_len, dtype=np.int32).reshape(B)
    Lk = L if Lk is None else int(Lk)
    shapes = [(B, H, L, d), (B, H, Lk, d), (B, H, Lk, d), (B, H, L, d)]
    draws = [rng.standard_normal(shape) for shape in shapes]
    Q, K, V = (x * qkv_std for x in draws[:3])
    dO = draws[3] * do_std
    arrs = [np.ascontiguousarray(x.astype(np.float32)) for x in (Q, K, V, dO)]
    bits = None
    if contract == "fast_bf16":
        bits = {}
        for name, i in zip(("Q", "K", "V", "dO"), range(4)):
            b = f32_to_bf16_bits(arrs[i])
            bits[name] = b
            arrs[i] = bf16_bits_to_f32(b)
    return AttnInputs(*arrs, key_len=kl, contract=contract, causal=bool(causal),
                      scale=(1.0 / math.sqrt(d)) if scale is None else float(scale),
                      bits=bits)


def workload_inputs(wid):
    """Inputs of one of the named workloads."""
    w = WORKLOADS[wid]
    return make_inputs(w.B, w.H, w.L, w.d, causal=w.causal, contract=w.contract,
                       seed=w.seed, qkv_std=w.qkv_std, do_std=w.do_std,
                       key_len_range=(w.key_len_lo, w.key_len_hi) if w.padded else None,
                       Lk=w.key_length)


def unmasked_pairs(B, H, L, causal, key_len=None, Lk=None):
    """Number of (query, key) pairs that attention must evaluate: the unit
    the credited FLOP and byte counts are quoted per.  L queries, Lk keys
    (None: L); the causal mask is aligned to the bottom-right corner."""
    Lk = L if Lk is None else Lk
    total = 0
    for b in range(B):
        n = Lk if key_len is None else max(0, min(int(key_len[b]), Lk))
        if causal:
            # rows i see keys j <= i + Lk - L and j < n
            per_head = sum(max(0, min(i + Lk - L + 1, n)) for i in range(L))
        else:
            per_head = L * n
        total += H * per_head
    return total
