"""Host checks of the seeded input generator and the pair counts the
benchmark credits (no GPU, no oracle)."""
import numpy as np
import pytest

from workloads import WORKLOADS, make_inputs, unmasked_pairs, workload_inputs


def brute_pairs(B, H, Lq, Lk, causal, key_len):
    """Count allowed (query, key) pairs from an explicit mask: key j < key
    length and, when causal, j <= i + Lk - Lq (bottom-right alignment)."""
    i = np.arange(Lq)[:, None]
    j = np.arange(Lk)[None, :]
    total = 0
    for b in range(B):
        n = Lk if key_len is None else max(0, min(int(key_len[b]), Lk))
        m = (j < n) & (i >= 0)          # broadcast to [Lq][Lk]
        if causal:
            m = m & (j <= i + (Lk - Lq))
        total += H * int(m.sum())
    return total


@pytest.mark.parametrize("Lq,Lk", [(7, 7), (50, 66), (66, 50), (1024, 77), (3, 1), (1, 9)])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("key_len", [None, [0, 5]])
def test_unmasked_pairs_matches_explicit_mask(Lq, Lk, causal, key_len):
    assert unmasked_pairs(2, 3, Lq, causal, key_len, Lk=Lk) == \
        brute_pairs(2, 3, Lq, Lk, causal, key_len)


def test_cross_inputs_shapes_and_self_attention_draws_unchanged():
    x = make_inputs(2, 3, 5, 32, causal=False, seed=4, Lk=9)
    assert x.Q.shape == x.dO.shape == (2, 3, 5, 32)
    assert x.K.shape == x.V.shape == (2, 3, 9, 32)
    a = make_inputs(2, 3, 5, 32, causal=True, seed=4)
    b = make_inputs(2, 3, 5, 32, causal=True, seed=4, Lk=5)
    for n in ("Q", "K", "V", "dO"):
        assert np.array_equal(getattr(a, n), getattr(b, n))


def test_named_workloads_shapes():
    for wid, w in WORKLOADS.items():
        if w.B * w.H * w.L * w.d > 1 << 24:
            continue   # drawn at full size in the GPU tests and the benchmark
        x = workload_inputs(wid)
        assert x.Q.shape == (w.B, w.H, w.L, w.d)
        assert x.K.shape == (w.B, w.H, w.key_length, w.d)
    assert WORKLOADS[7].key_length == 77 and WORKLOADS[8].L == 1500
