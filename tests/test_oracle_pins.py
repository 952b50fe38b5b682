"""Pins of the CPU oracle against facts fixed by the mathematics of exact
attention, independent of the oracle's own code: closed forms, library
routines (scipy softmax/logsumexp, torch autograd in f64), central finite
differences, brute force with the explicit softmax Jacobian, and invariants.

The paper prints no attention tensors or worked example, so every pin here is
self-made; tests/test_oracle_mutants.py checks that each plausible planted
mistake in the oracle fails at least one of these pins.
"""
import math

import numpy as np
import pytest
import scipy.special

from oracle import oracle_forward, oracle_backward, oracle_backward_from, \
    oracle_head_matrices, round_to_f16

RNG = np.random.default_rng(12345)


def normwise(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.max(np.abs(b))
    num = np.max(np.abs(a - b))
    return num / den if den > 0 else num


def rand(*shape, std=1.0):
    return RNG.standard_normal(shape) * std


def allowed_mask(L, causal, n):
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    m = j < n
    if causal:
        m = m & (j <= i)
    return np.broadcast_to(m, (L, L))


# ---------------------------------------------------------------- forward --

def test_fwd_single_key_returns_value():
    Q, K, V = rand(2, 3, 1, 5), rand(2, 3, 1, 5), rand(2, 3, 1, 5)
    for causal in (False, True):
        O, LSE = oracle_forward(Q, K, V, causal, 0.7)
        assert np.array_equal(O, V)
        assert np.allclose(LSE, 0.7 * np.sum(Q * K, axis=-1), rtol=0, atol=1e-15)


def test_fwd_zero_scale_gives_prefix_means():
    B, H, L, d = 2, 2, 9, 3
    Q, K, V = rand(B, H, L, d), rand(B, H, L, d), rand(B, H, L, d)
    # causal: row i averages V_0..V_i
    O, LSE = oracle_forward(Q, K, V, True, 0.0)
    counts = np.arange(1, L + 1)
    expect = np.cumsum(V, axis=2) / counts[None, None, :, None]
    assert normwise(O, expect) < 1e-14
    assert np.allclose(LSE, np.log(counts)[None, None, :], rtol=0, atol=1e-14)
    # padded, non-causal: every row averages the first n keys
    kl = np.array([4, 9], dtype=np.int32)
    O, LSE = oracle_forward(Q, K, V, False, 0.0, key_len=kl)
    for b in range(B):
        n = kl[b]
        mean = V[b, :, :n, :].mean(axis=1, keepdims=True)
        assert normwise(O[b], np.broadcast_to(mean, O[b].shape)) < 1e-14
        assert np.allclose(LSE[b], math.log(n), rtol=0, atol=1e-14)


def test_fwd_two_keys_is_logistic():
    # Two keys: P_i0 = 1 / (1 + exp(s_i1 - s_i0)); LSE = log(e^s0 + e^s1)
    B, H, L, d = 1, 1, 2, 1
    Q, K, V = rand(B, H, L, d), rand(B, H, L, d), rand(B, H, L, d)
    scale = 1.3
    O, LSE = oracle_forward(Q, K, V, False, scale)
    for i in range(2):
        s0 = scale * Q[0, 0, i, 0] * K[0, 0, 0, 0]
        s1 = scale * Q[0, 0, i, 0] * K[0, 0, 1, 0]
        p0 = 1.0 / (1.0 + math.exp(s1 - s0))
        assert abs(O[0, 0, i, 0] - (p0 * V[0, 0, 0, 0] + (1 - p0) * V[0, 0, 1, 0])) < 1e-15
        hi, lo = max(s0, s1), min(s0, s1)
        assert abs(LSE[0, 0, i] - (hi + math.log1p(math.exp(lo - hi)))) < 1e-15
    # causal: row 0 sees only key 0
    O, LSE = oracle_forward(Q, K, V, True, scale)
    assert O[0, 0, 0, 0] == V[0, 0, 0, 0]
    assert abs(LSE[0, 0, 0] - scale * Q[0, 0, 0, 0] * K[0, 0, 0, 0]) < 1e-15


def test_fwd_large_scale_is_hard_argmax():
    B, H, L, d = 1, 2, 12, 4
    Q, K, V = rand(B, H, L, d), rand(B, H, L, d), rand(B, H, L, d)
    S = np.einsum("bhid,bhjd->bhij", Q, K)
    srt = np.sort(S, axis=-1)
    scale = 80.0 / np.min(srt[..., -1] - srt[..., -2])   # winners clear by e^-80
    O, _ = oracle_forward(Q, K, V, False, scale)
    idx = np.argmax(S, axis=-1)
    expect = np.take_along_axis(V, idx[..., None], axis=2)
    assert normwise(O, expect) < 1e-12


def test_fwd_causal_first_row_is_first_value():
    Q, K, V = rand(2, 2, 7, 8), rand(2, 2, 7, 8), rand(2, 2, 7, 8)
    O, LSE = oracle_forward(Q, K, V, True, 0.35)
    assert np.array_equal(O[:, :, 0, :], V[:, :, 0, :])
    assert np.allclose(LSE[:, :, 0], 0.35 * np.sum(Q[:, :, 0] * K[:, :, 0], -1),
                       rtol=0, atol=1e-15)


@pytest.mark.parametrize("causal,padded", [(False, False), (True, False), (False, True),
                                           (True, True)])
def test_fwd_matches_scipy_softmax(causal, padded):
    B, H, L, d = 3, 2, 23, 6
    Q, K, V = rand(B, H, L, d), rand(B, H, L, d), rand(B, H, L, d)
    kl = np.array([23, 1, 11], dtype=np.int32) if padded else None
    scale = 1 / math.sqrt(d)
    O, LSE = oracle_forward(Q, K, V, causal, scale, key_len=kl)
    for b in range(B):
        n = L if kl is None else kl[b]
        m = allowed_mask(L, causal, n)
        S = scale * np.matmul(Q[b], np.swapaxes(K[b], -1, -2))
        S = np.where(m, S, -np.inf)
        P = scipy.special.softmax(S, axis=-1)
        assert normwise(O[b], np.matmul(P, V[b])) < 1e-13
        assert normwise(LSE[b], scipy.special.logsumexp(S, axis=-1)) < 1e-14


def test_fwd_row_shift_invariance():
    # A constant added to every score of a row leaves O unchanged and shifts
    # LSE by that constant.  K has a last column of ones, so adding a to the
    # last element of Q_i adds scale*a to every S_ij.
    B, H, L, d = 1, 1, 10, 5
    Q, K, V = rand(B, H, L, d), rand(B, H, L, d), rand(B, H, L, d)
    K[..., -1] = 1.0
    scale = 0.8
    O1, L1 = oracle_forward(Q, K, V, True, scale)
    shift = rand(L)
    Q2 = Q.copy()
    Q2[0, 0, :, -1] += shift
    O2, L2 = oracle_forward(Q2, K, V, True, scale)
    assert normwise(O2, O1) < 1e-14
    assert np.allclose(L2[0, 0] - L1[0, 0], scale * shift, rtol=0, atol=1e-13)


def test_fwd_key_permutation_and_value_linearity():
    B, H, L, d = 2, 2, 13, 4
    Q, K, V = rand(B, H, L, d), rand(B, H, L, d), rand(B, H, L, d)
    perm = RNG.permutation(L)
    O1, L1 = oracle_forward(Q, K, V, False, 0.6)
    O2, L2 = oracle_forward(Q, K[:, :, perm], V[:, :, perm], False, 0.6)
    assert normwise(O2, O1) < 1e-14 and normwise(L2, L1) < 1e-14
    qp = RNG.permutation(L)
    O3, _ = oracle_forward(Q[:, :, qp], K, V, False, 0.6)
    assert normwise(O3, O1[:, :, qp]) < 1e-14
    V2 = rand(B, H, L, d)
    Oa, _ = oracle_forward(Q, K, V + 2.5 * V2, True, 0.6)
    Ob, _ = oracle_forward(Q, K, V, True, 0.6)
    Oc, _ = oracle_forward(Q, K, V2, True, 0.6)
    assert normwise(Oa, Ob + 2.5 * Oc) < 1e-13


def test_fwd_invariants_from_matrices():
    B, H, L, d = 2, 2, 17, 4
    Q, K, V, dO = (rand(B, H, L, d) for _ in range(4))
    kl = np.array([17, 6], dtype=np.int32)
    scale = 0.9
    for causal in (False, True):
        _, LSE = oracle_forward(Q, K, V, causal, scale, key_len=kl)
        for b in range(B):
            for h in range(H):
                P, dS, Dalt = oracle_head_matrices(Q, K, V, dO, causal, scale, b, h, key_len=kl)
                m = allowed_mask(L, causal, kl[b])
                assert np.all(P[~m] == 0.0) and np.all(dS[~m] == 0.0)
                assert np.max(np.abs(P.sum(axis=1) - 1.0)) < 1e-14
                assert np.all(P >= 0)
                S = scale * Q[b, h] @ K[b, h].T
                S = np.where(m, S, -np.inf)
                smax = S.max(axis=1)
                nall = m.sum(axis=1)
                assert np.all(LSE[b, h] >= smax - 1e-14)
                assert np.all(LSE[b, h] <= smax + np.log(nall) + 1e-14)


def test_fwd_fully_masked_rows():
    B, H, L, d = 2, 1, 6, 3
    Q, K, V = rand(B, H, L, d), rand(B, H, L, d), rand(B, H, L, d)
    kl = np.array([0, 6], dtype=np.int32)
    for causal in (False, True):
        O, LSE = oracle_forward(Q, K, V, causal, 0.5, key_len=kl)
        assert np.all(O[0] == 0.0)
        assert np.all(LSE[0] == -np.inf)
        assert np.all(np.isfinite(O[1])) and np.all(np.isfinite(LSE[1]))


def test_fwd_head_selection_leaves_others_untouched():
    Q, K, V = rand(2, 3, 5, 4), rand(2, 3, 5, 4), rand(2, 3, 5, 4)
    O, LSE = oracle_forward(Q, K, V, True, 0.5, heads=[(1, 2)])
    Ofull, _ = oracle_forward(Q, K, V, True, 0.5)
    assert np.array_equal(O[1, 2], Ofull[1, 2])
    assert np.all(np.isnan(O[0])) and np.all(np.isnan(LSE[1, :2]))


# --------------------------------------------------------------- backward --

def _loss(Q, K, V, dO, causal, scale, kl):
    O, _ = oracle_forward(Q, K, V, causal, scale, key_len=kl)
    return float(np.sum(dO * O))


FD_CASES = [(L, d, causal, padded)
            for L in (1, 2, 3, 5, 8) for d in (1, 2, 4)
            for causal, padded in ((False, False), (True, False), (False, True))]


@pytest.mark.parametrize("L,d,causal,padded", FD_CASES)
def test_bwd_central_finite_differences(L, d, causal, padded):
    B, H = 1, 2
    Q, K, V, dO = (rand(B, H, L, d) for _ in range(4))
    kl = np.array([max(1, (L + 1) // 2)], dtype=np.int32) if padded else None
    scale = 0.77
    dQ, dK, dV, _ = oracle_backward(Q, K, V, dO, causal, scale, key_len=kl)
    h = 1e-5
    for X, G in ((Q, dQ), (K, dK), (V, dV)):
        num = np.zeros_like(X)
        it = np.nditer(X, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            old = X[idx]
            X[idx] = old + h
            fp = _loss(Q, K, V, dO, causal, scale, kl)
            X[idx] = old - h
            fm = _loss(Q, K, V, dO, causal, scale, kl)
            X[idx] = old
            num[idx] = (fp - fm) / (2 * h)
        assert np.max(np.abs(num - G)) <= 1e-7 * max(1.0, np.max(np.abs(G)))


def _torch_reference(Q, K, V, dO, causal, scale, kl):
    """Unfused f64 attention by torch autograd; Q [B,H,Lq,d], K, V [B,H,Lk,d],
    causal mask bottom-right aligned (the usual lower triangle when Lq == Lk)."""
    import torch
    B, H, Lq, d = Q.shape
    Lk = K.shape[2]
    q, k, v = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (Q, K, V))
    S = scale * torch.matmul(q, k.transpose(-1, -2))
    mask = torch.ones(B, 1, Lq, Lk, dtype=torch.bool)
    if causal:
        mask &= torch.ones(Lq, Lk, dtype=torch.bool).tril(diagonal=Lk - Lq)
    if kl is not None:
        for b in range(B):
            mask[b, :, :, int(kl[b]):] = False
    S = S.masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(S, dim=-1)
    O = torch.matmul(torch.softmax(S, dim=-1), v)
    O.backward(torch.tensor(dO, dtype=torch.float64))
    return (O.detach().numpy(), lse.detach().numpy(),
            q.grad.numpy(), k.grad.numpy(), v.grad.numpy())


@pytest.mark.parametrize("causal,padded,L,d", [(True, False, 37, 8), (False, False, 20, 16),
                                               (False, True, 33, 8), (True, True, 16, 4)])
def test_fwd_bwd_match_torch_autograd_f64(causal, padded, L, d):
    B, H = 2, 3
    Q, K, V, dO = (rand(B, H, L, d) for _ in range(4))
    kl = np.array([L, max(1, L // 3)], dtype=np.int32) if padded else None
    scale = 1 / math.sqrt(d)
    O, LSE = oracle_forward(Q, K, V, causal, scale, key_len=kl)
    dQ, dK, dV, _ = oracle_backward(Q, K, V, dO, causal, scale, key_len=kl)
    tO, tL, tdQ, tdK, tdV = _torch_reference(Q, K, V, dO, causal, scale, kl)
    assert normwise(O, tO) < 1e-13
    assert normwise(LSE, tL) < 1e-13
    assert normwise(dQ, tdQ) < 1e-12
    assert normwise(dK, tdK) < 1e-12
    assert normwise(dV, tdV) < 1e-12


def test_bwd_explicit_softmax_jacobian():
    B, H, L, d = 2, 2, 19, 5
    Q, K, V, dO = (rand(B, H, L, d) for _ in range(4))
    kl = np.array([19, 7], dtype=np.int32)
    scale = 0.45
    for causal in (False, True):
        dQ, dK, dV, _ = oracle_backward(Q, K, V, dO, causal, scale, key_len=kl)
        for b in range(B):
            m = allowed_mask(L, causal, kl[b])
            for h in range(H):
                S = np.where(m, scale * Q[b, h] @ K[b, h].T, -np.inf)
                P = scipy.special.softmax(S, axis=-1)
                dP = dO[b, h] @ V[b, h].T
                dS = np.stack([(np.diag(P[i]) - np.outer(P[i], P[i])) @ dP[i]
                               for i in range(L)])
                assert normwise(dQ[b, h], scale * dS @ K[b, h]) < 1e-12
                assert normwise(dK[b, h], scale * dS.T @ Q[b, h]) < 1e-12
                assert normwise(dV[b, h], P.T @ dO[b, h]) < 1e-12


def test_bwd_invariants():
    B, H, L, d = 2, 2, 21, 6
    Q, K, V, dO = (rand(B, H, L, d) for _ in range(4))
    kl = np.array([21, 9], dtype=np.int32)
    scale = 0.6
    for causal in (False, True):
        dQ, dK, dV, D = oracle_backward(Q, K, V, dO, causal, scale, key_len=kl)
        # a common shift of every key changes each score row by a constant
        assert np.max(np.abs(dK.sum(axis=2))) < 1e-12 * max(1, np.max(np.abs(dK)))
        # every row's probabilities sum to one
        assert normwise(dV.sum(axis=2), dO.sum(axis=2)) < 1e-12
        # padded keys get exactly zero gradient
        assert np.all(dK[1, :, 9:] == 0.0) and np.all(dV[1, :, 9:] == 0.0)
        for b in range(B):
            for h in range(H):
                P, dS, Dalt = oracle_head_matrices(Q, K, V, dO, causal, scale, b, h,
                                                   key_len=kl)
                assert np.max(np.abs(dS.sum(axis=1))) < 1e-13 * max(1, np.abs(dS).max())
                assert normwise(D[b, h], Dalt) < 1e-13


def test_bwd_single_key_special_case():
    Q, K, V, dO = (rand(2, 2, 1, 4) for _ in range(4))
    dQ, dK, dV, _ = oracle_backward(Q, K, V, dO, True, 0.5)
    assert np.array_equal(dV, dO)
    assert np.max(np.abs(dQ)) < 1e-15 and np.max(np.abs(dK)) < 1e-15


def test_bwd_linear_in_upstream_gradient_and_masked_batch():
    B, H, L, d = 2, 2, 11, 4
    Q, K, V, dO = (rand(B, H, L, d) for _ in range(4))
    kl = np.array([0, 11], dtype=np.int32)
    g1 = oracle_backward(Q, K, V, dO, True, 0.5, key_len=kl)
    g2 = oracle_backward(Q, K, V, 2 * dO, True, 0.5, key_len=kl)
    for a, b in zip(g1[:3], g2[:3]):
        assert np.array_equal(2 * a, b)
    for g in g1[:3]:
        assert np.all(g[0] == 0.0)


# ---- the backward equations at given saved outputs (a recompute-based
# backward consuming another forward's O and LSE: the accelerated contract's
# f32 backward after its rounded-input forward)

@pytest.mark.parametrize("causal,padded,Lq,Lk", [(True, False, 6, 6), (False, True, 5, 7),
                                                 (True, True, 7, 4)])
def test_bwd_from_exact_forward_is_the_backward(causal, padded, Lq, Lk):
    """At the forward's own O and LSE it is the pinned backward."""
    Q, dO = rand(2, 2, Lq, 3), rand(2, 2, Lq, 3)
    K, V = rand(2, 2, Lk, 3), rand(2, 2, Lk, 3)
    kl = np.array([Lk - 1, 2], dtype=np.int32) if padded else None
    O, LSE = oracle_forward(Q, K, V, causal, 0.6, key_len=kl)
    for a, b in zip(oracle_backward(Q, K, V, dO, causal, 0.6, key_len=kl),
                    oracle_backward_from(Q, K, V, O, LSE, dO, causal, 0.6, key_len=kl)):
        assert np.array_equal(a, b)


def test_bwd_from_single_key_closed_forms():
    """Every row sees key 0 only (key length 1), so P_i = exp(S_i0 - LSE_i).
    Given LSE_i = S_i0 + ln 2, P = 1/2: dV_0 = (1/2) sum_i dO_i.  Given O_i =
    V_0, D_i = dP_i and every dS vanishes: dQ = dK = 0.  Given O_i = V_0 +
    t u_i, dS_i = -(t/2) dO_i . u_i, dQ_i = scale dS_i K_0, dK_0 = scale sum_i
    dS_i Q_i.  Keys past the key length get nothing."""
    L, d, scale, t = 5, 3, 0.7, 0.3
    Q, K, V, dO = (rand(1, 1, L, d) for _ in range(4))
    kl = np.array([1], dtype=np.int32)
    S0 = scale * np.einsum("id,d->i", Q[0, 0], K[0, 0, 0])
    LSE = (S0 + math.log(2.0))[None, None]
    O = np.broadcast_to(V[0, 0, 0], (1, 1, L, d)).copy()
    dQ, dK, dV, D = oracle_backward_from(Q, K, V, O, LSE, dO, False, scale, key_len=kl)
    assert np.all(dQ == 0.0) and np.all(dK == 0.0)
    assert np.allclose(dV[0, 0, 0], 0.5 * dO[0, 0].sum(axis=0), rtol=1e-14, atol=1e-15)
    assert np.all(dV[0, 0, 1:] == 0.0)
    u = rand(1, 1, L, d)
    dQ, dK, dV, D = oracle_backward_from(Q, K, V, O + t * u, LSE, dO, False, scale, key_len=kl)
    dS = -(t / 2) * np.einsum("id,id->i", dO[0, 0], u[0, 0])
    assert normwise(dQ[0, 0], scale * dS[:, None] * K[0, 0, 0][None]) < 1e-13
    assert normwise(dK[0, 0, 0], scale * (dS[:, None] * Q[0, 0]).sum(axis=0)) < 1e-13
    assert np.all(dK[0, 0, 1:] == 0.0)


def test_bwd_from_linear_in_upstream_gradient():
    """With O and LSE fixed (here unrelated to Q, K, V), D and all three
    gradients are linear in dO."""
    Q, dO1, dO2 = rand(2, 1, 6, 4), rand(2, 1, 6, 4), rand(2, 1, 6, 4)
    K, V, O = rand(2, 1, 6, 4), rand(2, 1, 6, 4), rand(2, 1, 6, 4)
    LSE = rand(2, 1, 6) + 2.0
    g1 = oracle_backward_from(Q, K, V, O, LSE, dO1, True, 0.5)
    g2 = oracle_backward_from(Q, K, V, O, LSE, dO2, True, 0.5)
    g = oracle_backward_from(Q, K, V, O, LSE, 2.0 * dO1 - 3.0 * dO2, True, 0.5)
    for a, b, c in zip(g1, g2, g):
        assert normwise(c, 2.0 * a - 3.0 * b) < 1e-13


# ---- f16 input rounding of the accelerated contract (Sec. 4.2 permissions)

def test_round_to_f16_closed_forms():
    """IEEE binary16: 10 fraction bits, ties to even, max finite 65504,
    smallest subnormal 2^-24."""
    cases = [
        (1.0 + 2.0 ** -11, 1.0),                  # halfway, ties to the even 1.0
        (1.0 + 3 * 2.0 ** -11, 1.0 + 2.0 ** -9),  # halfway, ties to the even neighbour
        (1.0 + 2.0 ** -10, 1.0 + 2.0 ** -10),     # representable
        (-2049.0, -2048.0),                       # spacing 2 above 2048, tie to even
        (65504.0, 65504.0),                       # largest finite
        (65519.0, 65504.0),                       # below the overflow midpoint
        (65520.0, math.inf),                      # overflow midpoint rounds to inf
        (2.0 ** -24, 2.0 ** -24),                 # smallest subnormal
        (2.0 ** -25, 0.0),                        # half of it ties to zero
        (3 * 2.0 ** -25, 2.0 ** -23),             # 1.5 subnormal steps -> 2 (even)
        (1.0 / 3.0, 1365.0 / 4096.0),             # 0.0101010101|01... -> 1365/4096
    ]
    got = round_to_f16(np.array([c[0] for c in cases]))
    assert np.array_equal(got, np.array([c[1] for c in cases]))


def test_round_to_f16_error_bound_and_identity():
    rng = np.random.default_rng(11)
    x = rng.standard_normal(100000) * np.exp(rng.uniform(-8, 8, 100000))
    r = round_to_f16(x)
    normal = np.abs(x) >= 2.0 ** -14
    # relative error at most half an ulp: 2^-11 for normal numbers
    assert np.all(np.abs(r[normal] - x[normal]) <= 2.0 ** -11 * np.abs(x[normal]))
    # values already in binary16 are fixed points; rounding is idempotent
    assert np.array_equal(round_to_f16(r), r)
    ints = np.arange(-2048, 2049, dtype=np.float64)
    assert np.array_equal(round_to_f16(ints), ints)


def test_round_to_f16_inputs_change_attention_only_through_rounding():
    """The oracle on f16-rounded inputs equals the oracle on inputs that were
    f16-representable to begin with, and differs from the unrounded result by
    about the rounding size."""
    B, H, L, d = 1, 2, 9, 8
    Q, K, V = (round_to_f16(rand(B, H, L, d)) for _ in range(3))
    O1, L1 = oracle_forward(round_to_f16(Q), round_to_f16(K), round_to_f16(V), True, 0.5)
    O0, L0 = oracle_forward(Q, K, V, True, 0.5)
    assert np.array_equal(O1, O0) and np.array_equal(L1, L0)
    Qf, Kf, Vf = (rand(B, H, L, d) for _ in range(3))
    Or, _ = oracle_forward(round_to_f16(Qf), round_to_f16(Kf), round_to_f16(Vf), True, 0.5)
    Oe, _ = oracle_forward(Qf, Kf, Vf, True, 0.5)
    err = normwise(Or, Oe)
    assert 1e-6 < err < 2e-2


# ---- cross-attention: Lq != Lk, causal mask bottom-right aligned

CROSS_FD_CASES = [(Lq, Lk, causal, padded) for (Lq, Lk) in ((3, 5), (5, 2), (4, 7))
                  for causal, padded in ((True, False), (False, False), (False, True))]


def _loss_cross(Q, K, V, dO, causal, scale, kl):
    O, _ = oracle_forward(Q, K, V, causal, scale, key_len=kl)
    return float(np.sum(O * dO))


@pytest.mark.parametrize("Lq,Lk,causal,padded", CROSS_FD_CASES)
def test_cross_central_finite_differences(Lq, Lk, causal, padded):
    B, H, d = 1, 2, 3
    Q, dO = rand(B, H, Lq, d), rand(B, H, Lq, d)
    K, V = rand(B, H, Lk, d), rand(B, H, Lk, d)
    kl = np.array([max(1, (Lk + 1) // 2)], dtype=np.int32) if padded else None
    scale = 0.77
    dQ, dK, dV, _ = oracle_backward(Q, K, V, dO, causal, scale, key_len=kl)
    assert dQ.shape == Q.shape and dK.shape == K.shape and dV.shape == V.shape
    h = 1e-5
    for X, G in ((Q, dQ), (K, dK), (V, dV)):
        num = np.zeros_like(X)
        it = np.nditer(X, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            old = X[idx]
            X[idx] = old + h
            fp = _loss_cross(Q, K, V, dO, causal, scale, kl)
            X[idx] = old - h
            fm = _loss_cross(Q, K, V, dO, causal, scale, kl)
            X[idx] = old
            num[idx] = (fp - fm) / (2 * h)
        assert np.max(np.abs(num - G)) <= 1e-7 * max(1.0, np.max(np.abs(G)))


@pytest.mark.parametrize("Lq,Lk,causal,padded", [(9, 23, True, False), (17, 6, False, False),
                                                 (12, 30, False, True), (20, 20, True, False)])
def test_cross_matches_torch_autograd_f64(Lq, Lk, causal, padded):
    B, H, d = 2, 2, 8
    Q, dO = rand(B, H, Lq, d), rand(B, H, Lq, d)
    K, V = rand(B, H, Lk, d), rand(B, H, Lk, d)
    kl = np.array([Lk, max(1, Lk // 3)], dtype=np.int32) if padded else None
    scale = 1 / math.sqrt(d)
    O, LSE = oracle_forward(Q, K, V, causal, scale, key_len=kl)
    dQ, dK, dV, _ = oracle_backward(Q, K, V, dO, causal, scale, key_len=kl)
    tO, tL, tdQ, tdK, tdV = _torch_reference(Q, K, V, dO, causal, scale, kl)
    assert normwise(O, tO) < 1e-13 and normwise(LSE, tL) < 1e-13
    assert normwise(dQ, tdQ) < 1e-12 and normwise(dK, tdK) < 1e-12
    assert normwise(dV, tdV) < 1e-12


def test_cross_causal_is_the_bottom_rows_of_square_causal():
    """Bottom-right alignment: with Lq < Lk, causal cross-attention of the
    last Lq queries equals those rows of square causal attention over all Lk
    (and, with dO zero on the other rows, the same dK and dV); with Lq > Lk,
    the first Lq - Lk rows see no key and the rest are square causal
    attention of the last Lk queries."""
    B, H, d, Lk, Lq = 2, 2, 5, 13, 6
    Qall, dOall = rand(B, H, Lk, d), rand(B, H, Lk, d)
    K, V = rand(B, H, Lk, d), rand(B, H, Lk, d)
    dOall[:, :, :Lk - Lq] = 0.0
    Osq, Lsq = oracle_forward(Qall, K, V, True, 0.4)
    gsq = oracle_backward(Qall, K, V, dOall, True, 0.4)
    Q, dO = Qall[:, :, Lk - Lq:].copy(), dOall[:, :, Lk - Lq:].copy()
    O, LSE = oracle_forward(Q, K, V, True, 0.4)
    g = oracle_backward(Q, K, V, dO, True, 0.4)
    assert np.array_equal(O, Osq[:, :, Lk - Lq:]) and np.array_equal(LSE, Lsq[:, :, Lk - Lq:])
    assert np.array_equal(g[0], gsq[0][:, :, Lk - Lq:])
    assert np.array_equal(g[1], gsq[1]) and np.array_equal(g[2], gsq[2])
    # Lq > Lk: queries longer than keys
    Lq2, Lk2 = 11, 4
    Q2, K2, V2 = rand(B, H, Lq2, d), rand(B, H, Lk2, d), rand(B, H, Lk2, d)
    O2, L2 = oracle_forward(Q2, K2, V2, True, 0.4)
    assert np.all(O2[:, :, :Lq2 - Lk2] == 0.0) and np.all(L2[:, :, :Lq2 - Lk2] == -np.inf)
    O3, L3 = oracle_forward(Q2[:, :, Lq2 - Lk2:].copy(), K2, V2, True, 0.4)
    assert np.array_equal(O2[:, :, Lq2 - Lk2:], O3) and np.array_equal(L2[:, :, Lq2 - Lk2:], L3)


def test_cross_single_key():
    B, H, d = 1, 2, 4
    Q, K, V = rand(B, H, 5, d), rand(B, H, 1, d), rand(B, H, 1, d)
    O, LSE = oracle_forward(Q, K, V, False, 0.3)
    assert np.array_equal(O, np.broadcast_to(V, O.shape))
    assert normwise(LSE, 0.3 * np.einsum("bhid,bhjd->bhi", Q, K)) < 1e-15
    O, LSE = oracle_forward(Q, K, V, True, 0.3)   # only the last row sees the key
    assert np.all(O[:, :, :4] == 0.0) and np.all(LSE[:, :, :4] == -np.inf)
    assert np.array_equal(O[:, :, 4], V[:, :, 0])
