"""Pins of the convolution oracle (CPU only): each check ties the oracle to
something other than itself -- a library routine (scipy's 2-D correlation,
torch's f64 convolution and its autograd), a closed form (pointwise
convolution is a matrix product, a delta filter is a shift, a single output
position gives an outer product), or an identity that relates the three
functions (the adjoint identity, exact central differences of a bilinear
loss).  Layouts: X [N,H,W,C], dY [N,P,Q,K], W [K,R,S,C].
"""
import numpy as np
import pytest

from oracle.conv import (conv_out_size, oracle_conv2d_bwd_data, oracle_conv2d_bwd_data_at,
                         oracle_conv2d_bwd_filter, oracle_conv2d_bwd_filter_at,
                         oracle_conv2d_fwd, oracle_conv2d_fwd_at)

# (N, H, W, C, K, R, S, stride, pad): strides and pads that differ per axis,
# non-square filters, one channel, odd sizes
SHAPES = [
    (2, 7, 6, 3, 4, 3, 3, (1, 1), (1, 1)),
    (2, 9, 8, 2, 3, 3, 2, (2, 1), (1, 0)),
    (1, 11, 10, 3, 2, 7, 7, (2, 2), (3, 3)),
    (3, 5, 5, 1, 1, 1, 1, (1, 1), (0, 0)),
    (2, 8, 9, 4, 5, 1, 1, (2, 2), (0, 0)),
    (1, 6, 7, 2, 3, 2, 3, (1, 2), (0, 2)),
]


def draw(shape, seed):
    N, H, W, C, K, R, S, stride, pad = shape
    P, Q = conv_out_size(H, W, R, S, stride, pad)
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((N, H, W, C))
    Wt = rng.standard_normal((K, R, S, C))
    dY = rng.standard_normal((N, P, Q, K))
    return X, Wt, dY, stride, pad


@pytest.mark.parametrize("shape", SHAPES)
def test_fwd_matches_scipy_correlation(shape):
    """Forward = per (k, c) 2-D correlation of the zero-padded image with the
    filter plane, summed over c and subsampled by the stride."""
    from scipy.signal import correlate2d
    X, Wt, _, (sh, sw), (ph, pw) = draw(shape, 1)
    N, H, W, C = X.shape
    K, R, S, _ = Wt.shape
    Y = oracle_conv2d_fwd(X, Wt, (sh, sw), (ph, pw))
    P, Q = Y.shape[1:3]
    for n in range(N):
        for k in range(K):
            acc = 0.0
            for c in range(C):
                img = np.pad(X[n, :, :, c], ((ph, ph), (pw, pw)))
                acc = acc + correlate2d(img, Wt[k, :, :, c], mode="valid")
            np.testing.assert_allclose(Y[n, :, :, k], acc[::sh, ::sw][:P, :Q], rtol=1e-12,
                                       atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES)
def test_all_three_match_torch_autograd_f64(shape):
    """torch's f64 conv2d (NCHW) and its autograd give Y, dX and dW."""
    import torch
    X, Wt, dY, stride, pad = draw(shape, 2)
    xt = torch.tensor(X.transpose(0, 3, 1, 2), requires_grad=True)
    wt = torch.tensor(Wt.transpose(0, 3, 1, 2), requires_grad=True)
    y = torch.nn.functional.conv2d(xt, wt, stride=stride, padding=pad)
    y.backward(torch.tensor(dY.transpose(0, 3, 1, 2)))
    np.testing.assert_allclose(oracle_conv2d_fwd(X, Wt, stride, pad),
                               y.detach().numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle_conv2d_bwd_data(dY, Wt, X.shape, stride, pad),
                               xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle_conv2d_bwd_filter(X, dY, Wt.shape, stride, pad),
                               wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES)
def test_adjoint_identity(shape):
    """<conv(X, W), dY> = <X, dX(dY, W)> = <W, dW(X, dY)>: the two gradients
    are the adjoints of the forward in each argument."""
    X, Wt, dY, stride, pad = draw(shape, 3)
    lhs = np.sum(oracle_conv2d_fwd(X, Wt, stride, pad) * dY)
    via_x = np.sum(X * oracle_conv2d_bwd_data(dY, Wt, X.shape, stride, pad))
    via_w = np.sum(Wt * oracle_conv2d_bwd_filter(X, dY, Wt.shape, stride, pad))
    assert abs(lhs - via_x) <= 1e-11 * max(1.0, abs(lhs))
    assert abs(lhs - via_w) <= 1e-11 * max(1.0, abs(lhs))


@pytest.mark.parametrize("shape", SHAPES[:3])
def test_central_differences_of_bilinear_loss(shape):
    """The loss <dY, conv(X, W)> is linear in X and in W, so a central
    difference with step 1 recovers each gradient element exactly (up to
    rounding)."""
    X, Wt, dY, stride, pad = draw(shape, 4)
    dX = oracle_conv2d_bwd_data(dY, Wt, X.shape, stride, pad)
    dW = oracle_conv2d_bwd_filter(X, dY, Wt.shape, stride, pad)
    rng = np.random.default_rng(5)

    def loss(x, w):
        return np.sum(oracle_conv2d_fwd(x, w, stride, pad) * dY)

    for _ in range(12):
        i = tuple(rng.integers(0, n) for n in X.shape)
        e = np.zeros_like(X)
        e[i] = 1.0
        fd = (loss(X + e, Wt) - loss(X - e, Wt)) / 2.0
        assert abs(fd - dX[i]) <= 1e-10 * max(1.0, abs(fd))
        j = tuple(rng.integers(0, n) for n in Wt.shape)
        e = np.zeros_like(Wt)
        e[j] = 1.0
        fd = (loss(X, Wt + e) - loss(X, Wt - e)) / 2.0
        assert abs(fd - dW[j]) <= 1e-10 * max(1.0, abs(fd))


def test_pointwise_convolution_is_a_matrix_product():
    """1x1 filters, stride 1, no padding: Y = X W^T, dX = dY W, dW = dY^T X
    over the N*H*W pixel rows."""
    X, Wt, dY, stride, pad = draw((3, 5, 4, 6, 7, 1, 1, (1, 1), (0, 0)), 6)
    Xm, Wm, dYm = X.reshape(-1, 6), Wt.reshape(7, 6), dY.reshape(-1, 7)
    np.testing.assert_allclose(oracle_conv2d_fwd(X, Wt).reshape(-1, 7), Xm @ Wm.T, rtol=1e-12)
    np.testing.assert_allclose(oracle_conv2d_bwd_data(dY, Wt, X.shape).reshape(-1, 6), dYm @ Wm,
                               rtol=1e-12)
    np.testing.assert_allclose(oracle_conv2d_bwd_filter(X, dY, Wt.shape).reshape(7, 6),
                               dYm.T @ Xm, rtol=1e-12)


def test_strided_pointwise_data_gradient_skips_pixels():
    """1x1 filters with stride 2: dX is dY W on the even pixels and exactly 0
    on every pixel no output position reads."""
    X, Wt, dY, stride, pad = draw((2, 7, 6, 3, 4, 1, 1, (2, 2), (0, 0)), 7)
    dX = oracle_conv2d_bwd_data(dY, Wt, X.shape, stride, pad)
    np.testing.assert_allclose(dX[:, ::2, ::2, :], dY @ Wt.reshape(4, 3), rtol=1e-12)
    mask = np.ones(dX.shape, dtype=bool)
    mask[:, ::2, ::2, :] = False
    assert np.all(dX[mask] == 0.0)


def test_delta_filter_is_a_shift():
    """A filter that copies channel c from tap (r0, s0): with stride 1 and
    padding p the output is the input shifted by (r0 - p, s0 - p), zero
    outside; the data gradient shifts dY back the other way."""
    N, H, W, C, R, S, p = 2, 6, 5, 3, 3, 3, 1
    r0, s0 = 2, 0
    Wt = np.zeros((C, R, S, C))
    for c in range(C):
        Wt[c, r0, s0, c] = 1.0
    rng = np.random.default_rng(8)
    X = rng.standard_normal((N, H, W, C))
    Y = oracle_conv2d_fwd(X, Wt, (1, 1), (p, p))
    Xp = np.pad(X, ((0, 0), (p, p), (p, p), (0, 0)))
    np.testing.assert_array_equal(Y, Xp[:, r0:r0 + H, s0:s0 + W, :])
    dY = rng.standard_normal(Y.shape)
    dX = oracle_conv2d_bwd_data(dY, Wt, X.shape, (1, 1), (p, p))
    want = np.zeros_like(X)          # dX[h, w] = dY[h - (r0 - p), w - (s0 - p)]
    for h in range(H):
        for w in range(W):
            hp, wq = h - (r0 - p), w - (s0 - p)
            if 0 <= hp < Y.shape[1] and 0 <= wq < Y.shape[2]:
                want[:, h, w, :] = dY[:, hp, wq, :]
    np.testing.assert_array_equal(dX, want)


def test_single_output_position_gives_an_outer_product():
    """A filter as large as the unpadded input leaves one output position, so
    dW[k, r, s, c] = sum_n dY[n, 0, 0, k] X[n, r, s, c]."""
    X, Wt, dY, stride, pad = draw((3, 4, 5, 2, 3, 4, 5, (1, 1), (0, 0)), 9)
    assert dY.shape == (3, 1, 1, 3)
    dW = oracle_conv2d_bwd_filter(X, dY, Wt.shape)
    np.testing.assert_allclose(dW, np.einsum("nk,nrsc->krsc", dY[:, 0, 0, :], X), rtol=1e-12)


@pytest.mark.parametrize("shape", SHAPES[:3])
def test_sampled_elements_equal_the_full_gradients(shape):
    X, Wt, dY, stride, pad = draw(shape, 10)
    dX = oracle_conv2d_bwd_data(dY, Wt, X.shape, stride, pad)
    dW = oracle_conv2d_bwd_filter(X, dY, Wt.shape, stride, pad)
    rng = np.random.default_rng(11)
    ix = rng.integers(0, dX.size, 40)
    iw = rng.integers(0, dW.size, 40)
    np.testing.assert_array_equal(oracle_conv2d_bwd_data_at(dY, Wt, X.shape, ix, stride, pad),
                                  dX.reshape(-1)[ix])
    Y = oracle_conv2d_fwd(X, Wt, stride, pad)
    iy = rng.integers(0, Y.size, 40)
    np.testing.assert_array_equal(oracle_conv2d_fwd_at(X, Wt, iy, stride, pad), Y.reshape(-1)[iy])
    np.testing.assert_array_equal(oracle_conv2d_bwd_filter_at(X, dY, Wt.shape, iw, stride, pad),
                                  dW.reshape(-1)[iw])


def test_invalid_shapes_are_refused():
    X = np.zeros((1, 2, 2, 1))
    with pytest.raises(ValueError):
        oracle_conv2d_fwd(X, np.zeros((1, 3, 3, 1)))            # no output position
    with pytest.raises(ValueError):
        oracle_conv2d_fwd(X, np.zeros((1, 1, 1, 2)))            # channel mismatch
