"""GPU parity of the convolution derivatives (through the C ABI) against the
f64 convolution oracle on the same seeded inputs.

Tolerance: normwise, max|gpu - oracle| / max|oracle| <= 1e-4 per output
tensor.  Both derivatives are f32 sums of products with f32 accumulation; a
sum of n products of unit-scale values carries a rounding error of about
sqrt(n) * 2^-24 relative to its typical size (n up to 50176 here, about
1.3e-5), and the normwise metric divides by the largest output, so 1e-4
leaves a margin of several times over the measured errors.

Small shapes are compared element by element; the ResNet-50 layer shapes
(batch 4, 224x224) are run at full size and compared on sampled outputs that
the oracle computes one by one.
"""
import numpy as np
import pytest

from gpu_util import normwise_error, say
from workloads.conv import layer_inputs, make_conv_inputs, resnet50_layers

pytestmark = pytest.mark.gpu

TOL = 1e-4

# (N, H, W, C, K, R, S, stride, pad): odd sizes, channel counts off every
# vector width, per-axis strides and pads, filters larger than the tile of a
# dimension, single pixels and single channels
SMALL = [
    (2, 9, 7, 3, 5, 3, 3, (1, 1), (1, 1)),
    (1, 13, 11, 3, 64, 7, 7, (2, 2), (3, 3)),
    (2, 8, 8, 16, 24, 1, 1, (1, 1), (0, 0)),
    (2, 9, 9, 16, 20, 1, 1, (2, 2), (0, 0)),
    (1, 10, 12, 8, 12, 3, 3, (2, 2), (1, 1)),
    (3, 5, 6, 68, 70, 3, 3, (1, 1), (1, 1)),
    (1, 7, 9, 5, 7, 3, 2, (2, 1), (1, 0)),
    (2, 1, 1, 4, 8, 1, 1, (1, 1), (0, 0)),
    (1, 6, 6, 1, 1, 3, 3, (1, 1), (2, 2)),
    (2, 17, 15, 32, 130, 3, 3, (1, 1), (1, 1)),
    (1, 4, 4, 132, 36, 4, 4, (1, 1), (0, 0)),
    (4, 12, 12, 64, 64, 3, 3, (1, 1), (1, 1)),
    # stride-parity classes: stride 3 (9 classes), stride 5 (25 classes, more
    # than one launch holds), and an input shorter than its stride
    (1, 11, 13, 8, 12, 3, 3, (3, 3), (1, 1)),
    (1, 12, 12, 4, 8, 5, 5, (5, 5), (2, 2)),
    (2, 1, 5, 4, 4, 1, 3, (2, 2), (0, 1)),
]


def run_gpu(x, need_input_grad=True):
    import torch
    import paper_2608_01563_amd as mg
    X, W, dY = (torch.from_numpy(a.copy()).cuda() for a in (x.X, x.W, x.dY))
    dX, dW = mg.conv2d_backward(X, W, dY, stride=x.stride, pad=x.pad,
                                need_input_grad=need_input_grad)
    torch.cuda.synchronize()
    host = lambda t: None if t is None else t.cpu().numpy().astype(np.float64)
    return host(dX), host(dW)


@pytest.mark.parametrize("shape", SMALL)
def test_small_shapes(gpu_lib, shape):
    from oracle.conv import oracle_conv2d_bwd_data, oracle_conv2d_bwd_filter
    N, H, W, C, K, R, S, stride, pad = shape
    say("conv small N%d H%d W%d C%d K%d R%d S%d stride%s pad%s" % (N, H, W, C, K, R, S, stride,
                                                                    pad))
    x = make_conv_inputs(N, H, W, C, K, R, S, stride, pad, seed=H * 131 + C * 7 + K)
    dX, dW = run_gpu(x)
    rX = oracle_conv2d_bwd_data(x.dY, x.W, x.X.shape, stride, pad)
    rW = oracle_conv2d_bwd_filter(x.X, x.dY, x.W.shape, stride, pad)
    eX, eW = normwise_error(dX, rX), normwise_error(dW, rW)
    assert eX <= TOL and eW <= TOL, (eX, eW)
    # positions that no output reads (stride > filter) get exact zeros
    assert np.all(dX[rX == 0.0] == 0.0)


@pytest.mark.parametrize("shape", [SMALL[1], SMALL[4], SMALL[9], (4, 7, 7, 128, 128, 3, 3, 1, 1),
                                   (4, 14, 14, 64, 256, 1, 1, 2, 0)])
def test_fused_equals_separate_calls(gpu_lib, shape):
    """mg_conv2d_bwd (both derivatives in one launch) gives exactly the
    results of mg_conv2d_bwd_data and mg_conv2d_bwd_filter."""
    import torch
    mg = gpu_lib
    N, H, W, C, K, R, S, stride, pad = shape
    stride = (stride, stride) if isinstance(stride, int) else stride
    pad = (pad, pad) if isinstance(pad, int) else pad
    say("conv fused vs separate N%d H%d C%d K%d R%d stride%s" % (N, H, C, K, R, stride))
    x = make_conv_inputs(N, H, W, C, K, R, S, stride, pad, seed=11)
    X, Wt, dY = (torch.from_numpy(a.copy()).cuda() for a in (x.X, x.W, x.dY))
    dX1, dW1 = torch.empty_like(X), torch.empty_like(Wt)
    mg.mg_conv2d_bwd_data(dY, Wt, dX1, stride=stride, pad=pad)
    mg.mg_conv2d_bwd_filter(X, dY, dW1, stride=stride, pad=pad)
    dX2, dW2 = torch.empty_like(X), torch.empty_like(Wt)
    mg.mg_conv2d_bwd(X, Wt, dY, dX2, dW2, stride=stride, pad=pad)
    torch.cuda.synchronize()
    assert torch.equal(dX1, dX2) and torch.equal(dW1, dW2)


def test_repeatable_bit_for_bit(gpu_lib):
    x = make_conv_inputs(4, 28, 28, 64, 64, 3, 3, 1, 1, seed=3)
    a, b = run_gpu(x), run_gpu(x)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


LAYERS = resnet50_layers()
# one layer of every distinct shape
DISTINCT = {}
for _layer in LAYERS:
    DISTINCT.setdefault((_layer.H, _layer.C, _layer.K, _layer.R, _layer.stride), _layer)


def _edges(n, tile):
    """Indices in [0, n) at the edges of `tile`-wide tiles: the first and
    last index, both sides of the first two tile boundaries, and the first
    and last index of the last (possibly partial) tile."""
    last = (n - 1) // tile * tile
    cand = {0, 1, tile - 1, tile, 2 * tile - 1, 2 * tile, last, last + 1, n - 2, n - 1}
    return sorted(i for i in cand if 0 <= i < n)


def boundary_samples(rows, cols, tiles_r=(64,), tiles_c=(64, 128)):
    """Flat indices of a [rows][cols] output at the edges of its output
    tiles (64 rows by 64 or 128 columns) and of the split reduction's vector
    groups: the first and last 16 flat elements (the reduction's tail)."""
    rs = sorted({i for t in tiles_r for i in _edges(rows, t)})
    cs = sorted({i for t in tiles_c for i in _edges(cols, t)})
    idx = {r * cols + c for r in rs for c in cs}
    total = rows * cols
    idx.update(range(min(16, total)))
    idx.update(range(max(0, total - 16), total))
    return np.array(sorted(idx), dtype=np.int64)


def image_edge_samples(N, H, W, C):
    """Flat indices of dX [N,H,W,C] at the image borders (first and last two
    rows and columns of the first and last image, where the padding and
    every stride-parity class of pixels meet) on the channel tile edges."""
    cs = sorted({i for t in (64, 128) for i in _edges(C, t)})
    ns = sorted({0, N - 1})
    hs = sorted({h for h in (0, 1, H - 2, H - 1) if 0 <= h < H})
    ws = sorted({w for w in (0, 1, W - 2, W - 1) if 0 <= w < W})
    return np.array(sorted({((n * H + h) * W + w) * C + c for n in ns for h in hs for w in ws
                            for c in cs}), dtype=np.int64)


def sampled_error(got, flat_idx, ref_vals):
    """max |got - oracle| over the samples / max |oracle| over the samples
    (the denominator comes from the oracle only)."""
    den = np.max(np.abs(ref_vals))
    return np.max(np.abs(got.reshape(-1)[flat_idx] - ref_vals)) / den


@pytest.mark.parametrize("layer", list(DISTINCT.values()), ids=lambda l: l.name)
def test_resnet50_layer_sampled(gpu_lib, layer):
    """Full-size ResNet-50 layer (batch 4): 256 random elements of dX and of
    dW plus every element at a tile edge or at the ends of the flat arrays,
    against the oracle's one-by-one sums; finiteness everywhere."""
    from oracle.conv import oracle_conv2d_bwd_data_at, oracle_conv2d_bwd_filter_at
    say("resnet50 %s: N%d H%d C%d K%d R%d stride %d" % (layer.name, layer.N, layer.H, layer.C,
                                                       layer.K, layer.R, layer.stride))
    x = layer_inputs(layer, seed=len(layer.name) * 17 + layer.C)
    dX, dW = run_gpu(x, need_input_grad=layer.input_grad)
    rng = np.random.default_rng(layer.K + layer.H)
    rsc = layer.R * layer.S * layer.C
    iw = np.concatenate([rng.integers(0, dW.size, 256), boundary_samples(layer.K, rsc)])
    rW = oracle_conv2d_bwd_filter_at(x.X, x.dY, x.W.shape, iw, x.stride, x.pad)
    eW = sampled_error(dW, iw, rW)
    assert np.all(np.isfinite(dW)) and eW <= TOL, eW
    if layer.input_grad:
        pixels = layer.N * layer.H * layer.W
        ix = np.concatenate([rng.integers(0, dX.size, 256),
                             boundary_samples(pixels, layer.C),
                             image_edge_samples(layer.N, layer.H, layer.W, layer.C)])
        rX = oracle_conv2d_bwd_data_at(x.dY, x.W, x.X.shape, ix, x.stride, x.pad)
        eX = sampled_error(dX, ix, rX)
        assert np.all(np.isfinite(dX)) and eX <= TOL, eX


def test_argument_errors(gpu_lib):
    import torch
    mg = gpu_lib
    X = torch.zeros(1, 4, 4, 4, device="cuda")
    W = torch.zeros(8, 3, 3, 4, device="cuda")
    dY = torch.zeros(1, 2, 2, 8, device="cuda")
    dW = torch.empty_like(W)
    with pytest.raises(mg.MgError) as e:
        mg.mg_conv2d_bwd_filter(X, dY, dW, contract="fast_bf16")
    assert e.value.status == 2
    with pytest.raises(ValueError):
        mg.mg_conv2d_bwd_filter(X, dY[:, :1], dW)       # dY of the wrong shape
    big = mg.mg_conv2d_bwd_filter_workspace_bytes((4, 224, 224, 3), (64, 7, 7, 3), (2, 2),
                                                  (3, 3))
    assert big > 0
    Xb = torch.zeros(4, 224, 224, 3, device="cuda")
    dYb = torch.zeros(4, 112, 112, 64, device="cuda")
    dWb = torch.empty(64, 7, 7, 3, device="cuda")
    small = torch.empty(big - 4, dtype=torch.uint8, device="cuda")
    with pytest.raises(mg.MgError) as e:
        mg.mg_conv2d_bwd_filter(Xb, dYb, dWb, stride=(2, 2), pad=(3, 3), workspace=small)
    assert e.value.status == 4
