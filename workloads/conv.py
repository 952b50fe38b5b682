"""Seeded synthetic inputs for the convolution derivatives, with the layer
shapes of ResNet-50 at batch 4 and 224x224 input (the paper's ResNet-50
workload, Sec. 10; its per-dispatch profile, Sec. 7.3, attributes most of
the training step to these derivative kernels).

This module holds no convolution arithmetic: it lists layer shapes and
draws random tensors.  Layouts are channels-last: X [N,H,W,C],
W [K,R,S,C], dY [N,P,Q,K].

Draw recipe: rng = numpy.random.default_rng(seed); X, W, dY are three
successive rng.standard_normal draws (f64) of those shapes; W is scaled by
sqrt(2 / (R*S*C)) (He initialisation, the usual scale of a trained or
freshly initialised ResNet filter); all three are rounded to float32.
"""
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class ConvLayer:
    name: str
    N: int
    H: int
    W: int
    C: int
    K: int
    R: int
    S: int
    stride: int
    pad: int
    input_grad: bool = True   # False for the first layer: the image needs no gradient

    @property
    def P(self):
        return (self.H + 2 * self.pad - self.R) // self.stride + 1

    @property
    def Q(self):
        return (self.W + 2 * self.pad - self.S) // self.stride + 1

    def flops(self):
        """2 * N*P*Q*K*R*S*C per derivative (one multiply-add per tap)."""
        return 2.0 * self.N * self.P * self.Q * self.K * self.R * self.S * self.C


def resnet50_layers(N=4, size=224):
    """The 53 convolutions of ResNet-50 (bottleneck blocks with the stride on
    the 3x3 convolution) in forward order."""
    layers = [ConvLayer("conv1", N, size, size, 3, 64, 7, 7, 2, 3, input_grad=False)]
    h = (size + 2 * 3 - 7) // 2 + 1          # 112
    h = (h + 2 * 1 - 3) // 2 + 1              # 3x3 max pool, stride 2: 56
    cin = 64
    for stage, (width, blocks) in enumerate(((64, 3), (128, 4), (256, 6), (512, 3)), start=1):
        cout = 4 * width
        for b in range(blocks):
            stride = 2 if (b == 0 and stage > 1) else 1
            tag = "layer%d.%d" % (stage, b)
            layers.append(ConvLayer(tag + ".conv1", N, h, h, cin, width, 1, 1, 1, 0))
            layers.append(ConvLayer(tag + ".conv2", N, h, h, width, width, 3, 3, stride, 1))
            ho = (h + 2 - 3) // stride + 1
            layers.append(ConvLayer(tag + ".conv3", N, ho, ho, width, cout, 1, 1, 1, 0))
            if b == 0:
                layers.append(ConvLayer(tag + ".downsample", N, h, h, cin, cout, 1, 1, stride, 0))
            cin, h = cout, ho
    return layers


@dataclass
class ConvInputs:
    X: np.ndarray
    W: np.ndarray
    dY: np.ndarray
    stride: tuple
    pad: tuple


def make_conv_inputs(N, H, W, C, K, R, S, stride=(1, 1), pad=(0, 0), seed=0):
    """One seeded draw following the module recipe (float32 arrays)."""
    stride = (stride, stride) if isinstance(stride, int) else tuple(stride)
    pad = (pad, pad) if isinstance(pad, int) else tuple(pad)
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((N, H, W, C))
    Wt = rng.standard_normal((K, R, S, C)) * np.sqrt(2.0 / (R * S * C))
    dY = rng.standard_normal((N, P, Q, K))
    f = lambda a: np.ascontiguousarray(a.astype(np.float32))
    return ConvInputs(f(X), f(Wt), f(dY), stride, pad)


def layer_inputs(layer, seed):
    return make_conv_inputs(layer.N, layer.H, layer.W, layer.C, layer.K, layer.R, layer.S,
                            layer.stride, layer.pad, seed)
