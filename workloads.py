"""Seeded synthetic inputs for the sparse-input convolution.

This module only draws random numbers: it holds none of the convolution's
arithmetic, and both the oracle tests and the HIP-path tests / benchmark take
their inputs from here.

The paper measures ReLU outputs of LeNet (MNIST), AlexNet (CIFAR-10 and
ImageNet) and GoogLeNet (ImageNet) (Sec. "Sparsity of ReLUs", Sec.
"Experiments", Tab. 2).  Those datasets and trained weights are not available,
so the workloads below stand in for them: inputs that look like ReLU outputs
(exact zeros at a chosen sparsity, |N(0,1)| elsewhere) and Gaussian weights,
on Caffe-shaped layers.

Recipe (numpy PCG64 via default_rng):
  seed = 170407724 + 1000*config + 10*layer_or_branch + sweep_index
  draw order: weights, then the zero mask, then the nonzero values
  weights  ~ N(0, sigma) (sigma is a standard deviation)
  mask     i.i.d. Bernoulli(sparsity), or for the clustered workload a 3x3
           box-blurred N(0,1) field per (n, c) plane thresholded so that
           exactly ceil(sparsity * numel) entries are zero
  values   |N(0,1)|; a draw that rounds to 0 in fp32 is redrawn

Layer chain (conv3 -> ReLU -> conv4 -> ReLU -> conv5 of AlexNet, no pooling
between them): only the first layer's input is drawn; each later layer's
input is the rectified output of the one before.  Eq. 1 has no bias, so the
sparsity of a rectified output is set by the filters' mean instead: weights
~ N(mean, 0.01) with mean = -0.208, -0.187, -0.189 times sigma for conv3,
conv4, conv5, which leaves about 0.95 of each rectified output zero on the
drawn input (the sparsity the paper reports for those layers, Tab. 2).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

BASE_SEED = 170407724


@dataclass(frozen=True)
class Layer:
    """One convolution layer: Tab. 1 parameter names (T = stride, P = pad)."""
    name: str
    N: int
    C: int
    H: int
    W: int
    K: int
    R: int
    S: int
    T: int
    P: int
    sparsity: float
    sigma: float
    clustered: bool = False
    w_mean: float = 0.0      # mean of the weights (0 except in the layer chain)
    config: int = 0
    layer: int = 0
    sweep_index: int = 0

    @property
    def seed(self) -> int:
        return BASE_SEED + 1000 * self.config + 10 * self.layer + self.sweep_index

    @property
    def x_shape(self):
        return (self.N, self.C, self.H, self.W)

    @property
    def w_shape(self):
        return (self.K, self.C, self.R, self.S)

    def with_(self, **kw) -> "Layer":
        d = dict(self.__dict__)
        d.update(kw)
        return Layer(**d)


@dataclass(frozen=True)
class Workload:
    name: str
    layers: tuple = field(default_factory=tuple)


SWEEP = (0.5, 0.7, 0.9, 0.95, 0.99)


def _lenet(name, N, config, sparsity, sweep_index=0):
    return Layer(name, N, 20, 12, 12, 50, 5, 5, 1, 0, sparsity, 0.1,
                 config=config, sweep_index=sweep_index)


# Tab. 2 of the paper: name, C, H_in (= W_in), K, R (= S), P, T, sparsity
TAB2 = (
    ("lenet_conv2", 20, 11, 64, 5, 1, 2, 0.95),
    ("alexnetc_conv3", 32, 6, 64, 5, 2, 1, 0.9),
    ("alexneti_conv4", 384, 5, 384, 3, 1, 1, 0.9),
    ("inception4a_1", 480, 14, 192, 1, 0, 1, 0.9),
    ("inception4a_2", 192, 14, 96, 1, 0, 1, 0.9),
    ("inception4e_3", 160, 14, 320, 3, 1, 1, 0.9),
    ("inception5a_1", 832, 7, 256, 1, 0, 1, 0.95),
    ("inception5a_2", 256, 7, 160, 1, 0, 1, 0.9),
    ("inception5b_3", 192, 7, 384, 3, 1, 1, 0.95),
    ("inception5b_5", 48, 7, 128, 5, 2, 1, 0.95),
)


def _tab2(N, config):
    suffix = "" if N == 128 else "_n%d" % N
    return [Layer("tab2_%s%s" % (name, suffix), N, C, H, H, K, R, R, T, P, sp, 0.1 if name == "lenet_conv2" else 0.01,
                  config=config, layer=i)
            for i, (name, C, H, K, R, P, T, sp) in enumerate(TAB2)]


WORKLOADS = {
    # LeNet conv2, 20->50 maps at 12x12, 5x5, no pad: tiny batch
    "lenet_conv2_tiny": Workload("lenet_conv2_tiny", (_lenet("lenet_conv2", 8, 1, 0.9),)),
    # the same layer at batch 256 over the sparsity sweep 0.5 .. 0.99
    "lenet_conv2_batch": Workload("lenet_conv2_batch", tuple(
        _lenet("lenet_conv2_s%g" % s, 256, 2, s, i) for i, s in enumerate(SWEEP))),
    # AlexNet conv2: 96->256 maps at 27x27, 5x5, pad 2, batch 128
    "alexnet_conv2": Workload("alexnet_conv2", (
        Layer("alexnet_conv2", 128, 96, 27, 27, 256, 5, 5, 1, 2, 0.9, 0.01, config=3),)),
    # AlexNet conv3/conv4/conv5 at 13x13, 3x3, pad 1, each input drawn on its own
    "alexnet_conv345": Workload("alexnet_conv345", (
        Layer("alexnet_conv3", 128, 256, 13, 13, 384, 3, 3, 1, 1, 0.95, 0.01, config=4, layer=0),
        Layer("alexnet_conv4", 128, 384, 13, 13, 384, 3, 3, 1, 1, 0.95, 0.01, config=4, layer=1),
        Layer("alexnet_conv5", 128, 384, 13, 13, 256, 3, 3, 1, 1, 0.95, 0.01, config=4, layer=2),
    )),
    # conv3 -> ReLU -> conv4 -> ReLU -> conv5: only conv3's input is drawn
    "alexnet_chain345": Workload("alexnet_chain345", (
        Layer("chain_conv3", 128, 256, 13, 13, 384, 3, 3, 1, 1, 0.95, 0.01, w_mean=-0.208 * 0.01,
              config=6, layer=0),
        Layer("chain_conv4", 128, 384, 13, 13, 384, 3, 3, 1, 1, 0.95, 0.01, w_mean=-0.187 * 0.01,
              config=6, layer=1),
        Layer("chain_conv5", 128, 384, 13, 13, 256, 3, 3, 1, 1, 0.95, 0.01, w_mean=-0.189 * 0.01,
              config=6, layer=2),
    )),
    # the layers of the paper's Tab. 2 at their listed sparsity, batch 128 and
    # batch 1 (the paper's runs are one image at a time)
    "paper_tab2": Workload("paper_tab2", tuple(_tab2(128, 7))),
    "paper_tab2_n1": Workload("paper_tab2_n1", tuple(_tab2(1, 8))),
    # GoogLeNet inception-shaped, 28x28: 3x3 branch and 5x5 branch, clustered zeros
    "inception_28": Workload("inception_28", (
        Layer("inception_3x3", 128, 96, 28, 28, 128, 3, 3, 1, 1, 0.9, 0.01, True, config=5, layer=0),
        Layer("inception_5x5", 128, 16, 28, 28, 32, 5, 5, 1, 2, 0.9, 0.01, True, config=5, layer=1),
    )),
}


def _nonzero_values(rng, shape) -> np.ndarray:
    vals = np.abs(rng.standard_normal(shape)).astype(np.float32)
    bad = vals == 0
    while bad.any():  # a draw that rounds to zero in fp32 is drawn again
        vals[bad] = np.abs(rng.standard_normal(int(bad.sum()))).astype(np.float32)
        bad = vals == 0
    return vals


def _iid_mask(rng, shape, sparsity) -> np.ndarray:
    """True where the input is zero."""
    return rng.random(shape) < sparsity


def _clustered_mask(rng, shape, sparsity) -> np.ndarray:
    """Spatially clustered zeros: per (n, c) plane a (H+2)x(W+2) N(0,1) field,
    3x3 box mean ("valid") -> H x W, zero at the ceil(sparsity*numel) smallest
    blurred values over the whole tensor."""
    N, C, H, W = shape
    f = rng.standard_normal((N, C, H + 2, W + 2))
    b = np.zeros((N, C, H, W))
    for dy in range(3):
        for dx in range(3):
            b += f[:, :, dy:dy + H, dx:dx + W]
    b /= 9.0
    numel = N * C * H * W
    nz = int(math.ceil(sparsity * numel))
    mask = np.zeros(numel, dtype=bool)
    if nz > 0:
        order = np.argsort(b.ravel(), kind="stable")
        mask[order[:nz]] = True
    return mask.reshape(shape)


def make_inputs(layer: Layer, seed: int | None = None):
    """(x, w) as float32 numpy arrays for one layer, from its own seed."""
    rng = np.random.default_rng(layer.seed if seed is None else seed)
    w = rng.normal(layer.w_mean, layer.sigma, size=layer.w_shape).astype(np.float32)
    if layer.clustered:
        mask = _clustered_mask(rng, layer.x_shape, layer.sparsity)
    else:
        mask = _iid_mask(rng, layer.x_shape, layer.sparsity)
    vals = _nonzero_values(rng, layer.x_shape)
    x = np.where(mask, np.float32(0.0), vals).astype(np.float32)
    return x, w


def small_case(N, C, H, W, K, R, S, T, P, sparsity, seed, sigma=0.1,
               clustered=False) -> Layer:
    """A test-sized layer with its own seed."""
    return Layer("case", N, C, H, W, K, R, S, T, P, sparsity, sigma, clustered,
                 config=0, layer=0, sweep_index=0).with_(name="case_%d" % seed)


def make_case(N, C, H, W, K, R, S, T, P, sparsity, seed, sigma=0.1,
              clustered=False):
    layer = small_case(N, C, H, W, K, R, S, T, P, sparsity, seed, sigma, clustered)
    return make_inputs(layer, seed=seed)


def integer_case(N, C, H, W, K, R, S, seed, sparsity=0.8, xmax=7, wmax=4):
    """Integer-valued inputs (x in 0..xmax, w in -wmax..wmax): every partial
    sum of a convolution is an integer far below 2**24, so fp32 arithmetic in
    any order is exact."""
    rng = np.random.default_rng(seed)
    w = rng.integers(-wmax, wmax + 1, size=(K, C, R, S)).astype(np.float32)
    mask = rng.random((N, C, H, W)) < sparsity
    vals = rng.integers(1, xmax + 1, size=(N, C, H, W)).astype(np.float32)
    x = np.where(mask, np.float32(0.0), vals).astype(np.float32)
    return x, w


def make_chain(workload: Workload, N: int | None = None):
    """(x0, [w per layer]) of a layer chain: the first layer's input and
    every layer's weights, each layer's weights from its own seed (the first
    layer's input follows its weights, as in make_inputs).  N overrides the
    batch of the drawn input."""
    first = workload.layers[0] if N is None else workload.layers[0].with_(N=N)
    x0, w0 = make_inputs(first)
    ws = [w0]
    for layer in workload.layers[1:]:
        rng = np.random.default_rng(layer.seed)
        ws.append(rng.normal(layer.w_mean, layer.sigma, size=layer.w_shape).astype(np.float32))
    return x0, ws
