"""Seeded synthetic inputs and layer tables for the FCN workloads.

This module is shared by the tests, the benchmark and the oracle, and holds
none of the method's arithmetic: only random draws, the workload shapes and
the input recipes. Every tensor is drawn in fp64 with
``numpy.random.default_rng(seed)`` and rounded to fp16 (nearest-even) where
the workload stores fp16. No value here comes from the GPU path.

The paper's data (multislice-simulated diffraction stacks of 1024 channels
at 512x512 with a projected-density target, Section 6.2) is not available;
``diffraction_like`` stands in for it with the same structure: a bright
centred disk over a zero-count background, Poisson counting noise, log1p and
per-sample standardisation.
"""
from dataclasses import dataclass, field

import numpy as np

LOSS_SCALE = 2.0 ** 15
GROUP_CAP_BYTES = 25 * 1024 * 1024
GROUP_ALIGN_BYTES = 256
HUBER_DELTA = 10.0   # the Huber cutoff the paper starts from (Section 6.2)


@dataclass(frozen=True)
class Layer:
    name: str
    kind: str            # "conv" or "convT"
    x_shape: tuple       # N, H, W, C_in
    y_shape: tuple       # N, P, Q, C_out
    r: int
    s: int
    stride: int
    pad: int
    relu: bool

    @property
    def w_shape(self):
        if self.kind == "conv":
            return (self.y_shape[3], self.r, self.s, self.x_shape[3])
        return (self.x_shape[3], self.r, self.s, self.y_shape[3])

    @property
    def w_numel(self):
        a, b, c, d = self.w_shape
        return a * b * c * d

    @property
    def flops(self):
        """2 * (multiply-adds of one pass), direct-convolution count."""
        n, h, w, ci = self.x_shape
        _, p, q, co = self.y_shape
        if self.kind == "conv":
            return 2 * n * p * q * co * ci * self.r * self.s
        return 2 * n * h * w * ci * co * self.r * self.s


def _conv(name, n, h, c, k, r, stride, pad, relu):
    p = (h + 2 * pad - r) // stride + 1
    return Layer(name, "conv", (n, h, h, c), (n, p, p, k), r, r, stride, pad, relu)


def _convt(name, n, h, c, k, relu):
    return Layer(name, "convT", (n, h, h, c), (n, 2 * h, 2 * h, k), 4, 4, 2, 1,
                 relu)


def fcn_layers(n=4, h=256, c_in=256, widths=(512, 1024, 1024, 1024),
               dec=(1024, 1024, 512, 256)):
    """Encoder-decoder of the full workload, forward order.

    Encoder: 4 stages of [3x3 s2 conv, 3x3 s1 conv]; decoder: one 4x4 s2 p1
    transposed conv per stage; head: 1x1 conv to 1 channel. ReLU after
    every layer except the head. Defaults give the one-GPU per-step batch
    (4 x 256 x 256 x 256 input, 99,483,904 weights).
    """
    L = []
    c, hh = c_in, h
    for i, k in enumerate(widths):
        L.append(_conv(f"E{i + 1}a", n, hh, c, k, 3, 2, 1, True))
        hh //= 2
        L.append(_conv(f"E{i + 1}b", n, hh, k, k, 3, 1, 1, True))
        c = k
    for i, k in enumerate(dec):
        L.append(_convt(f"D{len(dec) - i}T", n, hh, c, k, True))
        hh *= 2
        c = k
    L.append(_conv("F1x1", n, hh, c, 1, 1, 1, 0, False))
    return L


def densenet_layers(n=4, h=128, c_in=256, c0=256, growth=256, levels=2, per_block=2):
    """Conv layers of the FC-DenseNet variant (Section 6.2: dense blocks
    with growth rate 256, average pooling), forward order. The paper gives
    no layer counts; this Tiramisu-shaped reading has:
      C0       3x3 stem conv, c_in -> c0, at h;
      D{d}.{l} dense layers of down level d (3x3, -> growth channels), each
               reading the concatenation of the block input and the
               block's earlier outputs;
      TD{d}    transition down: 1x1 conv over the block's full
               concatenation (channels kept), then 2x2 average pooling;
      B.{l}    dense layers of the bottleneck block;
      TU{d}    transition up: 4x4 stride-2 transposed conv of the previous
               block's new features (per_block * growth channels, kept);
      U{d}.{l} dense layers of up level d, whose block input is the
               concatenation of TU{d}'s output and the skip (the full
               concatenation of down level d);
      F1x1     1x1 head over the last block's new features -> 1 channel.
    A ReLU follows every layer except the head. Defaults: 4 x 128 x 128 x
    256 input, 38,928,896 weights."""
    L = [_conv("C0", n, h, c_in, c0, 3, 1, 1, True)]
    hh, c = h, c0
    skips = []
    for d in range(1, levels + 1):
        for l in range(1, per_block + 1):
            L.append(_conv(f"D{d}.{l}", n, hh, c, growth, 3, 1, 1, True))
            c += growth
        skips.append(c)
        L.append(_conv(f"TD{d}", n, hh, c, c, 1, 1, 0, True))
        hh //= 2
    for l in range(1, per_block + 1):
        L.append(_conv(f"B.{l}", n, hh, c, growth, 3, 1, 1, True))
        c += growth
    new = per_block * growth
    for d in range(levels, 0, -1):
        L.append(_convt(f"TU{d}", n, hh, new, new, True))
        hh *= 2
        c = new + skips[d - 1]
        for l in range(1, per_block + 1):
            L.append(_conv(f"U{d}.{l}", n, hh, c, growth, 3, 1, 1, True))
            c += growth
    L.append(_conv("F1x1", n, hh, new, 1, 1, 1, 0, False))
    return L


def single_conv_layer():
    """One 3x3 s1 p1 conv, N=2, C=K=16, 64x64, no epilogue."""
    return [_conv("C1", 2, 64, 16, 16, 3, 1, 1, False)]


def encoder_block_layers():
    """3x3 s2 p1 conv 64->128 at 128^2, then 3x3 s1 p1 128->128, each + ReLU."""
    return [_conv("Ea", 8, 128, 64, 128, 3, 2, 1, True),
            _conv("Eb", 8, 64, 128, 128, 3, 1, 1, True)]


def decoder_block_layers():
    """4x4 s2 p1 convT 256->128 from 32^2, then 1x1 conv 128->64 (no ReLU)."""
    return [_convt("DT", 8, 32, 256, 128, False),
            _conv("P1x1", 8, 64, 128, 64, 1, 1, 0, False)]


# ---- random draws ---------------------------------------------------------
def to_f16(a):
    return np.asarray(a, dtype=np.float64).astype(np.float16)


def uniform(rng, shape, lo=-1.0, hi=1.0):
    return to_f16(rng.uniform(lo, hi, size=shape))


def normal(rng, shape, std=1.0):
    return to_f16(rng.normal(0.0, std, size=shape))


def he_std(layer):
    """He-normal std: sqrt(2/fan), fan = R*S*C_in for a conv and the taps a
    transposed-conv output sees, (R/stride)*(S/stride)*C_in, for a convT."""
    ci = layer.x_shape[3]
    if layer.kind == "conv":
        fan = layer.r * layer.s * ci
    else:
        fan = (layer.r // layer.stride) * (layer.s // layer.stride) * ci
    return float(np.sqrt(2.0 / fan))


def he_weights(layers, seed=1):
    """fp16 He-normal weights for each layer, drawn in forward order."""
    rng = np.random.default_rng(seed)
    return [normal(rng, L.w_shape, he_std(L)) for L in layers]


def diffraction_like(n, h, c, seed=0, lam=50.0, sig_lo=8.0, sig_hi=24.0):
    """NHWC fp16 stand-in for stacked diffraction patterns.

    Per (sample, channel): a centred Gaussian disk with sigma ~ U[8, 24] px
    scales Poisson(lam) counts; then log1p and per-sample standardisation
    over (C, H, W) with the population std. All sigmas are drawn first, then
    the counts in (sample, channel) order.
    """
    rng = np.random.default_rng(seed)
    sig = rng.uniform(sig_lo, sig_hi, size=(n, c))
    c0 = (h - 1) / 2.0
    yy, xx = np.meshgrid(np.arange(h), np.arange(h), indexing="ij")
    d2 = (yy - c0) ** 2 + (xx - c0) ** 2
    out = np.empty((n, h, h, c), dtype=np.float16)
    for i in range(n):
        s = np.empty((c, h, h), dtype=np.float64)
        for j in range(c):
            inten = np.exp(-d2 / (2.0 * sig[i, j] ** 2))
            s[j] = np.log1p(rng.poisson(lam * inten))
        s = (s - s.mean()) / s.std()
        out[i] = to_f16(s.transpose(1, 2, 0))
    return out


def smooth_target(n, h, seed=4, sigma=4.0):
    """fp32 N x H x W x 1 target: Gaussian-filtered white noise (periodic),
    rescaled to unit std per sample."""
    rng = np.random.default_rng(seed)
    z = rng.normal(0.0, 1.0, size=(n, h, h))
    f = np.fft.fftfreq(h)
    k2 = f[:, None] ** 2 + f[None, :] ** 2
    filt = np.exp(-2.0 * np.pi ** 2 * sigma ** 2 * k2)
    sm = np.real(np.fft.ifft2(np.fft.fft2(z) * filt))
    sm = sm / sm.std(axis=(1, 2), keepdims=True)
    return sm.astype(np.float32)[..., None]


def injection_indices(total, rate=1e-6, seed=7):
    """Distinct flat indices (over the concatenated gradients) set to +inf."""
    k = int(round(total * rate))
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(total, size=k, replace=False))


# ---- whole workloads -------------------------------------------------------
@dataclass
class Workload:
    name: str
    layers: list
    x: np.ndarray
    weights: list
    dy: np.ndarray = None          # output-gradient (configs 1-3)
    target: np.ndarray = None      # L2 target (config 4)
    extra: dict = field(default_factory=dict)


def single_conv():
    """Single 3x3 conv, N=2, C=K=16, 64x64: x then dy from seed 0, W seed 1."""
    layers = single_conv_layer()
    rng = np.random.default_rng(0)
    x = uniform(rng, layers[0].x_shape)
    dy = uniform(rng, layers[0].y_shape)
    return Workload("single_conv_3x3_n2_c16_64", layers, x, he_weights(layers), dy=dy)


def encoder_block():
    layers = encoder_block_layers()
    x = diffraction_like(8, 128, 64, seed=0)
    dy = uniform(np.random.default_rng(3), layers[-1].y_shape)
    return Workload("encoder_block_n8_c64_128", layers, x, he_weights(layers), dy=dy)


def decoder_block():
    layers = decoder_block_layers()
    x = normal(np.random.default_rng(2), layers[0].x_shape)
    dy = normal(np.random.default_rng(3), layers[-1].y_shape, 1e-2)
    return Workload("decoder_block_n8_c256_32", layers, x, he_weights(layers), dy=dy)


def densenet(n=4, h=128, c_in=256, c0=256, growth=256, levels=2, per_block=2):
    layers = densenet_layers(n, h, c_in, c0, growth, levels, per_block)
    x = diffraction_like(n, h, c_in, seed=0)
    w = he_weights(layers, seed=1)
    t = smooth_target(n, h, seed=4)
    return Workload(f"densenet_n{n}_c{c_in}_{h}_k{growth}", layers, x, w, target=t,
                    extra=dict(levels=levels, per_block=per_block, growth=growth))


def fcn(n=4, h=256, c_in=256, widths=(512, 1024, 1024, 1024),
        dec=(1024, 1024, 512, 256)):
    layers = fcn_layers(n, h, c_in, widths, dec)
    x = diffraction_like(n, h, c_in, seed=0)
    w = he_weights(layers, seed=1)
    t = smooth_target(n, h, seed=4)
    return Workload(f"fcn_n{n}_c{c_in}_{h}", layers, x, w, target=t)
