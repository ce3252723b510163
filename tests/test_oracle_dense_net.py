"""Pin of the FC-DenseNet oracle's wiring (Section 6.2): in fp64, the
directional derivative of <g, y(W, x)> along a random direction of each
layer's weights and of the input must equal <dW, dir> (resp. <dX, dir>)
from the oracle's backward pass; central differences on a tiny network.
A wrong concatenation order, slice offset, gate or a dropped gradient
contribution (skip, dense reuse, transition) breaks it."""
import numpy as np
import pytest

import synth
from oracle import dense_net as DN

pytestmark = []


def _tiny():
    layers = synth.densenet_layers(n=1, h=8, c_in=8, c0=8, growth=8, levels=2, per_block=2)
    rng = np.random.default_rng(5)
    x = rng.normal(size=layers[0].x_shape)
    w = [rng.normal(size=L.w_shape) * np.sqrt(2.0 / (L.r * L.s * L.x_shape[3]))
         for L in layers]
    g = rng.normal(size=layers[-1].y_shape)
    return layers, x, w, g


def _obj(layers, x, w, g):
    return float(np.sum(DN.forward(layers, x, w, store_fp16=False)["y"] * g))


def test_weight_and_input_gradients_match_finite_differences():
    layers, x, w, g = _tiny()
    fwd = DN.forward(layers, x, w, store_fp16=False)
    dW, dX = DN.backward(layers, fwd, x, w, g, store_fp16=False)
    assert set(dW) == {L.name for L in layers}
    rng = np.random.default_rng(6)
    h = 1e-5
    for i, L in enumerate(layers):
        v = rng.normal(size=L.w_shape)
        wp = list(w); wp[i] = w[i] + h * v
        wm = list(w); wm[i] = w[i] - h * v
        fd = (_obj(layers, x, wp, g) - _obj(layers, x, wm, g)) / (2 * h)
        an = float(np.sum(dW[L.name] * v))
        assert an == pytest.approx(fd, rel=1e-5, abs=1e-7), L.name
    v = rng.normal(size=x.shape)
    fd = (_obj(layers, x + h * v, w, g) - _obj(layers, x - h * v, w, g)) / (2 * h)
    assert float(np.sum(dX * v)) == pytest.approx(fd, rel=1e-5, abs=1e-7)


def test_layer_table_shapes():
    L = {l.name: l for l in synth.densenet_layers()}
    assert sum(l.w_numel for l in L.values()) == 38928896
    # dense growth: each layer's input has growth more channels than the last
    assert L["D1.2"].x_shape[3] == L["D1.1"].x_shape[3] + 256
    # up block input = TU output (new features) + skip (full down concatenation)
    assert L["U1.1"].x_shape[3] == 512 + L["TD1"].x_shape[3]
    assert L["TD2"].x_shape[1] == 64 and L["B.1"].x_shape[1] == 32
