"""Pins of the oracle's decoder-stack pieces: RMS normalisation against
closed forms and invariants, and the stack composition against cases whose
result is known without running it (zero experts leave the residual stream
unchanged; a stack of two layers equals one layer applied twice in turn)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2504_15299_amd import workloads as wl


def test_rmsnorm_constant_rows():
    d, eps = 64, 1e-5
    c = np.array([3.0, -0.25, 1e-3, 0.0])
    x = np.repeat(c[:, None], d, axis=1)
    h = O.rmsnorm(x, eps)
    want = c / np.sqrt(c * c + eps)
    np.testing.assert_allclose(h, np.repeat(want[:, None], d, axis=1), rtol=1e-15, atol=0)


def test_rmsnorm_one_hot_row():
    d, v = 100, -2.5
    x = np.zeros((1, d))
    x[0, 17] = v
    h = O.rmsnorm(x, 0.0)
    assert h[0, 17] == pytest.approx(-np.sqrt(d), rel=1e-15)
    assert np.count_nonzero(h) == 1


def test_rmsnorm_mean_square_identity_and_scale_invariance():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((5, 333)) * np.array([[1e-3], [1.0], [7.0], [1e2], [0.5]])
    eps = 1e-5
    h = O.rmsnorm(x, eps)
    ms = (x * x).mean(axis=1)
    np.testing.assert_allclose((h * h).mean(axis=1), ms / (ms + eps), rtol=1e-12)
    h0 = O.rmsnorm(x, 0.0)
    np.testing.assert_allclose(O.rmsnorm(37.5 * x, 0.0), h0, rtol=1e-13)
    np.testing.assert_allclose(np.sign(h0), np.sign(x))


def _stack_layers(spec, n_layers, zero=False):
    layers = []
    for l in range(n_layers):
        Wg, _ = wl.gate(spec, l)
        c13, c2 = [], []
        for e in range(spec.E):
            W13 = wl.expert_w13(spec, e, l)
            W2 = wl.expert_w2(spec, e, l)
            if zero:
                W13, W2 = np.zeros_like(W13), np.zeros_like(W2)
            c13.append(O.mwq_quantize(W13, spec.group))
            c2.append(O.mwq_quantize(W2, spec.group))
        layers.append((Wg, c13, c2))
    return layers


def test_stack_of_zero_experts_keeps_the_residual_stream():
    spec = wl.scaled(wl.mixtral_decode(T=6), d=128, f=128, E=4)
    x0 = wl.activations(spec).astype(np.float64)
    req = wl.token_requests(spec)
    table = wl.bit_table(spec)
    x, _ = O.moe_stack(x0, _stack_layers(spec, 2, zero=True), spec.k, req, table)
    assert np.array_equal(x, x0)


def test_stack_composes_layer_by_layer():
    spec = wl.scaled(wl.mixtral_decode(T=5), d=128, f=128, E=4)
    x0 = wl.activations(spec).astype(np.float64)
    req = wl.token_requests(spec)
    table = wl.bit_table(spec)
    layers = _stack_layers(spec, 2)
    both, logits = O.moe_stack(x0, layers, spec.k, req, table)
    one, _ = O.moe_stack(x0, layers[:1], spec.k, req, table)
    two, _ = O.moe_stack(one, layers[1:], spec.k, req, table)
    assert np.array_equal(both, two)
    assert len(logits) == 2 and not np.array_equal(both, one)
