"""Pins of the CPU oracle's dual routing (Fig. 1; selection counts B_{j,k} of
Sec. 3.4.3) and of its SwiGLU expert FFN / combine, against exhaustive sorts,
library routines (numpy, scipy) and special cases."""
import numpy as np
import pytest
from scipy.special import softmax

from oracle import oracle as O


def _route_inputs(T, E, k, R, seed, ties=False):
    rng = np.random.default_rng(seed)
    logits = rng.standard_normal((T, E))
    if ties:
        logits = np.round(logits * 2) / 2          # many exact ties
        logits[0, :] = 0.25                         # a fully tied token
    req = rng.integers(0, R, T).astype(np.int32)
    table = rng.choice(np.array([2, 3, 4, 8], np.uint8), size=(R, E))
    return logits, req, table


@pytest.mark.parametrize("T,E,k,ties", [(50, 8, 2, False), (64, 8, 2, True), (40, 64, 6, True),
                                        (7, 5, 5, True), (1, 8, 1, False)])
def test_topk_matches_exhaustive_sort(T, E, k, ties):
    """Mandated test 3: the routed experts are the first k of a full sort by
    (logit descending, expert index ascending), all distinct; the routing
    weights are the softmax of the selected logits and sum to 1."""
    logits, req, table = _route_inputs(T, E, k, 3, 1 + T, ties)
    r = O.route_from_logits(logits, k, req, table)
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-logits[t, e], e))[:k]
        assert r["topk_idx"][t].tolist() == order
        assert len(set(order)) == k
        np.testing.assert_allclose(r["topk_w"][t], softmax(logits[t, order]), rtol=1e-14)
        assert abs(r["topk_w"][t].sum() - 1.0) < 1e-14
        assert r["topk_bits"][t].tolist() == [int(table[req[t], e]) for e in order]


def test_histogram_scan_permutation_brute_force():
    T, E, k, R = 300, 64, 6, 4
    logits, req, table = _route_inputs(T, E, k, R, 5, ties=True)
    r = O.route_from_logits(logits, k, req, table, b_min=2, b_max=8)
    L = 7
    keys = (r["topk_idx"] * L + (r["topk_bits"].astype(np.int64) - 2)).ravel()
    hist = np.bincount(keys, minlength=E * L).reshape(E, L)
    assert np.array_equal(r["hist"], hist)
    assert r["hist"].sum() == T * k
    assert np.array_equal(r["offsets"], np.concatenate([[0], np.cumsum(hist.ravel())]))
    assert np.array_equal(r["perm"], np.argsort(keys, kind="stable"))
    assert np.array_equal(r["slot_of"][r["perm"]], np.arange(T * k))
    for e in range(E):
        nz = np.nonzero(hist[e])[0]
        assert r["maxbit"][e] == (2 + nz.max() if nz.size else 0)


def test_route_rejects_out_of_range_bits():
    logits, req, table = _route_inputs(10, 8, 2, 2, 3)
    table = table.copy()
    table[:] = 9
    with pytest.raises(ValueError):
        O.route_from_logits(logits, 2, req, table)
    # request 2 does not exist; the memory after the 2-row table holds valid
    # bit-widths, so only an explicit range check rejects it
    _, req, big = _route_inputs(10, 8, 2, 4, 3)
    table = big[:2]
    req = req.copy()
    req[3] = 2
    with pytest.raises(ValueError):
        O.route_from_logits(logits, 2, req, table)


def test_gate_logits_match_numpy():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((33, 256)).astype(np.float32)
    Wg = (rng.standard_normal((8, 256)) * 0.02).astype(np.float32)
    bias = rng.standard_normal(8).astype(np.float32)
    ref = x.astype(np.float64) @ Wg.astype(np.float64).T + bias
    np.testing.assert_allclose(O.gate_logits(x, Wg, bias), ref, rtol=1e-12, atol=1e-12)


def _codes(f, d, group, seed, b_max=8):
    rng = np.random.default_rng(seed)
    W13 = (rng.standard_normal((2 * f, d)) * 0.02).astype(np.float32)
    W2 = (rng.standard_normal((d, f)) * 0.02).astype(np.float32)
    return O.mwq_quantize(W13, group, 2, b_max), O.mwq_quantize(W2, group, 2, b_max)


@pytest.mark.parametrize("b", [2, 3, 5, 8])
def test_expert_ffn_is_dense_swiglu(b):
    """E = 1, k = 1: the expert output is the textbook SwiGLU
    W2 (silu(W1 x) * (W3 x)) on the dequantized weights (numpy float64)."""
    d, f = 128, 192
    c13, c2 = _codes(f, d, 64, 20 + b)
    x = np.random.default_rng(3).standard_normal((5, d))
    W13 = O.mwq_dequant(c13, b)
    W2 = O.mwq_dequant(c2, b)
    a, c = x @ W13[:f].T, x @ W13[f:].T
    ref = (a / (1 + np.exp(-a)) * c) @ W2.T
    np.testing.assert_allclose(O.expert_ffn(c13, c2, b, x), ref, rtol=1e-11, atol=1e-14)


def test_expert_ffn_on_a_subset_of_w2_rows():
    """MWQ codes of a row depend on that row alone, so quantizing a subset of
    W2's rows gives the same codes as quantizing all of W2, and the expert
    output on those rows equals the matching columns of the full output."""
    d, f, g, b = 128, 192, 64, 5
    rng = np.random.default_rng(41)
    W13 = (rng.standard_normal((2 * f, d)) * 0.02).astype(np.float32)
    W2 = (rng.standard_normal((d, f)) * 0.02).astype(np.float32)
    rows = np.array([0, 5, 6, 77, d - 1])
    c13 = O.mwq_quantize(W13, g)
    c2 = O.mwq_quantize(W2, g)
    c2s = O.mwq_quantize(np.ascontiguousarray(W2[rows]), g)
    assert np.array_equal(c2s.q1, c2.q1[rows]) and np.array_equal(c2s.signs, c2.signs[:, rows])
    assert np.array_equal(c2s.scales, c2.scales[:, rows]) and np.array_equal(c2s.zeros, c2.zeros[rows])
    x = rng.standard_normal((3, d))
    full = O.expert_ffn(c13, c2, b, x)
    sub = O.expert_ffn(c13, c2s, b, x)
    assert sub.shape == (3, len(rows))
    assert np.array_equal(sub, full[:, rows])


def test_layer_equivariance_and_linearity():
    """Permuting tokens permutes the layer output exactly; the combine is
    linear in the routing weights; a top-1 layer with one bit-width equals the
    dense expert of each token."""
    d, f, E, k, T = 64, 64, 4, 2, 12
    codes = [_codes(f, d, 64, 40 + e) for e in range(E)]
    c13 = [c[0] for c in codes]
    c2 = [c[1] for c in codes]
    rng = np.random.default_rng(7)
    x = rng.standard_normal((T, d)).astype(np.float32)
    logits = rng.standard_normal((T, E))
    table = rng.choice(np.array([2, 4, 8], np.uint8), size=(1, E))
    r = O.route_from_logits(logits, k, None, table)
    out = O.moe_layer(x, r, c13, c2)
    p = rng.permutation(T)
    rp = O.route_from_logits(logits[p], k, None, table)
    outp = O.moe_layer(x[p], rp, c13, c2)
    assert np.array_equal(outp, out[p])
    r2 = dict(r)
    r2["topk_w"] = r["topk_w"] * 3.0
    np.testing.assert_allclose(O.moe_layer(x, r2, c13, c2), 3.0 * out, rtol=1e-13, atol=1e-15)
    r1 = O.route_from_logits(logits, 1, None, table)
    out1 = O.moe_layer(x, r1, c13, c2)
    for t in range(T):
        e = int(r1["topk_idx"][t, 0])
        y = O.expert_ffn(c13[e], c2[e], int(table[0, e]), x[t:t + 1].astype(np.float64))
        np.testing.assert_allclose(out1[t], y[0], rtol=1e-14, atol=1e-16)


def test_shared_expert_adds_with_weight_one():
    d, f, E = 64, 64, 4
    codes = [_codes(f, d, 64, 60 + e) for e in range(E)]
    sh = _codes(128, d, 64, 99)
    rng = np.random.default_rng(8)
    x = rng.standard_normal((6, d)).astype(np.float32)
    r = O.route_from_logits(rng.standard_normal((6, E)), 2, None,
                            np.full((1, E), 4, np.uint8))
    base = O.moe_layer(x, r, [c[0] for c in codes], [c[1] for c in codes])
    with_sh = O.moe_layer(x, r, [c[0] for c in codes], [c[1] for c in codes],
                          shared=(sh[0], sh[1], 8))
    ysh = O.expert_ffn(sh[0], sh[1], 8, x.astype(np.float64))
    np.testing.assert_allclose(with_sh - base, ysh, rtol=1e-10, atol=1e-15)


def _numpy_layer(x, r, c13, c2):
    """Fig. 1 written out with numpy on the dequantized weights: every token's
    output is the sum over its k slots of the slot's routing weight times the
    SwiGLU output of the slot's expert at the slot's bit-width."""
    T, k = r["topk_idx"].shape
    f = c2[0].cols
    out = np.zeros((T, x.shape[1]))
    for t in range(T):
        xt = x[t].astype(np.float64)
        for i in range(k):
            e, b = int(r["topk_idx"][t, i]), int(r["topk_bits"][t, i])
            W13, W2 = O.mwq_dequant(c13[e], b), O.mwq_dequant(c2[e], b)
            a, c = W13[:f] @ xt, W13[f:] @ xt
            out[t] += r["topk_w"][t, i] * (W2 @ (a / (1 + np.exp(-a)) * c))
    return out


def _check_weighted_combine(k, E, seed):
    d, f, T = 64, 64, 9
    codes = [_codes(f, d, 64, seed + e) for e in range(E)]
    c13, c2 = [c[0] for c in codes], [c[1] for c in codes]
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, d)).astype(np.float32)
    # well separated logits: distinct experts, clearly unequal slot weights
    logits = rng.permuted(np.tile(np.arange(E, dtype=np.float64) * 0.7, (T, 1)), axis=1)
    table = rng.choice(np.array([2, 3, 5, 8], np.uint8), size=(T, E))
    r = O.route_from_logits(logits, k, np.arange(T, dtype=np.int32), table)
    w = r["topk_w"]
    assert np.all(np.diff(w, axis=1) < -1e-3), "slot weights must differ"
    np.testing.assert_allclose(O.moe_layer(x, r, c13, c2), _numpy_layer(x, r, c13, c2),
                               rtol=1e-11, atol=1e-14)


@pytest.mark.parametrize("k,E", [(2, 8), (6, 64)])
def test_combine_pairs_each_weight_with_its_slot(k, E):
    """Pin of the weighted combine at k >= 2 (Fig. 1): the layer equals an
    independent numpy sum of w[t,i] * SwiGLU_{e(t,i), b(t,i)}(x_t) with
    distinct experts, widths and weights per slot."""
    _check_weighted_combine(k, E, 300 + k)


@pytest.mark.parametrize("k,E", [(2, 8), (6, 64)])
def test_combine_pin_catches_slot_swap(k, E, monkeypatch):
    """A combine that pairs w[t,i] with the output of slot k-1-i (planted in
    the oracle's combine) fails the pin above."""
    real = O.combine

    def swapped(topk_w, y_slot):
        return real(np.ascontiguousarray(np.asarray(topk_w)[:, ::-1]), y_slot)

    monkeypatch.setattr(O, "combine", swapped)
    with pytest.raises(AssertionError):
        _check_weighted_combine(k, E, 300 + k)
