"""Pins of the CPU oracle's MWQ quantizer (Sec. 3.3.1, Eq. 2-5, Algorithm 1 at
X = I) against facts fixed by the paper and by mathematics: a hand-worked
example, brute-force optimality of each code and scale, closed forms, the
nesting property the method is built on, residual invariants, degenerate
groups and the expected error statistics of uniform residuals.  None of these
re-types the oracle's formulas."""
import os

import numpy as np
import pytest
import torch

from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_w(rows, cols, seed, std=0.02):
    return (np.random.default_rng(seed).standard_normal((rows, cols)) * std).astype(np.float32)


# ---- number formats ---------------------------------------------------------

def test_f16_conversion_matches_numpy():
    rng = np.random.default_rng(1)
    vals = np.concatenate([
        rng.standard_normal(4000).astype(np.float32) * 10.0 ** rng.integers(-9, 5, 4000),
        np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, 70000.0, -70000.0, 6.1e-5,
                  5.96e-8, 2.98e-8, 2.99e-8, 1e-10, np.inf, -np.inf], np.float32),
        # exact ties between neighbouring binary16 values
        (np.arange(1024, 1100, dtype=np.float32) + 0.5) / 1024.0,
        (np.arange(1, 60, dtype=np.float32) + 0.5) * np.float32(2.0 ** -24),
    ]).astype(np.float32)
    ours = O.f32_to_f16_bits(vals)
    ref = vals.astype(np.float16).view(np.uint16)
    assert np.array_equal(ours, ref)


def test_f16_decode_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    finite = (bits & 0x7C00) != 0x7C00
    ours = O.f16_bits_to_f32(bits[finite])
    ref = bits[finite].view(np.float16).astype(np.float32)
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(2)
    v = (rng.standard_normal(3000) * 10.0 ** rng.integers(-6, 6, 3000)).astype(np.float32)
    v = np.concatenate([v, np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0], np.float32)])
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(O.round_bf16(v).view(np.uint32), ref.view(np.uint32))


# ---- hand-worked example ----------------------------------------------------

def _golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            key, *vals = line.split()
            out[key] = [float(v) for v in vals]
    return out


def test_hand_worked_example():
    g = _golden("mwq_hand_example.txt")
    W = np.array([g["W"]], np.float32)
    c = O.mwq_quantize(W, group=4, b_min=2, b_max=4)
    assert c.q1[0].tolist() == [int(v) for v in g["q1"]]
    assert int(c.zeros[0, 0]) == int(g["zero"][0])
    s = O.f16_bits_to_f32(c.scales[:, 0, 0])
    assert s.tolist() == [g["scale_b2"][0], g["scale_b3"][0], g["scale_b4"][0]]
    assert c.signs[0, 0].tolist() == [int(v) for v in g["sign_b3"]]
    assert c.signs[1, 0].tolist() == [int(v) for v in g["sign_b4"]]
    for b in (2, 3, 4):
        assert O.mwq_dequant(c, b)[0].tolist() == g[f"what_b{b}"]


# ---- base level (Eq. 2 / Eq. 3 at X = I) ------------------------------------

@pytest.mark.parametrize("b_min", [1, 2, 3, 4])
def test_base_codes_are_nearest_levels(b_min):
    """Each unclamped base code is the brute-force nearest level (q - z) s."""
    W = _rand_w(16, 128, 3 + b_min)
    c = O.mwq_quantize(W, group=64, b_min=b_min, b_max=b_min)
    s = O.f16_bits_to_f32(c.scales[0].ravel()).reshape(16, 2).astype(np.float64)
    qs = np.arange(2 ** b_min)
    for n in range(16):
        for k in range(128):
            G = k // 64
            z = int(c.zeros[n, G])
            err = np.abs(W[n, k] - (qs - z) * s[n, G])
            best = err.min()
            chosen = abs(W[n, k] - (int(c.q1[n, k]) - z) * s[n, G])
            assert chosen <= best + 1e-6 * s[n, G]


def test_base_scale_closed_form_and_zero_exact():
    """s1 = range / (2^b1 - 1) rounded to binary16, range including 0; an exact
    zero weight dequantizes to exactly 0; extremes reconstruct within s1/2
    plus the binary16 rounding of the scale."""
    W = _rand_w(32, 256, 5)
    W[:, 7] = 0.0
    c = O.mwq_quantize(W, group=128, b_min=2, b_max=2)
    Wd = O.mwq_dequant(c, 2)
    for n in range(32):
        for G in range(2):
            w = W[n, G * 128:(G + 1) * 128].astype(np.float64)
            rng_ = max(w.max(), 0.0) - min(w.min(), 0.0)
            s_ref = np.float32(np.float32(rng_) / np.float32(3.0))
            assert c.scales[0, n, G] == np.float16(s_ref).view(np.uint16)
            s = float(np.float16(s_ref))
            assert abs(s - rng_ / 3) <= 2 ** -11 * rng_ / 3 + 1e-12
            err = np.abs(w - Wd[n, G * 128:(G + 1) * 128])
            assert err.max() <= s / 2 + 3 * abs(s - rng_ / 3) + 1e-9
    assert np.all(Wd[:, 7] == 0.0)


def test_ranges():
    W = _rand_w(64, 256, 6)
    c = O.mwq_quantize(W, group=64, b_min=2, b_max=8)
    assert c.q1.max() <= 3 and c.zeros.max() <= 3
    assert set(np.unique(c.signs).tolist()) <= {0, 1}
    assert c.signs.shape == (6, 64, 256)


# ---- residual levels (Eq. 4-5) ------------------------------------------------

def test_residual_scale_is_least_squares_optimum():
    """For a sign code, mean |R| minimises ||R - s sign(R)||^2: compare with a
    brute-force scan of s, and the stored scale is its binary16 rounding."""
    W = _rand_w(4, 64, 7)
    c = O.mwq_quantize(W, group=64, b_min=2, b_max=5)
    for b in (3, 4, 5):
        prev = O.mwq_dequant(c, b - 1)
        for n in range(4):
            R = W[n].astype(np.float64) - prev[n]
            sig = np.where(R >= 0, 1.0, -1.0)
            assert np.array_equal((sig > 0).astype(np.uint8), c.signs[b - 3, n])
            grid = np.linspace(0, 2 * np.abs(R).max(), 20001)
            obj = ((R[None, :] - grid[:, None] * sig[None, :]) ** 2).sum(1)
            s_bf = grid[obj.argmin()]
            s_stored = float(O.f16_bits_to_f32([c.scales[b - 2, n, 0]])[0])
            step = grid[1] - grid[0]
            assert abs(s_stored - s_bf) <= step + 2 ** -11 * s_bf + 1e-7


def test_nesting_slice_equals_direct_quantization():
    """Mandated test 1: slicing the 8-bit nest to b bits (planes 0..b-1 and the
    scales of levels <= b) and dequantizing equals running MWQ to b bits
    directly, bit for bit, for every b.  The slice is taken from the canonical
    packed buffers, unpacked here by the layout definition."""
    rows, cols, group = 64, 256, 128
    W = _rand_w(rows, cols, 8)
    c8 = O.mwq_quantize(W, group=group, b_min=2, b_max=8)
    planes, scales, zeros = O.mwq_pack(c8)
    BR, KB = 2048 // group, cols // group
    P, L = 8, 7
    pl = planes.reshape(rows // BR, KB, P, 64)
    sc = scales.reshape(rows // BR, KB, L, BR)
    ze = zeros.reshape(rows // BR, KB, BR)
    n = np.arange(rows)[:, None]
    k = np.arange(cols)[None, :]
    rb, i, kb = n // BR, n % BR, k // group
    w = ((k % group) // 32) * BR + i
    bit = k % 32
    plane_bits = np.stack([(pl[rb, kb, p, w] >> bit.astype(np.uint32)) & 1 for p in range(P)])
    for b in range(2, 9):
        cb = O.mwq_quantize(W, group=group, b_min=2, b_max=b)
        # codes of the slice
        q1 = plane_bits[0] + 2 * plane_bits[1]
        assert np.array_equal(q1, cb.q1)
        assert np.array_equal(ze[rb[:, 0], :, i[:, 0]], cb.zeros)
        for lev in range(b - 1):
            assert np.array_equal(sc[rb[:, 0], :, lev, i[:, 0]], cb.scales[lev])
        for p in range(2, b):
            assert np.array_equal(plane_bits[p], cb.signs[p - 2])
        # dequant of the slice == dequant of the direct b-bit quantization
        assert np.array_equal(O.mwq_dequant(c8, b), O.mwq_dequant(cb, b))


def test_nesting_invariants():
    """Mandated test 2: per group the squared residual never grows with b, the
    identity ||R_b||^2 = ||R_{b-1}||^2 - g s^2 + g (s^ - s)^2 holds (s = mean
    |R_{b-1}|, s^ its binary16 rounding), and the error of W^_b falls with b."""
    g = 128
    W = _rand_w(32, 512, 9)
    c = O.mwq_quantize(W, group=g, b_min=2, b_max=8)
    rs = c.resid_sq
    assert np.all(rs[1:] <= rs[:-1] * (1 + 1e-6) + 1e-30)
    for b in range(3, 9):
        prev = W.astype(np.float64) - O.mwq_dequant(c, b - 1)
        for n in range(32):
            for G in range(4):
                R = prev[n, G * g:(G + 1) * g]
                s = np.abs(R).mean()
                sh = float(O.f16_bits_to_f32([c.scales[b - 2, n, G]])[0])
                lhs = rs[b - 2, n, G]
                rhs = (R ** 2).sum() - g * s * s + g * (sh - s) ** 2
                assert abs(lhs - rhs) <= 1e-4 * (R ** 2).sum() + 1e-18
    errs = [np.sqrt(((W - O.mwq_dequant(c, b)) ** 2).mean()) for b in range(2, 9)]
    assert all(a > b_ for a, b_ in zip(errs, errs[1:]))


def test_degenerate_groups():
    g = 64
    W = np.zeros((32, 3 * g), np.float32)
    W[:, g:2 * g] = 0.013                   # constant group
    W[:, 2 * g + 5] = 0.5                   # single outlier among zeros
    c = O.mwq_quantize(W, group=g, b_min=2, b_max=8)
    for b in range(2, 9):
        Wd = O.mwq_dequant(c, b)
        assert np.all(Wd[:, :g] == 0.0)      # all-zero group is exact at every b
        s1 = float(O.f16_bits_to_f32([c.scales[0, 0, 1]])[0])
        assert np.abs(Wd[:, g:2 * g] - 0.013).max() <= s1 / 2 + 1e-7
        # the outlier group's zeros stay within the base half-step
        s1o = float(O.f16_bits_to_f32([c.scales[0, 0, 2]])[0])
        assert np.abs(Wd[:, 2 * g + 5] - 0.5).max() <= s1o / 2 + 1e-7
    # the constant group's residual is constant, so one residual bit removes it
    Wd3 = O.mwq_dequant(c, 3)
    assert np.abs(Wd3[:, g:2 * g] - 0.013).max() <= 2e-6


def test_error_statistics_band():
    """Uniform-residual behaviour: a 2-bit min-max step over 128 Gaussian
    samples (range ~5.2 sigma) leaves an RMS error near step/sqrt(12) ~ 0.50
    sigma, and each binary residual level halves a uniform residual.  A 25 %
    band around 0.50 * 2^-(b-2) catches a dropped term or a wrong scale."""
    W = _rand_w(64, 1024, 10)
    c = O.mwq_quantize(W, group=128, b_min=2, b_max=8)
    sd = W.std()
    for b in range(2, 9):
        rel = np.sqrt(((W - O.mwq_dequant(c, b)) ** 2).mean()) / sd
        expect = 0.50 * 2.0 ** -(b - 2)
        assert 0.75 * expect <= rel <= 1.25 * expect, (b, rel, expect)


def test_pack_layout_roundtrip_all_groups():
    """Every packed bit, scale and zero lands where the layout definition puts
    it, for both supported group sizes (independent unpack in the test)."""
    for group in (64, 128):
        rows, cols = 2048 // group * 2, group * 3
        W = _rand_w(rows, cols, 11 + group)
        c = O.mwq_quantize(W, group=group, b_min=2, b_max=8)
        planes, scales, zeros = O.mwq_pack(c)
        BR, KB = 2048 // group, cols // group
        assert planes.size == rows * cols * 8 // 32
        pl = planes.reshape(rows // BR, KB, 8, 64)
        for n in range(0, rows, 7):
            for k in range(0, cols, 5):
                rb, i, kb = n // BR, n % BR, k // group
                w = ((k % group) // 32) * BR + i
                bits = [(int(pl[rb, kb, p, w]) >> (k % 32)) & 1 for p in range(8)]
                assert bits[0] + 2 * bits[1] == c.q1[n, k]
                assert bits[2:] == [int(c.signs[p, n, k]) for p in range(6)]
        sc = scales.reshape(rows // BR, KB, 7, BR)
        ze = zeros.reshape(rows // BR, KB, BR)
        for n in range(rows):
            for G in range(KB):
                assert ze[n // BR, G, n % BR] == c.zeros[n, G]
                assert np.array_equal(sc[n // BR, G, :, n % BR], c.scales[:, n, G])
