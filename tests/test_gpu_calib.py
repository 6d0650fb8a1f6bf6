"""Calibration-aware MWQ on the GPU (Sec. 3.3.1: Eq. 3 and Eq. 5 with
calibration activations; Algorithm 1) against the CPU oracle.

The factor U (upper Cholesky factor of (2 X^T X + lambda I)^-1) is computed
on the GPU in binary64 and compared with the oracle's binary64 factor within
binary32 rounding.  The calibrated pack is compared bit for bit with the
oracle's codes, both computed from the same seeded weights and the same
factor (the oracle's, rounded to binary32), so that no GPU value enters the
oracle."""
import time

import numpy as np
import pytest
import torch

from layer_cases import DEV
from oracle import oracle as O
from paper_2504_15299_amd import api
from paper_2504_15299_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _calib(r, h, seed, corr=0.9):
    rng = np.random.default_rng(seed)
    Z = rng.standard_normal((r, h))
    X = np.empty_like(Z)
    X[:, 0] = Z[:, 0]
    for c in range(1, h):
        X[:, c] = corr * X[:, c - 1] + np.sqrt(1 - corr * corr) * Z[:, c]
    return X.astype(np.float32)


def _lam(X):
    return 0.01 * float(np.mean(2.0 * np.sum(X.astype(np.float64) ** 2, axis=0)))


@pytest.mark.parametrize("r,h", [(512, 256), (300, 640), (2048, 128)])
def test_factor_matches_oracle(r, h):
    X = _calib(r, h, r + h)
    lam = _lam(X)
    ref = O.mwq_inv_chol_upper(O.mwq_hessian(X, lam))
    U, info = api.mwq_calib_factor(torch.from_numpy(X).to(DEV), lam)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    got = U.cpu().numpy().astype(np.float64)
    # binary32 rounding of a binary64 factor, plus the two binary64 routes
    tol = 2.0 ** -23 * np.abs(ref) + 1e-9 * np.abs(ref).max()
    assert np.all(np.abs(got - ref) <= tol), np.abs(got - ref).max()
    assert np.all(np.tril(got, -1) == 0)


def test_factor_flags_a_singular_hessian():
    """No tokens and lambda 0: H = 0, the first pivot is not positive."""
    X = torch.zeros((0, 128), dtype=torch.float32, device=DEV)
    _, info = api.mwq_calib_factor(X, 0.0)
    torch.cuda.synchronize()
    assert int(info.item()) == 1


def _packed_ref(c):
    return O.mwq_pack(c)


@pytest.mark.parametrize("group,gamma,b_min,b_max,E,rows,cols", [
    (64, 64, 2, 8, 2, 96, 512), (64, 128, 2, 8, 1, 64, 384), (128, 128, 2, 8, 2, 48, 512),
    (64, 128, 1, 5, 1, 64, 256), (128, 128, 3, 8, 1, 32, 256)])
def test_calibrated_pack_bit_exact(group, gamma, b_min, b_max, E, rows, cols):
    X = _calib(4 * cols, cols, cols + group)
    U = O.mwq_inv_chol_upper(O.mwq_hessian(X, _lam(X))).astype(np.float32)
    rng = np.random.default_rng(rows + cols)
    W = (rng.standard_normal((E, rows, cols)) * 0.02).astype(np.float32)
    W[0, 0, :group] = 0.0                       # all-zero group
    W[0, 1, :] = 0.013                          # constant row
    W[-1, -1, -group:] = 40.0 * rng.standard_normal(group)
    m = api.MWQ.empty(E, rows, cols, group, b_min, b_max, device=DEV)
    api.pack_mwq_calibrated(torch.from_numpy(W).to(DEV), torch.from_numpy(U).to(DEV), gamma, m)
    torch.cuda.synchronize()
    planes = m.planes.cpu().numpy().view(np.uint32)
    scales = m.scales.cpu().numpy().view(np.uint16)
    zeros = m.zeros.cpu().numpy()
    nw, ns, nz = O.mwq_sizes(rows, cols, group, b_min, b_max)
    for e in range(E):
        c = O.mwq_quantize_calibrated(W[e], U, group, gamma, b_min, b_max)
        rp, rs, rz = O.mwq_pack(c)
        assert np.array_equal(planes[e * nw:(e + 1) * nw], rp), f"planes expert {e}"
        assert np.array_equal(scales[e * ns:(e + 1) * ns], rs), f"scales expert {e}"
        assert np.array_equal(zeros[e * nz:(e + 1) * nz], rz), f"zeros expert {e}"


def test_calibrated_pack_with_diagonal_factor_equals_plain_pack():
    rows, cols, group = 64, 512, 128
    W = (np.random.default_rng(1).standard_normal((2, rows, cols)) * 0.02).astype(np.float32)
    U = np.diag(np.random.default_rng(2).uniform(0.1, 3.0, cols)).astype(np.float32)
    a = api.MWQ.empty(2, rows, cols, group, device=DEV)
    b = api.MWQ.empty(2, rows, cols, group, device=DEV)
    Wt = torch.from_numpy(W).to(DEV)
    api.pack_mwq_calibrated(Wt, torch.from_numpy(U).to(DEV), 128, a)
    api.pack_mwq(Wt, b)
    torch.cuda.synchronize()
    for name in ("planes", "scales", "zeros"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name


def _row_codes(m, e, rows_sel, levels):
    """Scales [levels][k][groups] and zeros [k][groups] of the selected rows
    of expert e, read out of the tiled layout."""
    BR, KB = 2048 // m.group, m.cols // m.group
    RB = m.rows // BR
    scales = m.scales.cpu().numpy().view(np.uint16)
    zeros = m.zeros.cpu().numpy()
    sc = np.zeros((levels, len(rows_sel), KB), np.uint16)
    zz = np.zeros((len(rows_sel), KB), np.uint8)
    for j, n in enumerate(rows_sel):
        for kb in range(KB):
            blk = (e * RB + n // BR) * KB + kb
            zz[j, kb] = zeros[blk * BR + n % BR]
            for lev in range(levels):
                sc[lev, j, kb] = scales[(blk * levels + lev) * BR + n % BR]
    return sc, zz


def test_calibrated_pack_full_size_sampled_rows():
    """One Mixtral-8x7B-shaped W1/W3 expert (28672 x 4096, group 128, nest
    2..8, blocks of 128 columns) with its factor from 2048 correlated
    calibration tokens: the GPU factor within rounding of the oracle's, and
    the GPU codes of 16 sampled rows (one per 1792-row band, every position
    of a 16-row block) bit-exact with the oracle's from the oracle's factor
    (rows are quantized independently given U)."""
    t0 = time.time()
    s = wl.mixtral_decode(T=1)
    h, N, group, gamma = s.d, 2 * s.f, 128, 128
    X = _calib(2048, h, 77, corr=0.8)
    lam = _lam(X)
    ref = O.mwq_inv_chol_upper(O.mwq_hessian(X, lam))
    U32 = ref.astype(np.float32)
    Ug, info = api.mwq_calib_factor(torch.from_numpy(X).to(DEV), lam)
    W = wl.expert_w13(s, 0)
    m = api.MWQ.empty(1, N, h, group, device=DEV)
    api.pack_mwq_calibrated(torch.from_numpy(W[None]).to(DEV), torch.from_numpy(U32).to(DEV),
                            gamma, m)
    torch.cuda.synchronize()
    print(f"[{time.time() - t0:.1f} s] GPU factor and calibrated pack done", flush=True)
    assert int(info.item()) == 0
    got = Ug.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref) <= 2.0 ** -23 * np.abs(ref) + 1e-9 * np.abs(ref).max())
    rows_sel = np.arange(16) * (N // 16) + np.arange(16)
    c = O.mwq_quantize_calibrated(np.ascontiguousarray(W[rows_sel]), U32, group, gamma)
    print(f"[{time.time() - t0:.1f} s] oracle rows done", flush=True)
    q1, signs = api.debug_unpack(m, 0, 8)
    torch.cuda.synchronize()
    assert np.array_equal(q1.cpu().numpy()[rows_sel], c.q1)
    want = np.where(c.signs > 0, 1, -1).astype(np.int8)
    assert np.array_equal(signs.cpu().numpy()[:, rows_sel], want)
    sc, zz = _row_codes(m, 0, rows_sel, c.levels)
    assert np.array_equal(zz, c.zeros)
    assert np.array_equal(sc, c.scales)
