"""Pins of the Eq. (3) noise oracle: the RMS against a brute-force loop and
closed forms, the size of the perturbation, per-head independence and the
degenerate cases."""
import math

import numpy as np
import pytest

from oracle import noise as NZ


def _xz(shape, seed, spread=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(shape).astype(np.float32)
    if spread:
        x *= (10.0 ** rng.uniform(-3, 3, size=(shape[0], 1, shape[2], 1))).astype(np.float32)
    return x, rng.standard_normal(shape).astype(np.float32)


def test_rms_matches_a_brute_force_loop():
    x, _ = _xz((2, 7, 3, 5), 1)
    rho = NZ.rms_per_head(x)
    for b in range(2):
        for h in range(3):
            acc = 0.0
            for i in range(7):
                for j in range(5):
                    acc += float(x[b, i, h, j]) ** 2
            assert math.isclose(rho[b, h], math.sqrt(acc / 35), rel_tol=1e-14)


def test_rms_closed_forms():
    x = np.full((1, 10, 2, 8), 3.0, np.float32)
    x[..., 1, :] = -0.5
    assert np.allclose(NZ.rms_per_head(x), [[3.0, 0.5]], rtol=1e-15)
    # a single non-zero entry c in an S x d head: rho = |c| / sqrt(S d)
    y = np.zeros((1, 4, 1, 16), np.float32)
    y[0, 2, 0, 5] = -8.0
    assert np.isclose(NZ.rms_per_head(y)[0, 0], 8.0 / 8.0)
    # rho is absolutely homogeneous and invariant to row and channel permutations
    x, _ = _xz((1, 33, 2, 12), 2)
    r = NZ.rms_per_head(x)
    assert np.allclose(NZ.rms_per_head(-4.0 * x), 4.0 * r, rtol=1e-14)
    assert np.allclose(NZ.rms_per_head(x[:, ::-1, :, ::-1]), r, rtol=1e-14)


def test_perturbation_size_is_eps_times_rms_times_field_norm():
    # ||X~ - X||_F = eps rho ||Z||_F per head, exactly; with ||Z||_F^2 ~ S d the relative
    # perturbation ||X~ - X|| / ||X|| is about eps for every head, whatever its magnitude.
    x, z = _xz((2, 4000, 3, 16), 3)
    eps = 0.0265
    xt, rho = NZ.perturb_per_head(x, z, eps)
    for b in range(2):
        for h in range(3):
            d = np.linalg.norm(xt[b, :, h] - x[b, :, h].astype(np.float64))
            assert math.isclose(d, eps * rho[b, h] * np.linalg.norm(z[b, :, h].astype(np.float64)), rel_tol=1e-12)
            rel = d / np.linalg.norm(x[b, :, h].astype(np.float64))
            assert abs(rel / eps - 1) < 0.02
    # the heads span six orders of magnitude, yet their relative perturbations agree
    assert rho.max() / rho.min() > 1e3


def test_heads_are_perturbed_independently():
    x, z = _xz((1, 50, 4, 8), 4)
    xt, rho = NZ.perturb_per_head(x, z, 0.1)
    x2 = x.copy()
    x2[:, :, 2] *= 1024.0
    xt2, rho2 = NZ.perturb_per_head(x2, z, 0.1)
    keep = [0, 1, 3]
    assert np.array_equal(xt2[:, :, keep], xt[:, :, keep]) and np.array_equal(rho2[:, keep], rho[:, keep])
    assert np.allclose(xt2[:, :, 2], 1024.0 * xt[:, :, 2], rtol=1e-13)


def test_degenerate_cases():
    x, z = _xz((1, 20, 2, 8), 5)
    xt, _ = NZ.perturb_per_head(x, z, 0.0)
    assert np.array_equal(xt, x.astype(np.float64))                     # eps = 0: identity
    xz = x.copy()
    xz[:, :, 1] = 0.0
    xt, rho = NZ.perturb_per_head(xz, z, 0.5)
    assert rho[0, 1] == 0.0 and np.all(xt[:, :, 1] == 0.0)               # a zero head stays zero
    # Z = X: every entry is scaled by 1 + eps rho
    xt, rho = NZ.perturb_per_head(x, x, 0.25)
    assert np.allclose(xt, x * (1 + 0.25 * rho[:, None, :, None]), rtol=1e-14)
    e, rho = NZ.perturb_per_head(np.zeros((2, 0, 3, 8), np.float32), np.zeros((2, 0, 3, 8), np.float32), 1.0)
    assert e.shape == (2, 0, 3, 8) and np.array_equal(rho, np.zeros((2, 3)))
    with pytest.raises(ValueError):
        NZ.perturb_per_head(x, z[:, :10], 0.1)
