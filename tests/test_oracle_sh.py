"""Pins for the oracle's real spherical-harmonic basis (Sec. 3.1 radiance).

The basis is pinned to scipy's complex spherical harmonics (a library
routine), to the constant band-0 value, and to orthonormality on the sphere.
"""
import math

import numpy as np
import pytest
from scipy import special

import oracle


def _unit_dirs(n, seed=0):
    d = np.random.default_rng(seed).standard_normal((n, 3))
    return d / np.linalg.norm(d, axis=1, keepdims=True)


def test_band0_constant():
    Y = oracle.sh_basis(0, _unit_dirs(50))
    assert np.allclose(Y[:, 0], 1.0 / (2.0 * math.sqrt(math.pi)), rtol=0, atol=1e-15)


@pytest.mark.parametrize("deg", [1, 2, 3])
def test_matches_scipy_real_form(deg):
    d = _unit_dirs(400, seed=deg)
    Y = oracle.sh_basis(deg, d)
    polar = np.arccos(np.clip(d[:, 2], -1, 1))
    azim = np.arctan2(d[:, 1], d[:, 0])
    for l in range(deg + 1):
        for m in range(-l, l + 1):
            c = special.sph_harm_y(l, abs(m), polar, azim)  # includes the Condon-Shortley phase
            if m > 0:
                ref = math.sqrt(2.0) * (-1) ** m * c.real
            elif m < 0:
                ref = math.sqrt(2.0) * (-1) ** m * c.imag
            else:
                ref = c.real
            assert np.abs(Y[:, l * l + l + m] - ref).max() < 1e-13, (l, m)


def test_orthonormal_by_quadrature():
    # Gauss-Legendre in cos(theta) x uniform azimuth integrates products of
    # degree-3 harmonics exactly.
    x, w = np.polynomial.legendre.leggauss(16)
    nphi = 32
    phi = (np.arange(nphi) + 0.5) * 2 * math.pi / nphi
    ct = np.repeat(x, nphi)
    wt = np.repeat(w, nphi) * (2 * math.pi / nphi)
    st = np.sqrt(1 - ct ** 2)
    ph = np.tile(phi, x.shape[0])
    d = np.stack([st * np.cos(ph), st * np.sin(ph), ct], 1)
    Y = oracle.sh_basis(3, d)
    G = (Y * wt[:, None]).T @ Y
    assert np.abs(G - np.eye(16)).max() < 1e-12
