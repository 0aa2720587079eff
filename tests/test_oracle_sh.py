"""Pins for the oracle's spherical harmonics: textbook closed forms, scipy, identities."""

import numpy as np
import pytest

from oracle import sh


def unit(rng, n):
    v = rng.normal(size=(n, 3))
    return v / np.linalg.norm(v, axis=1, keepdims=True)


def closed_forms(v):
    """Textbook real orthonormal SH (l <= 3) times sqrt(4 pi), m = -l..l."""
    x, y, z = v[:, 0], v[:, 1], v[:, 2]
    s = np.sqrt
    cols = [np.ones_like(x),
            s(3) * y, s(3) * z, s(3) * x,
            s(15) * x * y, s(15) * y * z, s(5) / 2 * (3 * z ** 2 - 1), s(15) * x * z, s(15) / 2 * (x ** 2 - y ** 2),
            s(70) / 4 * y * (3 * x ** 2 - y ** 2), s(105) * x * y * z, s(42) / 4 * y * (5 * z ** 2 - 1),
            s(7) / 2 * (5 * z ** 3 - 3 * z), s(42) / 4 * x * (5 * z ** 2 - 1), s(105) / 2 * z * (x ** 2 - y ** 2),
            s(70) / 4 * x * (x ** 2 - 3 * y ** 2)]
    return np.stack(cols, axis=1)


def test_closed_forms_l_le_3():
    v = unit(np.random.default_rng(0), 50)
    np.testing.assert_allclose(sh.sh(3, v), closed_forms(v), atol=1e-13)


def test_scipy_sph_harm_y():
    from scipy.special import sph_harm_y
    v = unit(np.random.default_rng(1), 40)
    theta = np.arccos(np.clip(v[:, 2], -1, 1))
    phi = np.arctan2(v[:, 1], v[:, 0])
    Y = sh.sh(5, v)
    k = 0
    for l in range(6):
        for m in range(-l, l + 1):
            if m > 0:
                ref = np.sqrt(2) * (-1) ** m * sph_harm_y(l, m, theta, phi).real
            elif m == 0:
                ref = sph_harm_y(l, 0, theta, phi).real
            else:
                ref = np.sqrt(2) * (-1) ** m * sph_harm_y(l, -m, theta, phi).imag
            np.testing.assert_allclose(Y[:, k], np.sqrt(4 * np.pi) * ref, atol=1e-12, err_msg=f"l={l} m={m}")
            k += 1


def test_addition_theorem_and_scale_invariance():
    rng = np.random.default_rng(2)
    v = rng.normal(size=(30, 3))
    Y = sh.sh(4, v)
    for l in range(5):
        np.testing.assert_allclose((Y[:, l * l:(l + 1) ** 2] ** 2).sum(1), 2 * l + 1, rtol=1e-13)
    np.testing.assert_allclose(sh.sh(4, 3.7 * v), Y, atol=1e-13)


def test_orthonormality_quadrature():
    # Gauss-Legendre in cos(theta) x uniform phi: exact for the products below
    t, w = np.polynomial.legendre.leggauss(12)
    ph = np.arange(24) * 2 * np.pi / 24
    T, P = np.meshgrid(t, ph, indexing="ij")
    Wt = np.repeat(w[:, None], 24, 1) * (2 * np.pi / 24)
    st = np.sqrt(1 - T ** 2)
    v = np.stack([st * np.cos(P), st * np.sin(P), T], -1).reshape(-1, 3)
    Y = sh.sh(3, v)
    G = (Y * Wt.reshape(-1, 1)).T @ Y / (4 * np.pi)
    np.testing.assert_allclose(G, np.eye(16), atol=1e-13)


def test_jacobian_matches_finite_differences():
    rng = np.random.default_rng(3)
    v = rng.normal(size=(10, 3))
    J = sh.sh_jacobian(3, v)
    h = 1e-6
    for a in range(3):
        d = np.zeros(3)
        d[a] = h
        fd = (sh.sh(3, v + d) - sh.sh(3, v - d)) / (2 * h)
        np.testing.assert_allclose(J[:, :, a], fd, atol=2e-8)


def test_hessian_matches_finite_differences():
    rng = np.random.default_rng(4)
    v = rng.normal(size=(10, 3))
    H = sh.sh_hessian(3, v)
    h = 1e-5
    for a in range(3):
        d = np.zeros(3)
        d[a] = h
        fd = (sh.sh_jacobian(3, v + d) - sh.sh_jacobian(3, v - d)) / (2 * h)
        np.testing.assert_allclose(H[:, :, :, a], fd, atol=1e-7)
    np.testing.assert_allclose(H, np.swapaxes(H, -1, -2), atol=1e-12)


def test_homogeneity_identities():
    # Y depends on the direction only: v . grad Y = 0 and Hess(Y) v = -grad Y
    rng = np.random.default_rng(5)
    v = rng.normal(size=(10, 3))
    J = sh.sh_jacobian(3, v)
    H = sh.sh_hessian(3, v)
    np.testing.assert_allclose(np.einsum("ejk,ek->ej", J, v), 0, atol=1e-12)
    np.testing.assert_allclose(np.einsum("ejkl,el->ejk", H, v), -J, atol=1e-11)


@pytest.mark.parametrize("l", [1, 2, 3])
def test_parity(l):
    v = unit(np.random.default_rng(6), 8)
    sl = slice(l * l, (l + 1) ** 2)
    np.testing.assert_allclose(sh.sh(3, -v)[:, sl], (-1) ** l * sh.sh(3, v)[:, sl], atol=1e-13)
