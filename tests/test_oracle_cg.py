"""Pins for the oracle's Clebsch-Gordan tensors: sympy, orthonormality, equivariance."""

import itertools

import numpy as np
import pytest

from oracle import cg, sh

NNZ_TABLE = {  # non-zero counts of the real coupling tensors, l <= 3
    (0, 0, 0): 1, (0, 1, 1): 3, (0, 2, 2): 5, (0, 3, 3): 7, (1, 0, 1): 3, (1, 1, 0): 3, (1, 1, 1): 6,
    (1, 1, 2): 11, (1, 2, 1): 11, (1, 2, 2): 16, (1, 2, 3): 21, (1, 3, 2): 21, (1, 3, 3): 26,
    (2, 0, 2): 5, (2, 1, 1): 11, (2, 1, 2): 16, (2, 1, 3): 21, (2, 2, 0): 5, (2, 2, 1): 16, (2, 2, 2): 25,
    (2, 2, 3): 28, (2, 3, 1): 21, (2, 3, 2): 28, (2, 3, 3): 41, (3, 0, 3): 7, (3, 1, 2): 21, (3, 1, 3): 26,
    (3, 2, 1): 21, (3, 2, 2): 28, (3, 2, 3): 41, (3, 3, 0): 7, (3, 3, 1): 26, (3, 3, 2): 41, (3, 3, 3): 42}


def triples(lmax=3):
    for l1, l2 in itertools.product(range(lmax + 1), repeat=2):
        for l3 in range(abs(l1 - l2), min(l1 + l2, lmax) + 1):
            yield l1, l2, l3


def test_complex_cg_matches_sympy():
    from sympy import S
    from sympy.physics.wigner import clebsch_gordan
    for l1, l2, l3 in triples():
        for m1 in range(-l1, l1 + 1):
            for m2 in range(-l2, l2 + 1):
                m3 = m1 + m2
                if abs(m3) > l3:
                    continue
                ref = float(clebsch_gordan(S(l1), S(l2), S(l3), S(m1), S(m2), S(m3)))
                assert abs(cg.complex_cg(l1, m1, l2, m2, l3, m3) - ref) < 1e-14


def test_orthonormality_and_completeness():
    for l1, l2 in itertools.product(range(4), repeat=2):
        total = np.zeros(((2 * l1 + 1) * (2 * l2 + 1),) * 2)
        for l3 in range(abs(l1 - l2), l1 + l2 + 1):
            Q = cg.real_cg(l1, l2, l3)
            np.testing.assert_allclose(np.einsum("abc,abd->cd", Q, Q), np.eye(2 * l3 + 1), atol=1e-14)
            Qf = Q.reshape(-1, 2 * l3 + 1)
            total += Qf @ Qf.T
        np.testing.assert_allclose(total, np.eye(total.shape[0]), atol=1e-13)


def test_nonzero_counts():
    for key, n in NNZ_TABLE.items():
        assert int((cg.real_cg(*key) != 0).sum()) == n, key


def wigner_from_sh(l, R):
    """D^l(R) by least squares from Y(R n) = D Y(n) over generic points."""
    rng = np.random.default_rng(123)
    n = rng.normal(size=(4 * l + 8, 3))
    n /= np.linalg.norm(n, axis=1, keepdims=True)
    sl = slice(l * l, (l + 1) ** 2)
    A = sh.sh(l, n)[:, sl]
    B = sh.sh(l, n @ R.T)[:, sl]
    D, *_ = np.linalg.lstsq(A, B, rcond=None)
    return D.T


def random_rotation(rng):
    q, r = np.linalg.qr(rng.normal(size=(3, 3)))
    q = q * np.sign(np.diag(r))
    if np.linalg.det(q) < 0:
        q[:, 0] = -q[:, 0]
    return q


def test_equivariance():
    rng = np.random.default_rng(7)
    R = random_rotation(rng)
    D = {l: wigner_from_sh(l, R) for l in range(4)}
    for l in range(4):
        np.testing.assert_allclose(D[l] @ D[l].T, np.eye(2 * l + 1), atol=1e-12)
    for l1, l2, l3 in triples():
        Q = cg.real_cg(l1, l2, l3)
        x = rng.normal(size=2 * l1 + 1)
        y = rng.normal(size=2 * l2 + 1)
        lhs = np.einsum("abc,a,b->c", Q, D[l1] @ x, D[l2] @ y)
        rhs = D[l3] @ np.einsum("abc,a,b->c", Q, x, y)
        np.testing.assert_allclose(lhs, rhs, atol=1e-12, err_msg=str((l1, l2, l3)))


def test_special_cases_and_sign_rule():
    np.testing.assert_allclose(cg.real_cg(1, 1, 0)[:, :, 0], np.eye(3) / np.sqrt(3), atol=1e-15)
    for l in range(4):
        np.testing.assert_allclose(cg.real_cg(0, l, l)[0], np.eye(2 * l + 1), atol=1e-15)
        np.testing.assert_allclose(cg.real_cg(l, 0, l)[:, 0, :], np.eye(2 * l + 1), atol=1e-15)
    # 1 x 1 -> 1 is the normalised cross product in the (y, z, x) component order
    eps = np.zeros((3, 3, 3))
    for (a, b, c), s in {(0, 1, 2): 1, (1, 2, 0): 1, (2, 0, 1): 1, (1, 0, 2): -1, (2, 1, 0): -1, (0, 2, 1): -1}.items():
        eps[a, b, c] = s
    np.testing.assert_allclose(cg.real_cg(1, 1, 1), eps / np.sqrt(2), atol=1e-15)
    for key in NNZ_TABLE:
        flat = cg.real_cg(*key).reshape(-1)
        assert flat[np.nonzero(flat)[0][0]] > 0


@pytest.mark.parametrize("norm", ["none", "fan_in"])
def test_path_coefficient_normalisation(norm):
    from oracle import irreps as ir
    irr = ir.parse_irreps("3x0e+2x1o")
    paths = ir.enumerate_paths(irr, ir.sh_irreps(1), irr)
    cs = cg.path_coefficients(paths, norm)
    for p, c in zip(paths, cs):
        Q = cg.real_cg(p["l_in"], p["l_sh"], p["l_out"])
        fan = sum(q["c_in"] for q in paths if q["i_out"] == p["i_out"])
        alpha = 1.0 if norm == "none" else 1.0 / np.sqrt(fan)
        np.testing.assert_allclose(c, alpha * Q)
