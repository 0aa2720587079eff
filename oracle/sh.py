"""Real spherical harmonics of an edge vector, with Jacobian and Hessian.

Test infrastructure only (see ``oracle/__init__``).

The paper's angular input Y_ij is "spherical harmonics of the unit direction"
(§2.4) with no normalisation or ordering stated.  Reading taken (and used by the
HIP library too): real basis, component normalisation sum_m Y_lm^2 = 2l+1,
components ordered m = -l..l, which gives Y_1 = sqrt(3) (y, z, x).

Construction (the textbook definition, written out): with
P_l(t) = 2^-l sum_k (-1)^k binom(l,k) binom(2l-2k,l) t^(l-2k) (Legendre),
mu = |m| and K = sqrt((2l+1) (l-mu)!/(l+mu)!) (x sqrt(2) when mu > 0):

    r^l Y_lm = K * Hom[d^mu P_l/dt^mu](z, r) * { Re (x+iy)^mu   m >= 0
                                                 { Im (x+iy)^mu   m <  0

where Hom[.] turns t^n into z^n r^(l-mu-n) so that every term is a homogeneous
polynomial of degree l in (x, y, z).  Hence Y(v) = P(v) / |v|^l for any
non-zero v, which makes the derivatives exact:

    grad Y = grad P / rho^l - l P v / rho^(l+2)
    Hess Y = Hess P / rho^l - l (grad P v^T + v grad P^T) / rho^(l+2)
             - l P I / rho^(l+2) + l (l+2) P v v^T / rho^(l+4).
"""

from __future__ import annotations

from math import comb, factorial, sqrt

import numpy as np

_CACHE = {}


def _padd(a, b, s=1.0):
    out = dict(a)
    for k, v in b.items():
        out[k] = out.get(k, 0.0) + s * v
    return {k: v for k, v in out.items() if v != 0.0}


def _pmul(a, b):
    out = {}
    for (i1, j1, k1), v1 in a.items():
        for (i2, j2, k2), v2 in b.items():
            key = (i1 + i2, j1 + j2, k1 + k2)
            out[key] = out.get(key, 0.0) + v1 * v2
    return {k: v for k, v in out.items() if v != 0.0}


def _ppow(a, n):
    out = {(0, 0, 0): 1.0}
    for _ in range(n):
        out = _pmul(out, a)
    return out


def sh_polynomial(l, m):
    """Homogeneous degree-l polynomial {(px,py,pz): coeff} with Y_lm = P/|v|^l."""
    key = (l, m)
    if key in _CACHE:
        return _CACHE[key]
    mu = abs(m)
    # Legendre coefficients: power n -> coeff
    leg = {}
    for k in range(l // 2 + 1):
        n = l - 2 * k
        leg[n] = leg.get(n, 0.0) + (-1) ** k * comb(l, k) * comb(2 * l - 2 * k, l) / 2.0 ** l
    # mu-th derivative
    der = {}
    for n, c in leg.items():
        if n >= mu:
            der[n - mu] = der.get(n - mu, 0.0) + c * factorial(n) / factorial(n - mu)
    r2 = {(2, 0, 0): 1.0, (0, 2, 0): 1.0, (0, 0, 2): 1.0}
    hom = {}
    for n, c in der.items():
        rest = l - mu - n  # even by parity of the Legendre polynomial
        assert rest % 2 == 0
        term = _pmul({(0, 0, n): c}, _ppow(r2, rest // 2))
        hom = _padd(hom, term)
    # Re / Im of (x + i y)^mu
    ab = {}
    for j in range(mu + 1):
        c = comb(mu, j)
        if m >= 0 and j % 2 == 0:
            ab[(mu - j, j, 0)] = ab.get((mu - j, j, 0), 0.0) + c * (-1) ** (j // 2)
        if m < 0 and j % 2 == 1:
            ab[(mu - j, j, 0)] = ab.get((mu - j, j, 0), 0.0) + c * (-1) ** ((j - 1) // 2)
    norm = sqrt((2 * l + 1) * factorial(l - mu) / factorial(l + mu))
    if mu > 0:
        norm *= sqrt(2.0)
    poly = {k: v * norm for k, v in _pmul(hom, ab).items()}
    _CACHE[key] = poly
    return poly


def _deriv(poly, axis):
    out = {}
    for k, v in poly.items():
        if k[axis] == 0:
            continue
        nk = list(k)
        nk[axis] -= 1
        nk = tuple(nk)
        out[nk] = out.get(nk, 0.0) + v * k[axis]
    return out


def _eval(poly, v):
    v = np.asarray(v, dtype=np.float64)
    x, y, z = v[..., 0], v[..., 1], v[..., 2]
    out = np.zeros(v.shape[:-1])
    for (i, j, k), c in poly.items():
        out = out + c * x ** i * y ** j * z ** k
    return out


def sh(lmax, evec):
    """Y[..., (lmax+1)^2] of the (not necessarily unit) vectors evec[..., 3]."""
    evec = np.asarray(evec, dtype=np.float64)
    rho = np.linalg.norm(evec, axis=-1)
    cols = []
    for l in range(lmax + 1):
        for m in range(-l, l + 1):
            cols.append(_eval(sh_polynomial(l, m), evec) / rho ** l)
    return np.stack(cols, axis=-1)


def sh_jacobian(lmax, evec):
    """J[..., (lmax+1)^2, 3] = dY/d evec."""
    evec = np.asarray(evec, dtype=np.float64)
    rho = np.linalg.norm(evec, axis=-1)
    out = []
    for l in range(lmax + 1):
        for m in range(-l, l + 1):
            P = sh_polynomial(l, m)
            p = _eval(P, evec)
            g = np.stack([_eval(_deriv(P, a), evec) for a in range(3)], axis=-1)
            out.append(g / rho[..., None] ** l - l * p[..., None] * evec / rho[..., None] ** (l + 2))
    return np.stack(out, axis=-2)


def sh_hessian(lmax, evec):
    """H[..., (lmax+1)^2, 3, 3] = d^2 Y / d evec^2."""
    evec = np.asarray(evec, dtype=np.float64)
    rho = np.linalg.norm(evec, axis=-1)[..., None, None]
    eye = np.eye(3)
    out = []
    for l in range(lmax + 1):
        for m in range(-l, l + 1):
            P = sh_polynomial(l, m)
            p = _eval(P, evec)[..., None, None]
            g = np.stack([_eval(_deriv(P, a), evec) for a in range(3)], axis=-1)
            h = np.stack([np.stack([_eval(_deriv(_deriv(P, a), b), evec) for b in range(3)], axis=-1)
                          for a in range(3)], axis=-2)
            vg = evec[..., :, None] * g[..., None, :]
            gv = g[..., :, None] * evec[..., None, :]
            vv = evec[..., :, None] * evec[..., None, :]
            H = (h / rho ** l - l * (gv + vg) / rho ** (l + 2) - l * p * eye / rho ** (l + 2)
                 + l * (l + 2) * p * vv / rho ** (l + 4))
            out.append(H)
    return np.stack(out, axis=-3)
