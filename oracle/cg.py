"""Real-basis Clebsch-Gordan coupling tensors (oracle side).

Test infrastructure only (see ``oracle/__init__``).

§4.2 (eq. ``angular_path_contraction``) names c^pi only as "the path
normalisation and sparse Clebsch-Gordan coefficient".  Reading taken:

1. Complex CG <l1 m1 l2 m2 | l3 m3> by Racah's closed formula, summed exactly
   in rational arithmetic (Condon-Shortley convention).
2. Real coupling Q[a,b,c] = sum conj(U1[a,m1]) conj(U2[b,m2]) U3[c,m3] CG,
   with U the unitary that maps complex spherical harmonics (with the
   Condon-Shortley phase) to the real ones of ``oracle.sh``:
       m > 0 : U[m, m] = (-1)^m / sqrt2,      U[m, -m] = 1/sqrt2
       m < 0 : U[m, |m|] = -i (-1)^|m| / sqrt2, U[m, m] = i / sqrt2
       m = 0 : U[0, 0] = 1.
   Q is purely real when l1+l2+l3 is even and purely imaginary when it is
   odd; the non-zero part is taken (a global constant factor keeps
   equivariance).
3. Sign: the first non-zero entry in lexicographic (a, b, c) order is made
   positive.  Any sign is equally correct (it is absorbed by the learned
   weights); the HIP library's generator uses the same rule.
4. Path normalisation alpha_pi = 1 by default; with ``fan_in`` normalisation
   alpha_pi = 1/sqrt(sum of C_in over the paths into the same output irrep).

Q is orthonormal: sum_ab Q[a,b,c] Q[a,b,c'] = delta(c,c').
"""

from __future__ import annotations

from fractions import Fraction
from math import factorial, sqrt

import numpy as np

_CACHE = {}


def _f(n):
    return factorial(n)


def complex_cg(j1, m1, j2, m2, J, M):
    """<j1 m1 j2 m2 | J M> by Racah's formula (integer angular momenta)."""
    if M != m1 + m2 or not (abs(j1 - j2) <= J <= j1 + j2):
        return 0.0
    if abs(m1) > j1 or abs(m2) > j2 or abs(M) > J:
        return 0.0
    pre = Fraction((2 * J + 1) * _f(J + j1 - j2) * _f(J - j1 + j2) * _f(j1 + j2 - J),
                   _f(j1 + j2 + J + 1))
    pre *= _f(J + M) * _f(J - M) * _f(j1 - m1) * _f(j1 + m1) * _f(j2 - m2) * _f(j2 + m2)
    s = Fraction(0)
    for k in range(0, j1 + j2 - J + 1):
        args = [k, j1 + j2 - J - k, j1 - m1 - k, j2 + m2 - k, J - j2 + m1 + k, J - j1 - m2 + k]
        if min(args) < 0:
            continue
        den = 1
        for a in args:
            den *= _f(a)
        s += Fraction((-1) ** k, den)
    return float(s) * sqrt(float(pre))


def real_from_complex(l):
    """U[(2l+1) x (2l+1)], rows real m = -l..l, columns complex m = -l..l."""
    d = 2 * l + 1
    U = np.zeros((d, d), dtype=np.complex128)
    U[l, l] = 1.0
    for mu in range(1, l + 1):
        U[l + mu, l + mu] = (-1) ** mu / sqrt(2.0)
        U[l + mu, l - mu] = 1.0 / sqrt(2.0)
        U[l - mu, l + mu] = -1j * (-1) ** mu / sqrt(2.0)
        U[l - mu, l - mu] = 1j / sqrt(2.0)
    return U


def real_cg(l1, l2, l3):
    """Q[2l1+1, 2l2+1, 2l3+1] real, orthonormal, sign-fixed coupling tensor."""
    key = (l1, l2, l3)
    if key in _CACHE:
        return _CACHE[key]
    if not (abs(l1 - l2) <= l3 <= l1 + l2):
        raise ValueError(f"triangle rule violated for {key}")
    d1, d2, d3 = 2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1
    C = np.zeros((d1, d2, d3))
    for m1 in range(-l1, l1 + 1):
        for m2 in range(-l2, l2 + 1):
            M = m1 + m2
            if abs(M) <= l3:
                C[m1 + l1, m2 + l2, M + l3] = complex_cg(l1, m1, l2, m2, l3, M)
    U1, U2, U3 = real_from_complex(l1), real_from_complex(l2), real_from_complex(l3)
    Q = np.einsum("am,bn,ck,mnk->abc", U1.conj(), U2.conj(), U3, C)
    if np.abs(Q.real).max() >= np.abs(Q.imag).max():
        Q = Q.real.copy()
    else:
        Q = Q.imag.copy()
    Q[np.abs(Q) < 1e-14] = 0.0
    flat = Q.reshape(-1)
    first = flat[np.nonzero(flat)[0][0]]
    if first < 0:
        Q = -Q
    _CACHE[key] = Q
    return Q


def path_coefficients(paths, normalization="none", mode="uvw"):
    """c^pi = alpha_pi Q^(l_in, l_sh, l_out) for every path (eq. angular_path_contraction).

    With "fan_in" normalisation alpha = 1/sqrt(fan_in), fan_in being the number of
    terms summed into one output channel: C_in per path into the output irrep for
    fully connected mixing, one per path for channelwise mixing.
    """
    fan = {}
    for p in paths:
        fan[p["i_out"]] = fan.get(p["i_out"], 0) + (1 if mode == "uvu" else p["c_in"])
    out = []
    for p in paths:
        Q = real_cg(p["l_in"], p["l_sh"], p["l_out"])
        if normalization == "none":
            alpha = 1.0
        elif normalization == "fan_in":
            alpha = 1.0 / sqrt(fan[p["i_out"]])
        else:
            raise ValueError(normalization)
        out.append(alpha * Q)
    return out
