"""Irreps descriptors and tensor-product path enumeration (oracle side).

Test infrastructure only (see ``oracle/__init__``).

Definitions followed
--------------------
* A feature is a direct sum of irreps x_{l,sigma} in R^{C x (2l+1)}; its
  flattened width is C_x = sum C (2l+1)  (§2.2, eq. ``flattened_feature_dimension``).
* A path couples one input irrep, one spherical-harmonic irrep and one output
  irrep when |l_in - l_sh| <= l_out <= l_in + l_sh and sigma_out =
  sigma_in sigma_sh  (§2.2, eq. ``cg_selection_rules``).  Spherical harmonics
  of order l carry parity (-1)^l and multiplicity one (§2.4).
* In fully connected (uvw) mode a path owns n_pi = C_in C_out weights and the
  total is N_w = sum n_pi  (§2.4, eq. ``num_weights``).

Readings where the paper is silent
----------------------------------
* Path order: lexicographic in (input index, SH index, output index).
* Flattening of (pi, a) in A (§2.4 says only "after flattening"): path-major in
  that order, then input multiplicity u, then output multiplicity w, i.e.
  A[q, off_pi + u * C_out + w].
* Flat node layout ``ir_mul``: irrep blocks in descriptor order, and inside a
  block the element (u, m) sits at off + m * C + u (adjacent multiplicity
  channels contiguous, the layout of §4.5).  ``mul_ir`` puts it at
  off + u * (2l+1) + m.
"""

from __future__ import annotations

import re

import numpy as np


def parse_irreps(spec):
    """'8x0e+8x1o' -> [(8, 0, 1), (8, 1, -1)].  Accepts a list of triples too."""
    if not isinstance(spec, str):
        return [(int(m), int(l), int(p)) for (m, l, p) in spec]
    out = []
    for tok in spec.replace(" ", "").split("+"):
        if not tok:
            continue
        m = re.fullmatch(r"(?:(\d+)x)?(\d+)([eo])", tok)
        if m is None:
            raise ValueError(f"bad irrep token {tok!r}")
        mul = int(m.group(1) or 1)
        out.append((mul, int(m.group(2)), 1 if m.group(3) == "e" else -1))
    return out


def sh_irreps(lmax):
    """Spherical harmonics 1x0e + 1x1o + ... up to lmax, parity (-1)^l (§2.4)."""
    return [(1, l, (-1) ** l) for l in range(lmax + 1)]


def dim(irreps):
    """Flattened width C_x = sum C (2l+1)  (eq. flattened_feature_dimension)."""
    return sum(mul * (2 * l + 1) for (mul, l, _p) in irreps)


def offsets(irreps):
    """Start of each irrep block in the flattened vector."""
    offs, o = [], 0
    for (mul, l, _p) in irreps:
        offs.append(o)
        o += mul * (2 * l + 1)
    return offs


def enumerate_paths(irreps_in, irreps_sh, irreps_out, mode="uvw"):
    """All paths allowed by eq. cg_selection_rules, lexicographic order.

    Returns dicts with the irrep indices, orders, multiplicities, the path's
    weight count and its offset in the flattened weight axis.  The count is
    C_in C_out for fully connected mixing (eq. uvw_connection, eq. num_weights)
    and C_in for channelwise mixing (eq. uvu_connection), which ties the output
    multiplicity to the input one: a channelwise path with C_out != C_in is an
    error.
    """
    paths, off = [], 0
    for ia, (ca, la, pa) in enumerate(irreps_in):
        for ib, (cb, lb, pb) in enumerate(irreps_sh):
            if cb != 1:
                raise ValueError("spherical-harmonic irreps have multiplicity one")
            for ic, (cc, lc, pc) in enumerate(irreps_out):
                if not (abs(la - lb) <= lc <= la + lb):
                    continue
                if pc != pa * pb:
                    continue
                if mode == "uvu":
                    if cc != ca:
                        raise ValueError(f"uvu path {ia}->{ic} needs C_out = C_in, got {ca} and {cc}")
                    n = ca
                elif mode == "uvw":
                    n = ca * cc
                else:
                    raise ValueError(mode)
                paths.append(dict(i_in=ia, i_sh=ib, i_out=ic, l_in=la, l_sh=lb,
                                  l_out=lc, c_in=ca, c_out=cc, n_w=n, w_off=off))
                off += n
    return paths


def num_weights(paths):
    """N_w = sum over paths of their weight counts (C_in C_out each for uvw, eq. num_weights; C_in for uvu)."""
    return sum(p["n_w"] for p in paths)


def flat_to_blocks(x, irreps, layout="ir_mul"):
    """Flat [..., C_x] array -> list of [..., C, 2l+1] blocks indexed (u, m)."""
    x = np.asarray(x)
    blocks = []
    for (mul, l, _p), o in zip(irreps, offsets(irreps)):
        d = 2 * l + 1
        seg = x[..., o:o + mul * d]
        if layout == "ir_mul":
            b = seg.reshape(seg.shape[:-1] + (d, mul))
            b = np.swapaxes(b, -1, -2)
        elif layout == "mul_ir":
            b = seg.reshape(seg.shape[:-1] + (mul, d))
        else:
            raise ValueError(layout)
        blocks.append(np.ascontiguousarray(b))
    return blocks


def blocks_to_flat(blocks, irreps, layout="ir_mul"):
    """Inverse of flat_to_blocks."""
    parts = []
    for b, (mul, l, _p) in zip(blocks, irreps):
        b = np.asarray(b)
        if layout == "ir_mul":
            parts.append(np.swapaxes(b, -1, -2).reshape(b.shape[:-2] + (mul * (2 * l + 1),)))
        elif layout == "mul_ir":
            parts.append(b.reshape(b.shape[:-2] + (mul * (2 * l + 1),)))
        else:
            raise ValueError(layout)
    return np.concatenate(parts, axis=-1)

