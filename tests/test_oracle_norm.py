"""Pin of the oracle's ``fan_in`` path normalisation by the property it exists for.

§4.2 (eq. ``angular_path_contraction``) puts a "path normalisation" inside c^pi
without giving its value; the reading taken is alpha_pi = 1/sqrt(fan_in_g), with
fan_in_g the number of terms summed into one output channel of output irrep g
(sum of C_in over the paths into g for fully connected mixing, the number of
such paths for channelwise mixing).

What fixes it independently of the oracle's own formula: with node features
x ~ N(0, 1), weights A ~ N(0, 1/K) and radial features phi ~ N(0, 1), all
independent, and edge directions uniform on the sphere, the forward output of a
receiver with one edge has, per component,

    E[m^2] = sum_{pi into g} alpha_pi^2 * (terms of pi per output channel) * E[|phi|^2] / K
             * sum_{m_i, m_y} Q[m_i, m_y, m_o]^2

and the real coupling is orthonormal in its first two indices (each output
component has unit norm), while component-normalised harmonics of a uniform
direction have E[Y_m Y_m'] = delta.  So every output irrep has E[m^2] = 1 with
the fan-in normalisation, whatever its fan-in, and E[m^2] = fan_in_g without
normalisation.  The tests estimate E[m^2] by Monte Carlo through the oracle's
forward and check both, on signatures whose output irreps have very different
fan-ins (a normalisation that counted paths, or output channels, would be off
by factors of 3 to 6 there).
"""

import numpy as np
import pytest

from oracle import conv
from oracle import irreps as ir


def _moments(irr_in, lmax, irr_out, K, norm, mode, trials=16, N=1000, seed=0):
    prob = conv.Problem(irr_in, lmax, irr_out, K, normalization=norm, mode=mode)
    rng = np.random.default_rng(seed)
    acc = np.zeros(len(prob.irreps_out))
    cnt = np.zeros(len(prob.irreps_out))
    outs = ir.offsets(prob.irreps_out)
    for _ in range(trials):
        # N receivers with one edge each, senders uniform, directions uniform
        sender = rng.integers(0, N, size=N).astype(np.int32)
        rowptr = np.arange(N + 1, dtype=np.int32)
        v = rng.standard_normal((N, 3))
        evec = v / np.linalg.norm(v, axis=1, keepdims=True) * rng.uniform(0.5, 5.0, size=(N, 1))
        phi = rng.standard_normal((N, K))
        x = rng.standard_normal((N, prob.dim_in))
        W = rng.standard_normal((K, prob.n_w)) / np.sqrt(K)
        m = conv.fwd(prob, x, evec, phi, W, rowptr, sender)
        for g, ((mul, l, _p), o) in enumerate(zip(prob.irreps_out, outs)):
            blk = m[:, o:o + mul * (2 * l + 1)]
            acc[g] += np.sum(blk * blk)
            cnt[g] += blk.size
    return prob, acc / cnt


def _fan_in(prob, mode):
    f = np.zeros(len(prob.irreps_out))
    for p in prob.paths:
        f[p["i_out"]] += 1 if mode == "uvu" else p["c_in"]
    return f


# output fan-ins (uvw): 0e <- 4 + 12 + 2 = 18 over 3 paths, 1o <- 4 + 12 + 12 + 2 = 30 over 4 paths,
# 2e <- 4 + 12 + 2 + 2 = 20 over 4 paths
UVW = ("4x0e+12x1o+2x2e", 2, "3x0e+5x1o+2x2e", 4)
# channelwise: 0e is reached by 3 paths, 1o by 4, 2e by 4 (equal multiplicities along every path)
UVU = ("16x0e+16x1o+16x2e", 2, "16x0e+16x1o+16x2e", 4)


@pytest.mark.parametrize("mode,sig", [("uvw", UVW), ("uvu", UVU)])
def test_fan_in_gives_unit_output_variance(mode, sig):
    prob, m2 = _moments(*sig, "fan_in", mode)
    fan = _fan_in(prob, mode)
    assert len(set(fan.tolist())) > 1, "the signature must mix different fan-ins"
    # seeded Monte Carlo; its spread over seeds is about 2%, so 12% is five standard deviations
    np.testing.assert_allclose(m2, 1.0, rtol=0.12)


@pytest.mark.parametrize("mode,sig", [("uvw", UVW), ("uvu", UVU)])
def test_no_normalisation_gives_fan_in_variance(mode, sig):
    prob, m2 = _moments(*sig, "none", mode)
    np.testing.assert_allclose(m2, _fan_in(prob, mode), rtol=0.12)
