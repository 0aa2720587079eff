// Host-side generation of the constant tables the kernels are specialised on:
// real-basis Clebsch-Gordan coupling tensors and real spherical-harmonic
// polynomials (with their first and second derivatives).
#pragma once

#include <array>
#include <vector>

namespace sobek {

// Dense real coupling tensor Q[(2l1+1)][(2l2+1)][(2l3+1)], row-major, orthonormal
// over (a, b) for each c, first non-zero entry (lexicographic) positive.
const std::vector<double> &real_cg(int l1, int l2, int l3);

// One monomial term c * x^px * y^py * z^pz.
struct Mono {
  double c;
  int px, py, pz;
};

// Homogeneous degree-l polynomial P_lm with Y_lm(v) = P_lm(v) / |v|^l
// (component normalised real spherical harmonics, m = -l..l).
const std::vector<Mono> &sh_poly(int l, int m);

}  // namespace sobek
