// Table generation for the kernel generator.
//
// Clebsch-Gordan (Section 4.2, eq. angular_path_contraction: c^pi holds the
// sparse CG coefficient of the path).  The complex coefficients are built by
// the ladder-operator construction: the highest state |J, J> of each total
// angular momentum J is the unit vector of the m1 + m2 = J subspace orthogonal
// to the states of every larger J (phase: the |m1 = l1> component positive,
// the Condon-Shortley choice), and |J, M-1> = J_- |J, M> / sqrt(J(J+1) - M(M-1)).
// The real tensor is Q[a,b,c] = sum conj(U1[a,m1]) conj(U2[b,m2]) U3[c,m3] <..|..>,
// U the unitary that maps complex harmonics (Condon-Shortley phase) to the real
// ones below; Q is purely real or purely imaginary and its non-zero part is
// kept, with the first non-zero entry in (a, b, c) order made positive.
//
// Spherical harmonics (Section 2.4: Y_ij are spherical harmonics of the edge
// direction).  Real, component normalised, m = -l..l.  With mu = |m| and the
// homogeneous Legendre family Q_l^mu(z, r^2) given by the three-term recurrence
//   Q_mu^mu = (2mu-1)!!,  Q_{mu+1}^mu = (2mu+1) z Q_mu^mu,
//   (l - mu) Q_l^mu = (2l-1) z Q_{l-1}^mu - (l+mu-1) r^2 Q_{l-2}^mu,
// and A_mu + i B_mu = (x + i y)^mu (A_{mu+1} = x A_mu - y B_mu,
// B_{mu+1} = x B_mu + y A_mu):
//   P_lm = N_l^mu Q_l^mu * (A_mu if m >= 0 else B_mu),
//   N_l^mu = sqrt((2l+1) (l-mu)! / (l+mu)!) * (sqrt2 if mu > 0).
#include "tables.h"

#include <cmath>
#include <complex>
#include <map>
#include <mutex>
#include <stdexcept>

namespace sobek {
namespace {

using cd = std::complex<double>;

// Complex CG matrix for fixed (l1, l2, J): C[m1 + l1][m2 + l2][M + J].
std::vector<double> complex_cg_ladder(int l1, int l2, int J) {
  const int d1 = 2 * l1 + 1, d2 = 2 * l2 + 1;
  const int dim = d1 * d2;
  auto idx = [&](int m1, int m2) { return (m1 + l1) * d2 + (m2 + l2); };
  // states[Jp][M] for Jp > J already built, each a vector over product basis
  std::map<int, std::map<int, std::vector<double>>> states;
  std::vector<double> out((size_t)d1 * d2 * (2 * J + 1), 0.0);
  for (int Jc = l1 + l2; Jc >= J; --Jc) {
    // highest state of Jc: start from |m1 = l1, m2 = Jc - l1>
    std::vector<double> v(dim, 0.0);
    v[idx(l1, Jc - l1)] = 1.0;
    for (auto &kv : states) {
      const std::vector<double> &w = kv.second.at(Jc);
      double dot = 0.0;
      for (int t = 0; t < dim; ++t) dot += w[t] * v[t];
      for (int t = 0; t < dim; ++t) v[t] -= dot * w[t];
    }
    double nrm = 0.0;
    for (double a : v) nrm += a * a;
    nrm = std::sqrt(nrm);
    for (double &a : v) a /= nrm;
    std::map<int, std::vector<double>> mine;
    mine[Jc] = v;
    for (int M = Jc; M > -Jc; --M) {
      const std::vector<double> &cur = mine[M];
      std::vector<double> nxt(dim, 0.0);
      for (int m1 = -l1; m1 <= l1; ++m1)
        for (int m2 = -l2; m2 <= l2; ++m2) {
          double a = cur[idx(m1, m2)];
          if (a == 0.0) continue;
          if (m1 > -l1) nxt[idx(m1 - 1, m2)] += a * std::sqrt((double)(l1 * (l1 + 1) - m1 * (m1 - 1)));
          if (m2 > -l2) nxt[idx(m1, m2 - 1)] += a * std::sqrt((double)(l2 * (l2 + 1) - m2 * (m2 - 1)));
        }
      double s = std::sqrt((double)(Jc * (Jc + 1) - M * (M - 1)));
      for (double &a : nxt) a /= s;
      mine[M - 1] = nxt;
    }
    if (Jc == J) {
      for (int M = -J; M <= J; ++M)
        for (int m1 = -l1; m1 <= l1; ++m1)
          for (int m2 = -l2; m2 <= l2; ++m2)
            out[((size_t)(m1 + l1) * d2 + (m2 + l2)) * (2 * J + 1) + (M + J)] = mine[M][idx(m1, m2)];
    }
    states[Jc] = std::move(mine);
  }
  return out;
}

// Row a (real m = a - l), column (complex m = k - l).
std::vector<cd> real_unitary(int l) {
  const int d = 2 * l + 1;
  std::vector<cd> U((size_t)d * d, cd(0, 0));
  const double r2 = 1.0 / std::sqrt(2.0);
  U[(size_t)l * d + l] = 1.0;
  for (int mu = 1; mu <= l; ++mu) {
    double sg = (mu % 2) ? -1.0 : 1.0;
    U[(size_t)(l + mu) * d + (l + mu)] = sg * r2;
    U[(size_t)(l + mu) * d + (l - mu)] = r2;
    U[(size_t)(l - mu) * d + (l + mu)] = cd(0, -sg * r2);
    U[(size_t)(l - mu) * d + (l - mu)] = cd(0, r2);
  }
  return U;
}

std::vector<double> build_real_cg(int l1, int l2, int l3) {
  if (l3 < std::abs(l1 - l2) || l3 > l1 + l2) throw std::invalid_argument("triangle rule");
  const int d1 = 2 * l1 + 1, d2 = 2 * l2 + 1, d3 = 2 * l3 + 1;
  std::vector<double> C = complex_cg_ladder(l1, l2, l3);
  std::vector<cd> U1 = real_unitary(l1), U2 = real_unitary(l2), U3 = real_unitary(l3);
  std::vector<cd> Q((size_t)d1 * d2 * d3, cd(0, 0));
  for (int a = 0; a < d1; ++a)
    for (int b = 0; b < d2; ++b)
      for (int c = 0; c < d3; ++c) {
        cd s(0, 0);
        for (int m1 = 0; m1 < d1; ++m1) {
          cd u1 = std::conj(U1[(size_t)a * d1 + m1]);
          if (u1 == cd(0, 0)) continue;
          for (int m2 = 0; m2 < d2; ++m2) {
            cd u2 = std::conj(U2[(size_t)b * d2 + m2]);
            if (u2 == cd(0, 0)) continue;
            for (int m3 = 0; m3 < d3; ++m3) {
              double cgv = C[((size_t)m1 * d2 + m2) * d3 + m3];
              if (cgv == 0.0) continue;
              s += u1 * u2 * U3[(size_t)c * d3 + m3] * cgv;
            }
          }
        }
        Q[((size_t)a * d2 + b) * d3 + c] = s;
      }
  double mre = 0, mim = 0;
  for (const cd &q : Q) {
    mre = std::max(mre, std::abs(q.real()));
    mim = std::max(mim, std::abs(q.imag()));
  }
  std::vector<double> R(Q.size());
  for (size_t t = 0; t < Q.size(); ++t) {
    double v = (mre >= mim) ? Q[t].real() : Q[t].imag();
    R[t] = (std::abs(v) < 1e-14) ? 0.0 : v;
  }
  for (double v : R) {
    if (v != 0.0) {
      if (v < 0)
        for (double &w : R) w = -w;
      break;
    }
  }
  return R;
}

// Polynomial in (x, y, z) as a map from exponents to coefficient.
using Poly = std::map<std::array<int, 3>, double>;

Poly pmul(const Poly &a, const Poly &b) {
  Poly o;
  for (auto &ka : a)
    for (auto &kb : b) {
      std::array<int, 3> k{ka.first[0] + kb.first[0], ka.first[1] + kb.first[1], ka.first[2] + kb.first[2]};
      o[k] += ka.second * kb.second;
    }
  return o;
}
Poly padd(const Poly &a, const Poly &b, double sa, double sb) {
  Poly o;
  for (auto &k : a) o[k.first] += sa * k.second;
  for (auto &k : b) o[k.first] += sb * k.second;
  return o;
}
Poly pconst(double c) { return Poly{{{0, 0, 0}, c}}; }

std::vector<Mono> build_sh(int l, int m) {
  const int mu = std::abs(m);
  if (mu > l) throw std::invalid_argument("|m| > l");
  const Poly Z{{{0, 0, 1}, 1.0}}, R2{{{2, 0, 0}, 1.0}, {{0, 2, 0}, 1.0}, {{0, 0, 2}, 1.0}};
  const Poly X{{{1, 0, 0}, 1.0}}, Yv{{{0, 1, 0}, 1.0}};
  double dfact = 1.0;
  for (int k = 2 * mu - 1; k > 1; k -= 2) dfact *= k;
  Poly qm2, qm1 = pconst(dfact), q = qm1;  // Q_mu^mu
  if (l > mu) {
    q = pmul(Z, qm1);
    for (auto &kv : q) kv.second *= (2 * mu + 1);
    qm2 = qm1;
    qm1 = q;
    for (int ll = mu + 2; ll <= l; ++ll) {
      Poly a = pmul(Z, qm1), b = pmul(R2, qm2);
      q = padd(a, b, (2.0 * ll - 1) / (ll - mu), -(double)(ll + mu - 1) / (ll - mu));
      qm2 = qm1;
      qm1 = q;
    }
  }
  Poly A = pconst(1.0), B = pconst(0.0);
  for (int k = 0; k < mu; ++k) {
    Poly An = padd(pmul(X, A), pmul(Yv, B), 1.0, -1.0);
    Poly Bn = padd(pmul(X, B), pmul(Yv, A), 1.0, 1.0);
    A = An;
    B = Bn;
  }
  double fr = 1.0;  // (l-mu)!/(l+mu)!
  for (int k = l - mu + 1; k <= l + mu; ++k) fr /= k;
  double norm = std::sqrt((2 * l + 1) * fr) * (mu > 0 ? std::sqrt(2.0) : 1.0);
  Poly P = pmul(q, m >= 0 ? A : B);
  std::vector<Mono> out;
  for (auto &kv : P)
    if (std::abs(kv.second) > 1e-14) out.push_back({kv.second * norm, kv.first[0], kv.first[1], kv.first[2]});
  return out;
}

std::mutex g_mu;
std::map<std::array<int, 3>, std::vector<double>> g_cg;
std::map<std::array<int, 2>, std::vector<Mono>> g_sh;

}  // namespace

const std::vector<double> &real_cg(int l1, int l2, int l3) {
  std::lock_guard<std::mutex> lk(g_mu);
  auto key = std::array<int, 3>{l1, l2, l3};
  auto it = g_cg.find(key);
  if (it != g_cg.end()) return it->second;
  return g_cg.emplace(key, build_real_cg(l1, l2, l3)).first->second;
}

const std::vector<Mono> &sh_poly(int l, int m) {
  std::lock_guard<std::mutex> lk(g_mu);
  auto key = std::array<int, 2>{l, m};
  auto it = g_sh.find(key);
  if (it != g_sh.end()) return it->second;
  return g_sh.emplace(key, build_sh(l, m)).first->second;
}

}  // namespace sobek
