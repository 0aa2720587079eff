// Plan construction and kernel generation.
//
// The generated translation unit is specialised on the static signature only
// (irreps, K, normalisation), never on the graph (Appendix B.1: node and edge
// counts, degrees and chunking select launches, not code).  Per path it holds
// the sparse CG coefficients as immediates; per wave unit it holds loop
// bounds, offsets and register-resident receiver-state accumulators.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <sstream>
#include <stdexcept>

#include "plan.h"
#include "tables.h"

namespace sobek {

namespace {
constexpr int kAccMax = 128;        // forward accumulators per lane per wave unit
constexpr int kSlabFloats = 8192;   // backward LDS budget for one slab of adjoint state (32 KiB)
constexpr int kWaves = 4;           // waves per backward block

bool pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

// channel blocks of an input irrep of multiplicity C: (U, U0, ES)
std::vector<std::array<int, 3>> channel_blocks(int C) {
  std::vector<std::array<int, 3>> out;
  if (C <= 64) {
    int es = (pow2(C) && 64 % C == 0) ? 64 / C : 1;
    out.push_back({C, 0, es});
  } else {
    for (int u0 = 0; u0 < C; u0 += 64) out.push_back({64, u0, 1});
  }
  return out;
}
}  // namespace

void build_plan(Plan& p) {
  int off = 0;
  for (auto& r : p.in) { r.off = off; off += r.dim(); }
  p.dim_in = off;
  off = 0;
  for (auto& r : p.out) { r.off = off; off += r.dim(); }
  p.dim_out = off;
  p.nsh = (p.lmax + 1) * (p.lmax + 1);

  // paths (Section 2.2 eq. cg_selection_rules; lexicographic (in, sh, out) order)
  p.paths.clear();
  int64_t woff = 0;
  for (int a = 0; a < (int)p.in.size(); ++a)
    for (int b = 0; b <= p.lmax; ++b)
      for (int c = 0; c < (int)p.out.size(); ++c) {
        const Irrep &ri = p.in[a], &ro = p.out[c];
        int psh = (b % 2) ? -1 : 1;
        if (ro.l < std::abs(ri.l - b) || ro.l > ri.l + b) continue;
        if (ro.p != ri.p * psh) continue;
        Path q;
        q.i_in = a; q.i_sh = b; q.i_out = c;
        q.l_in = ri.l; q.l_sh = b; q.l_out = ro.l;
        q.c_in = ri.mul; q.c_out = ro.mul;
        q.w_off = woff;
        woff += (int64_t)ri.mul * ro.mul;
        p.paths.push_back(q);
      }
  p.n_w = woff;

  // groups, normalisation, receiver-state column offsets
  p.groups.clear();
  std::vector<int> gidx(p.out.size(), -1);
  for (int c = 0; c < (int)p.out.size(); ++c) {
    std::vector<int> ps;
    for (int t = 0; t < (int)p.paths.size(); ++t)
      if (p.paths[t].i_out == c) ps.push_back(t);
    if (ps.empty()) { p.dead_out.push_back(c); continue; }
    Group g;
    g.i_out = c; g.l = p.out[c].l; g.d = 2 * g.l + 1; g.C = p.out[c].mul; g.off = p.out[c].off;
    g.paths = ps;
    int64_t fan = 0, k = 0;
    for (int t : ps) fan += p.paths[t].c_in;
    for (int t : ps) {
      Path& q = p.paths[t];
      q.alpha = (p.norm == 1) ? 1.0 / std::sqrt((double)fan) : 1.0;
      q.group = (int)p.groups.size();
      q.koff = k;
      k += (int64_t)p.K * q.c_in;
    }
    g.D = k;
    gidx[c] = (int)p.groups.size();
    p.groups.push_back(g);
  }
  int64_t soff = 0, koff = 0;
  p.ktab.clear();
  for (auto& g : p.groups) {
    g.s_off = soff;
    soff += (int64_t)g.d * g.D;
    g.ktab_off = koff;
    koff += g.D;
    for (int t : g.paths) {
      const Path& q = p.paths[t];
      for (int qq = 0; qq < p.K; ++qq)
        for (int u = 0; u < q.c_in; ++u) p.ktab.push_back((int32_t)(qq * p.n_w + q.w_off + (int64_t)u * q.c_out));
    }
  }
  p.srow = soff;
  for (auto& q : p.paths) {
    const std::vector<double>& Q = real_cg(q.l_in, q.l_sh, q.l_out);
    q.cg.resize(Q.size());
    for (size_t t = 0; t < Q.size(); ++t) q.cg[t] = q.alpha * Q[t];
  }

  // forward wave units: per input irrep and channel block, paths packed while
  // K * sum(d_out) accumulators fit the register budget
  p.fwd_units.clear();
  for (int a = 0; a < (int)p.in.size(); ++a) {
    std::vector<int> ps;
    for (int t = 0; t < (int)p.paths.size(); ++t)
      if (p.paths[t].i_in == a) ps.push_back(t);
    if (ps.empty()) { p.dead_in.push_back(a); continue; }
    for (auto blk : channel_blocks(p.in[a].mul)) {
      Unit cur;
      cur.a = a; cur.U = blk[0]; cur.U0 = blk[1]; cur.ES = blk[2];
      int acc = 0;
      for (int t : ps) {
        int need = p.K * (2 * p.paths[t].l_out + 1);
        if (!cur.paths.empty() && acc + need > kAccMax) {
          p.fwd_units.push_back(cur);
          cur.paths.clear();
          acc = 0;
        }
        cur.paths.push_back(t);
        acc += need;
      }
      p.fwd_units.push_back(cur);
    }
  }

  // backward slabs: wave units (input irrep, channel block, path subset) whose
  // adjoint-state slices fit the LDS budget; a given (irrep, block) always runs
  // on the same wave index, so contribution read-modify-writes stay in one thread
  p.slabs.clear();
  struct Item { Unit u; int floats; };
  std::vector<std::vector<Item>> per_pair;  // per (a, block): chunks in order
  for (int a = 0; a < (int)p.in.size(); ++a) {
    std::vector<int> ps;
    for (int t = 0; t < (int)p.paths.size(); ++t)
      if (p.paths[t].i_in == a) ps.push_back(t);
    if (ps.empty()) continue;
    for (auto blk : channel_blocks(p.in[a].mul)) {
      std::vector<Item> chunks;
      Unit cur;
      cur.a = a; cur.U = blk[0]; cur.U0 = blk[1]; cur.ES = blk[2];
      int fl = 0;
      for (int t : ps) {
        int need = p.K * (2 * p.paths[t].l_out + 1) * cur.U;
        if (need > kSlabFloats) throw std::runtime_error("path adjoint slice exceeds the LDS slab budget");
        if (!cur.paths.empty() && fl + need > kSlabFloats) {
          chunks.push_back({cur, fl});
          cur.paths.clear();
          fl = 0;
        }
        cur.paths.push_back(t);
        fl += need;
      }
      chunks.push_back({cur, fl});
      for (size_t c = 0; c < chunks.size(); ++c) chunks[c].u.first = (c == 0);
      per_pair.push_back(chunks);
    }
  }
  {
    Slab cur;
    cur.waves.assign(kWaves, Unit{-1, 0, 0, 0, {}, true, {}});
    auto flush = [&]() {
      bool any = false;
      for (auto& w : cur.waves) any |= (w.a >= 0);
      if (any) p.slabs.push_back(cur);
      cur = Slab();
      cur.waves.assign(kWaves, Unit{-1, 0, 0, 0, {}, true, {}});
    };
    for (size_t i = 0; i < per_pair.size(); ++i) {
      int w = (int)(i % kWaves);
      for (auto& it : per_pair[i]) {
        if (cur.waves[w].a >= 0 || cur.lds_floats + it.floats > kSlabFloats) flush();
        Unit u = it.u;
        int o = cur.lds_floats;
        for (int t : u.paths) {
          u.lds_off.push_back(o);
          o += p.K * (2 * p.paths[t].l_out + 1) * u.U;
        }
        cur.waves[w] = u;
        cur.lds_floats = o;
      }
    }
    flush();
  }
  p.bwd_lds_max = 0;
  for (auto& s : p.slabs) p.bwd_lds_max = std::max(p.bwd_lds_max, s.lds_floats);
}

// ---------------------------------------------------------------------------
// code generation
// ---------------------------------------------------------------------------
namespace {

std::string fl(double v) {
  char b[64];
  std::snprintf(b, sizeof(b), "%.9e", v);
  return std::string(b) + "f";
}

std::string mono(int px, int py, int pz) {
  std::string s;
  auto add = [&](const char* v, int k) {
    if (k == 0) return;
    if (!s.empty()) s += "*";
    s += std::string(v) + std::to_string(k);
  };
  add("x", px); add("y", py); add("z", pz);
  return s.empty() ? "1.0f" : s;
}

// sum of terms c * x^a y^b z^c as an expression
std::string poly_expr(const std::vector<Mono>& P) {
  if (P.empty()) return "0.0f";
  std::string s;
  for (size_t t = 0; t < P.size(); ++t) {
    if (t) s += " + ";
    s += fl(P[t].c) + "*" + mono(P[t].px, P[t].py, P[t].pz);
  }
  return s;
}

std::vector<Mono> dpoly(const std::vector<Mono>& P, int axis) {
  std::vector<Mono> o;
  for (auto m : P) {
    int e = axis == 0 ? m.px : axis == 1 ? m.py : m.pz;
    if (e == 0) continue;
    Mono d = m;
    d.c *= e;
    if (axis == 0) d.px--; else if (axis == 1) d.py--; else d.pz--;
    o.push_back(d);
  }
  return o;
}

std::string powers(int L) {
  std::ostringstream o;
  o << "  const float x0 = 1.0f, y0 = 1.0f, z0 = 1.0f; (void)x0; (void)y0; (void)z0;\n";
  o << "  const float x1 = x, y1 = y, z1 = z; (void)x1; (void)y1; (void)z1;\n";
  for (int k = 2; k <= std::max(L, 1); ++k)
    o << "  const float x" << k << " = x" << k - 1 << "*x, y" << k << " = y" << k - 1 << "*y, z" << k << " = z" << k - 1
      << "*z; (void)x" << k << "; (void)y" << k << "; (void)z" << k << ";\n";
  return o.str();
}

void emit_sh(std::ostringstream& o, int lmax) {
  // Y[0 .. (L+1)^2) on the unit sphere
  for (int L = 0; L <= lmax; ++L) {
    o << "SB_DEV void sb_sh_eval_L" << L << "(float x, float y, float z, float* Y) {\n" << powers(L);
    for (int l = 0, k = 0; l <= L; ++l)
      for (int m = -l; m <= l; ++m, ++k) o << "  Y[" << k << "] = " << poly_expr(sh_poly(l, m)) << ";\n";
    o << "}\n";
  }
  // tangent: Yd_m = (grad P_m . d - l P_m (u . d)) / rho
  for (int L = 0; L <= lmax; ++L) {
    o << "SB_DEV void sb_sh_jvp_L" << L
      << "(float x, float y, float z, float rinv, float dx, float dy, float dz, const float* Y, float* Yd) {\n"
      << powers(L) << "  const float ud = x*dx + y*dy + z*dz; (void)ud;\n";
    for (int l = 0, k = 0; l <= L; ++l)
      for (int m = -l; m <= l; ++m, ++k) {
        const auto& P = sh_poly(l, m);
        o << "  Yd[" << k << "] = ((" << poly_expr(dpoly(P, 0)) << ")*dx + (" << poly_expr(dpoly(P, 1)) << ")*dy + ("
          << poly_expr(dpoly(P, 2)) << ")*dz - " << fl((double)l) << "*Y[" << k << "]*ud)*rinv;\n";
      }
    o << "}\n";
  }
  // cotangent: r_bar = (sum_m Yb_m grad P_m - (sum_m l Yb_m P_m) u) / rho
  o << "SB_DEV void sb_sh_vjp(float x, float y, float z, float rinv, const float* Yb, float* g) {\n" << powers(lmax)
    << "  float gx = 0.f, gy = 0.f, gz = 0.f, s = 0.f;\n";
  for (int l = 0, k = 0; l <= lmax; ++l)
    for (int m = -l; m <= l; ++m, ++k) {
      const auto& P = sh_poly(l, m);
      if (l == 0) continue;
      o << "  { const float b = Yb[" << k << "];\n"
        << "    gx += b*(" << poly_expr(dpoly(P, 0)) << ");\n"
        << "    gy += b*(" << poly_expr(dpoly(P, 1)) << ");\n"
        << "    gz += b*(" << poly_expr(dpoly(P, 2)) << ");\n"
        << "    s += " << fl((double)l) << "*b*(" << poly_expr(P) << "); }\n";
    }
  o << "  g[0] = (gx - s*x)*rinv; g[1] = (gy - s*y)*rinv; g[2] = (gz - s*z)*rinv;\n}\n";
  // Hessian-vector: sum_m Yb_m Hess(Y_m) d, with
  // Hess Y = [Hess P - l (grad P u^T + u grad P^T) - l P I + l (l+2) P u u^T] / rho^2
  o << "SB_DEV void sb_sh_hvp(float x, float y, float z, float rinv, const float* Yb, float dx, float dy, float dz,"
       " float* h) {\n"
    << powers(lmax)
    << "  const float ud = x*dx + y*dy + z*dz;\n"
       "  float t1x = 0.f, t1y = 0.f, t1z = 0.f, t2x = 0.f, t2y = 0.f, t2z = 0.f, t3 = 0.f, t4 = 0.f, t5 = 0.f;\n";
  for (int l = 0, k = 0; l <= lmax; ++l)
    for (int m = -l; m <= l; ++m, ++k) {
      if (l == 0) continue;
      const auto& P = sh_poly(l, m);
      auto Px = dpoly(P, 0), Py = dpoly(P, 1), Pz = dpoly(P, 2);
      o << "  { const float b = Yb[" << k << "];\n"
        << "    const float px = " << poly_expr(Px) << ", py = " << poly_expr(Py) << ", pz = " << poly_expr(Pz)
        << ", pv = " << poly_expr(P) << ";\n"
        << "    const float hxx = " << poly_expr(dpoly(Px, 0)) << ", hxy = " << poly_expr(dpoly(Px, 1))
        << ", hxz = " << poly_expr(dpoly(Px, 2)) << ";\n"
        << "    const float hyy = " << poly_expr(dpoly(Py, 1)) << ", hyz = " << poly_expr(dpoly(Py, 2))
        << ", hzz = " << poly_expr(dpoly(Pz, 2)) << ";\n"
        << "    t1x += b*(hxx*dx + hxy*dy + hxz*dz); t1y += b*(hxy*dx + hyy*dy + hyz*dz); t1z += b*(hxz*dx + hyz*dy + hzz*dz);\n"
        << "    const float lb = " << fl((double)l) << "*b;\n"
        << "    t2x += lb*px; t2y += lb*py; t2z += lb*pz;\n"
        << "    t3 += lb*(px*dx + py*dy + pz*dz);\n"
        << "    t4 += lb*pv;\n"
        << "    t5 += " << fl((double)(l * (l + 2))) << "*b*pv; }\n";
    }
  o << "  const float r2 = rinv*rinv;\n"
       "  h[0] = (t1x - t2x*ud - x*t3 - dx*t4 + x*ud*t5)*r2;\n"
       "  h[1] = (t1y - t2y*ud - y*t3 - dy*t4 + y*ud*t5)*r2;\n"
       "  h[2] = (t1z - t2z*ud - z*t3 - dz*t4 + z*ud*t5)*r2;\n}\n";
}

struct PairTerm { int my; double c; };

// Path p: M[(mi,mo) pairs] = sum_my c Y[my];  C[mo] = sum_mi x[mi] M[mi,mo];
// X: xb[mi] += sum_mo M[mi,mo] G[mo];  Yb[my] += sum c x[mi] G[mo].
void emit_path(std::ostringstream& o, const Plan& P, int t) {
  const Path& q = P.paths[t];
  const int di = 2 * q.l_in + 1, ds = 2 * q.l_sh + 1, dd = 2 * q.l_out + 1;
  std::vector<std::pair<int, int>> pairs;
  std::vector<std::vector<PairTerm>> terms;
  for (int mi = 0; mi < di; ++mi)
    for (int mo = 0; mo < dd; ++mo) {
      std::vector<PairTerm> tt;
      for (int my = 0; my < ds; ++my) {
        double c = q.cg[((size_t)mi * ds + my) * dd + mo];
        if (std::abs(c) > 1e-14) tt.push_back({my, c});
      }
      if (!tt.empty()) { pairs.push_back({mi, mo}); terms.push_back(tt); }
    }
  const int np = (int)pairs.size();
  o << "// path " << t << ": l_in=" << q.l_in << " l_sh=" << q.l_sh << " l_out=" << q.l_out << " alpha=" << q.alpha
    << "\n#define P" << t << "_NP " << np << "\n";
  o << "SB_DEV void sb_M" << t << "(const float* Y, float* M) {\n";
  for (int k = 0; k < np; ++k) {
    o << "  M[" << k << "] = ";
    for (size_t s = 0; s < terms[k].size(); ++s)
      o << (s ? " + " : "") << fl(terms[k][s].c) << "*Y[" << terms[k][s].my << "]";
    o << ";\n";
  }
  o << "}\nSB_DEV void sb_C" << t << "(const float* x, const float* M, float* C) {\n";
  for (int mo = 0; mo < dd; ++mo) {
    o << "  C[" << mo << "] = 0.0f";
    for (int k = 0; k < np; ++k)
      if (pairs[k].second == mo) o << " + x[" << pairs[k].first << "]*M[" << k << "]";
    o << ";\n";
  }
  o << "}\nSB_DEV void sb_X" << t << "(const float* G, const float* M, float* xb) {\n";
  for (int mi = 0; mi < di; ++mi) {
    bool any = false;
    for (int k = 0; k < np; ++k) any |= pairs[k].first == mi;
    if (!any) continue;
    o << "  xb[" << mi << "] +=";
    bool first = true;
    for (int k = 0; k < np; ++k)
      if (pairs[k].first == mi) { o << (first ? " " : " + ") << "M[" << k << "]*G[" << pairs[k].second << "]"; first = false; }
    o << ";\n";
  }
  o << "}\nSB_DEV void sb_Y" << t << "(const float* x, const float* G, float* yb) {\n";
  for (int my = 0; my < ds; ++my) {
    std::ostringstream e;
    bool first = true;
    for (int k = 0; k < np; ++k)
      for (auto& tt : terms[k])
        if (tt.my == my) {
          e << (first ? " " : " + ") << fl(tt.c) << "*(x[" << pairs[k].first << "]*G[" << pairs[k].second << "])";
          first = false;
        }
    if (!first) o << "  yb[" << my << "] +=" << e.str() << ";\n";
  }
  o << "}\n";
}

int unit_lsh(const Plan& P, const Unit& u) {
  int L = 0;
  for (int t : u.paths) L = std::max(L, P.paths[t].l_sh);
  return L;
}

void emit_fwd_unit(std::ostringstream& o, const Plan& P, const Unit& u, int id) {
  const Irrep& ri = P.in[u.a];
  const int DA = 2 * ri.l + 1, L = unit_lsh(P, u), NS = (L + 1) * (L + 1);
  o << "template <bool TAN>\nSB_DEV void sb_fwd_u" << id
    << "(int lane, int il, int beg, int end, const int* __restrict__ sender, const float* __restrict__ evec,"
       " const float* __restrict__ phi, const float* __restrict__ x, float* __restrict__ S, sb_i64 ncap,"
       " const float* __restrict__ xdot, const float* __restrict__ evdot, const float* __restrict__ phidot, int flags) {\n";
  o << "  constexpr int U = " << u.U << ", U0 = " << u.U0 << ", ES = " << u.ES << ", CA = " << ri.mul
    << ", AOFF = " << ri.off << ";\n";
  o << "  const int sub = lane / U, u = U0 + lane % U;\n"
       "  const bool act = (lane < ES * U) && (u < CA);\n";
  for (int t : u.paths) o << "  float acc" << t << "[K * " << 2 * P.paths[t].l_out + 1 << "] = {};\n";
  o << "  if (act) {\n"
       "    for (int e = beg + sub; e < end; e += ES) {\n"
       "      const float vx = evec[3 * (sb_i64)e], vy = evec[3 * (sb_i64)e + 1], vz = evec[3 * (sb_i64)e + 2];\n"
       "      const float rinv = 1.0f / sqrtf(vx * vx + vy * vy + vz * vz);\n"
       "      const float ux = vx * rinv, uy = vy * rinv, uz = vz * rinv;\n"
    << "      float Y[" << NS << "];\n      sb_sh_eval_L" << L << "(ux, uy, uz, Y);\n"
    << "      float ph[K];\n"
       "#pragma unroll\n      for (int q = 0; q < K; ++q) ph[q] = phi[(sb_i64)e * K + q];\n"
       "      const sb_i64 xrow = (sb_i64)sender[e] * CXI + AOFF + u;\n"
    << "      float xv[" << DA << "];\n"
    << "#pragma unroll\n      for (int m = 0; m < " << DA << "; ++m) xv[m] = x[xrow + m * CA];\n";
  o << "      float Yd[" << NS << "], phd[K], xdv[" << DA << "];\n"
       "      if (TAN) {\n"
       "        if (flags & 4) {\n"
       "          const float dx = evdot[3 * (sb_i64)e], dy = evdot[3 * (sb_i64)e + 1], dz = evdot[3 * (sb_i64)e + 2];\n"
    << "          sb_sh_jvp_L" << L << "(ux, uy, uz, rinv, dx, dy, dz, Y, Yd);\n"
    << "        }\n"
       "        if (flags & 1) {\n#pragma unroll\n          for (int q = 0; q < K; ++q) phd[q] = phidot[(sb_i64)e * K + q];\n        }\n"
       "        if (flags & 2) {\n#pragma unroll\n"
    << "          for (int m = 0; m < " << DA << "; ++m) xdv[m] = xdot[xrow + m * CA];\n        }\n      }\n";
  for (int t : u.paths) {
    const Path& q = P.paths[t];
    const int DO = 2 * q.l_out + 1, Y0 = q.l_sh * q.l_sh;
    o << "      {\n        float M[P" << t << "_NP], C[" << DO << "];\n"
      << "        sb_M" << t << "(Y + " << Y0 << ", M);\n"
      << "        if (!TAN) {\n          sb_C" << t << "(xv, M, C);\n"
      << "#pragma unroll\n          for (int q = 0; q < K; ++q)\n#pragma unroll\n"
      << "            for (int m = 0; m < " << DO << "; ++m) acc" << t << "[q * " << DO << " + m] = fmaf(ph[q], C[m], acc"
      << t << "[q * " << DO << " + m]);\n"
      << "        } else {\n"
      << "          float C2[" << DO << "] = {};\n"
      << "          if (flags & 2) { sb_C" << t << "(xdv, M, C); for (int m = 0; m < " << DO << "; ++m) C2[m] += C[m]; }\n"
      << "          if (flags & 4) { float Md[P" << t << "_NP]; sb_M" << t << "(Yd + " << Y0 << ", Md); sb_C" << t
      << "(xv, Md, C); for (int m = 0; m < " << DO << "; ++m) C2[m] += C[m]; }\n"
      << "#pragma unroll\n          for (int q = 0; q < K; ++q)\n#pragma unroll\n"
      << "            for (int m = 0; m < " << DO << "; ++m) acc" << t << "[q * " << DO << " + m] = fmaf(ph[q], C2[m], acc"
      << t << "[q * " << DO << " + m]);\n"
      << "          if (flags & 1) {\n            sb_C" << t << "(xv, M, C);\n"
      << "#pragma unroll\n            for (int q = 0; q < K; ++q)\n#pragma unroll\n"
      << "              for (int m = 0; m < " << DO << "; ++m) acc" << t << "[q * " << DO << " + m] = fmaf(phd[q], C[m], acc"
      << t << "[q * " << DO << " + m]);\n          }\n        }\n      }\n";
  }
  o << "    }\n  }\n";
  if (u.ES > 1) {
    for (int t : u.paths)
      o << "#pragma unroll\n  for (int v = 0; v < K * " << 2 * P.paths[t].l_out + 1 << "; ++v)\n"
        << "    for (int s = U; s < 64; s <<= 1) acc" << t << "[v] += __shfl_xor(acc" << t << "[v], s);\n";
  }
  o << "  if (act && sub == 0) {\n";
  for (int t : u.paths) {
    const Path& q = P.paths[t];
    const Group& g = P.groups[q.group];
    const int DO = 2 * q.l_out + 1;
    o << "    {\n      float* Sg = S + ncap * " << g.s_off << "LL + (sb_i64)il * " << (int64_t)g.d * g.D << "LL + "
      << q.koff << " + u;\n"
      << "#pragma unroll\n      for (int q = 0; q < K; ++q)\n#pragma unroll\n"
      << "        for (int m = 0; m < " << DO << "; ++m) Sg[(sb_i64)m * " << g.D << " + q * " << q.c_in << "] = acc" << t
      << "[q * " << DO << " + m];\n    }\n";
  }
  o << "  }\n}\n";
}

// Backward / double-backward wave unit of one slab.
void emit_bwd_wave(std::ostringstream& o, const Plan& P, const Unit& u, int s, int w) {
  const Irrep& ri = P.in[u.a];
  const int DA = 2 * ri.l + 1, L = unit_lsh(P, u), NS = (L + 1) * (L + 1);
  const int RW = u.ES > 1 ? u.U : 64;
  o << "template <bool DB>\nSB_DEV void sb_bw_" << s << "_" << w
    << "(int lane, int eb, int nb, int e0, const int* __restrict__ sender, const float* __restrict__ evec,"
       " const float* __restrict__ phi, const float* __restrict__ x, const float* __restrict__ xdot,"
       " const float* __restrict__ evdot, const float* __restrict__ phidot, const float* sS, const float* sS2,"
       " float* spart, float* __restrict__ contrib, int flags) {\n";
  o << "  constexpr int U = " << u.U << ", U0 = " << u.U0 << ", ES = " << u.ES << ", CA = " << ri.mul
    << ", AOFF = " << ri.off << ", RW = " << RW << ";\n"
    << "  constexpr int NV = DB ? (K + 2 * NSH) : (K + NSH);\n"
       "  const int sub = lane / U, uu = lane % U, u = U0 + uu;\n"
       "  const bool act = (lane < ES * U) && (u < CA);\n"
       "  for (int k0 = 0; k0 < nb; k0 += ES) {\n"
       "    const int kk = k0 + sub;\n"
       "    const bool ev = act && kk < nb;\n"
       "    const int e = eb + kk;\n"
       "    float pv[NV];\n#pragma unroll\n    for (int v = 0; v < NV; ++v) pv[v] = 0.f;\n"
    << "    float xc[" << DA << "] = {};\n"
    << "    if (ev) {\n"
       "      const float vx = evec[3 * (sb_i64)e], vy = evec[3 * (sb_i64)e + 1], vz = evec[3 * (sb_i64)e + 2];\n"
       "      const float rinv = 1.0f / sqrtf(vx * vx + vy * vy + vz * vz);\n"
       "      const float ux = vx * rinv, uy = vy * rinv, uz = vz * rinv;\n"
    << "      float Y[" << NS << "];\n      sb_sh_eval_L" << L << "(ux, uy, uz, Y);\n"
    << "      float ph[K];\n#pragma unroll\n      for (int q = 0; q < K; ++q) ph[q] = phi[(sb_i64)e * K + q];\n"
       "      const sb_i64 xrow = (sb_i64)sender[e] * CXI + AOFF + u;\n"
    << "      float xv[" << DA << "];\n#pragma unroll\n      for (int m = 0; m < " << DA << "; ++m) xv[m] = x[xrow + m * CA];\n"
    << "      float Yd[" << NS << "], phd[K], xdv[" << DA << "];\n"
    << "      if (DB) {\n"
       "        if (flags & 4) {\n"
       "          const float dx = evdot[3 * (sb_i64)e], dy = evdot[3 * (sb_i64)e + 1], dz = evdot[3 * (sb_i64)e + 2];\n"
    << "          sb_sh_jvp_L" << L << "(ux, uy, uz, rinv, dx, dy, dz, Y, Yd);\n        }\n"
    << "        if (flags & 1) {\n#pragma unroll\n          for (int q = 0; q < K; ++q) phd[q] = phidot[(sb_i64)e * K + q];\n        }\n"
    << "        if (flags & 2) {\n#pragma unroll\n          for (int m = 0; m < " << DA << "; ++m) xdv[m] = xdot[xrow + m * CA];\n        }\n"
    << "      }\n";
  for (size_t pi = 0; pi < u.paths.size(); ++pi) {
    const int t = u.paths[pi];
    const Path& q = P.paths[t];
    const int DO = 2 * q.l_out + 1, Y0 = q.l_sh * q.l_sh;
    const int lo = u.lds_off[pi];
    o << "      {\n"
      << "        const float* Sp = sS + " << lo << " + uu;\n"
      << "        float M[P" << t << "_NP], C[" << DO << "], G[" << DO << "];\n"
      << "        sb_M" << t << "(Y + " << Y0 << ", M);\n"
      << "#pragma unroll\n        for (int m = 0; m < " << DO << "; ++m) {\n"
      << "          float g = 0.f;\n#pragma unroll\n          for (int q = 0; q < K; ++q) g = fmaf(ph[q], Sp[(q * " << DO
      << " + m) * U], g);\n          G[m] = g;\n        }\n"
      << "        if (!DB) {\n"
      << "          sb_C" << t << "(xv, M, C);\n"
      << "#pragma unroll\n          for (int q = 0; q < K; ++q) {\n            float a = 0.f;\n#pragma unroll\n"
      << "            for (int m = 0; m < " << DO << "; ++m) a = fmaf(Sp[(q * " << DO << " + m) * U], C[m], a);\n"
      << "            pv[q] += a;\n          }\n"
      << "          sb_Y" << t << "(xv, G, pv + K + " << Y0 << ");\n"
      << "          sb_X" << t << "(G, M, xc);\n"
      << "        } else {\n"
      << "          const float* Sp2 = sS2 + " << lo << " + uu;\n"
      << "          float Gd[" << DO << "] = {}, Cd[" << DO << "] = {};\n"
      << "          if (flags & 1) {\n#pragma unroll\n            for (int m = 0; m < " << DO << "; ++m) {\n"
      << "              float g = 0.f;\n#pragma unroll\n              for (int q = 0; q < K; ++q) g = fmaf(phd[q], Sp[(q * " << DO
      << " + m) * U], g);\n              Gd[m] += g;\n            }\n          }\n"
      << "          if (flags & 8) {\n#pragma unroll\n            for (int m = 0; m < " << DO << "; ++m) {\n"
      << "              float g = 0.f;\n#pragma unroll\n              for (int q = 0; q < K; ++q) g = fmaf(ph[q], Sp2[(q * " << DO
      << " + m) * U], g);\n              Gd[m] += g;\n            }\n          }\n"
      << "          float Md[P" << t << "_NP];\n"
      << "          if (flags & 2) { sb_C" << t << "(xdv, M, C); for (int m = 0; m < " << DO << "; ++m) Cd[m] += C[m]; }\n"
      << "          if (flags & 4) { sb_M" << t << "(Yd + " << Y0 << ", Md); sb_C" << t << "(xv, Md, C); for (int m = 0; m < "
      << DO << "; ++m) Cd[m] += C[m]; }\n"
      << "#pragma unroll\n          for (int q = 0; q < K; ++q) {\n            float a = 0.f;\n#pragma unroll\n"
      << "            for (int m = 0; m < " << DO << "; ++m) a = fmaf(Sp[(q * " << DO << " + m) * U], Cd[m], a);\n"
      << "            pv[q] += a;\n          }\n"
      << "          if (flags & 8) {\n            sb_C" << t << "(xv, M, C);\n"
      << "#pragma unroll\n            for (int q = 0; q < K; ++q) {\n              float a = 0.f;\n#pragma unroll\n"
      << "              for (int m = 0; m < " << DO << "; ++m) a = fmaf(Sp2[(q * " << DO << " + m) * U], C[m], a);\n"
      << "              pv[q] += a;\n            }\n          }\n"
      << "          sb_Y" << t << "(xv, Gd, pv + K + " << Y0 << ");\n"
      << "          if (flags & 2) sb_Y" << t << "(xdv, G, pv + K + " << Y0 << ");\n"
      << "          if (flags & 4) sb_Y" << t << "(xv, G, pv + K + NSH + " << Y0 << ");\n"
      << "          sb_X" << t << "(Gd, M, xc);\n"
      << "          if (flags & 4) sb_X" << t << "(G, Md, xc);\n"
      << "        }\n      }\n";
  }
  o << "    }\n"
       "#pragma unroll\n    for (int v = 0; v < NV; ++v)\n"
       "      for (int sft = 1; sft < RW; sft <<= 1) pv[v] += __shfl_xor(pv[v], sft);\n"
       "    if ((lane % RW) == 0 && lane < ES * U && kk < nb) {\n"
    << "#pragma unroll\n      for (int v = 0; v < NV; ++v) spart[(" << w << " * EB + kk) * NV + v] = pv[v];\n    }\n"
    << "    if (ev && contrib) {\n"
       "      float* cr = contrib + (sb_i64)(e - e0) * CXI + AOFF + u;\n"
    << "#pragma unroll\n      for (int m = 0; m < " << DA << "; ++m) cr[m * CA] = " << (u.first ? "xc[m]" : "cr[m * CA] + xc[m]")
    << ";\n    }\n  }\n}\n";
}

}  // namespace

std::string generate_source(const Plan& P) {
  std::ostringstream o;
  o.precision(17);
  o << "\n// ---- generated for: K=" << P.K << " lmax=" << P.lmax << " in=";
  for (auto& r : P.in) o << r.mul << "x" << r.l << (r.p > 0 ? "e" : "o") << " ";
  o << "out=";
  for (auto& r : P.out) o << r.mul << "x" << r.l << (r.p > 0 ? "e" : "o") << " ";
  o << "norm=" << P.norm << "\n";
  o << "#define K " << P.K << "\n#define NSH " << P.nsh << "\n#define CXI " << P.dim_in << "\n#define CXO " << P.dim_out
    << "\n#define EB " << P.bwd_eb << "\n";
  emit_sh(o, P.lmax);
  for (int t = 0; t < (int)P.paths.size(); ++t) emit_path(o, P, t);

  // forward S / dS kernels: one wave per (receiver, unit)
  for (int t = 0; t < (int)P.fwd_units.size(); ++t) emit_fwd_unit(o, P, P.fwd_units[t], t);
  const int NU = (int)P.fwd_units.size();
  for (int tan = 0; tan < 2; ++tan) {
    o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_fwd_" << (tan ? "dS" : "S")
      << "(const int* __restrict__ rowptr, const int* __restrict__ sender, const float* __restrict__ evec,"
         " const float* __restrict__ phi, const float* __restrict__ x, float* __restrict__ S, int r0, int n_recv,"
         " sb_i64 ncap, const float* __restrict__ xdot, const float* __restrict__ evdot,"
         " const float* __restrict__ phidot, int flags) {\n"
      << "  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;\n"
      << "  const int il = gw / " << NU << ", t = gw % " << NU << ";\n"
      << "  if (il >= n_recv) return;\n"
         "  const int beg = rowptr[r0 + il], end = rowptr[r0 + il + 1];\n"
         "  switch (t) {\n";
    for (int t = 0; t < NU; ++t)
      o << "    case " << t << ": sb_fwd_u" << t << "<" << (tan ? "true" : "false")
        << ">(lane, il, beg, end, sender, evec, phi, x, S, ncap, xdot, evdot, phidot, flags); break;\n";
    o << "  }\n}\n";
  }

  // backward / double-backward edge kernels: one block per receiver, slabs of
  // adjoint state staged in LDS, per-edge partials reduced in a fixed order
  for (int s = 0; s < (int)P.slabs.size(); ++s)
    for (int w = 0; w < (int)P.slabs[s].waves.size(); ++w)
      if (P.slabs[s].waves[w].a >= 0) emit_bwd_wave(o, P, P.slabs[s].waves[w], s, w);
  const int LDSF = std::max(1, P.bwd_lds_max);
  o << "template <bool DB>\nSB_DEV void sb_edge_body(const int* __restrict__ rowptr, const int* __restrict__ sender,"
       " const float* __restrict__ evec, const float* __restrict__ phi, const float* __restrict__ x,"
       " const float* __restrict__ Sb, const float* __restrict__ Sb2, const float* __restrict__ xdot,"
       " const float* __restrict__ evdot, const float* __restrict__ phidot, float* __restrict__ gphi,"
       " float* __restrict__ gevec, float* __restrict__ contrib, int r0, int n_recv, sb_i64 ncap, int e0, int flags,"
       " float* sS, float* sS2, float* sacc, float* spart) {\n"
    << "  constexpr int NV = DB ? (K + 2 * NSH) : (K + NSH);\n"
       "  const int il = blockIdx.x;\n"
       "  if (il >= n_recv) return;\n"
       "  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;\n"
       "  const int beg = rowptr[r0 + il], end = rowptr[r0 + il + 1];\n"
       "  for (int eb = beg; eb < end; eb += EB) {\n"
       "    const int nb = min(EB, end - eb);\n"
       "    for (int t = tid; t < EB * NV; t += 256) sacc[t] = 0.f;\n";
  for (int s = 0; s < (int)P.slabs.size(); ++s) {
    const Slab& sl = P.slabs[s];
    o << "    // slab " << s << "\n    __syncthreads();\n";
    for (int w = 0; w < (int)sl.waves.size(); ++w) {
      const Unit& u = sl.waves[w];
      if (u.a < 0) continue;
      for (size_t pi = 0; pi < u.paths.size(); ++pi) {
        const Path& q = P.paths[u.paths[pi]];
        const Group& g = P.groups[q.group];
        const int DO = 2 * q.l_out + 1, n = P.K * DO * u.U;
        o << "    for (int t = tid; t < " << n << "; t += 256) {\n"
          << "      const int q = t / " << DO * u.U << ", r = t % " << DO * u.U << ", m = r / " << u.U << ", uu = r % "
          << u.U << ";\n"
          << "      const int uc = " << u.U0 << " + uu;\n"
          << "      const sb_i64 src = ncap * " << g.s_off << "LL + ((sb_i64)il * " << g.d << " + m) * " << g.D << "LL + "
          << q.koff << " + q * " << q.c_in << " + uc;\n"
          << "      sS[" << u.lds_off[pi] << " + t] = (uc < " << q.c_in << ") ? Sb[src] : 0.f;\n"
          << "      if (DB && (flags & 8)) sS2[" << u.lds_off[pi] << " + t] = (uc < " << q.c_in << ") ? Sb2[src] : 0.f;\n"
          << "    }\n";
      }
    }
    o << "    __syncthreads();\n    switch (wave) {\n";
    for (int w = 0; w < (int)sl.waves.size(); ++w)
      if (sl.waves[w].a >= 0)
        o << "      case " << w << ": sb_bw_" << s << "_" << w
          << "<DB>(lane, eb, nb, e0, sender, evec, phi, x, xdot, evdot, phidot, sS, sS2, spart, contrib, flags); break;\n";
    o << "      default: break;\n    }\n    __syncthreads();\n"
      << "    for (int t = tid; t < nb * NV; t += 256) {\n      float s = 0.f;\n";
    for (int w = 0; w < (int)sl.waves.size(); ++w)
      if (sl.waves[w].a >= 0) o << "      s += spart[" << w << " * EB * NV + t];\n";
    o << "      sacc[t] += s;\n    }\n";
  }
  o << "    __syncthreads();\n";
  // zero contributions of input irreps that no path reads
  for (int a : P.dead_in) {
    o << "    if (contrib) for (int t = tid; t < nb * " << P.in[a].dim() << "; t += 256)\n"
      << "      contrib[(sb_i64)(eb + t / " << P.in[a].dim() << " - e0) * CXI + " << P.in[a].off << " + t % "
      << P.in[a].dim() << "] = 0.f;\n";
  }
  o << "    if (tid < nb) {\n"
       "      const int e = eb + tid;\n"
       "      const float* a = sacc + tid * NV;\n"
       "      if (gphi) {\n#pragma unroll\n        for (int q = 0; q < K; ++q) gphi[(sb_i64)e * K + q] = a[q];\n      }\n"
       "      if (gevec) {\n"
       "        const float vx = evec[3 * (sb_i64)e], vy = evec[3 * (sb_i64)e + 1], vz = evec[3 * (sb_i64)e + 2];\n"
       "        const float rinv = 1.0f / sqrtf(vx * vx + vy * vy + vz * vz);\n"
       "        const float ux = vx * rinv, uy = vy * rinv, uz = vz * rinv;\n"
       "        float g[3];\n"
       "        sb_sh_vjp(ux, uy, uz, rinv, a + K, g);\n"
       "        if (DB && (flags & 4)) {\n"
       "          float h[3];\n"
       "          sb_sh_hvp(ux, uy, uz, rinv, a + K + NSH, evdot[3 * (sb_i64)e], evdot[3 * (sb_i64)e + 1],"
       " evdot[3 * (sb_i64)e + 2], h);\n"
       "          g[0] += h[0]; g[1] += h[1]; g[2] += h[2];\n"
       "        }\n"
       "        gevec[3 * (sb_i64)e] = g[0]; gevec[3 * (sb_i64)e + 1] = g[1]; gevec[3 * (sb_i64)e + 2] = g[2];\n"
       "      }\n"
       "    }\n"
       "    __syncthreads();\n"
       "  }\n}\n";
  for (int db = 0; db < 2; ++db) {
    o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_" << (db ? "dbwd" : "bwd")
      << "_E(const int* __restrict__ rowptr, const int* __restrict__ sender, const float* __restrict__ evec,"
         " const float* __restrict__ phi, const float* __restrict__ x, const float* __restrict__ Sb,"
         " const float* __restrict__ Sb2, const float* __restrict__ xdot, const float* __restrict__ evdot,"
         " const float* __restrict__ phidot, float* __restrict__ gphi, float* __restrict__ gevec,"
         " float* __restrict__ contrib, int r0, int n_recv, sb_i64 ncap, int e0, int flags) {\n"
      << "  constexpr int NV = " << (db ? "K + 2 * NSH" : "K + NSH") << ";\n"
      << "  __shared__ float sS[" << LDSF * (db ? 2 : 1) << "];\n"
      << "  __shared__ float sacc[EB * NV];\n  __shared__ float spart[4 * EB * NV];\n"
      << "  sb_edge_body<" << (db ? "true" : "false")
      << ">(rowptr, sender, evec, phi, x, Sb, Sb2, xdot, evdot, phidot, gphi, gevec, contrib, r0, n_recv, ncap, e0,"
         " flags, sS, sS + " << (db ? LDSF : 0) << ", sacc, spart);\n}\n";
  }
  return o.str();
}

}  // namespace sobek
