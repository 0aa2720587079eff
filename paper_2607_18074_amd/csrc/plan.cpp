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
// device/gemm_bf16.hip, embedded by the build
const char* kGemmBf16 =
#include "gemm_bf16_embed.inc"
    ;

constexpr int kAccMax = 128;        // forward accumulators per lane per wave unit
constexpr int kFetchRing = 2;       // forward edge-data register sets in flight
constexpr int kSlabFloats = 10240;  // backward LDS budget for one slab of adjoint state (40 KiB)
constexpr int kAdjWaves = 2;        // waves per adjoint block

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

// Forward wave units: per input irrep and channel block, the paths (all of them, or those into
// output group `group` only) packed while K * sum(d_out) accumulators fit the register budget.
std::vector<Unit> pack_fwd_units(const Plan& p, int group, std::vector<int>* dead_in) {
  std::vector<Unit> units;
  for (int a = 0; a < (int)p.in.size(); ++a) {
    std::vector<int> ps;
    for (int t = 0; t < (int)p.paths.size(); ++t)
      if (p.paths[t].i_in == a && (group < 0 || p.paths[t].group == group)) ps.push_back(t);
    if (ps.empty()) {
      if (dead_in) dead_in->push_back(a);
      continue;
    }
    for (auto blk : channel_blocks(p.in[a].mul)) {
      Unit cur;
      cur.a = a; cur.U = blk[0]; cur.U0 = blk[1]; cur.ES = blk[2];
      int acc = 0;
      for (int t : ps) {
        int need = p.K * (2 * p.paths[t].l_out + 1);
        if (!cur.paths.empty() && acc + need > kAccMax) {
          units.push_back(cur);
          cur.paths.clear();
          acc = 0;
        }
        cur.paths.push_back(t);
        acc += need;
      }
      units.push_back(cur);
    }
  }
  return units;
}

void build_plan(Plan& p) {
  int off = 0;
  for (auto& r : p.in) { r.off = off; off += r.dim(); }
  p.dim_in = off;
  off = 0;
  for (auto& r : p.out) { r.off = off; off += r.dim(); }
  p.dim_out = off;
  p.nsh = (p.lmax + 1) * (p.lmax + 1);
  p.vec4 = true;
  for (auto& r : p.in) p.vec4 = p.vec4 && r.mul % 4 == 0;
  for (auto& r : p.out) p.vec4 = p.vec4 && r.mul % 4 == 0;

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
        if (p.mode == 1 && ro.mul != ri.mul)
          throw std::invalid_argument("uvu path " + std::to_string(a) + " -> " + std::to_string(c) +
                                      " needs equal input and output multiplicities");
        Path q;
        q.i_in = a; q.i_sh = b; q.i_out = c;
        q.l_in = ri.l; q.l_sh = b; q.l_out = ro.l;
        q.c_in = ri.mul; q.c_out = ro.mul;
        q.w_off = woff;
        woff += p.mode == 1 ? (int64_t)ri.mul : (int64_t)ri.mul * ro.mul;
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
    for (int t : ps) fan += p.mode == 1 ? 1 : p.paths[t].c_in;  // terms summed into one output channel
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
        for (int u = 0; u < q.c_in; ++u)  // W row of (q, path, u): uvw mixes C_out columns from it, uvu reads one
          p.ktab.push_back((int32_t)(qq * p.n_w + q.w_off + (int64_t)u * (p.mode == 1 ? 1 : q.c_out)));
    }
  }
  p.srow = soff;
  p.uvu_C = 0;
  if (p.mode == 1) {
    int C = p.paths.empty() ? 0 : p.paths[0].c_in;
    for (auto& q : p.paths) if (q.c_in != C || q.c_out != C) C = 0;
    // the kernels stage A [path][q][64 channels] in LDS: keep it within 96 KB
    if ((int64_t)p.paths.size() * p.K * std::min(C, 64) * 4 > 96 * 1024) C = 0;
    p.uvu_C = C;
    p.uvu_NB = C > 0 ? (C + 63) / 64 : 0;
    p.uvu_NA = 0;
    for (size_t a = 0; a < p.in.size(); ++a)
      for (auto& q : p.paths)
        if (q.i_in == (int)a) { ++p.uvu_NA; break; }
  }
  for (auto& q : p.paths) {
    const std::vector<double>& Q = real_cg(q.l_in, q.l_sh, q.l_out);
    q.cg.resize(Q.size());
    for (size_t t = 0; t < Q.size(); ++t) q.cg[t] = q.alpha * Q[t];
  }

  // forward wave units: per input irrep and channel block, paths packed while
  // K * sum(d_out) accumulators fit the register budget
  p.fwd_units = pack_fwd_units(p, -1, &p.dead_in);

  // adjoint tiles: 16 channels per item, radial index padded to a multiple of 4
  p.adj_U = 16;
  p.adj_KP = (p.K + 3) / 4 * 4;
  p.adj_waves = kAdjWaves;
  p.bwd_eb = 16 * kAdjWaves * 2;
  auto slice = [&](int t) { return p.adj_KP * (2 * p.paths[t].l_out + 1) * p.adj_U; };
  // items (input irrep, channel tile, path chunk) packed into LDS slabs in order
  p.slabs.clear();
  std::vector<AdjItem> items;
  std::vector<int> item_floats;
  for (int a = 0; a < (int)p.in.size(); ++a) {
    std::vector<int> ps;
    for (int t = 0; t < (int)p.paths.size(); ++t)
      if (p.paths[t].i_in == a) ps.push_back(t);
    if (ps.empty()) continue;
    for (int u0 = 0; u0 < p.in[a].mul; u0 += p.adj_U) {
      AdjItem cur;
      cur.a = a; cur.u0 = u0;
      int fl = 0;
      bool first = true;
      for (int t : ps) {
        int need = slice(t);
        if (need > kSlabFloats) throw std::runtime_error("path adjoint slice exceeds the LDS slab budget");
        if (!cur.paths.empty() && fl + need > kSlabFloats) {
          cur.first = first;
          first = false;
          items.push_back(cur);
          item_floats.push_back(fl);
          cur.paths.clear();
          fl = 0;
        }
        cur.paths.push_back(t);
        fl += need;
      }
      cur.first = first;
      items.push_back(cur);
      item_floats.push_back(fl);
    }
  }
  {
    AdjSlab cur;
    for (size_t i = 0; i < items.size(); ++i) {
      if (!cur.items.empty() && cur.floats + item_floats[i] > kSlabFloats) {
        p.slabs.push_back(cur);
        cur = AdjSlab();
      }
      AdjItem it = items[i];
      int o = cur.floats;
      for (int t : it.paths) {
        it.lds_off.push_back(o);
        o += slice(t);
      }
      cur.items.push_back(it);
      cur.floats = o;
    }
    if (!cur.items.empty()) p.slabs.push_back(cur);
  }
  p.bwd_lds_max = 0;
  for (auto& s : p.slabs) p.bwd_lds_max = std::max(p.bwd_lds_max, s.floats);
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

// Sparse structure of a path's coupling: the (m_i, m_o) pairs with a nonzero
// coefficient, each with its (m_y, c) terms.
struct PathTerms {
  std::vector<std::pair<int, int>> pairs;
  std::vector<std::vector<PairTerm>> terms;
};

PathTerms path_terms(const Path& q) {
  const int di = 2 * q.l_in + 1, ds = 2 * q.l_sh + 1, dd = 2 * q.l_out + 1;
  PathTerms r;
  for (int mi = 0; mi < di; ++mi)
    for (int mo = 0; mo < dd; ++mo) {
      std::vector<PairTerm> tt;
      for (int my = 0; my < ds; ++my) {
        double c = q.cg[((size_t)mi * ds + my) * dd + mo];
        if (std::abs(c) > 1e-14) tt.push_back({my, c});
      }
      if (!tt.empty()) { r.pairs.push_back({mi, mo}); r.terms.push_back(tt); }
    }
  return r;
}

// Path p: M[(mi,mo) pairs] = sum_my c Y[my];  C[mo] = sum_mi x[mi] M[mi,mo].
void emit_path(std::ostringstream& o, const Plan& P, int t) {
  const Path& q = P.paths[t];
  const int dd = 2 * q.l_out + 1;
  const PathTerms pt = path_terms(q);
  const std::vector<std::pair<int, int>>& pairs = pt.pairs;
  const std::vector<std::vector<PairTerm>>& terms = pt.terms;
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
    o << "  C[" << mo << "] =";
    bool any = false;
    for (int k = 0; k < np; ++k)
      if (pairs[k].second == mo) { o << (any ? " + " : " ") << "x[" << pairs[k].first << "]*M[" << k << "]"; any = true; }
    o << (any ? ";\n" : " 0.0f;\n");
  }
  o << "}\n";
}

int unit_lsh(const Plan& P, const Unit& u) {
  int L = 0;
  for (int t : u.paths) L = std::max(L, P.paths[t].l_sh);
  return L;
}

// Forward state (S) or directional state (dS) of one wave unit.  Lane = sub * U + u:
// ES edges in flight, one input channel u per lane.  Every lane runs the same
// number of edge iterations: a lane past the receiver's last edge takes that
// edge again with zero radial features, so the rank-1 accumulation
// S[u, q] += C[u] phi[q] can run on v_mfma_f32_4x4x1_16b_f32 when U and K are
// multiples of 4: each 4-lane block multiplies its 4 channel values (A) by a
// quad of radial features (B), and lane 4b + j, register i accumulates
// S[u = 4b + i][q = 4 qq + j].  Otherwise it runs on the VALU, one channel per
// lane.  Edge data is fetched three iterations ahead into a ring of three
// register sets (the loop is unrolled by three, so no set is ever copied): while
// one iteration is computed, the loads of the next two are in flight.  The
// receiver's sender ids are held 64 at a time in one register per lane, the
// next block already loaded, and handed to the lanes of an edge by a shuffle.
void emit_fwd_unit(std::ostringstream& o, const Plan& P, const Unit& u, int id, bool group_only = false) {
  const Irrep& ri = P.in[u.a];
  const char* st = P.dtype == 1 ? "__bf16" : "float";  // the state's storage type (bf16 for bf16-GEMM plans)
  const int DA = 2 * ri.l + 1, L = unit_lsh(P, u), NS = (L + 1) * (L + 1);
  const bool mf = (u.U % 4 == 0) && (P.K % 4 == 0);
  const int KQ = P.K / 4;
  const int NPH = mf ? KQ : P.K;
  o << "template <bool TAN, int FL>\nSB_DEV void sb_fwd_u" << id
    << "(int lane, int il, int beg, int end, const int* __restrict__ sender, const float* __restrict__ evec,"
       " const float* __restrict__ phi, const float* __restrict__ x, " << st << "* __restrict__ S, sb_i64 ncap,"
       " const float* __restrict__ xdot, const float* __restrict__ evdot, const float* __restrict__ phidot, int flags,"
       " int* ids) {\n";
  o << "  const int fl = FL >= 0 ? FL : flags;\n";
  o << "  constexpr int U = " << u.U << ", U0 = " << u.U0 << ", ES = " << u.ES << ", CA = " << ri.mul
    << ", AOFF = " << ri.off << ", DA = " << DA << ", NPH = " << NPH << ";\n";
  o << "  const int sub = lane / U, u = U0 + lane % U;\n"
       "  const int sl = sub < ES ? sub : ES - 1, uu = u < CA ? u : CA - 1;\n"
       "  const int deg = end - beg;\n";
  for (int t : u.paths) {
    const int DO = 2 * P.paths[t].l_out + 1;
    if (mf)
      o << "  sb_f4 acc" << t << "[" << DO * KQ << "];\n"
        << "#pragma unroll\n  for (int v = 0; v < " << DO * KQ << "; ++v) acc" << t << "[v] = (sb_f4){0.f, 0.f, 0.f, 0.f};\n";
    else
      o << "  float acc" << t << "[K * " << DO << "] = {};\n";
  }
  // The receiver's edges are taken in segments of up to 256.  A segment's
  // sender ids go to this wave's LDS slice first (clamped addresses: every load
  // is in bounds); read back with LDS loads, they never make the edge loop wait
  // on its own global loads.
  o << "  for (int seg = 0; seg < deg; seg += 256) {\n"
       "  const int sdeg = min(256, deg - seg), sbeg = beg + seg;\n"
       "  const int niter = (sdeg + ES - 1) / ES;\n"
       "#pragma unroll\n  for (int i = 0; i < 4; ++i) ids[64 * i + lane] = sender[sbeg + min(64 * i + lane, sdeg - 1)];\n";
  const std::string pidx = mf ? "e * K + 4 * q + (lane & 3)" : "e * K + q";
  // edge data of ring slot r for iteration `itn`; the edge weight w is applied
  // at use, so nothing here waits for a load
  auto fetch = [&](int r, const std::string& itn) {
    const std::string R = std::to_string(r);
    o << "    {\n"
         "      const int kb = (" << itn << ") * ES;\n"
         "      const int k = kb + sl;\n"
         "      const int kc = k < sdeg ? k : sdeg - 1;\n"
         "      w" << R << " = k < sdeg ? 1.f : 0.f;\n"
         "      const int j = ids[kc];\n"
         "      const sb_i64 e = sbeg + kc;\n"
         "      vx" << R << " = evec[3 * e]; vy" << R << " = evec[3 * e + 1]; vz" << R << " = evec[3 * e + 2];\n"
         "      if (TAN && (fl & 4)) { dx" << R << " = evdot[3 * e]; dy" << R << " = evdot[3 * e + 1]; dz" << R
      << " = evdot[3 * e + 2]; }\n"
         "#pragma unroll\n      for (int q = 0; q < NPH; ++q) pa" << R << "[q] = phi[" << pidx << "];\n"
         "      if (TAN && (fl & 1)) {\n"
         "#pragma unroll\n        for (int q = 0; q < NPH; ++q) pd" << R << "[q] = phidot[" << pidx << "];\n"
         "      }\n";
    o << "      const sb_i64 xrow = (sb_i64)j * CXI + AOFF + uu;\n"
         "#pragma unroll\n      for (int m = 0; m < DA; ++m) xa" << R << "[m] = x[xrow + m * CA];\n"
         "      if (TAN && (fl & 2)) {\n"
         "#pragma unroll\n        for (int m = 0; m < DA; ++m) xd" << R << "[m] = xdot[xrow + m * CA];\n"
         "      }\n"
         "    }\n";
  };
  auto compute = [&](int r) {
    const std::string R = std::to_string(r);
    o << "    {\n"
         "      float ph[NPH], phd[NPH];\n"
         "#pragma unroll\n      for (int q = 0; q < NPH; ++q) {\n"
         "        ph[q] = pa" << R << "[q] * w" << R << ";\n"
         "        phd[q] = (TAN && (fl & 1)) ? pd" << R << "[q] * w" << R << " : 0.f;\n"
         "      }\n"
         "      const float rinv = __builtin_amdgcn_rsqf(vx" << R << " * vx" << R << " + vy" << R << " * vy" << R << " + vz" << R
      << " * vz" << R << ");\n"
         "      const float ux = vx" << R << " * rinv, uy = vy" << R << " * rinv, uz = vz" << R << " * rinv;\n"
      << "      float Y[" << NS << "], Yd[" << NS << "];\n      sb_sh_eval_L" << L << "(ux, uy, uz, Y);\n"
      << "      if (TAN && (fl & 4)) sb_sh_jvp_L" << L << "(ux, uy, uz, rinv, dx" << R << ", dy" << R << ", dz" << R
      << ", Y, Yd);\n";
    for (int t : u.paths) {
      const Path& q = P.paths[t];
      const int DO = 2 * q.l_out + 1, Y0 = q.l_sh * q.l_sh;
      o << "      {  // path " << t << "\n"
        << "        constexpr int DO = " << DO << ";\n"
        << "        float M[P" << t << "_NP], C[DO], C2[DO];\n"
        << "        sb_M" << t << "(Y + " << Y0 << ", M);\n"
        << "        if (!TAN) {\n          sb_C" << t << "(xa" << R << ", M, C2);\n        } else {\n"
        << "#pragma unroll\n          for (int m = 0; m < DO; ++m) C2[m] = 0.f;\n"
        << "          if (fl & 2) { sb_C" << t << "(xd" << R << ", M, C); for (int m = 0; m < DO; ++m) C2[m] += C[m]; }\n"
        << "          if (fl & 4) { float Md[P" << t << "_NP]; sb_M" << t << "(Yd + " << Y0 << ", Md); sb_C" << t
        << "(xa" << R << ", Md, C); for (int m = 0; m < DO; ++m) C2[m] += C[m]; }\n"
        << "          if (fl & 1) sb_C" << t << "(xa" << R << ", M, C);\n"
        << "        }\n";
      if (mf) {
        o << "#pragma unroll\n        for (int m = 0; m < DO; ++m)\n#pragma unroll\n"
          << "          for (int qq = 0; qq < " << KQ << "; ++qq) {\n"
          << "            acc" << t << "[m * " << KQ << " + qq] = __builtin_amdgcn_mfma_f32_4x4x1f32(C2[m], ph[qq], acc" << t
          << "[m * " << KQ << " + qq], 0, 0, 0);\n"
          << "            if (TAN && (fl & 1)) acc" << t << "[m * " << KQ
          << " + qq] = __builtin_amdgcn_mfma_f32_4x4x1f32(C[m], phd[qq], acc" << t << "[m * " << KQ << " + qq], 0, 0, 0);\n"
          << "          }\n";
      } else {
        o << "#pragma unroll\n        for (int q = 0; q < K; ++q)\n#pragma unroll\n"
          << "          for (int m = 0; m < DO; ++m) {\n"
          << "            acc" << t << "[q * DO + m] = fmaf(ph[q], C2[m], acc" << t << "[q * DO + m]);\n"
          << "            if (TAN && (fl & 1)) acc" << t << "[q * DO + m] = fmaf(phd[q], C[m], acc" << t << "[q * DO + m]);\n"
          << "          }\n";
      }
      o << "      }\n";
    }
    o << "    }\n";
  };
  // ring of register sets: slot r holds iteration it + r; fetches past the last
  // iteration re-read the last edge with weight 0, which keeps them unconditional
  // and the number of loads in flight the same on every path
  const int NR = kFetchRing;
  o << "  {\n";
  for (int r = 0; r < NR; ++r)
    o << "    float vx" << r << ", vy" << r << ", vz" << r << ", dx" << r << " = 0.f, dy" << r << " = 0.f, dz" << r
      << " = 0.f, w" << r << ", xa" << r << "[DA], xd" << r << "[DA], pa" << r << "[NPH], pd" << r << "[NPH];\n";
  for (int r = 0; r < NR; ++r) fetch(r, std::to_string(r));
  o << "    int it = 0;\n    for (; it + " << NR << " <= niter; it += " << NR << ") {\n";
  for (int r = 0; r < NR; ++r) {
    compute(r);
    fetch(r, "it + " + std::to_string(NR + r));
  }
  o << "    }\n";
  for (int r = 0; r + 1 < NR; ++r) {
    o << "    if (it + " << r << " < niter) {\n";
    compute(r);
    o << "    }\n";
  }
  o << "  }\n  }  // segment\n";
  if (u.ES > 1) {
    for (int t : u.paths) {
      const int DO = 2 * P.paths[t].l_out + 1;
      if (mf)
        o << "#pragma unroll\n  for (int v = 0; v < " << DO * KQ << "; ++v)\n#pragma unroll\n    for (int i = 0; i < 4; ++i)\n"
          << "      for (int s = U; s < 64; s <<= 1) acc" << t << "[v][i] += __shfl_xor(acc" << t << "[v][i], s);\n";
      else
        o << "#pragma unroll\n  for (int v = 0; v < K * " << DO << "; ++v)\n"
          << "    for (int s = U; s < 64; s <<= 1) acc" << t << "[v] += __shfl_xor(acc" << t << "[v], s);\n";
    }
  }
  o << "  if (sub == 0 && lane < U) {\n";
  for (int t : u.paths) {
    const Path& q = P.paths[t];
    const Group& g = P.groups[q.group];
    const int DO = 2 * q.l_out + 1;
    o << "    {\n      constexpr int DO = " << DO << ";\n      " << st << "* Sg = S + ncap * " << (group_only ? 0 : g.s_off)
      << "LL + (sb_i64)il * " << (int64_t)g.d * g.D << "LL + " << q.koff << ";\n";
    if (mf) {
      o << "      const int ub = U0 + 4 * ((lane % U) >> 2), j = lane & 3;\n"
        << "#pragma unroll\n      for (int m = 0; m < DO; ++m)\n#pragma unroll\n"
        << "        for (int qq = 0; qq < " << KQ << "; ++qq)\n#pragma unroll\n"
        << "          for (int i = 0; i < 4; ++i)\n"
        << "            if (ub + i < CA) Sg[(sb_i64)m * " << g.D << " + (4 * qq + j) * " << q.c_in << " + ub + i] = acc" << t
        << "[m * " << KQ << " + qq][i];\n";
    } else {
      o << "      if (u < CA) {\n#pragma unroll\n        for (int q = 0; q < K; ++q)\n#pragma unroll\n"
        << "          for (int m = 0; m < DO; ++m) Sg[(sb_i64)m * " << g.D << " + q * " << q.c_in << " + u] = acc" << t
        << "[q * DO + m];\n      }\n";
    }
    o << "    }\n";
  }
  o << "  }\n}\n\n";
}

// One path of an adjoint item, output component by output component so that
// only one m_o's coupling values, channel values and G tile are live at a time.
// For output component m the lane computes, for its edge and its 4 channels r:
//   M_k = sum c Y[m_y]               (pairs k = (m_i, m) of the path)
//   G[r] = sum_q phi[q] Sbar[q][m][u_r]                       (16x16x4 MFMA)
//   C[r] = sum_k x[r][m_i] M_k;  phibar[q] += Sbar[q][m][u_r] C[r]  (4x4x1)
//   xbar[r][m_i] += M_k G[r];   Ybar[m_y] += c sum_r x[r][m_i] G[r]
// and the double-backward analogues with the tangents of Y, phi, x and A.
// One (path, m_o) block of an adjoint slab: the unit whose adjoint-state
// operands are loaded from LDS together.
struct AdjBlock {
  int t, off, DO, m;
};

// The blocks of a slab in emission order (items, their paths, output components
// with a nonzero coupling).
std::vector<AdjBlock> adj_blocks(const Plan& P, const AdjSlab& sl) {
  std::vector<AdjBlock> v;
  for (const AdjItem& it : sl.items)
    for (size_t pi = 0; pi < it.paths.size(); ++pi) {
      const Path& q = P.paths[it.paths[pi]];
      const PathTerms pt = path_terms(q);
      const int DO = 2 * q.l_out + 1;
      for (int m = 0; m < DO; ++m) {
        bool any = false;
        for (auto& pr : pt.pairs) any = any || pr.second == m;
        if (any) v.push_back({it.paths[pi], it.lds_off[pi], DO, m});
      }
    }
  return v;
}

// Backward (DB = false) block pipeline.  Block b's G tile (sum_q phi[q] Sbar[q][m][u],
// 16x16x4 MFMA) is issued by block b - 1 (by the iteration start for b = 0), from
// operands gA<b> that block b - 2 loaded from LDS; so each block's VALU work finds
// its G tile finished and overlaps the next block's MFMAs.  The double-backward
// kernels keep more per-edge state live and compute G in-block from LDS.
void emit_adj_gload(std::ostringstream& o, const std::vector<AdjBlock>& bl, int b, const char* ind) {
  const AdjBlock& x = bl[b];
  o << ind << "if (!DB) {\n"
    << "#pragma unroll\n" << ind << "  for (int v = 0; v < KQ; ++v) gA" << b << "[v] = (sS + " << x.off << " + zz)[((4 * v + g) * "
    << x.DO << " + " << x.m << ") * 16 + es];\n" << ind << "}\n";
}

void emit_adj_gtile(std::ostringstream& o, int b, const char* ind) {
  o << ind << "if (!DB) {\n" << ind << "  G" << b << " = (sb_f4){0.f, 0.f, 0.f, 0.f};\n"
    << "#pragma unroll\n" << ind << "  for (int v = 0; v < KQ; ++v) G" << b << " = sb_mfma(gA" << b << "[v], phB[v], G" << b
    << ");\n" << ind << "}\n";
}

// Path t of an adjoint item; `bl`/`b` are the slab's blocks and the index of the
// path's first block, advanced past its blocks.  A block's adjoint-state operands
// are in registers when it starts (loaded by the previous block, the last block
// loading the first one's for the next iteration), so no block waits on LDS.
void emit_adj_path(std::ostringstream& o, const Plan& P, int t, int off, const std::vector<AdjBlock>& bl, int& b) {
  const Path& q = P.paths[t];
  const int DO = 2 * q.l_out + 1, Y0 = q.l_sh * q.l_sh;
  const PathTerms pt = path_terms(q);
  auto yexpr = [&](const std::vector<PairTerm>& tt, const char* Yn) {
    std::ostringstream e;
    for (size_t j = 0; j < tt.size(); ++j) e << (j ? " + " : "") << fl(tt[j].c) << "*" << Yn << "[" << Y0 + tt[j].my << "]";
    return e.str();
  };
  auto cexpr = [&](const std::vector<int>& ks, const char* xn, const char* Mn, int r) {
    std::ostringstream e;
    for (size_t j = 0; j < ks.size(); ++j)
      e << (j ? " + " : "") << xn << "[" << r << "][" << pt.pairs[ks[j]].first << "]*" << Mn << ks[j];
    return e.str();
  };
  // G tile of component m against radial features `ph` and adjoint state `sp`
  auto gtile = [&](const char* dst, const char* sp, const char* ph, int m) {
    std::ostringstream e;
    e << "#pragma unroll\n            for (int v = 0; v < KQ; ++v) " << dst << " = sb_mfma(" << sp << "[((4 * v + g) * " << DO
        << " + " << m << ") * 16 + es], " << ph << "[v], " << dst << ");\n";
    return e.str();
  };
  // phibar[q] += sum_r Sbar[q][m][u_r] c[r]
  auto ptile = [&](const char* sp, const char* cn, int m) {
    std::ostringstream e;
    e << "#pragma unroll\n            for (int v = 0; v < KQ; ++v) {\n";
    if (std::string(sp) == "Sp")  // the backward loaded this block's operands at its start
      e << "              const sb_f4 a = DB ? *(const sb_f4*)(" << sp << " + ((4 * v + l3) * " << DO << " + " << m
        << ") * 16 + 4 * g) : pA[v];\n";
    else
      e << "              const sb_f4 a = *(const sb_f4*)(" << sp << " + ((4 * v + l3) * " << DO << " + " << m << ") * 16 + 4 * g);\n";
    e
      << "              pacc[v] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[0], " << cn << "0, pacc[v], 0, 0, 0);\n"
      << "              pacc[v] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[1], " << cn << "1, pacc[v], 0, 0, 0);\n"
      << "              pacc[v] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[2], " << cn << "2, pacc[v], 0, 0, 0);\n"
      << "              pacc[v] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[3], " << cn << "3, pacc[v], 0, 0, 0);\n"
      << "            }\n";
    return e.str();
  };
  // xbar[r][m_i] += Mk G[r] over the pairs
  auto xupd = [&](const std::vector<int>& ks, const char* Mn, const char* Gn) {
    std::ostringstream e;
    for (int k : ks)
      for (int r = 0; r < 4; ++r)
        e << "            xc[" << r << "][" << pt.pairs[k].first << "] = fmaf(" << Mn << k << ", " << Gn << "[" << r
          << "], xc[" << r << "][" << pt.pairs[k].first << "]);\n";
    return e.str();
  };
  // acc[Y0 + m_y] += c sum_r xs[r][m_i] G[r]
  auto yupd = [&](const std::vector<int>& ks, const char* xs, const char* Gn, const char* acc) {
    std::ostringstream e;
    for (int k : ks) {
      const int mi = pt.pairs[k].first;
      e << "            {\n              float pp = " << xs << "[0][" << mi << "] * " << Gn << "[0];\n";
      for (int r = 1; r < 4; ++r)
        e << "              pp = fmaf(" << xs << "[" << r << "][" << mi << "], " << Gn << "[" << r << "], pp);\n";
      for (auto& tt : pt.terms[k])
        e << "              " << acc << "[" << Y0 + tt.my << "] = fmaf(" << fl(tt.c) << ", pp, " << acc << "[" << Y0 + tt.my
          << "]);\n";
      e << "            }\n";
    }
    return e.str();
  };
  o << "      {  // path " << t << ": l_in=" << q.l_in << " l_sh=" << q.l_sh << " l_out=" << q.l_out << "\n"
    << "        const float* Sp = sS + " << off << " + zz;\n"
    << "        const float* Sp2 = sS2 + " << off << " + zz;\n"
    << "        (void)Sp2;\n";
  for (int m = 0; m < DO; ++m) {
    std::vector<int> ks;
    for (int k = 0; k < (int)pt.pairs.size(); ++k)
      if (pt.pairs[k].second == m) ks.push_back(k);
    if (ks.empty()) continue;
    if (bl[b].t != t || bl[b].m != m) throw std::runtime_error("adjoint block order mismatch");
    const int nbk = (int)bl.size();
    o << "        {  // m_o = " << m << "\n";
    // backward pipeline: operands two blocks ahead, the next block's G tile, this block's 4x4x1 operands
    emit_adj_gload(o, bl, (b + 2) % nbk, "          ");
    if (b + 1 < nbk) emit_adj_gtile(o, b + 1, "          ");
    o << "          sb_f4 pA[KQ];\n"
      << "          if (!DB) {\n"
      << "#pragma unroll\n            for (int v = 0; v < KQ; ++v) pA[v] = *(const sb_f4*)(Sp + ((4 * v + l3) * " << DO << " + "
      << m << ") * 16 + 4 * g);\n"
      << "          }\n";
    for (int k : ks) o << "          const float M" << k << " = " << yexpr(pt.terms[k], "Y") << ";\n";
    o << "          sb_f4 G = (sb_f4){0.f, 0.f, 0.f, 0.f};\n"
      << "          if (!DB) {\n            G = G" << b << ";\n          } else {\n  " << gtile("G", "Sp", "phB", m)
      << "          }\n";
    o << "          if (!DB) {\n";
    for (int r = 0; r < 4; ++r) o << "            const float c" << r << " = " << cexpr(ks, "xv", "M", r) << ";\n";
    o << ptile("Sp", "c", m) << xupd(ks, "M", "G") << yupd(ks, "xv", "G", "gy");
    o << "          } else {\n";
    for (int k : ks) o << "            float D" << k << " = 0.f;\n";
    o << "            if (fl & 4) {\n";
    for (int k : ks) o << "              D" << k << " = " << yexpr(pt.terms[k], "Yd") << ";\n";
    o << "            }\n"
      << "            sb_f4 Gd = (sb_f4){0.f, 0.f, 0.f, 0.f};\n"
      << "            if (fl & 1) {\n" << "  " << gtile("Gd", "Sp", "phdB", m) << "            }\n"
      << "            if (fl & 8) {\n" << "  " << gtile("Gd", "Sp2", "phB", m) << "            }\n";
    for (int r = 0; r < 4; ++r)
      o << "            float d" << r << " = 0.f, z" << r << " = 0.f;\n";
    o << "            if (fl & 2) {\n";
    for (int r = 0; r < 4; ++r) o << "              d" << r << " += " << cexpr(ks, "xdv", "M", r) << ";\n";
    o << "            }\n            if (fl & 4) {\n";
    for (int r = 0; r < 4; ++r) o << "              d" << r << " += " << cexpr(ks, "xv", "D", r) << ";\n";
    o << "            }\n            if (fl & 8) {\n";
    for (int r = 0; r < 4; ++r) o << "              z" << r << " = " << cexpr(ks, "xv", "M", r) << ";\n";
    o << "            }\n"
      << ptile("Sp", "d", m)
      << "            if (fl & 8) {\n" << ptile("Sp2", "z", m) << "            }\n"
      << "            if (HAS_GY && (fl & 9)) {\n" << yupd(ks, "xv", "Gd", "gy") << "            }\n"
      << "            if (HAS_GY && (fl & 2)) {\n" << yupd(ks, "xdv", "G", "gy") << "            }\n"
      << "            if (HAS_YB && (fl & 4)) {\n" << yupd(ks, "xv", "G", "yb") << "            }\n"
      << "            if (fl & 9) {\n" << xupd(ks, "M", "Gd") << "            }\n"
      << "            if (fl & 4) {\n" << xupd(ks, "D", "G") << "            }\n"
      << "          }\n";
    // pin the updated partial sums here: left alone, the compiler sinks these
    // multiply-adds into the conditional blocks that finally use them, which
    // keeps every G tile of the item alive until then
    {
      std::vector<int> mis, mys;
      for (int k : ks) {
        if (std::find(mis.begin(), mis.end(), pt.pairs[k].first) == mis.end()) mis.push_back(pt.pairs[k].first);
        for (auto& tt : pt.terms[k])
          if (std::find(mys.begin(), mys.end(), tt.my) == mys.end()) mys.push_back(tt.my);
      }
      for (int mi : mis)
        for (int r = 0; r < 4; ++r) o << "          asm volatile(\"\" : \"+v\"(xc[" << r << "][" << mi << "]));\n";
      for (int my : mys) {
        o << "          if (HAS_GY) asm volatile(\"\" : \"+v\"(gy[" << Y0 + my << "]));\n";
        o << "          if (HAS_YB) asm volatile(\"\" : \"+v\"(yb[" << Y0 + my << "]));\n";
      }
    }
    ++b;
    o << "          __builtin_amdgcn_sched_barrier(0);\n"
      << "        }\n";
  }
  o << "      }\n";
}

// Adjoint (backward / double-backward) code for one slab.  A wave takes 16
// edges per iteration (edge k of the batch -> wave (k / 16) % ADJ_W, slot
// k % 16); lane l holds slot l % 16 and channels 4 (l / 16) .. 4 (l / 16) + 3 of
// each 16-channel tile.  The products with the staged adjoint state run on MFMA:
//   G[e][u][m_o] = sum_q phi[e][q] Sbar[q][m_o][u]
//     16x16x4: rows = the tile's channels, columns = edge slots, k = q;
//   phibar[e][q] += sum_{m_o, u} Sbar[q][m_o][u] C[e][u][m_o]
//     4x4x1 blocks of 4 lanes: rows = q, columns = the block's 4 edge slots,
//     one channel per step;
// and the CG contractions of each lane's 4 channels on the VALU.  Per-edge
// partial sums are reduced over the 4 channel quads once per edge.  MFMAs run
// with the whole wave: lanes past the last edge carry zero radial features and
// zero channel values, never a branch around a matrix instruction.
void emit_adj_slab(std::ostringstream& o, const Plan& P, int s) {
  const AdjSlab& sl = P.slabs[s];
  const bool first = s == 0, last = s + 1 == (int)P.slabs.size();
  int L = 0;
  for (auto& it : sl.items)
    for (int t : it.paths) L = std::max(L, P.paths[t].l_sh);
  const int NS = (L + 1) * (L + 1);
  auto is_v4 = [&](const AdjItem& it) {
    const Irrep& ri = P.in[it.a];
    return ri.mul % 4 == 0 && ri.off % 4 == 0 && P.dim_in % 4 == 0;
  };
  o << "template <bool DB, int FL>\nSB_DEV void sb_adj_s" << s
    << "(int w, int lane, int ebase, int nb, int e0, const int* __restrict__ sender, const float* __restrict__ evec,"
       " const float* __restrict__ phi, const float* __restrict__ x, const float* __restrict__ xdot,"
       " const float* __restrict__ evdot, const float* __restrict__ phidot, const float* sS, const float* sS2,"
       " float* sacc, float* __restrict__ gphi, float* __restrict__ gevec, float* __restrict__ contrib, int flags,"
       " bool multi, int* wids) {\n"
    << "  const int fl = FL >= 0 ? FL : flags;\n"
       "  constexpr bool HAS_GY = !DB || FL < 0 || (FL & 11);\n"
       "  constexpr bool HAS_YB = DB && (FL < 0 || (FL & 4));\n"
       "  constexpr int GY = K, YB = K + (HAS_GY ? NSH : 0);\n"
       "  constexpr int NV = K + (HAS_GY ? NSH : 0) + (HAS_YB ? NSH : 0);\n"
       "  constexpr int KQ = KP / 4;\n"
       "  const int es = lane & 15, g = lane >> 4, l3 = lane & 3;\n"
       // the batch's edges in segments of up to 256: a segment's sender ids go to
       // this wave's LDS slice first, so the edge loop never waits on them
       "  for (int seg = 0; seg < nb; seg += 256) {\n"
       "  const int sn = min(256, nb - seg), sbase = ebase + seg;\n"
       "#pragma unroll\n  for (int i = 0; i < 4; ++i) wids[64 * i + lane] = sender[sbase + min(64 * i + lane, sn - 1)];\n"
       // this wave's 16-edge batches are w, w + ADJ_W, ...: a wave whose last batch would
       // be empty stops one iteration early instead of computing on padding
       "  const int niter = ((sn + 15) / 16 - w + ADJ_W - 1) / ADJ_W;\n"
       // edge data and sender rows of the next iteration, loaded one iteration
       // ahead (clamped to the segment's last edge, masked at use)
       "  float nvx, nvy, nvz, ndx = 0.f, ndy = 0.f, ndz = 0.f, nph[KQ], nphd[KQ];\n"
       "  sb_i64 nrow;\n";
  for (size_t i = 0; i < sl.items.size(); ++i) {
    const int DA = 2 * P.in[sl.items[i].a].l + 1;
    if (is_v4(sl.items[i])) o << "  sb_f4 xn" << i << "[" << DA << "];\n";
    else o << "  float xn" << i << "[4][" << DA << "];\n";
  }
  // loads of the next iteration's edge data (and its sender's row offset)
  auto fetch_edge = [&](const std::string& itn) {
    o << "    {\n"
         "      const int kf = ((" << itn << ") * ADJ_W + w) * 16 + es;\n"
         "      const int kc = kf < sn ? kf : sn - 1;\n"
         "      const sb_i64 ef = sbase + kc;\n"
         "      nvx = evec[3 * ef]; nvy = evec[3 * ef + 1]; nvz = evec[3 * ef + 2];\n"
         "#pragma unroll\n      for (int v = 0; v < KQ; ++v) nph[v] = phi[ef * K + min(4 * v + g, K - 1)];\n"
         "      if (DB && (fl & 1)) {\n"
         "#pragma unroll\n        for (int v = 0; v < KQ; ++v) nphd[v] = phidot[ef * K + min(4 * v + g, K - 1)];\n"
         "      }\n"
         "      if (DB && (fl & 4)) { ndx = evdot[3 * ef]; ndy = evdot[3 * ef + 1]; ndz = evdot[3 * ef + 2]; }\n"
         "      nrow = (sb_i64)wids[kc] * CXI;\n"
         "    }\n";
  };
  // loads of item i's sender-row slice at row offset nrow (channel index clamped into the irrep)
  auto fetch_x = [&](size_t i, const char* ind) {
    const AdjItem& it = sl.items[i];
    const Irrep& ri = P.in[it.a];
    const int DA = 2 * ri.l + 1;
    if (is_v4(it))
      o << ind << "{\n" << ind << "  const int uc = min(" << it.u0 << " + 4 * g, " << ri.mul - 4 << ");\n"
        << "#pragma unroll\n" << ind << "  for (int m = 0; m < " << DA << "; ++m) xn" << i << "[m] = *(const sb_f4*)(x + nrow + "
        << ri.off << " + m * " << ri.mul << " + uc);\n" << ind << "}\n";
    else
      o << "#pragma unroll\n" << ind << "for (int r = 0; r < 4; ++r) {\n"
        << ind << "  const int uc = min(" << it.u0 << " + 4 * g + r, " << ri.mul - 1 << ");\n"
        << "#pragma unroll\n" << ind << "  for (int m = 0; m < " << DA << "; ++m) xn" << i << "[r][m] = x[nrow + " << ri.off
        << " + m * " << ri.mul << " + uc];\n" << ind << "}\n";
  };
  fetch_edge("0");
  for (size_t i = 0; i < sl.items.size(); ++i) fetch_x(i, "  ");
  const std::vector<AdjBlock> bl = adj_blocks(P, sl);
  for (size_t bi = 0; bi < bl.size(); ++bi) o << "  float gA" << bi << "[KQ]; sb_f4 G" << bi << ";\n";
  o << "  {\n    int zz = 0;\n    asm volatile(\"\" : \"+v\"(zz));\n";
  emit_adj_gload(o, bl, 0, "    ");
  if (bl.size() > 1) emit_adj_gload(o, bl, 1, "    ");
  o << "  }\n";
  int blk = 0;
  o << "  for (int it = 0; it < niter; ++it) {\n"
       "    const int kl = (it * ADJ_W + w) * 16 + es;\n"
       "    const int k = seg + kl;\n"
       "    const bool ev = kl < sn;\n"
       "    const int e = sbase + kl;\n"
       "    sb_f4 pacc[KQ];\n"
       "#pragma unroll\n    for (int v = 0; v < KQ; ++v) pacc[v] = (sb_f4){0.f, 0.f, 0.f, 0.f};\n"
       "    float gy[NSH], yb[NSH];\n"
       "#pragma unroll\n    for (int v = 0; v < NSH; ++v) { gy[v] = 0.f; yb[v] = 0.f; }\n"
       "    // this iteration's edge data (masked), then the next iteration's loads\n"
       "    const float vx = nvx, vy = nvy, vz = nvz;\n"
       "    const float dx = ev ? ndx : 0.f, dy = ev ? ndy : 0.f, dz = ev ? ndz : 0.f;\n"
       "    float phB[KQ], phdB[KQ];\n"
       "#pragma unroll\n    for (int v = 0; v < KQ; ++v) {\n"
       "      const bool ok = ev && 4 * v + g < K;\n"
       "      phB[v] = ok ? nph[v] : 0.f;\n"
       "      phdB[v] = (DB && (fl & 1) && ok) ? nphd[v] : 0.f;\n"
       "    }\n"
       "    const sb_i64 srow = nrow;\n"
       "    (void)srow;\n";
  fetch_edge("it + 1");
  o << "    const float rinv = __builtin_amdgcn_rsqf(vx * vx + vy * vy + vz * vz);\n"
       "    const float ux = vx * rinv, uy = vy * rinv, uz = vz * rinv;\n"
       "    // opaque zero: keeps the adjoint-state reads inside the loop (LDS), instead of\n"
       "    // hoisting the whole slab into registers\n"
       "    int zz = 0;\n    asm volatile(\"\" : \"+v\"(zz));\n"
    << "    float Y[" << NS << "], Yd[" << NS << "];\n    sb_sh_eval_L" << L << "(ux, uy, uz, Y);\n"
    << "    if (DB && (fl & 4)) sb_sh_jvp_L" << L << "(ux, uy, uz, rinv, dx, dy, dz, Y, Yd);\n";
  emit_adj_gtile(o, 0, "    ");
  for (size_t ii = 0; ii < sl.items.size(); ++ii) {
    const AdjItem& it = sl.items[ii];
    const Irrep& ri = P.in[it.a];
    const int DA = 2 * ri.l + 1;
    const bool v4 = is_v4(it);
    o << "    {  // input irrep " << it.a << ", channels " << it.u0 << " .. " << it.u0 + 15 << "\n"
      << "      constexpr int CA = " << ri.mul << ", AOFF = " << ri.off << ", U0 = " << it.u0 << ", DA = " << DA << ";\n"
      << "      const int u = U0 + 4 * g;\n"
      << "      float xv[4][DA], xdv[4][DA], xc[4][DA];\n";
    // the prefetched row slice of this iteration (zero for lanes past the edges or past C_in),
    // then the same slice of the next iteration
    if (v4)
      o << "#pragma unroll\n      for (int m = 0; m < DA; ++m) {\n"
        << "        const bool ok = ev && u < CA;\n"
        << "#pragma unroll\n        for (int r = 0; r < 4; ++r) xv[r][m] = ok ? xn" << ii << "[m][r] : 0.f;\n"
        << "      }\n";
    else
      o << "#pragma unroll\n      for (int r = 0; r < 4; ++r)\n#pragma unroll\n"
        << "        for (int m = 0; m < DA; ++m) xv[r][m] = (ev && u + r < CA) ? xn" << ii << "[r][m] : 0.f;\n";
    fetch_x(ii, "      ");
    o << "#pragma unroll\n      for (int r = 0; r < 4; ++r)\n#pragma unroll\n"
      << "        for (int m = 0; m < DA; ++m) { xdv[r][m] = 0.f; xc[r][m] = 0.f; }\n";
    if (v4)
      o << "      if (DB && (fl & 2) && ev && u < CA) {\n"
        << "#pragma unroll\n        for (int m = 0; m < DA; ++m) {\n"
        << "          const sb_f4 v = *(const sb_f4*)(xdot + srow + AOFF + m * CA + u);\n"
        << "          xdv[0][m] = v[0]; xdv[1][m] = v[1]; xdv[2][m] = v[2]; xdv[3][m] = v[3];\n"
        << "        }\n      }\n";
    else
      o << "      if (DB && (fl & 2) && ev) {\n"
        << "#pragma unroll\n        for (int r = 0; r < 4; ++r)\n"
        << "          if (u + r < CA) {\n"
        << "#pragma unroll\n            for (int m = 0; m < DA; ++m) xdv[r][m] = xdot[srow + AOFF + m * CA + u + r];\n"
        << "          }\n      }\n";
    for (size_t pi = 0; pi < it.paths.size(); ++pi) emit_adj_path(o, P, it.paths[pi], it.lds_off[pi], bl, blk);
    o << "      if (contrib && ev) {\n"
      << "        float* cr = contrib + (sb_i64)(e - e0) * CXI + AOFF + u;\n";
    if (v4)
      o << "        if (u < CA) {\n"
        << "#pragma unroll\n          for (int m = 0; m < DA; ++m) {\n"
        << "            sb_f4 v = (sb_f4){xc[0][m], xc[1][m], xc[2][m], xc[3][m]};\n"
        << (it.first ? "" : "            v += *(const sb_f4*)(cr + m * CA);\n")
        << "            *(sb_f4*)(cr + m * CA) = v;\n"
        << "          }\n        }\n";
    else
      o << "#pragma unroll\n        for (int r = 0; r < 4; ++r)\n"
        << "          if (u + r < CA) {\n"
        << "#pragma unroll\n            for (int m = 0; m < DA; ++m) cr[m * CA + r] = "
        << (it.first ? "xc[r][m]" : "cr[m * CA + r] + xc[r][m]") << ";\n"
        << "          }\n";
    o << "      }\n    }\n";
  }
  if (first) {
    for (int a : P.dead_in)
      o << "    if (contrib && ev) for (int t = g; t < " << P.in[a].dim() << "; t += 4) contrib[(sb_i64)(e - e0) * CXI + "
        << P.in[a].off << " + t] = 0.f;\n";
  }
  o << "    // sum the four channel quads of each edge slot\n"
       "#pragma unroll\n    for (int v = 0; v < KQ; ++v)\n#pragma unroll\n"
       "      for (int i = 0; i < 4; ++i) {\n"
       "        pacc[v][i] += __shfl_xor(pacc[v][i], 16);\n"
       "        pacc[v][i] += __shfl_xor(pacc[v][i], 32);\n"
       "      }\n"
       "    if (HAS_GY) {\n#pragma unroll\n      for (int v = 0; v < NSH; ++v) { gy[v] += __shfl_xor(gy[v], 16); gy[v] += __shfl_xor(gy[v], 32); }\n    }\n"
       "    if (HAS_YB) {\n#pragma unroll\n      for (int v = 0; v < NSH; ++v) { yb[v] += __shfl_xor(yb[v], 16); yb[v] += __shfl_xor(yb[v], 32); }\n    }\n"
       "    if (ev && g == 0) {\n"
       "      float pv[NV];\n"
       "#pragma unroll\n      for (int q = 0; q < K; ++q) pv[q] = pacc[q >> 2][q & 3];\n"
       "      if (HAS_GY) {\n#pragma unroll\n        for (int v = 0; v < NSH; ++v) pv[GY + v] = gy[v];\n      }\n"
       "      if (HAS_YB) {\n#pragma unroll\n        for (int v = 0; v < NSH; ++v) pv[YB + v] = yb[v];\n      }\n"
       "      if (multi) {\n"
       "#pragma unroll\n        for (int v = 0; v < NV; ++v) {\n"
    << "          float tv = pv[v];\n"
    << (first ? "" : "          tv += sacc[k * NV + v];\n")
    << (last ? "          pv[v] = tv;\n" : "          sacc[k * NV + v] = tv;\n")
    << "        }\n      }\n";
  if (last) {
    o << "      if (gphi) {\n#pragma unroll\n        for (int q = 0; q < K; ++q) gphi[(sb_i64)e * K + q] = pv[q];\n      }\n"
         "      if (gevec) {\n"
         "        float gg[3] = {0.f, 0.f, 0.f};\n"
         "        if (HAS_GY) sb_sh_vjp(ux, uy, uz, rinv, pv + GY, gg);\n"
         "        if (HAS_YB && (fl & 4)) {\n"
         "          float h[3];\n"
         "          sb_sh_hvp(ux, uy, uz, rinv, pv + YB, dx, dy, dz, h);\n"
         "          gg[0] += h[0]; gg[1] += h[1]; gg[2] += h[2];\n"
         "        }\n"
         "        gevec[3 * (sb_i64)e] = gg[0]; gevec[3 * (sb_i64)e + 1] = gg[1]; gevec[3 * (sb_i64)e + 2] = gg[2];\n"
         "      }\n";
  }
  o << "    }\n  }\n  }  // segment\n}\n";
}

// Staging of one slab's adjoint-state slices (and the second slice set when dA
// is active): [q < KP][m_o][16 channels] per path, zero past K and past C_in.
// Every load of the slab is issued before the first LDS write, so a block pays
// one memory round trip for its receiver's state instead of one per element.
// With every multiplicity a multiple of 4 the copy moves float4s (a channel
// quad never straddles C_in and every source offset is 16-byte aligned).
void emit_adj_stage(std::ostringstream& o, const Plan& P, int s, const char* indent) {
  const int NT = 64 * P.adj_waves;
  struct Sl { const Path* q; const Group* g; int u0, off, DO; };
  std::vector<Sl> sls;
  for (const AdjItem& it : P.slabs[s].items)
    for (size_t pi = 0; pi < it.paths.size(); ++pi) {
      const Path& q = P.paths[it.paths[pi]];
      sls.push_back({&q, &P.groups[q.group], it.u0, it.lds_off[pi], 2 * q.l_out + 1});
    }
  const int W = P.vec4 ? 4 : 1;  // floats per copy unit
  // Sbar: group blocks sb_ncap receivers apart, this receiver at row sb_r0 + il (a
  // workspace chunk slot, or a state kept for every receiver); Sbar': the chunk slot,
  // row sub_off + il
  auto src_expr = [&](const Sl& x, const std::string& t, int pass) {
    std::ostringstream e;
    const int per_q = x.DO * 16 / W;   // copy units per q row
    e << "const int q = " << t << " / " << per_q << ", r = " << t << " % " << per_q << ", m = r / " << 16 / W
      << ", uc = " << x.u0 << " + " << W << " * (r % " << 16 / W << ");\n"
      << indent << "    const bool ok = q < K && uc < " << x.q->c_in << ";\n"
      << indent << "    const sb_i64 src = " << (pass ? "ncap" : "sb_ncap") << " * " << x.g->s_off << "LL + ((sb_i64)"
      << (pass ? "(sub_off + il)" : "(sb_r0 + il)") << " * " << x.g->d << " + m) * " << x.g->D << "LL + " << x.q->koff << " + q * "
      << x.q->c_in << " + uc;\n";
    return e.str();
  };
  const char* T = W == 4 ? "sb_f4" : "float";
  const char* Z = W == 4 ? "(sb_f4){0.f, 0.f, 0.f, 0.f}" : "0.f";
  for (int pass = 0; pass < 2; ++pass) {   // pass 0: Sbar, pass 1: Sbar' (dA active)
    const char* src = pass ? "Sb2" : "Sb";
    const char* dst = pass ? "sS2" : "sS";
    o << indent << (pass ? "if (DB && (fl & 8)) {\n" : "{\n");
    int reg = 0;
    std::ostringstream stores;
    for (const Sl& x : sls) {
      const int n = P.adj_KP * x.DO * 16 / W;
      for (int j = 0; j * NT < n; ++j, ++reg) {
        const std::string t = "t" + std::to_string(reg);
        o << indent << "  " << T << " v" << reg << " = " << Z << ";\n"
          << indent << "  const int " << t << " = tid + " << j * NT << ";\n"
          << indent << "  if (" << t << " < " << n << ") {\n"
          << indent << "    " << src_expr(x, t, pass)
          << indent << "    if (ok) v" << reg << " = " << (W == 4 ? "*(const sb_f4*)(" : "*(") << src << " + src);\n"
          << indent << "  }\n";
        stores << indent << "  if (" << t << " < " << n << ") *(" << T << "*)(" << dst << " + " << x.off << " + " << W
               << " * " << t << ") = v" << reg << ";\n";
      }
    }
    o << stores.str() << indent << "}\n";
  }
}

}  // namespace

// Channelwise (uvu) forward without receiver state, for plans whose paths all have
// one multiplicity C: with channel u tied through every path (eq. uvu_connection),
// the edge weight of (path, u) is w = sum_q phi_q A[q, path, u] and the message of
// channel u is w times the path's CG contraction of channel u alone, so a lane owns
// one channel of one receiver and accumulates its output components directly
// (state-free: the receiver state would be K times larger than the output).  Blocks
// are (4 receivers, 64-channel block); the block's A slice [path][q][channel] is
// staged in LDS once.  C < 64 puts 64 / C edges in flight per wave (lane = edge
// slot * C + u), combined by cross-lane adds in a fixed order.
void emit_uvu_fwd(std::ostringstream& o, const Plan& P, bool tan) {
  const int C = P.uvu_C, UB = std::min(C, 64);
  const int ES = (64 % UB == 0) ? 64 / UB : 1;
  const int NPt = (int)P.paths.size();
  const int L = P.lmax, NS = (L + 1) * (L + 1);
  o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_uvu_fwd" << (tan ? "_t" : "") << "(const int* __restrict__ rowptr,"
       " const int* __restrict__ sender, const float* __restrict__ evec, const float* __restrict__ phi,"
       " const float* __restrict__ x, const float* __restrict__ W, float* __restrict__ out, int r0, int n_recv,"
       " const float* __restrict__ evd) {\n"
    << "  constexpr int C_ = " << C << ", UB_ = " << UB << ", ES_ = " << ES << ";\n"
    << "  __shared__ float sA[" << NPt * P.K * UB << "];\n"
    << "  const int cb = blockIdx.y, tid = threadIdx.x, lane = tid & 63;\n";
  for (int t = 0; t < NPt; ++t)
    o << "  for (int i = tid; i < K * UB_; i += 256) {\n"
      << "    const int q = i / UB_, uc = cb * UB_ + i % UB_;\n"
      << "    sA[" << t * P.K * UB << " + i] = uc < C_ ? W[(sb_i64)q * " << P.n_w << "LL + " << P.paths[t].w_off
      << "LL + uc] : 0.f;\n  }\n";
  o << "  __syncthreads();\n"
       "  const int il = blockIdx.x * 4 + (tid >> 6);\n"
       "  if (il >= n_recv) return;\n"
       "  const int sub = lane / UB_, u = lane % UB_, uc = cb * UB_ + u;\n"
       "  const bool lane_ok = sub < ES_ && uc < C_;\n";
  for (size_t g = 0; g < P.groups.size(); ++g)
    o << "  float acc" << g << "[" << P.groups[g].d << "];\n"
      << "#pragma unroll\n  for (int m = 0; m < " << P.groups[g].d << "; ++m) acc" << g << "[m] = 0.f;\n";
  o << "  const int beg = rowptr[r0 + il], end = rowptr[r0 + il + 1];\n"
       "  for (int e = beg + sub; lane_ok && e < end; e += ES_) {\n"
       // an opaque copy of the lane's channel offset keeps the A reads inside the loop
       // (hoisted, they would hold K x paths registers per lane)
       "    int ul = u;\n    asm volatile(\"\" : \"+v\"(ul));\n"
       "    const int j = sender[e];\n"
       "    const float vx = evec[3 * (sb_i64)e], vy = evec[3 * (sb_i64)e + 1], vz = evec[3 * (sb_i64)e + 2];\n"
       "    const float rinv = __builtin_amdgcn_rsqf(vx * vx + vy * vy + vz * vz);\n"
       "    float Y[" << NS << "];\n    sb_sh_eval_L" << L << "(vx * rinv, vy * rinv, vz * rinv, Y);\n"
       "    float ph[K];\n#pragma unroll\n    for (int q = 0; q < K; ++q) ph[q] = phi[(sb_i64)e * K + q];\n"
       "    const sb_i64 xrow = (sb_i64)j * CXI + uc;\n";
  if (tan)  // the tangent variant takes the message along Ydot = J evd (the tangent output)
    o << "    {\n      float Yd[" << NS << "];\n      sb_sh_jvp_L" << L << "(vx * rinv, vy * rinv, vz * rinv, rinv,"
         " evd[3 * (sb_i64)e], evd[3 * (sb_i64)e + 1], evd[3 * (sb_i64)e + 2], Y, Yd);\n"
         "#pragma unroll\n      for (int m = 0; m < " << NS << "; ++m) Y[m] = Yd[m];\n    }\n";
  std::vector<bool> used(P.in.size(), false);
  for (auto& q : P.paths) used[q.i_in] = true;
  for (size_t a = 0; a < P.in.size(); ++a)
    if (used[a]) {
      const int d = 2 * P.in[a].l + 1;
      o << "    float x" << a << "[" << d << "];\n#pragma unroll\n    for (int m = 0; m < " << d << "; ++m) x" << a
        << "[m] = x[xrow + " << P.in[a].off << " + m * C_];\n";
    }
  for (int t = 0; t < NPt; ++t) {
    const Path& q = P.paths[t];
    const int dd = 2 * q.l_out + 1;
    o << "    {\n      float M[P" << t << "_NP], Cc[" << dd << "];\n      sb_M" << t << "(Y + " << q.l_sh * q.l_sh
      << ", M);\n      sb_C" << t << "(x"
      << q.i_in << ", M, Cc);\n      int ua = ul;\n      asm volatile(\"\" : \"+v\"(ua) :: \"memory\");\n"
      << "      float w = 0.f;\n#pragma unroll\n      for (int q = 0; q < K; ++q) w += ph[q] * sA["
      << t * P.K * UB << " + q * UB_ + ua];\n#pragma unroll\n      for (int m = 0; m < " << dd << "; ++m) acc" << q.group
      << "[m] += w * Cc[m];\n    }\n    __builtin_amdgcn_sched_barrier(0);\n";
  }
  o << "  }\n";
  if (ES > 1) {
    o << "#pragma unroll\n  for (int s = UB_; s < 64; s <<= 1) {\n";
    for (size_t g = 0; g < P.groups.size(); ++g)
      o << "#pragma unroll\n    for (int m = 0; m < " << P.groups[g].d << "; ++m) acc" << g << "[m] += __shfl_xor(acc" << g
        << "[m], s);\n";
    o << "  }\n";
  }
  o << "  if (sub == 0 && uc < C_) {\n    const sb_i64 orow = (sb_i64)(r0 + il) * CXO + uc;\n";
  for (size_t g = 0; g < P.groups.size(); ++g)
    o << "#pragma unroll\n    for (int m = 0; m < " << P.groups[g].d << "; ++m) out[orow + " << P.groups[g].off
      << " + m * C_] = acc" << g << "[m];\n";
  o << "  }\n}\n";
}

// Transposed couplings of one path for the channelwise backward:
// X[m_i] += sum_{m_o} M[(m_i, m_o)] G[m_o]   (x-gradient, M = sum_y c Y_y), and
// Yb[m_y] += sum_{(m_i, m_o)} c x[m_i] G[m_o] (SH adjoint of the path's slice).
void emit_path_transposes(std::ostringstream& o, const Plan& P, int t) {
  const Path& q = P.paths[t];
  const PathTerms pt = path_terms(q);
  o << "SB_DEV void sb_XT" << t << "(const float* M, const float* G, float* X) {\n";
  for (size_t k = 0; k < pt.pairs.size(); ++k)
    o << "  X[" << pt.pairs[k].first << "] += M[" << k << "]*G[" << pt.pairs[k].second << "];\n";
  o << "}\nSB_DEV void sb_YT" << t << "(const float* x, const float* G, float* Yb) {\n";
  for (size_t k = 0; k < pt.pairs.size(); ++k) {
    o << "  { const float xg = x[" << pt.pairs[k].first << "]*G[" << pt.pairs[k].second << "];";
    for (const PairTerm& tm : pt.terms[k]) o << " Yb[" << tm.my << "] += " << fl(tm.c) << "*xg;";
    o << " }\n";
  }
  o << "}\n";
}

// Channelwise (uvu) backward without adjoint state, same plans as the state-free
// forward: with G = w mbar_i (tied channel), the edge adjoints are
//   h[path, u] = <mbar_i[u], C_path[u]>,  phi_bar[q] = sum_{path, u} A[q, path, u] h,
//   x_bar contribution = C^T(G, Y), Y_bar = C^T(x_j, G), evec_bar = J^T Y_bar.
// A lane owns one channel of one receiver and one edge at a time (64 / C edges in
// flight below 64 channels).  Slices (blockIdx.z, blockIdx.y = 64-channel block) hold
// all input irreps (suffix _u) or one input irrep each (suffix _s, fewer registers for
// plans with many paths, at one more pass over the edges per irrep): each slice
// writes its own columns of the x-gradient contribution rows, and its phi_bar and
// Y_bar summed over the lane group's channels (fixed order); with one slice they are
// final, else each slice writes per-edge partials that sobek_uvu_bwd_fin adds in
// slice order.  Edges are those of the receiver inside [win0, win1); the
// contribution row of edge e sits at e - e0.
void emit_uvu_bwd(std::ostringstream& o, const Plan& P, bool sliced, bool tan) {
  const int C = P.uvu_C, NB = P.uvu_NB;
  const std::string sfx = std::string(sliced ? "_s" : "_u") + (tan ? "t" : "");
  int UBP = 64;
  if (C < 64) { UBP = 1; while (UBP < C) UBP <<= 1; }
  const int ES = 64 / UBP;
  const int NPt = (int)P.paths.size();
  const int L = P.lmax, NS = (L + 1) * (L + 1), NV = P.K + NS;
  std::vector<int> ins;
  std::vector<bool> used(P.in.size(), false);
  for (auto& q : P.paths) used[q.i_in] = true;
  for (size_t a = 0; a < P.in.size(); ++a)
    if (used[a]) ins.push_back((int)a);
  // slices: one input irrep each (sliced), or all of them in one (unsliced)
  std::vector<std::vector<int>> slices;
  if (sliced) for (int a : ins) slices.push_back({a});
  else slices.push_back(ins);
  const int NA = (int)slices.size(), NPART = NA * NB;
  int maxp = 1;
  for (auto& sl : slices) {
    int n = 0;
    for (auto& q : P.paths) n += std::find(sl.begin(), sl.end(), q.i_in) != sl.end();
    maxp = std::max(maxp, n);
  }
  if (!sliced && !tan)
    for (int t = 0; t < NPt; ++t) emit_path_transposes(o, P, t);
  o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_uvu_bwd" << sfx << "(const int* __restrict__ rowptr,"
       " const int* __restrict__ sender, const float* __restrict__ evec, const float* __restrict__ phi,"
       " const float* __restrict__ x, const float* __restrict__ W, const float* __restrict__ Mb,"
       " float* __restrict__ gphi, float* __restrict__ gevec, float* __restrict__ contrib, float* __restrict__ part,"
       " int r0, int n_recv, int e0, int win0, int win1, const float* __restrict__ evd) {\n"
    << "  constexpr int C_ = " << C << ", UB_ = " << UBP << ", ES_ = " << ES << ", NB_ = " << NB << ", NV_ = " << NV
    << ", NPART_ = " << NPART << ";\n  __shared__ float sA[" << maxp * P.K * UBP << "];\n"
    << "  const int cb = blockIdx.y, tid = threadIdx.x, lane = tid & 63;\n"
    << "  const int il = blockIdx.x * 4 + (tid >> 6);\n"
    << "  const int sub = lane / UB_, u = lane % UB_, uc = cb * UB_ + u;\n"
    << "  const bool cv = uc < C_;\n"
    << "  const sb_i64 mrow = (sb_i64)(r0 + il) * CXO + uc;\n"
    << "  switch (blockIdx.z) {\n";
  for (int ia = 0; ia < NA; ++ia) {
    const std::vector<int>& sl = slices[ia];
    std::vector<int> ts, gs;
    for (int t = 0; t < NPt; ++t)
      if (std::find(sl.begin(), sl.end(), P.paths[t].i_in) != sl.end()) {
        ts.push_back(t);
        if (std::find(gs.begin(), gs.end(), P.paths[t].group) == gs.end()) gs.push_back(P.paths[t].group);
      }
    o << "  case " << ia << ": {\n";
    for (size_t k = 0; k < ts.size(); ++k)
      o << "    for (int i = tid; i < K * UB_; i += 256) {\n"
        << "      const int q = i / UB_, uc2 = cb * UB_ + i % UB_;\n"
        << "      sA[" << k * P.K * UBP << " + i] = uc2 < C_ ? W[(sb_i64)q * " << P.n_w << "LL + " << P.paths[ts[k]].w_off
        << "LL + uc2] : 0.f;\n    }\n";
    o << "    __syncthreads();\n    if (il >= n_recv) return;\n";
    for (int g : gs)
      o << "    float mb" << g << "[" << P.groups[g].d << "];\n#pragma unroll\n    for (int m = 0; m < " << P.groups[g].d
        << "; ++m) mb" << g << "[m] = cv ? Mb[mrow + " << P.groups[g].off << " + m * C_] : 0.f;\n";
    o << "    const int wb = max(rowptr[r0 + il], win0), we = min(rowptr[r0 + il + 1], win1);\n"
         "    for (int e = wb + sub; e < we; e += ES_) {\n"
         "      int ul = u;\n      asm volatile(\"\" : \"+v\"(ul));\n"
         "      const int j = sender[e];\n"
         "      const float vx = evec[3 * (sb_i64)e], vy = evec[3 * (sb_i64)e + 1], vz = evec[3 * (sb_i64)e + 2];\n"
         "      const float rinv = __builtin_amdgcn_rsqf(vx * vx + vy * vy + vz * vz);\n"
         "      const float ux = vx * rinv, uy = vy * rinv, uz = vz * rinv;\n"
         "      float Y[" << NS << "], yb[" << NS << "], pb[K];\n      sb_sh_eval_L" << L << "(ux, uy, uz, Y);\n"
         // double backward along an edge-vector tangent (no other cotangent): h and the
         // x-gradient contribution are taken along Ydot = J evd, Y_bar stays the backward's
         // and the edge-vector output is its Hessian term sum_m Y_bar_m Hess(Y_m) evd
         << (tan ? std::string("      const float tx = evd[3 * (sb_i64)e], ty = evd[3 * (sb_i64)e + 1], tz = evd[3 * (sb_i64)e + 2];\n"
                               "      {\n        float Yd[") + std::to_string(NS) + "];\n        sb_sh_jvp_L" + std::to_string(L) +
                       "(ux, uy, uz, rinv, tx, ty, tz, Y, Yd);\n#pragma unroll\n        for (int m = 0; m < " +
                       std::to_string(NS) + "; ++m) Y[m] = Yd[m];\n      }\n"
                 : std::string())
      << "#pragma unroll\n      for (int m = 0; m < " << NS << "; ++m) yb[m] = 0.f;\n"
         "      float ph[K];\n#pragma unroll\n      for (int q = 0; q < K; ++q) { ph[q] = phi[(sb_i64)e * K + q]; pb[q] = 0.f; }\n"
         "      const sb_i64 xrow = (sb_i64)j * CXI + uc;\n";
    for (int a : sl) {
      const int d = 2 * P.in[a].l + 1;
      o << "      float x" << a << "[" << d << "], xb" << a << "[" << d << "];\n#pragma unroll\n      for (int m = 0; m < " << d
        << "; ++m) { x" << a << "[m] = cv ? x[xrow + " << P.in[a].off << " + m * C_] : 0.f; xb" << a << "[m] = 0.f; }\n";
    }
    for (size_t k = 0; k < ts.size(); ++k) {
      const int t = ts[k];
      const Path& q = P.paths[t];
      const int dd = 2 * q.l_out + 1;
      o << "      {\n        float M[P" << t << "_NP], Cc[" << dd << "], G[" << dd << "];\n        sb_M" << t << "(Y + "
        << q.l_sh * q.l_sh << ", M);\n        sb_C" << t << "(x" << q.i_in << ", M, Cc);\n"
        << "        int ua = ul;\n        asm volatile(\"\" : \"+v\"(ua) :: \"memory\");\n"
        << "        const float* At = sA + " << k * P.K * UBP << " + ua;\n        float w = 0.f, h = 0.f;\n"
        << "#pragma unroll\n        for (int q = 0; q < K; ++q) w += ph[q] * At[q * UB_];\n"
        << "#pragma unroll\n        for (int m = 0; m < " << dd << "; ++m) { h += mb" << q.group << "[m] * Cc[m]; G[m] = w * mb"
        << q.group << "[m]; }\n"
        << "#pragma unroll\n        for (int q = 0; q < K; ++q) pb[q] += At[q * UB_] * h;\n"
        << "        sb_XT" << t << "(M, G, xb" << q.i_in << ");\n        sb_YT" << t << "(x" << q.i_in << ", G, yb + "
        << q.l_sh * q.l_sh << ");\n      }\n"
        << "      __builtin_amdgcn_sched_barrier(0);\n";
    }
    o << "      if (contrib) {\n        float* cr = contrib + (sb_i64)(e - e0) * CXI;\n        if (cv) {\n";
    for (int a : sl)
      o << "#pragma unroll\n          for (int m = 0; m < " << 2 * P.in[a].l + 1 << "; ++m) cr[" << P.in[a].off
        << " + m * C_ + uc] = xb" << a << "[m];\n";
    o << "        }\n";
    if (ia == 0)  // dead input irreps: zero columns, written by the first slice's first channel block
      for (size_t a2 = 0; a2 < P.in.size(); ++a2)
        if (!used[a2])
          o << "        if (cb == 0)\n          for (int c = u; c < " << P.in[a2].dim() << "; c += UB_) cr[" << P.in[a2].off
            << " + c] = 0.f;\n";
    o << "      }\n"
         "#pragma unroll\n      for (int s = 1; s < UB_; s <<= 1) {\n"
         "#pragma unroll\n        for (int q = 0; q < K; ++q) pb[q] += __shfl_xor(pb[q], s);\n"
         "#pragma unroll\n        for (int m = 0; m < " << NS << "; ++m) yb[m] += __shfl_xor(yb[m], s);\n      }\n";
    if (NPART == 1)
      o << "      if (u == 0) {\n"
           "        if (gphi) {\n#pragma unroll\n          for (int q = 0; q < K; ++q) gphi[(sb_i64)e * K + q] = pb[q];\n        }\n"
           "        if (gevec) {\n          float gg[3];\n"
        << (tan ? "          sb_sh_hvp(ux, uy, uz, rinv, yb, tx, ty, tz, gg);\n" : "          sb_sh_vjp(ux, uy, uz, rinv, yb, gg);\n")
        << "          gevec[3 * (sb_i64)e] = gg[0]; gevec[3 * (sb_i64)e + 1] = gg[1]; gevec[3 * (sb_i64)e + 2] = gg[2];\n"
           "        }\n      }\n";
    else
      o << "      if (u == 0) {\n        float* pp = part + ((sb_i64)(e - e0) * NPART_ + " << ia << " * NB_ + cb) * NV_;\n"
           "#pragma unroll\n        for (int q = 0; q < K; ++q) pp[q] = pb[q];\n"
           "#pragma unroll\n        for (int m = 0; m < " << NS << "; ++m) pp[K + m] = yb[m];\n      }\n";
    o << "    }\n    break;\n  }\n";
  }
  o << "  }\n}\n";
  if (NPART > 1) {
    o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_uvu_bwd_fin" << sfx << "(const float* __restrict__ evec,"
         " const float* __restrict__ part, float* __restrict__ gphi, float* __restrict__ gevec, int e0, int e1,"
         " const float* __restrict__ evd) {\n"
      << "  constexpr int NPART_ = " << NPART << ", NV_ = " << NV << ";\n"
      << "  const int e = e0 + blockIdx.x * 256 + threadIdx.x;\n  if (e >= e1) return;\n"
      << "  const float* pp = part + (sb_i64)(e - e0) * NPART_ * NV_;\n"
      << "  float v[NV_];\n#pragma unroll\n  for (int k = 0; k < NV_; ++k) v[k] = pp[k];\n"
      << "  for (int b = 1; b < NPART_; ++b) {\n#pragma unroll\n    for (int k = 0; k < NV_; ++k) v[k] += pp[b * NV_ + k];\n  }\n"
      << "  if (gphi) {\n#pragma unroll\n    for (int q = 0; q < K; ++q) gphi[(sb_i64)e * K + q] = v[q];\n  }\n"
      << "  if (gevec) {\n"
      << "    const float vx = evec[3 * (sb_i64)e], vy = evec[3 * (sb_i64)e + 1], vz = evec[3 * (sb_i64)e + 2];\n"
      << "    const float rinv = __builtin_amdgcn_rsqf(vx * vx + vy * vy + vz * vz);\n"
      << "    float gg[3];\n"
      << (tan ? "    sb_sh_hvp(vx * rinv, vy * rinv, vz * rinv, rinv, v + K, evd[3 * (sb_i64)e], evd[3 * (sb_i64)e + 1],"
                " evd[3 * (sb_i64)e + 2], gg);\n"
              : "    sb_sh_vjp(vx * rinv, vy * rinv, vz * rinv, rinv, v + K, gg);\n")
      << "    gevec[3 * (sb_i64)e] = gg[0]; gevec[3 * (sb_i64)e + 1] = gg[1]; gevec[3 * (sb_i64)e + 2] = gg[2];\n  }\n}\n";
  }
}

// Channelwise weight gradient without receiver state: A_bar[q, path, u] is the sum
// over all edges of phi_e[q] h_e[path, u], h = <mbar_i[u], C_path[u]> (tied channel).
// Grid (nwv / 4, 64-channel blocks, input irreps with paths): wave w of the
// slice (input irrep a, channel block) takes receivers w, w + nwv, ... and
// keeps K accumulators per path of a and channel in registers; each wave writes
// its own partial row part[w][q * N_w + w_off + u], which sobek_uvu_wreduce adds
// in wave order.
void emit_uvu_wgrad(std::ostringstream& o, const Plan& P, bool tan) {
  const int C = P.uvu_C;
  int UBP = 64;
  if (C < 64) { UBP = 1; while (UBP < C) UBP <<= 1; }
  const int ES = 64 / UBP;
  const int L = P.lmax, NS = (L + 1) * (L + 1);
  std::vector<int> ins;
  for (size_t a = 0; a < P.in.size(); ++a)
    for (auto& q : P.paths)
      if (q.i_in == (int)a) { ins.push_back((int)a); break; }
  o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_uvu_wgrad" << (tan ? "_t" : "") << "(const int* __restrict__ rowptr,"
       " const int* __restrict__ sender, const float* __restrict__ evec, const float* __restrict__ phi,"
       " const float* __restrict__ x, const float* __restrict__ Mb, float* __restrict__ part, int n_recv,"
       " const float* __restrict__ evd, int nwv) {\n"
    << "  constexpr int C_ = " << C << ", UB_ = " << UBP << ", ES_ = " << ES << ";\n"
    << "  const int cb = blockIdx.y, lane = threadIdx.x & 63, wv = blockIdx.x * 4 + (threadIdx.x >> 6);\n"
    << "  const int sub = lane / UB_, u = lane % UB_, uc = cb * UB_ + u;\n"
    << "  const bool cv = uc < C_;\n"
    << "  float* prow = part + (sb_i64)wv * " << (int64_t)P.K * P.n_w << "LL;\n"
    << "  switch (blockIdx.z) {\n";
  for (size_t ia = 0; ia < ins.size(); ++ia) {
    const int a = ins[ia];
    const int d = 2 * P.in[a].l + 1;
    std::vector<int> ts, gs;
    for (int t = 0; t < (int)P.paths.size(); ++t)
      if (P.paths[t].i_in == a) {
        ts.push_back(t);
        if (std::find(gs.begin(), gs.end(), P.paths[t].group) == gs.end()) gs.push_back(P.paths[t].group);
      }
    o << "  case " << ia << ": {\n";
    for (int t : ts) o << "    float acc" << t << "[K];\n#pragma unroll\n    for (int q = 0; q < K; ++q) acc" << t << "[q] = 0.f;\n";
    o << "    for (int r = wv; r < n_recv; r += nwv) {\n"
         "      const sb_i64 mrow = (sb_i64)r * CXO + uc;\n";
    for (int g : gs)
      o << "      float mb" << g << "[" << P.groups[g].d << "];\n#pragma unroll\n      for (int m = 0; m < "
        << P.groups[g].d << "; ++m) mb" << g << "[m] = cv ? Mb[mrow + " << P.groups[g].off << " + m * C_] : 0.f;\n";
    o << "      const int beg = rowptr[r], end = rowptr[r + 1];\n"
         "      for (int e = beg + sub; e < end; e += ES_) {\n"
         "        const int j = sender[e];\n"
         "        const float vx = evec[3 * (sb_i64)e], vy = evec[3 * (sb_i64)e + 1], vz = evec[3 * (sb_i64)e + 2];\n"
         "        const float rinv = __builtin_amdgcn_rsqf(vx * vx + vy * vy + vz * vz);\n"
         "        float Y[" << NS << "];\n        sb_sh_eval_L" << L << "(vx * rinv, vy * rinv, vz * rinv, Y);\n"
         << (tan ? std::string("        {\n          float Yd[") + std::to_string(NS) + "];\n          sb_sh_jvp_L" +
                       std::to_string(L) + "(vx * rinv, vy * rinv, vz * rinv, rinv, evd[3 * (sb_i64)e], evd[3 * (sb_i64)e + 1],"
                       " evd[3 * (sb_i64)e + 2], Y, Yd);\n#pragma unroll\n          for (int m = 0; m < " + std::to_string(NS) +
                       "; ++m) Y[m] = Yd[m];\n        }\n"
                     : std::string())
      << "        float ph[K];\n#pragma unroll\n        for (int q = 0; q < K; ++q) ph[q] = phi[(sb_i64)e * K + q];\n"
         "        float xa[" << d << "];\n#pragma unroll\n        for (int m = 0; m < " << d << "; ++m) xa[m] = cv ? x[(sb_i64)j * CXI + "
      << P.in[a].off << " + m * C_ + uc] : 0.f;\n";
    for (int t : ts) {
      const Path& q = P.paths[t];
      const int dd = 2 * q.l_out + 1;
      o << "        {\n          float M[P" << t << "_NP], Cc[" << dd << "];\n          sb_M" << t << "(Y + " << q.l_sh * q.l_sh
        << ", M);\n          sb_C" << t << "(xa, M, Cc);\n          float h = 0.f;\n#pragma unroll\n          for (int m = 0; m < "
        << dd << "; ++m) h += mb" << q.group << "[m] * Cc[m];\n#pragma unroll\n          for (int q = 0; q < K; ++q) acc" << t
        << "[q] += ph[q] * h;\n        }\n";
    }
    o << "      }\n    }\n";
    if (ES > 1) {
      o << "#pragma unroll\n    for (int s = UB_; s < 64; s <<= 1) {\n";
      for (int t : ts) o << "#pragma unroll\n      for (int q = 0; q < K; ++q) acc" << t << "[q] += __shfl_xor(acc" << t << "[q], s);\n";
      o << "    }\n";
    }
    o << "    if (sub == 0 && cv) {\n";
    for (int t : ts)
      o << "#pragma unroll\n      for (int q = 0; q < K; ++q) prow[(sb_i64)q * " << P.n_w << "LL + " << P.paths[t].w_off
        << "LL + uc] = acc" << t << "[q];\n";
    o << "    }\n    break;\n  }\n";
  }
  o << "  }\n}\n";
}

// The materialized baseline (Section 2.4 eq. radial_projection_background, Section 2.5): the
// conventional evaluation order that forms the per-edge weights W = phi A (E x N_w) and the
// per-edge messages M (E x C_out) in memory and then reduces M over each receiver's edges.  It is
// a comparison system for the memory law of Section 2.5 and a second route to the same forward;
// a module of its own, compiled on first use, so that no streamed kernel's source changes.
//   sobek_mat_w      W[e][n] = sum_q phi[e][q] A[q][n] for the window's edges (one column per
//                    thread, A's column in registers, a tile of edges per block)
//   sobek_mat_msg    one block per edge: the coupling values C_pi[u][m_o] of every path and input
//                    channel in LDS, then M[e][off_g + m_o C_g + w] = sum_{pi in g} sum_u
//                    W[e][off_pi + u C_g + w] C_pi[u][m_o] with one thread per output channel w
//   sobek_mat_reduce out[i][c] = sum of M[e][c] over receiver i's edges
std::string generate_materialized_source(const Plan& P) {
  std::ostringstream o;
  o.precision(17);
  o << "\n// ---- materialized forward, K=" << P.K << " lmax=" << P.lmax << " N_w=" << P.n_w << "\n";
  o << "#define K " << P.K << "\n#define NSH " << P.nsh << "\n#define CXI " << P.dim_in << "\n#define CXO " << P.dim_out
    << "\n#define NWT " << P.n_w << "LL\n#define MAT_ET 32\n";
  emit_sh(o, P.lmax);
  for (int t = 0; t < (int)P.paths.size(); ++t) emit_path(o, P, t);
  // W = phi A: blockIdx.x = 256 columns, blockIdx.y = MAT_ET edges of the window
  o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_mat_w(const float* __restrict__ phi,"
       " const float* __restrict__ A, float* __restrict__ Wm, sb_i64 e0, int ne) {\n"
       "  const sb_i64 col = (sb_i64)blockIdx.x * 256 + threadIdx.x;\n"
       "  if (col >= NWT) return;\n"
       "  float a[K];\n"
       "#pragma unroll\n  for (int q = 0; q < K; ++q) a[q] = A[q * NWT + col];\n"
       "  const int eb = blockIdx.y * MAT_ET, ee = min(ne, eb + MAT_ET);\n"
       "  for (int e = eb; e < ee; ++e) {\n"
       "    const float* ph = phi + (e0 + e) * K;\n"
       "    float s = 0.f;\n"
       "#pragma unroll\n    for (int q = 0; q < K; ++q) s = fmaf(ph[q], a[q], s);\n"
       "    Wm[(sb_i64)e * NWT + col] = s;\n"
       "  }\n}\n";
  // per-edge messages
  int ct = 0;
  std::vector<int> ctoff(P.paths.size());
  for (size_t t = 0; t < P.paths.size(); ++t) {
    ctoff[t] = ct;
    ct += P.paths[t].c_in * (2 * P.paths[t].l_out + 1);
  }
  int nch = 0;
  for (auto& g : P.groups) nch += g.C;
  o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_mat_msg(const int* __restrict__ sender,"
       " const float* __restrict__ evec, const float* __restrict__ x, const float* __restrict__ Wm,"
       " float* __restrict__ Mm, sb_i64 e0, int ne) {\n"
       "  __shared__ float sC[" << std::max(1, ct) << "];\n"
       "  const int e = blockIdx.x, tid = threadIdx.x;\n"
       "  if (e >= ne) return;\n"
       "  const sb_i64 ge = e0 + e;\n"
       "  const sb_i64 xrow = (sb_i64)sender[ge] * CXI;\n"
       "  const float vx = evec[3 * ge], vy = evec[3 * ge + 1], vz = evec[3 * ge + 2];\n"
       "  const float rinv = __builtin_amdgcn_rsqf(vx * vx + vy * vy + vz * vz);\n"
       "  float Y[" << (P.lmax + 1) * (P.lmax + 1) << "];\n"
       "  sb_sh_eval_L" << P.lmax << "(vx * rinv, vy * rinv, vz * rinv, Y);\n";
  for (size_t t = 0; t < P.paths.size(); ++t) {
    const Path& q = P.paths[t];
    const Irrep& ri = P.in[q.i_in];
    const int DI = 2 * q.l_in + 1, DO = 2 * q.l_out + 1;
    const int np = (int)path_terms(q).pairs.size();
    o << "  for (int u = tid; u < " << q.c_in << "; u += 256) {  // path " << t << "\n"
      << "    float xv[" << DI << "], M[" << std::max(1, np) << "], C[" << DO << "];\n"
      << "#pragma unroll\n    for (int m = 0; m < " << DI << "; ++m) xv[m] = x[xrow + " << ri.off << " + m * " << ri.mul
      << " + u];\n"
      << "    sb_M" << t << "(Y + " << q.l_sh * q.l_sh << ", M);\n"
      << "    sb_C" << t << "(xv, M, C);\n"
      << "#pragma unroll\n    for (int m = 0; m < " << DO << "; ++m) sC[" << ctoff[t] << " + u * " << DO << " + m] = C[m];\n"
      << "  }\n";
  }
  o << "  __syncthreads();\n"
       "  const float* We = Wm + (sb_i64)e * NWT;\n"
       "  float* Me = Mm + (sb_i64)e * CXO;\n"
       "  for (int idx = tid; idx < " << nch << "; idx += 256) {\n";
  int base = 0;
  for (auto& g : P.groups) {
    o << "    if (idx >= " << base << " && idx < " << base + g.C << ") {  // output irrep " << g.i_out << "\n"
      << "      const int w = idx - " << base << ";\n"
      << "      float acc[" << g.d << "] = {};\n";
    for (int t : g.paths) {
      const Path& q = P.paths[t];
      o << "      for (int u = 0; u < " << q.c_in << "; ++u) {  // path " << t << "\n"
        << "        const float wv = We[" << q.w_off << "LL + u * " << g.C << " + w];\n"
        << "#pragma unroll\n        for (int m = 0; m < " << g.d << "; ++m) acc[m] = fmaf(wv, sC[" << ctoff[t] << " + u * "
        << g.d << " + m], acc[m]);\n"
        << "      }\n";
    }
    o << "#pragma unroll\n      for (int m = 0; m < " << g.d << "; ++m) Me[" << g.off << " + m * " << g.C << " + w] = acc[m];\n"
      << "    }\n";
    base += g.C;
  }
  o << "  }\n}\n";
  // segment sum over each receiver's edges (every output column; irreps no path reaches are
  // cleared by the host afterwards)
  o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_mat_reduce(const int* __restrict__ rowptr,"
       " const float* __restrict__ Mm, float* __restrict__ out, int r0, int nr, sb_i64 e0) {\n"
       "  const int i = blockIdx.x, c = blockIdx.y * 256 + threadIdx.x;\n"
       "  if (c >= CXO || i >= nr) return;\n"
       "  const int beg = rowptr[r0 + i], end = rowptr[r0 + i + 1];\n"
       "  float s = 0.f;\n"
       "  for (int e = beg; e < end; ++e) s += Mm[(e - e0) * CXO + c];\n"
       "  out[(sb_i64)(r0 + i) * CXO + c] = s;\n"
       "}\n";
  return o.str();
}

// State kernels of one output group at a time (the per-group scratch policy, Appendix B.2 eq.
// receiver_chunk_budget): for every output group g, the forward units of g's paths alone and
// sobek_fwdg<g>_{S,dS_r,dS}, the same kernels as sobek_fwd_* restricted to g, writing S_g at the
// start of S (receiver il at il * d_g * D_g).  A module of its own, compiled on first use, so that
// the plan's main source does not change.
std::string generate_group_source(const Plan& P) {
  std::ostringstream o;
  o.precision(17);
  o << "\n// ---- per-group state kernels, K=" << P.K << " lmax=" << P.lmax << "\n";
  o << "#define K " << P.K << "\n#define NSH " << P.nsh << "\n#define CXI " << P.dim_in << "\n#define CXO " << P.dim_out
    << "\n#define EB " << P.bwd_eb << "\n#define KP " << P.adj_KP << "\n#define ADJ_W " << P.adj_waves << "\n";
  emit_sh(o, P.lmax);
  for (int t = 0; t < (int)P.paths.size(); ++t) emit_path(o, P, t);
  const char* st = P.dtype == 1 ? "__bf16" : "float";
  struct FV { const char* name; bool tan; int fl; };
  const FV fvs[] = {{"S", false, 0}, {"dS_r", true, 4}, {"dS", true, -1}};
  int id = 0;
  for (int gi = 0; gi < (int)P.groups.size(); ++gi) {
    const std::vector<Unit> units = pack_fwd_units(P, gi, nullptr);
    const int id0 = id;
    for (const Unit& u : units) emit_fwd_unit(o, P, u, id++, true);
    const int NU = (int)units.size();
    for (const FV& fv : fvs) {
      o << "extern \"C\" __global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void sobek_fwdg" << gi
        << "_" << fv.name
        << "(const int* __restrict__ rowptr, const int* __restrict__ sender, const float* __restrict__ evec,"
           " const float* __restrict__ phi, const float* __restrict__ x, " << st << "* __restrict__ S, int r0, int n_recv,"
           " sb_i64 ncap, const float* __restrict__ xdot, const float* __restrict__ evdot,"
           " const float* __restrict__ phidot, int flags) {\n"
        << "  __shared__ int sids[4][256];\n"
        << "  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;\n"
        << "  const int il = gw / " << NU << ", t = gw % " << NU << ";\n"
        << "  if (il >= n_recv) return;\n"
           "  const int beg = rowptr[r0 + il], end = rowptr[r0 + il + 1];\n"
           "  switch (t) {\n";
      for (int t = 0; t < NU; ++t)
        o << "    case " << t << ": sb_fwd_u" << id0 + t << "<" << (fv.tan ? "true" : "false") << ", " << fv.fl
          << ">(lane, il, beg, end, sender, evec, phi, x, S, ncap, xdot, evdot, phidot, flags, sids[threadIdx.x >> 6]); break;\n";
      o << "  }\n}\n";
    }
  }
  return o.str();
}

std::string generate_source(const Plan& P, bool receiver_route) {
  std::ostringstream o;
  o.precision(17);
  o << "\n// ---- generated for: K=" << P.K << " lmax=" << P.lmax << " in=";
  for (auto& r : P.in) o << r.mul << "x" << r.l << (r.p > 0 ? "e" : "o") << " ";
  o << "out=";
  for (auto& r : P.out) o << r.mul << "x" << r.l << (r.p > 0 ? "e" : "o") << " ";
  o << "norm=" << P.norm << "\n";
  o << "#define K " << P.K << "\n#define NSH " << P.nsh << "\n#define CXI " << P.dim_in << "\n#define CXO " << P.dim_out
    << "\n#define EB " << P.bwd_eb << "\n#define KP " << P.adj_KP << "\n#define ADJ_W " << P.adj_waves << "\n";
  emit_sh(o, P.lmax);
  for (int t = 0; t < (int)P.paths.size(); ++t) emit_path(o, P, t);
  if (P.mode == 1 && P.uvu_C > 0) {
    for (int tan = 0; tan < 2; ++tan) {  // plain and edge-vector-tangent (double backward) variants
      emit_uvu_fwd(o, P, tan);
      emit_uvu_bwd(o, P, false, tan);
      emit_uvu_bwd(o, P, true, tan);
      emit_uvu_wgrad(o, P, tan);
    }
  }

  // streaming adjoint-state GEMM, one instantiation per output multiplicity
  if (P.vec4) {
    std::vector<int> cgs;
    for (auto& g : P.groups)
      if (sbar_streams(P.vec4, g.C) && std::find(cgs.begin(), cgs.end(), g.C) == cgs.end()) cgs.push_back(g.C);
    for (int C : cgs)
      o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_gemm_sbar_c" << C
        << "(const float* M, int nrows, int D, const float* W, const int* ktab, float* Sbar, int dg, int off, int CX,"
           " int r0) {\n  sb_gemm_sbar_s<" << C << ">(M, nrows, D, W, ktab, Sbar, dg, off, CX, r0);\n}\n";
  }

  // x-gradient gather over the sender-sorted view, specialised on the input width
  o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_sender_reduce(const int* send_rowptr,"
       " const int* send_perm, const float* contrib, float* gx, int* cursor, int N, int CX, int e0, int e1,"
       " int first) {\n"
       "  (void)CX;\n"
       "  sb_sender_reduce<CXI>(send_rowptr, send_perm, contrib, gx, cursor, N, e0, e1, first);\n"
       "}\n";
  if (!receiver_route) return o.str();
  // reduced-precision plans: the bf16 variants of the vec4 channel GEMMs, and of the streaming
  // adjoint-state GEMM for output multiplicities in multiples of 32
  if (P.dtype == 1) {
    o << kGemmBf16;
    std::vector<int> cgs;
    for (auto& g : P.groups)
      if (sbar_bf16(P, g.C) && std::find(cgs.begin(), cgs.end(), g.C) == cgs.end()) cgs.push_back(g.C);
    for (int C : cgs)
      o << "extern \"C\" __global__ __launch_bounds__(256) void sobek_gemm_sbar_cb" << C
        << "(const float* M, int nrows, int D, const float* W, const int* ktab, float* Sbar, int dg, int off, int CX,"
           " int r0) {\n  sb_gemm_sbar_sb<" << C << ">(M, nrows, D, W, ktab, Sbar, dg, off, CX, r0);\n}\n";
  }

  // forward S / dS kernels: one wave per (receiver, unit); bf16-GEMM plans store the state in bf16
  const char* st = P.dtype == 1 ? "__bf16" : "float";
  for (int t = 0; t < (int)P.fwd_units.size(); ++t) emit_fwd_unit(o, P, P.fwd_units[t], t);
  const int NU = (int)P.fwd_units.size();
  struct FV { const char* name; bool tan; int fl; };
  const FV fvs[] = {{"S", false, 0}, {"dS_r", true, 4}, {"dS", true, -1}};
  for (const FV& fv : fvs) {
    // two waves per SIMD: keeps the MFMA accumulators in VGPRs without spilling
    o << "extern \"C\" __global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void sobek_fwd_"
      << fv.name
      << "(const int* __restrict__ rowptr, const int* __restrict__ sender, const float* __restrict__ evec,"
         " const float* __restrict__ phi, const float* __restrict__ x, " << st << "* __restrict__ S, int r0, int n_recv,"
         " sb_i64 ncap, const float* __restrict__ xdot, const float* __restrict__ evdot,"
         " const float* __restrict__ phidot, int flags) {\n"
      << "  __shared__ int sids[4][256];\n"
      << "  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;\n"
      << "  const int il = gw / " << NU << ", t = gw % " << NU << ";\n"
      << "  if (il >= n_recv) return;\n"
         "  const int beg = rowptr[r0 + il], end = rowptr[r0 + il + 1];\n"
         "  switch (t) {\n";
    for (int t = 0; t < NU; ++t)
      o << "    case " << t << ": sb_fwd_u" << t << "<" << (fv.tan ? "true" : "false") << ", " << fv.fl
        << ">(lane, il, beg, end, sender, evec, phi, x, S, ncap, xdot, evdot, phidot, flags, sids[threadIdx.x >> 6]); break;\n";
    o << "  }\n}\n";
  }

  // adjoint edge kernels: blocks of ADJ_W waves over (receiver, share of its edges),
  // adjoint state staged in LDS slab by slab, every wave owning a disjoint set of
  // the block's edges
  for (int s = 0; s < (int)P.slabs.size(); ++s) emit_adj_slab(o, P, s);
  const int LDSF = std::max(1, P.bwd_lds_max);
  const int NSL = (int)P.slabs.size();
  o << "template <bool DB, int FL>\nSB_DEV void sb_adj_body(const int* __restrict__ rowptr, const int* __restrict__ sender,"
       " const float* __restrict__ evec, const float* __restrict__ phi, const float* __restrict__ x,"
       " const float* __restrict__ Sb, const float* __restrict__ Sb2, const float* __restrict__ xdot,"
       " const float* __restrict__ evdot, const float* __restrict__ phidot, float* __restrict__ gphi,"
       " float* __restrict__ gevec, float* __restrict__ contrib, int r0, int n_recv, sb_i64 ncap, int e0, int flags,"
       " sb_i64 sb_ncap, int sb_r0, int win0, int win1, int sub_off, float* sS, float* sS2, float* sacc, int* sids) {\n"
       "  const int il = blockIdx.x;\n"
       "  if (il >= n_recv) return;\n"
       "  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;\n"
       "  const int fl = FL >= 0 ? FL : flags;\n"
       // the receiver's edges inside the launch's edge window [win0, win1), split evenly over
       // blockIdx.y in whole 16-edge batches (edge outputs need no reduction)
       "  const int wb = max(rowptr[r0 + il], win0), we = min(rowptr[r0 + il + 1], win1);\n"
       "  const int span = ((we - wb + (int)gridDim.y - 1) / (int)gridDim.y + 15) / 16 * 16;\n"
       "  const int beg = wb + (int)blockIdx.y * span, end = min(we, beg + span);\n"
       "  if (beg >= end) return;\n";
  if (NSL == 1) {
    emit_adj_stage(o, P, 0, "  ");
    o << "  __syncthreads();\n"
         "  sb_adj_s0<DB, FL>(w, lane, beg, end - beg, e0, sender, evec, phi, x, xdot, evdot, phidot, sS, sS2, sacc, gphi,"
         " gevec, contrib, flags, false, sids + 256 * w);\n";
  } else {
    o << "  for (int eb = beg; eb < end; eb += EB) {\n"
         "    const int nb = min(EB, end - eb);\n";
    for (int s = 0; s < NSL; ++s) {
      o << "    __syncthreads();\n";
      emit_adj_stage(o, P, s, "    ");
      o << "    __syncthreads();\n"
        << "    sb_adj_s" << s << "<DB, FL>(w, lane, eb, nb, e0, sender, evec, phi, x, xdot, evdot, phidot, sS, sS2, sacc,"
           " gphi, gevec, contrib, flags, true, sids + 256 * w);\n";
    }
    o << "  }\n";
  }
  o << "}\n";
  o << "#define SB_ADJ_NV(DB, FL) (K + ((!(DB) || (FL) < 0 || ((FL) & 11)) ? NSH : 0) + (((DB) && ((FL) < 0 || ((FL) & 4))) ? NSH : 0))\n";
  struct KV { const char* name; bool db; int fl; int lds_mult; };
  const KV kvs[] = {{"sobek_bwd_E", false, 0, 1}, {"sobek_dbwd_E_r", true, 4, 1}, {"sobek_dbwd_E", true, -1, 2}};
  for (const KV& kv : kvs) {
    o << "extern \"C\" __global__ __launch_bounds__(" << 64 * P.adj_waves << ") __attribute__((amdgpu_waves_per_eu(2))) void " << kv.name
      << "(const int* __restrict__ rowptr, const int* __restrict__ sender, const float* __restrict__ evec,"
         " const float* __restrict__ phi, const float* __restrict__ x, const float* __restrict__ Sb,"
         " const float* __restrict__ Sb2, const float* __restrict__ xdot, const float* __restrict__ evdot,"
         " const float* __restrict__ phidot, float* __restrict__ gphi, float* __restrict__ gevec,"
         " float* __restrict__ contrib, int r0, int n_recv, sb_i64 ncap, int e0, int flags, sb_i64 sb_ncap,"
         " int sb_r0, int win0, int win1, int sub_off) {\n"
      << "  __shared__ __attribute__((aligned(16))) float sS[" << LDSF * kv.lds_mult << "];\n"
      << "  __shared__ int sids[ADJ_W * 256];  // per-wave sender ids of the current segment\n";
    if (NSL > 1)
      o << "  __shared__ float sacc[EB * SB_ADJ_NV(" << (kv.db ? "true" : "false") << ", " << kv.fl << ")];\n";
    else
      o << "  float* sacc = nullptr;\n";
    o << "  sb_adj_body<" << (kv.db ? "true" : "false") << ", " << kv.fl
      << ">(rowptr, sender, evec, phi, x, Sb, Sb2, xdot, evdot, phidot, gphi, gevec, contrib, r0, n_recv, ncap, e0,"
         " flags, sb_ncap, sb_r0, win0, win1, sub_off, sS, sS + " << (kv.lds_mult == 2 ? LDSF : 0) << ", sacc, sids);\n}\n";
  }
  return o.str();
}

}  // namespace sobek
