// Host-side table builder (float64).  See builder.h for the conventions.
#include "builder.h"

#include <algorithm>
#include <cmath>
#include <map>
#include <sstream>
#include <stdexcept>

namespace e3b {

using cd = std::complex<double>;
using Mono = std::array<int, 3>;
using Poly = std::map<Mono, cd>;  // homogeneous polynomial in (x, y, z)

// ---------------------------------------------------------------- irreps
bool parse_irreps(const std::string& s, std::vector<Block>& out, std::string& err) {
  out.clear();
  if (s.empty()) {
    err = "empty irreps string";
    return false;
  }
  std::stringstream ss(s);
  std::string tok;
  while (std::getline(ss, tok, '+')) {
    // strip spaces
    std::string t;
    for (char c : tok)
      if (c != ' ' && c != '\t') t.push_back(c);
    if (t.empty()) {
      err = "empty irreps token";
      return false;
    }
    int mul = 1;
    size_t pos = t.find('x');
    std::string lp = t;
    if (pos != std::string::npos) {
      std::string m = t.substr(0, pos);
      if (m.empty() || m.find_first_not_of("0123456789") != std::string::npos) {
        err = "bad multiplicity in '" + t + "'";
        return false;
      }
      mul = std::stoi(m);
      lp = t.substr(pos + 1);
    }
    if (lp.size() < 2 || (lp.back() != 'e' && lp.back() != 'o')) {
      err = "bad irrep '" + t + "'";
      return false;
    }
    std::string ls = lp.substr(0, lp.size() - 1);
    if (ls.empty() || ls.find_first_not_of("0123456789") != std::string::npos || ls.size() > 3) {
      err = "bad degree in '" + t + "'";
      return false;
    }
    if (mul <= 0) {
      err = "multiplicity must be positive";
      return false;
    }
    out.push_back(Block{mul, std::stoi(ls), lp.back() == 'e' ? 1 : -1});
  }
  return true;
}

bool make_layout(const std::string& irreps, int lmax_sh, int lmax_out, bool natural,
                 Layout& lay, std::string& err) {
  lay = Layout();
  if (!parse_irreps(irreps, lay.blocks, err)) return false;
  if (lmax_sh < 0 || lmax_out < 0) {
    err = "negative degree";
    return false;
  }
  lay.C = lay.blocks[0].mul;
  for (const auto& b : lay.blocks)
    if (b.mul != lay.C) {
      err = "channelwise coupling needs one multiplicity for every block";
      return false;
    }
  lay.lmax_sh = lmax_sh;
  lay.lmax_out = lmax_out;
  lay.natural = natural;
  lay.d_sh = (lmax_sh + 1) * (lmax_sh + 1);
  int xoff = 0, ooff = 0;
  for (size_t xb = 0; xb < lay.blocks.size(); ++xb) {
    const Block& b = lay.blocks[xb];
    for (int l2 = 0; l2 <= lmax_sh; ++l2) {
      int p2 = (l2 % 2) ? -1 : 1;
      for (int l3 = std::abs(b.l - l2); l3 <= std::min(b.l + l2, lmax_out); ++l3) {
        int p3 = b.p * p2;
        if (natural && p3 != ((l3 % 2) ? -1 : 1)) continue;
        Path p{(int)lay.paths.size(), (int)xb, b.l, b.p, l2, l3, p3, xoff, l2 * l2, ooff};
        lay.paths.push_back(p);
        ooff += 2 * l3 + 1;
      }
    }
    xoff += 2 * b.l + 1;
  }
  lay.d_in = xoff;
  lay.d_out = ooff;
  return true;
}

// Everything the generated kernels depend on: the x axis length and, per path
// in order, its degrees and the first x row it reads (parities only select
// which paths exist; the coefficients do not depend on them).
std::string path_signature(const Layout& lay) {
  std::string s = "D" + std::to_string(lay.d_in) + ":";
  for (size_t i = 0; i < lay.paths.size(); ++i) {
    const Path& p = lay.paths[i];
    if (i) s += ",";
    s += std::to_string(p.l1) + "." + std::to_string(p.l2) + "." + std::to_string(p.l3) + "@" +
         std::to_string(p.x_off);
  }
  return s;
}

// ---------------------------------------------------------------- polynomials
static void add(Poly& p, const Mono& m, cd v) {
  auto it = p.find(m);
  if (it == p.end())
    p.emplace(m, v);
  else
    it->second += v;
}

static Poly deriv(const Poly& p, int axis) {
  Poly out;
  for (const auto& [m, v] : p) {
    if (m[axis] == 0) continue;
    Mono n = m;
    n[axis] -= 1;
    add(out, n, v * (double)m[axis]);
  }
  return out;
}

static Poly mul_lin(const Poly& p, cd cx, cd cy, cd cz) {  // (cx x + cy y + cz z) * p
  Poly out;
  for (const auto& [m, v] : p) {
    const cd c[3] = {cx, cy, cz};
    for (int a = 0; a < 3; ++a) {
      if (c[a] == cd(0.0)) continue;
      Mono n = m;
      n[a] += 1;
      add(out, n, v * c[a]);
    }
  }
  return out;
}

static Poly scale(const Poly& p, cd s) {
  Poly out;
  for (const auto& [m, v] : p) out.emplace(m, v * s);
  return out;
}

static Poly sum(const Poly& a, const Poly& b) {
  Poly out = a;
  for (const auto& [m, v] : b) add(out, m, v);
  return out;
}

static cd eval(const Poly& p, const double u[3]) {
  cd s = 0.0;
  for (const auto& [m, v] : p) s += v * std::pow(u[0], m[0]) * std::pow(u[1], m[1]) * std::pow(u[2], m[2]);
  return s;
}

// Lowering operator L_- = (x - i y) d/dz - z (d/dx - i d/dy).
static Poly lower(const Poly& p) {
  const cd I(0.0, 1.0);
  Poly a = mul_lin(deriv(p, 2), 1.0, -I, 0.0);
  Poly b = mul_lin(sum(deriv(p, 0), scale(deriv(p, 1), -I)), 0.0, 0.0, -1.0);
  return sum(a, b);
}

// Complex harmonics Y_l^m, m = -l..l, Condon-Shortley phase, component
// normalisation, as polynomials in (x, y, z).  Top state (-1)^l (x+iy)^l,
// then repeated lowering (App. G.1).
static std::vector<Poly> complex_sh(int l) {
  const cd I(0.0, 1.0);
  std::vector<Poly> Y(2 * l + 1);
  Poly top;
  top[{0, 0, 0}] = (l % 2) ? -1.0 : 1.0;
  for (int i = 0; i < l; ++i) top = mul_lin(top, 1.0, I, 0.0);
  Y[2 * l] = top;
  for (int m = l; m > -l; --m) {
    double a = std::sqrt((double)(l * (l + 1) - m * (m - 1)));
    Y[m - 1 + l] = scale(lower(Y[m + l]), 1.0 / a);
  }
  // normalise: sum_m |Y_l^m(u)|^2 = 2l+1 on the unit sphere (rotation invariant,
  // so one generic point suffices)
  double u[3] = {0.3, -0.5, 0.8};
  double n = std::sqrt(u[0] * u[0] + u[1] * u[1] + u[2] * u[2]);
  for (double& c : u) c /= n;
  double S = 0.0;
  for (const auto& p : Y) S += std::norm(eval(p, u));
  double c = std::sqrt((2.0 * l + 1.0) / S);
  for (auto& p : Y) p = scale(p, c);
  return Y;
}

// Real harmonics in the adopted axes: S_l (textbook axes) with x -> uz, y -> ux,
// z -> uy; as polynomials in (ux, uy, uz).
static std::vector<Poly> real_sh_polys(int l) {
  std::vector<Poly> C = complex_sh(l);
  std::vector<Poly> R(2 * l + 1);
  const double s2 = std::sqrt(2.0);
  for (int m = -l; m <= l; ++m) {
    Poly out;
    const Poly& src = C[std::abs(m) + l];
    double sign = (std::abs(m) % 2) ? -1.0 : 1.0;
    for (const auto& [mono, v] : src) {
      double val;
      if (m > 0)
        val = s2 * sign * v.real();
      else if (m < 0)
        val = s2 * sign * v.imag();
      else
        val = v.real();
      if (val == 0.0) continue;
      // (a, b, c) in (x, y, z) -> exponents (b, c, a) of (ux, uy, uz)
      Mono n = {mono[1], mono[2], mono[0]};
      add(out, n, val);
    }
    R[m + l] = out;
  }
  return R;
}

static std::vector<Mono> monomials(int l) {
  std::vector<Mono> out;
  for (int a = l; a >= 0; --a)
    for (int b = l - a; b >= 0; --b) out.push_back({a, b, l - a - b});
  return out;
}

// Solves A X = B (A n x n, B n x k), complex, partial pivoting.
static std::vector<cd> solve(std::vector<cd> A, std::vector<cd> B, int n, int k) {
  for (int c = 0; c < n; ++c) {
    int piv = c;
    for (int r = c + 1; r < n; ++r)
      if (std::abs(A[r * n + c]) > std::abs(A[piv * n + c])) piv = r;
    if (std::abs(A[piv * n + c]) < 1e-300) throw std::runtime_error("singular system");
    if (piv != c) {
      for (int j = 0; j < n; ++j) std::swap(A[c * n + j], A[piv * n + j]);
      for (int j = 0; j < k; ++j) std::swap(B[c * k + j], B[piv * k + j]);
    }
    for (int r = 0; r < n; ++r) {
      if (r == c) continue;
      cd f = A[r * n + c] / A[c * n + c];
      if (f == cd(0.0)) continue;
      for (int j = 0; j < n; ++j) A[r * n + j] -= f * A[c * n + j];
      for (int j = 0; j < k; ++j) B[r * k + j] -= f * B[c * k + j];
    }
  }
  for (int r = 0; r < n; ++r)
    for (int j = 0; j < k; ++j) B[r * k + j] /= A[r * n + r];
  return B;
}

std::vector<cd> real_basis(int l) {
  // real = U . complex, both polynomials of degree l in (ux, uy, uz); solve in the
  // monomial basis: U (Cx Cx^H) = R Cx^H.
  const int d = 2 * l + 1;
  std::vector<Poly> Cx = complex_sh(l);  // variables (x, y, z) == (ux, uy, uz)
  std::vector<Poly> R = real_sh_polys(l);
  std::vector<Mono> mon = monomials(l);
  const int nm = (int)mon.size();
  std::vector<cd> Cm(d * nm), Rm(d * nm);
  for (int i = 0; i < d; ++i)
    for (int j = 0; j < nm; ++j) {
      auto it = Cx[i].find(mon[j]);
      Cm[i * nm + j] = it == Cx[i].end() ? cd(0.0) : it->second;
      auto jt = R[i].find(mon[j]);
      Rm[i * nm + j] = jt == R[i].end() ? cd(0.0) : jt->second;
    }
  std::vector<cd> G(d * d), B(d * d);  // G = Cx Cx^H, B = R Cx^H
  for (int i = 0; i < d; ++i)
    for (int k = 0; k < d; ++k) {
      cd g = 0.0, b = 0.0;
      for (int j = 0; j < nm; ++j) {
        g += Cm[i * nm + j] * std::conj(Cm[k * nm + j]);
        b += Rm[i * nm + j] * std::conj(Cm[k * nm + j]);
      }
      G[i * d + k] = g;
      B[i * d + k] = b;
    }
  // U G = B  ->  G^T U^T = B^T
  std::vector<cd> GT(d * d), BT(d * d);
  for (int i = 0; i < d; ++i)
    for (int k = 0; k < d; ++k) {
      GT[i * d + k] = G[k * d + i];
      BT[i * d + k] = B[k * d + i];
    }
  std::vector<cd> UT = solve(GT, BT, d, d);
  std::vector<cd> U(d * d);
  for (int i = 0; i < d; ++i)
    for (int k = 0; k < d; ++k) U[i * d + k] = UT[k * d + i];
  // the representation is exact: check U Cx == R
  double worst = 0.0;
  for (int i = 0; i < d; ++i)
    for (int j = 0; j < nm; ++j) {
      cd s = 0.0;
      for (int k = 0; k < d; ++k) s += U[i * d + k] * Cm[k * nm + j];
      worst = std::max(worst, std::abs(s - Rm[i * nm + j]));
    }
  if (worst > 1e-10) throw std::runtime_error("real-basis change is not exact");
  return U;
}

// ---------------------------------------------------------------- Clebsch-Gordan
static double a_plus(int l, int m) { return std::sqrt((double)(l * (l + 1) - m * (m + 1))); }
static double a_minus(int l, int m) { return std::sqrt((double)(l * (l + 1) - m * (m - 1))); }

std::vector<double> complex_cg_block(int l1, int l2, int L) {
  const int d1 = 2 * l1 + 1, d2 = 2 * l2 + 1, dL = 2 * L + 1;
  std::vector<double> out((size_t)dL * d1 * d2, 0.0);
  if (L < std::abs(l1 - l2) || L > l1 + l2) return out;
  // Top state |L L> = sum V_m1 |m1, L-m1>: the eigenvector of J^2 with eigenvalue
  // L(L+1) in the M = L subspace (App. G.2).  On product states
  //   J^2 |m1 m2> = [l1(l1+1) + l2(l2+1) + 2 m1 m2] |m1 m2>
  //               + a-(l1,m1) a+(l2,m2) |m1-1, m2+1> + a+(l1,m1) a-(l2,m2) |m1+1, m2-1>,
  // a tridiagonal system solved by forward recursion from its first row.
  const int lo = std::max(-l1, L - l2), hi = std::min(l1, L + l2);
  const int n = hi - lo + 1;
  std::vector<double> V(n, 0.0);
  const double target = (double)L * (L + 1);
  auto diag = [&](int m1) { return (double)(l1 * (l1 + 1) + l2 * (l2 + 1) + 2 * m1 * (L - m1)); };
  // coupling from |mu+1, L-mu-1> into row mu, and from |mu-1, L-mu+1> into row mu
  auto up = [&](int mu) { return a_minus(l1, mu + 1) * a_plus(l2, L - mu - 1); };
  auto dn = [&](int mu) { return a_plus(l1, mu - 1) * a_minus(l2, L - mu + 1); };
  V[0] = 1.0;
  for (int i = 0; i + 1 < n; ++i) {
    int mu = lo + i;
    double r = (target - diag(mu)) * V[i];
    if (i > 0) r -= dn(mu) * V[i - 1];
    V[i + 1] = r / up(mu);
  }
  {  // last row must hold too
    int mu = hi, i = n - 1;
    double r = (diag(mu) - target) * V[i] + (i > 0 ? dn(mu) * V[i - 1] : 0.0);
    double nv = 0.0;
    for (double v : V) nv += v * v;
    if (std::abs(r) > 1e-9 * std::sqrt(nv)) throw std::runtime_error("top state recursion failed");
  }
  double nv = 0.0;
  for (double v : V) nv += v * v;
  nv = std::sqrt(nv);
  // Condon-Shortley: <l1 l1, l2 L-l1 | L L> > 0 (m1 = l1 is the last entry)
  double sg = V[n - 1] > 0 ? 1.0 : -1.0;
  std::vector<double> cur((size_t)d1 * d2, 0.0);  // |L M> in the product basis
  for (int i = 0; i < n; ++i) {
    int m1 = lo + i, m2 = L - m1;
    cur[(m1 + l1) * d2 + (m2 + l2)] = sg * V[i] / nv;
  }
  for (int M = L; M >= -L; --M) {
    for (int i = 0; i < d1 * d2; ++i) out[(size_t)(M + L) * d1 * d2 + i] = cur[i];
    if (M == -L) break;
    // |L, M-1> = J_- |L, M> / a-(L, M)
    std::vector<double> nxt((size_t)d1 * d2, 0.0);
    for (int m1 = -l1; m1 <= l1; ++m1)
      for (int m2 = -l2; m2 <= l2; ++m2) {
        double v = cur[(m1 + l1) * d2 + (m2 + l2)];
        if (v == 0.0) continue;
        if (m1 > -l1) nxt[(m1 - 1 + l1) * d2 + (m2 + l2)] += a_minus(l1, m1) * v;
        if (m2 > -l2) nxt[(m1 + l1) * d2 + (m2 - 1 + l2)] += a_minus(l2, m2) * v;
      }
    double a = a_minus(L, M);
    for (auto& v : nxt) v /= a;
    cur.swap(nxt);
  }
  return out;
}

std::vector<double> real_cg_block(int l1, int l2, int l3) {
  const int d1 = 2 * l1 + 1, d2 = 2 * l2 + 1, d3 = 2 * l3 + 1;
  std::vector<double> C = complex_cg_block(l1, l2, l3);
  std::vector<cd> U1 = real_basis(l1), U2 = real_basis(l2), U3 = real_basis(l3);
  // R[M][a][b] = sum U3[M][M'] C[M'][m1][m2] conj(U1[a][m1]) conj(U2[b][m2])
  std::vector<cd> T1((size_t)d3 * d1 * d2, 0.0);  // contract M'
  for (int M = 0; M < d3; ++M)
    for (int Mp = 0; Mp < d3; ++Mp) {
      cd u = U3[M * d3 + Mp];
      if (u == cd(0.0)) continue;
      for (int i = 0; i < d1 * d2; ++i) T1[(size_t)M * d1 * d2 + i] += u * C[(size_t)Mp * d1 * d2 + i];
    }
  std::vector<cd> T2((size_t)d3 * d1 * d2, 0.0);  // contract m1 -> a
  for (int M = 0; M < d3; ++M)
    for (int a = 0; a < d1; ++a)
      for (int m1 = 0; m1 < d1; ++m1) {
        cd u = std::conj(U1[a * d1 + m1]);
        if (u == cd(0.0)) continue;
        for (int m2 = 0; m2 < d2; ++m2)
          T2[((size_t)M * d1 + a) * d2 + m2] += u * T1[((size_t)M * d1 + m1) * d2 + m2];
      }
  std::vector<cd> R((size_t)d3 * d1 * d2, 0.0);  // contract m2 -> b
  for (int M = 0; M < d3; ++M)
    for (int a = 0; a < d1; ++a)
      for (int b = 0; b < d2; ++b) {
        cd s = 0.0;
        for (int m2 = 0; m2 < d2; ++m2) s += std::conj(U2[b * d2 + m2]) * T2[((size_t)M * d1 + a) * d2 + m2];
        R[((size_t)M * d1 + a) * d2 + b] = s;
      }
  double re = 0.0, im = 0.0;
  for (const cd& v : R) {
    re = std::max(re, std::abs(v.real()));
    im = std::max(im, std::abs(v.imag()));
  }
  if (im > re)
    for (cd& v : R) v *= cd(0.0, -1.0);
  std::vector<double> out(R.size());
  for (size_t i = 0; i < R.size(); ++i) {
    if (std::abs(R[i].imag()) > 1e-12) throw std::runtime_error("coupling block is not real up to a phase");
    out[i] = std::abs(R[i].real()) < 1e-13 ? 0.0 : R[i].real();
  }
  for (double v : out)
    if (std::abs(v) > 1e-12) {
      if (v < 0)
        for (double& w : out) w = -w;
      break;
    }
  return out;
}

// ---------------------------------------------------------------- tables
ShTable sh_table(int lmax) {
  ShTable t;
  t.lmax = lmax;
  std::vector<std::vector<Poly>> polys;
  std::map<Mono, int> index;
  for (int l = 0; l <= lmax; ++l) {
    polys.push_back(real_sh_polys(l));
    for (const auto& p : polys.back())
      for (const auto& [m, v] : p)
        if (std::abs(v) > 1e-14 && !index.count(m)) index.emplace(m, 0);
  }
  for (auto& [m, i] : index) {
    i = (int)t.mono.size();
    t.mono.push_back(m);
  }
  const int nrow = (lmax + 1) * (lmax + 1);
  t.coef.assign((size_t)nrow * t.mono.size(), 0.0);
  int row = 0;
  for (int l = 0; l <= lmax; ++l)
    for (const auto& p : polys[l]) {
      for (const auto& [m, v] : p)
        if (std::abs(v) > 1e-14) t.coef[(size_t)row * t.mono.size() + index.at(m)] = v.real();
      ++row;
    }
  return t;
}

void sh_eval(const ShTable& t, const double u[3], double* y) {
  const int nrow = (t.lmax + 1) * (t.lmax + 1);
  const size_t nm = t.mono.size();
  for (int r = 0; r < nrow; ++r) {
    double s = 0.0;
    for (size_t j = 0; j < nm; ++j) {
      double c = t.coef[r * nm + j];
      if (c == 0.0) continue;
      s += c * std::pow(u[0], t.mono[j][0]) * std::pow(u[1], t.mono[j][1]) * std::pow(u[2], t.mono[j][2]);
    }
    y[r] = s;
  }
}

std::vector<Record> coo(const Layout& lay) {
  std::vector<Record> out;
  for (const Path& p : lay.paths) {
    std::vector<double> B = real_cg_block(p.l1, p.l2, p.l3);
    const int d1 = 2 * p.l1 + 1, d2 = 2 * p.l2 + 1, d3 = 2 * p.l3 + 1;
    for (int M = 0; M < d3; ++M)
      for (int a = 0; a < d1; ++a)
        for (int b = 0; b < d2; ++b) {
          double v = B[((size_t)M * d1 + a) * d2 + b];
          if (v != 0.0) out.push_back(Record{p.out_off + M, p.x_off + a, p.y_off + b, v});
        }
  }
  std::sort(out.begin(), out.end(), [](const Record& a, const Record& b) {
    if (a.i0 != b.i0) return a.i0 < b.i0;
    if (a.i1 != b.i1) return a.i1 < b.i1;
    return a.i2 < b.i2;
  });
  return out;
}

}  // namespace e3b
