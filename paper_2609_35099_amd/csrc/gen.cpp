// Build-time generator of the straight-line device code for each supported
// irreps variant.
//
// The coupling records depend only on the irreps descriptors, so they are
// fixed before the kernels are compiled and written into the code as literal
// constants (the same idea as the trace-time specialisation of the paper's
// App. E.3, done ahead of time): no coefficient table is read at run time.
// For each variant this emits
//   * the real harmonics of a unit vector and the transposed gradient of the
//     harmonic polynomials (from the builder's polynomial table, App. G.1);
//   * per wave group of paths, the per-edge pre-contraction A = C . y
//     (entries (path, M, m1), App. E.4's grouping of records by i0 then i1),
//     the forward contraction z = A x with the path weight, the backward
//     contraction (cotangents of x, s and y), and the tensor-product rows.
// The same code is emitted for every single x block kind (degree <= 3, all
// or natural-parity paths, harmonics and outputs to degree 3) with its row
// strides left to run time, so that any other layout runs block by block.
//
// usage: gen <out_dir> [irreps/lmax_sh/lmax_out/parity ...]
#include <algorithm>
#include <cctype>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <set>
#include <sstream>
#include <string>
#include <vector>

#include "builder.h"

using namespace e3b;

namespace {

std::string flit(double v) {
  char buf[64];
  std::snprintf(buf, sizeof(buf), "T(%.17e)", v);
  return buf;
}

struct Rec {
  int m2;      // global row on the D_sh axis
  double c;
};

struct Entry {     // one non-zero A[(path, M), m1]
  int k;           // path
  int M;           // row within the path's output block
  int m1;          // row within the x block
  std::vector<Rec> recs;
};

struct VariantSpec {
  std::string blocks;  // x blocks without multiplicities, e.g. "0e+1o+2e+3o"
  int lmax_sh, lmax_out;
  bool natural;
};

// "0e+1o" -> "1x0e+1x1o" (the multiplicity does not change the kernels)
std::string irreps_of(const std::string& blocks) {
  std::string s, tok;
  std::stringstream in(blocks);
  while (std::getline(in, tok, '+')) s += (s.empty() ? "1x" : "+1x") + tok;
  return s;
}

// "irreps/lmax_sh/lmax_out/parity", parity "all" or "natural"
bool parse_spec(const std::string& t, VariantSpec& v) {
  std::vector<std::string> f;
  std::string tok;
  std::stringstream in(t);
  while (std::getline(in, tok, '/')) f.push_back(tok);
  if (f.size() != 4 || (f[3] != "all" && f[3] != "natural")) return false;
  v.blocks = f[0];
  v.lmax_sh = std::atoi(f[1].c_str());
  v.lmax_out = std::atoi(f[2].c_str());
  v.natural = f[3] == "natural";
  return v.lmax_sh >= 0 && v.lmax_sh <= 3 && v.lmax_out >= 0 && v.lmax_out <= 3;
}

struct PathInfo {
  Path p;
  std::vector<double> blk;  // [d3][d1][d2]
  std::vector<Entry> entries;
  int nnz = 0;
};

std::vector<PathInfo> path_infos(const Layout& lay) {
  std::vector<PathInfo> out;
  for (const Path& p : lay.paths) {
    PathInfo pi;
    pi.p = p;
    pi.blk = real_cg_block(p.l1, p.l2, p.l3);
    const int d1 = 2 * p.l1 + 1, d2 = 2 * p.l2 + 1, d3 = 2 * p.l3 + 1;
    for (int M = 0; M < d3; ++M)
      for (int a = 0; a < d1; ++a) {
        Entry e{p.k, M, a, {}};
        for (int b = 0; b < d2; ++b) {
          double v = pi.blk[((size_t)M * d1 + a) * d2 + b];
          if (v != 0.0) e.recs.push_back(Rec{p.y_off + b, v});
        }
        if (!e.recs.empty()) {
          pi.nnz += (int)e.recs.size();
          pi.entries.push_back(e);
        }
      }
    out.push_back(pi);
  }
  return out;
}

int fwd_cost(const PathInfo& pi) { return (int)pi.entries.size() + 2 * pi.p.l3 + 1; }

// Backward contraction routes of one path, per edge and channel.  Every route
// forms B[m2] = sum_{M,m1} C[M,m1,m2] dm[M] x[m1] (then ds = y . B and
// dy += s B) and adds the path's share of the x cotangent,
// t[m1] += s sum_M A[M,m1] dm[M]; they differ in the order of the sums:
//   kRouteA: B through the products dm[M] x[m1] of the path's A entries;
//   kRouteB: B through U[M,m2] = sum_{m1} C x[m1], then dm[M] U[M,m2];
//   kRouteC: per m1, V[m2] = sum_M C dm[M], then B[m2] += x[m1] V[m2] and the
//            unweighted cotangent sum_{m2} y[m2] V[m2]: no A entry is used.
// Routes A and B take t through A: s dm[M] first when the output block is no
// larger than the x block, the sum over M first otherwise.  Two shortcuts
// cover the paths whose coupling is the identity between two of the three
// blocks (unit coefficients, one per entry, a one-to-one map), that is the
// (0, l, l) and (l, 0, l) paths:
//   kRouteX0: a scalar x block (d1 = 1): with T = sum_M y[m2(M)] dm[M],
//             t += s T, ds = x T and dy[m2(M)] += (s x) dm[M];
//   kRouteY0: a scalar harmonic (d2 = 1): with B = sum_M dm[M] x[m1(M)],
//             ds = y B, dy += s B and t[m1(M)] += (s y) dm[M].
// Neither uses A entries.
enum Route { kRouteA, kRouteB, kRouteC, kRouteX0, kRouteY0 };

// The path's coupling as a one-to-one map with unit coefficients between the
// output rows and the rows of the x block (want_x) or of the harmonic block:
// map[M] = partner row, empty if the path has no such structure.
std::vector<int> unit_map(const PathInfo& pi, bool want_x) {
  const int d3 = 2 * pi.p.l3 + 1;
  std::vector<int> map(d3, -1);
  std::set<int> seen;
  if ((int)pi.entries.size() != d3) return {};
  for (const Entry& en : pi.entries) {
    if (en.recs.size() != 1 || std::fabs(en.recs[0].c - 1.0) > 1e-12) return {};
    const int partner = want_x ? en.m1 : en.recs[0].m2 - pi.p.y_off;
    if (map[en.M] != -1 || !seen.insert(partner).second) return {};
    map[en.M] = partner;
  }
  return map;
}

struct RouteCost {
  Route r;
  int cost;  // multiply-adds per edge and channel, ds and dy included
};

RouteCost bwd_route(const PathInfo& pi) {
  const Path& p = pi.p;
  const int d1 = 2 * p.l1 + 1, d2 = 2 * p.l2 + 1, d3 = 2 * p.l3 + 1;
  const int nE = (int)pi.entries.size();
  std::set<std::pair<int, int>> Mm2, m1m2;
  for (const Entry& en : pi.entries)
    for (const Rec& r : en.recs) Mm2.insert({en.M, r.m2}), m1m2.insert({en.m1, r.m2});
  const int common = 2 * d2;
  const int ca = 2 * nE + pi.nnz + std::min(d1, d3) + common;
  const int cb = nE + pi.nnz + (int)Mm2.size() + std::min(d1, d3) + common;
  const int cc = pi.nnz + 2 * (int)m1m2.size() + d1 + common;
  if (d1 == 1 && !unit_map(pi, false).empty()) return {kRouteX0, 2 * d3 + 3};
  if (d2 == 1 && !unit_map(pi, true).empty()) return {kRouteY0, 2 * d3 + 3};
  if (ca <= cb && ca <= cc) return {kRouteA, ca};
  if (cb <= cc) return {kRouteB, cb};
  return {kRouteC, cc};
}

int bwd_cost(const PathInfo& pi) { return bwd_route(pi).cost; }

// Contiguous partition of [0, n) into g parts minimising the largest cost,
// each part [s, i) satisfying fits(s, i).
template <class Fits>
std::vector<std::pair<int, int>> partition(const std::vector<int>& cost, int g, Fits fits) {
  const int n = (int)cost.size();
  const int INF = 1 << 29;
  std::vector<std::vector<int>> best(g + 1, std::vector<int>(n + 1, INF));
  std::vector<std::vector<int>> cut(g + 1, std::vector<int>(n + 1, -1));
  best[0][0] = 0;
  for (int j = 1; j <= g; ++j)
    for (int i = 1; i <= n; ++i)
      for (int s = i - 1; s >= 0; --s) {
        if (!fits(s, i)) continue;
        int c = 0;
        for (int t = s; t < i; ++t) c += cost[t];
        if (best[j - 1][s] >= INF) continue;
        int v = std::max(best[j - 1][s], c);
        if (v < best[j][i]) best[j][i] = v, cut[j][i] = s;
      }
  if (best[g][n] >= INF) return {};
  std::vector<std::pair<int, int>> parts;
  int i = n;
  for (int j = g; j >= 1; --j) {
    int s = cut[j][i];
    parts.push_back({s, i});
    i = s;
  }
  std::reverse(parts.begin(), parts.end());
  return parts;
}

struct Group {
  std::vector<int> paths;      // path indices (global)
  std::vector<int> xrows;      // global D_in rows used, ascending
  std::vector<int> orows;      // global D_out rows, in path order
  std::vector<int> yrows;      // global D_sh rows touched (backward)
  std::vector<Entry> entries;  // A entries in use order
  int na_pad = 0;
};

// with_A(k): whether path k's A entries are staged for the group
template <class WithA>
Group make_group(const Layout& lay, const std::vector<PathInfo>& pis, int b, int e, WithA with_A) {
  Group g;
  std::set<int> xs, ys;
  for (int k = b; k < e; ++k) {
    const PathInfo& pi = pis[k];
    g.paths.push_back(k);
    for (int a = 0; a < 2 * pi.p.l1 + 1; ++a) xs.insert(pi.p.x_off + a);
    for (int M = 0; M < 2 * pi.p.l3 + 1; ++M) g.orows.push_back(pi.p.out_off + M);
    for (int m2 = 0; m2 < 2 * pi.p.l2 + 1; ++m2) ys.insert(pi.p.y_off + m2);
    if (with_A(k))
      for (const Entry& en : pi.entries) g.entries.push_back(en);
  }
  g.xrows.assign(xs.begin(), xs.end());
  g.yrows.assign(ys.begin(), ys.end());
  int na = (int)g.entries.size();
  g.na_pad = (na + 3) / 4 * 4;
  if (g.na_pad % 32 == 0) g.na_pad += 4;  // stagger LDS rows across banks
  (void)lay;
  return g;
}

Group make_group(const Layout& lay, const std::vector<PathInfo>& pis, int b, int e) {
  return make_group(lay, pis, b, e, [](int) { return true; });
}

int index_of(const std::vector<int>& v, int x) {
  auto it = std::find(v.begin(), v.end(), x);
  return it == v.end() ? -1 : (int)(it - v.begin());
}

std::string int_list(const std::vector<int>& v) {
  std::string s = "{";
  for (size_t i = 0; i < v.size(); ++i) s += (i ? ", " : "") + std::to_string(v[i]);
  if (v.empty()) s += "0";
  return s + "}";
}

// ------------------------------------------------------------------ harmonics
void emit_sh(std::ostream& o, int lmax) {
  ShTable t = sh_table(lmax);
  const int nrow = (lmax + 1) * (lmax + 1);
  const size_t nm = t.mono.size();
  auto powname = [](int axis, int e) {
    const char* a = axis == 0 ? "x" : (axis == 1 ? "y" : "z");
    return e == 0 ? std::string("T(1)") : std::string(a) + std::to_string(e);
  };
  auto emit_pows = [&](int upto) {
    for (int e = 2; e <= upto; ++e)
      for (int a = 0; a < 3; ++a) {
        const char* n = a == 0 ? "x" : (a == 1 ? "y" : "z");
        o << "  const T " << n << e << " = " << n << (e - 1 == 1 ? std::string("") : std::to_string(e - 1))
          << " * " << n << ";\n";
      }
    o << "  const T x1 = x, y1 = y, z1 = z; (void)x1; (void)y1; (void)z1;\n";
  };
  auto mono_expr = [&](const std::array<int, 3>& m) {
    std::vector<std::string> f;
    for (int a = 0; a < 3; ++a)
      if (m[a]) f.push_back(powname(a, m[a]));
    if (f.empty()) return std::string("T(1)");
    std::string s;
    for (size_t i = 0; i < f.size(); ++i) s += (i ? " * " : "") + f[i];
    return s;
  };
  // values
  o << "// Real harmonics l <= " << lmax << " of a unit vector (x, y, z); rows l-major, m = -l..l.\n";
  o << "template <class T>\n__device__ __forceinline__ void sh_l" << lmax
    << "(const T x, const T y, const T z, T* __restrict__ Y) {\n";
  emit_pows(lmax);
  for (int r = 0; r < nrow; ++r) {
    std::string acc;
    for (size_t j = 0; j < nm; ++j) {
      double c = t.coef[r * nm + j];
      if (c == 0.0) continue;
      std::string term = flit(c) + " * (" + mono_expr(t.mono[j]) + ")";
      acc += acc.empty() ? term : " + " + term;
    }
    if (acc.empty()) acc = "T(0)";
    o << "  Y[" << r << "] = " << acc << ";\n";
  }
  o << "}\n\n";
  // gradient of sum_r dY[r] P_r(u) with respect to u (polynomial gradient)
  o << "// g = sum_r dY[r] grad P_r(x, y, z), P_r the harmonic polynomials above.\n";
  o << "template <class T>\n__device__ __forceinline__ void sh_grad_l" << lmax
    << "(const T x, const T y, const T z, const T* __restrict__ dY, T& gx, T& gy, T& gz) {\n";
  emit_pows(std::max(lmax - 1, 1));
  const char* gn[3] = {"gx", "gy", "gz"};
  for (int a = 0; a < 3; ++a) {
    // collect: derivative monomial -> list of (row, coef * exponent)
    std::map<std::array<int, 3>, std::vector<std::pair<int, double>>> terms;
    for (int r = 0; r < nrow; ++r)
      for (size_t j = 0; j < nm; ++j) {
        double c = t.coef[r * nm + j];
        if (c == 0.0 || t.mono[j][a] == 0) continue;
        std::array<int, 3> d = t.mono[j];
        double f = c * d[a];
        d[a] -= 1;
        terms[d].push_back({r, f});
      }
    o << "  " << gn[a] << " = T(0);\n";
    for (const auto& [m, lst] : terms) {
      std::string w;
      for (const auto& [r, f] : lst) w += (w.empty() ? "" : " + ") + flit(f) + " * dY[" + std::to_string(r) + "]";
      o << "  " << gn[a] << " = e3fma(" << mono_expr(m) << ", " << w << ", " << gn[a] << ");\n";
    }
  }
  o << "}\n\n";
}

// ------------------------------------------------------------------ groups
void emit_make_A(std::ostream& o, const Group& g) {
  o << "  // A[entry] = sum_m2 C[M, m1, m2] y[m2] for entries (path, M, m1) of this group\n";
  o << "  template <class T>\n  __device__ __forceinline__ static void make_A(const T* __restrict__ y, T* __restrict__ A) {\n";
  o << "    using T4 = typename Vec4<T>::type;\n";
  const int na = (int)g.entries.size();
  for (int q = 0; q < g.na_pad / 4; ++q) {
    o << "    { T4 v;\n";
    const char* comp[4] = {"x", "y", "z", "w"};
    for (int c = 0; c < 4; ++c) {
      int i = 4 * q + c;
      std::string expr = "T(0)";
      if (i < na) {
        const Entry& e = g.entries[i];
        expr = flit(e.recs[0].c) + " * y[" + std::to_string(e.recs[0].m2) + "]";
        for (size_t r = 1; r < e.recs.size(); ++r)
          expr = "e3fma(" + flit(e.recs[r].c) + ", y[" + std::to_string(e.recs[r].m2) + "], " + expr + ")";
      }
      o << "      v." << comp[c] << " = " << expr << ";\n";
    }
    o << "      reinterpret_cast<T4*>(A)[" << q << "] = v; }\n";
  }
  o << "  }\n";
}

std::string aval(int i) {
  const char* comp[4] = {"x", "y", "z", "w"};
  return "a" + std::to_string(i / 4) + "." + comp[i % 4];
}

// emits loads of float4 chunks covering entries [lo, hi) that are not loaded yet
void emit_A_loads(std::ostream& o, int lo, int hi, std::vector<bool>& loaded, const char* ind) {
  for (int q = lo / 4; q <= (hi - 1) / 4; ++q) {
    if (q < (int)loaded.size() && !loaded[q]) {
      o << ind << "const T4 a" << q << " = A4[" << q << "];\n";
      loaded[q] = true;
    }
  }
}

// kFwdLead: float4 chunks of A values requested beyond the last one the
// current row reads (emitted before its products; E3_FWD_PIN() between them
// can keep the compiler from moving them).
int kFwdLead = 4;
// kBwdLead: float4 chunks of A values requested beyond a backward path's own,
// before its code (held there by a scheduling barrier when PIN is set).
int kBwdLead = 2;

void emit_fwd_group(std::ostream& o, const Layout& lay, const std::vector<PathInfo>& pis, const Group& g) {
  o << "  template <int CPL, class T>\n";
  o << "  __device__ __forceinline__ static void edge(const T* __restrict__ A, const T (&x)[NXR][CPL],\n"
       "      const T (&s)[NPATH][CPL], T (&acc)[NROW][CPL]) {\n";
  o << "    using T4 = typename Vec4<T>::type;\n";
  o << "    const T4* __restrict__ A4 = reinterpret_cast<const T4*>(A);\n";
  struct Row {
    int pl, M, orow, lo, hi;
  };
  std::vector<Row> rows;
  int ei = 0, orow = 0;
  for (size_t pl = 0; pl < g.paths.size(); ++pl) {
    const PathInfo& pi = pis[g.paths[pl]];
    for (int M = 0; M < 2 * pi.p.l3 + 1; ++M, ++orow) {
      const int lo = ei;
      while (ei < (int)g.entries.size() && g.entries[ei].k == pi.p.k && g.entries[ei].M == M) ++ei;
      if (ei > lo) rows.push_back({(int)pl, M, orow, lo, ei});
    }
  }
  std::vector<bool> loaded(g.na_pad / 4, false);
  const int nr = (int)rows.size();
  const int nchunk = (int)g.entries.size() > 0 ? ((int)g.entries.size() - 1) / 4 + 1 : 0;
  for (int r = 0; r < nr; ++r) {
    // the chunks this row reads and kFwdLead more (within the entries in use)
    const int last = std::min((rows[r].hi - 1) / 4 + kFwdLead, nchunk - 1);
    emit_A_loads(o, 0, 4 * last + 1, loaded, "    ");
    o << "    E3_FWD_PIN();\n";
    const Row& rw = rows[r];
    const PathInfo& pi = pis[g.paths[rw.pl]];
    o << "    {  // path " << pi.p.k << " (" << pi.p.l1 << "," << pi.p.l2 << "," << pi.p.l3 << ") row " << rw.M << "\n";
    o << "#pragma unroll\n      for (int c = 0; c < CPL; ++c) {\n";
    for (int i = rw.lo; i < rw.hi; ++i) {
      const int xl = index_of(g.xrows, pi.p.x_off + g.entries[i].m1);
      if (i == rw.lo)
        o << "        T z = " << aval(i) << " * x[" << xl << "][c];\n";
      else
        o << "        z = e3fma(" << aval(i) << ", x[" << xl << "][c], z);\n";
    }
    o << "        acc[" << rw.orow << "][c] = e3fma(s[" << rw.pl << "][c], z, acc[" << rw.orow << "][c]);\n";
    o << "      }\n    }\n";
  }
  o << "  }\n";
  (void)lay;
}

// The three forward terms of the double backward's output cotangent in one
// pass: acc += s (A xd + A2 x) + sd (A x), with A from the harmonics y and A2
// from their tangent yd (same entry layout).
void emit_fwd3_group(std::ostream& o, const std::vector<PathInfo>& pis, const Group& g) {
  o << "  template <int CPL, class T>\n";
  o << "  __device__ __forceinline__ static void edge3(const T* __restrict__ A, const T* __restrict__ A2,\n"
       "      const T (&x)[NXR][CPL], const T (&xd)[NXR][CPL], const T (&s)[NPATH][CPL],\n"
       "      const T (&sd)[NPATH][CPL], T (&acc)[NROW][CPL]) {\n";
  o << "    using T4 = typename Vec4<T>::type;\n";
  o << "    const T4* __restrict__ A4 = reinterpret_cast<const T4*>(A);\n";
  o << "    const T4* __restrict__ B4 = reinterpret_cast<const T4*>(A2);\n";
  // The path weights are folded into the x rows first: with
  // u = s xd + sd x and v = s x (per channel, per x row of the path),
  // acc[M] += sum A[M,m1] u[m1] + sum A2[M,m1] v[m1].  Each path is a block
  // of its own, which loads the A chunks it reads (a chunk shared by two
  // paths is read twice).
  int ei = 0, orow = 0;
  for (size_t pl = 0; pl < g.paths.size(); ++pl) {
    const PathInfo& pi = pis[g.paths[pl]];
    const int d1 = 2 * pi.p.l1 + 1;
    std::vector<bool> loaded(g.na_pad / 4, false);
    o << "    {  // path " << pi.p.k << " (" << pi.p.l1 << "," << pi.p.l2 << "," << pi.p.l3 << ")\n";
    o << "      T u[" << d1 << "][CPL], v[" << d1 << "][CPL];\n";
    o << "#pragma unroll\n      for (int c = 0; c < CPL; ++c) {\n";
    for (int m1 = 0; m1 < d1; ++m1) {
      const int xl = index_of(g.xrows, pi.p.x_off + m1);
      o << "        u[" << m1 << "][c] = e3fma(sd[" << pl << "][c], x[" << xl << "][c], s[" << pl << "][c] * xd[" << xl
        << "][c]);\n";
      o << "        v[" << m1 << "][c] = s[" << pl << "][c] * x[" << xl << "][c];\n";
    }
    o << "      }\n";
    for (int M = 0; M < 2 * pi.p.l3 + 1; ++M, ++orow) {
      const int lo = ei;
      while (ei < (int)g.entries.size() && g.entries[ei].k == pi.p.k && g.entries[ei].M == M) ++ei;
      if (ei == lo) continue;
      for (int q = lo / 4; q <= (ei - 1) / 4; ++q)
        if (!loaded[q]) {
          o << "      const T4 a" << q << " = A4[" << q << "], b" << q << " = B4[" << q << "];\n";
          loaded[q] = true;
        }
      o << "#pragma unroll\n      for (int c = 0; c < CPL; ++c) {  // row " << M << "\n";
      o << "        T r = acc[" << orow << "][c];\n";
      for (int i = lo; i < ei; ++i) {
        const int m1 = g.entries[i].m1;
        o << "        r = e3fma(" << aval(i) << ", u[" << m1 << "][c], r);\n";
      }
      for (int i = lo; i < ei; ++i) {
        const int m1 = g.entries[i].m1;
        o << "        r = e3fma(b" << aval(i).substr(1) << ", v[" << m1 << "][c], r);\n";
      }
      o << "        acc[" << orow << "][c] = r;\n";
      o << "      }\n";
    }
    o << "    }\n";
  }
  o << "  }\n";
}

void emit_bwd_group(std::ostream& o, const Layout& lay, const std::vector<PathInfo>& pis, const Group& g) {
  o << "  // Per edge and channel, path by path: B[m2] = sum C dm x, ds = y . B, dy += s B\n"
       "  // (summed over this lane's channels), and t, the x cotangent before the sender\n"
       "  // reduction, += s sum_M A dm; the order of each path's sums is its cheapest route.\n";
  o << "  template <bool PIN, int CPL, class DS, class T>\n";
  o << "  __device__ __forceinline__ static void edge(const T* __restrict__ A, const T (&Y)[D_SH],\n"
       "      const T (&x)[NXR][CPL], const T (&s)[NPATH][CPL], const T (&dm)[NROW][CPL],\n"
       "      T (&t)[NXR][CPL], T (&dy)[D_SH], DS& st_ds) {\n";
  o << "    using T4 = typename Vec4<T>::type;\n";
  o << "    const T4* __restrict__ A4 = reinterpret_cast<const T4*>(A);\n";
  o << "    (void)A4;\n";
  std::vector<bool> loaded(g.na_pad / 4, false);
  int ei = 0, orow0 = 0;
  for (size_t pl = 0; pl < g.paths.size(); ++pl) {
    const PathInfo& pi = pis[g.paths[pl]];
    const Path& p = pi.p;
    const int d1 = 2 * p.l1 + 1, d2 = 2 * p.l2 + 1, d3 = 2 * p.l3 + 1;
    const Route route = bwd_route(pi).r;
    const std::string S = "s[" + std::to_string(pl) + "][c]";
    auto DM = [&](int M) { return "dm[" + std::to_string(orow0 + M) + "][c]"; };
    auto X = [&](int m1) { return "x[" + std::to_string(index_of(g.xrows, p.x_off + m1)) + "][c]"; };
    auto Tt = [&](int m1) { return "t[" + std::to_string(index_of(g.xrows, p.x_off + m1)) + "][c]"; };
    int lo = ei;
    const bool uses_A = route == kRouteA || route == kRouteB;
    if (uses_A) {
      while (ei < (int)g.entries.size() && g.entries[ei].k == p.k) ++ei;
      if (ei > lo) {
        // this path's chunks and kBwdLead more
        const int nchunk = ((int)g.entries.size() - 1) / 4 + 1;
        emit_A_loads(o, 0, 4 * std::min((ei - 1) / 4 + kBwdLead, nchunk - 1) + 1, loaded, "    ");
        o << "    if constexpr (PIN) __builtin_amdgcn_sched_barrier(0);\n";
      }
    }
    static const char* rname[5] = {"A", "B", "C", "X0", "Y0"};
    if (route == kRouteX0 || route == kRouteY0) {
      // identity coupling between the output block and the harmonic (X0) or x (Y0) block
      const std::vector<int> map = unit_map(pi, route == kRouteY0);
      o << "    {  // path " << p.k << " (" << p.l1 << "," << p.l2 << "," << p.l3 << "), route " << rname[route] << "\n";
      o << "      T dsv[CPL];\n";
      o << "#pragma unroll\n      for (int c = 0; c < CPL; ++c) {\n";
      if (route == kRouteX0) {
        auto Yr = [&](int b) { return "Y[" + std::to_string(p.y_off + b) + "]"; };
        std::string tt = Yr(map[0]) + " * " + DM(0);
        for (int M = 1; M < d3; ++M) tt = "e3fma(" + Yr(map[M]) + ", " + DM(M) + ", " + tt + ")";
        o << "        const T Tv = " << tt << ";\n";
        o << "        " << Tt(0) << " = e3fma(" << S << ", Tv, " << Tt(0) << ");\n";
        o << "        dsv[c] = " << X(0) << " * Tv;\n";
        o << "        const T sx = " << S << " * " << X(0) << ";\n";
        for (int M = 0; M < d3; ++M)
          o << "        dy[" << p.y_off + map[M] << "] = e3fma(sx, " << DM(M) << ", dy[" << p.y_off + map[M] << "]);\n";
      } else {
        std::string bb = DM(0) + " * " + X(map[0]);
        for (int M = 1; M < d3; ++M) bb = "e3fma(" + DM(M) + ", " + X(map[M]) + ", " + bb + ")";
        const std::string y0 = "Y[" + std::to_string(p.y_off) + "]";
        o << "        const T B = " << bb << ";\n";
        o << "        dsv[c] = " << y0 << " * B;\n";
        o << "        dy[" << p.y_off << "] = e3fma(" << S << ", B, dy[" << p.y_off << "]);\n";
        o << "        const T sy = " << S << " * " << y0 << ";\n";
        for (int M = 0; M < d3; ++M)
          o << "        " << Tt(map[M]) << " = e3fma(sy, " << DM(M) << ", " << Tt(map[M]) << ");\n";
      }
      o << "      }\n";
      o << "      st_ds(" << pl << ", dsv);\n";
      o << "    }\n";
      orow0 += d3;
      continue;
    }
    o << "    {  // path " << p.k << " (" << p.l1 << "," << p.l2 << "," << p.l3 << "), route " << rname[route] << "\n";
    o << "      T dsv[CPL];\n";
    o << "#pragma unroll\n      for (int c = 0; c < CPL; ++c) {\n";
    std::vector<bool> binit(d2, false);
    std::string decl;
    for (int b = 0; b < d2; ++b) decl += (b ? ", b" : "b") + std::to_string(b);
    o << "        T " << decl << ";\n";
    auto acc_b = [&](int b, const std::string& term_a, const std::string& term_b) {
      // b_b += term_a * term_b
      if (!binit[b]) {
        o << "          b" << b << " = " << term_a << " * " << term_b << ";\n";
        binit[b] = true;
      } else {
        o << "          b" << b << " = e3fma(" << term_a << ", " << term_b << ", b" << b << ");\n";
      }
    };
    if (uses_A) {
      // x cotangent through the A entries [lo, ei)
      if (d3 <= d1) {
        std::set<int> Ms;
        for (int i = lo; i < ei; ++i) Ms.insert(g.entries[i].M);
        for (int M : Ms) o << "        const T w" << M << " = " << S << " * " << DM(M) << ";\n";
        for (int i = lo; i < ei; ++i)
          o << "        " << Tt(g.entries[i].m1) << " = e3fma(" << aval(i) << ", w" << g.entries[i].M << ", "
            << Tt(g.entries[i].m1) << ");\n";
      } else {
        for (int m1 = 0; m1 < d1; ++m1) {
          bool first = true;
          for (int i = lo; i < ei; ++i) {
            if (g.entries[i].m1 != m1) continue;
            if (first)
              o << "        {\n          T u = " << aval(i) << " * " << DM(g.entries[i].M) << ";\n";
            else
              o << "          u = e3fma(" << aval(i) << ", " << DM(g.entries[i].M) << ", u);\n";
            first = false;
          }
          if (!first) o << "          " << Tt(m1) << " = e3fma(" << S << ", u, " << Tt(m1) << ");\n        }\n";
        }
      }
    }
    if (route == kRouteA) {
      for (int i = lo; i < ei; ++i) {
        const Entry& en = g.entries[i];
        o << "        {\n          const T pr = " << DM(en.M) << " * " << X(en.m1) << ";\n";
        for (const Rec& r : en.recs) acc_b(r.m2 - p.y_off, flit(r.c), "pr");
        o << "        }\n";
      }
    } else if (route == kRouteB) {
      // U[M, m2] = sum_m1 C x[m1], then b[m2] += dm[M] U[M, m2]
      for (int M = 0; M < d3; ++M) {
        std::map<int, std::vector<std::pair<int, double>>> u;  // m2 -> (m1, c)
        for (const Entry& en : pi.entries)
          if (en.M == M)
            for (const Rec& r : en.recs) u[r.m2 - p.y_off].push_back({en.m1, r.c});
        for (const auto& [b, lst] : u) {
          o << "        {\n          T u = " << flit(lst[0].second) << " * " << X(lst[0].first) << ";\n";
          for (size_t j = 1; j < lst.size(); ++j)
            o << "          u = e3fma(" << flit(lst[j].second) << ", " << X(lst[j].first) << ", u);\n";
          acc_b(b, DM(M), "u");
          o << "        }\n";
        }
      }
    } else {
      // per m1: V[m2] = sum_M C dm[M]; b[m2] += x[m1] V[m2]; t[m1] += s sum_m2 y[m2] V[m2]
      for (int m1 = 0; m1 < d1; ++m1) {
        std::map<int, std::vector<std::pair<int, double>>> v;  // m2 -> (M, c)
        for (const Entry& en : pi.entries)
          if (en.m1 == m1)
            for (const Rec& r : en.recs) v[r.m2 - p.y_off].push_back({en.M, r.c});
        if (v.empty()) continue;
        o << "        {\n";
        std::string ty;
        for (const auto& [b, lst] : v) {
          const std::string vn = "v" + std::to_string(b);
          o << "          T " << vn << " = " << flit(lst[0].second) << " * " << DM(lst[0].first) << ";\n";
          for (size_t j = 1; j < lst.size(); ++j)
            o << "          " << vn << " = e3fma(" << flit(lst[j].second) << ", " << DM(lst[j].first) << ", " << vn
              << ");\n";
          acc_b(b, X(m1), vn);
          const std::string yb = "Y[" + std::to_string(p.y_off + b) + "]";
          ty = ty.empty() ? yb + " * " + vn : "e3fma(" + yb + ", " + vn + ", " + ty + ")";
        }
        o << "          " << Tt(m1) << " = e3fma(" << S << ", " << ty << ", " << Tt(m1) << ");\n";
        o << "        }\n";
      }
    }
    std::string ds;
    for (int b = 0; b < d2; ++b) {
      if (!binit[b]) continue;
      std::string yb = "Y[" + std::to_string(p.y_off + b) + "]";
      ds = ds.empty() ? yb + " * b" + std::to_string(b) : "e3fma(" + yb + ", b" + std::to_string(b) + ", " + ds + ")";
    }
    o << "        dsv[c] = " << (ds.empty() ? std::string("T(0)") : ds) << ";\n";
    for (int b = 0; b < d2; ++b) {
      if (!binit[b]) continue;
      o << "        dy[" << p.y_off + b << "] = e3fma(" << S << ", b" << b << ", dy[" << p.y_off + b << "]);\n";
    }
    for (int b = 0; b < d2; ++b)
      if (!binit[b]) o << "        (void)b" << b << ";\n";
    o << "      }\n";
    o << "      st_ds(" << pl << ", dsv);\n";
    o << "    }\n";
    orow0 += d3;
  }
  o << "  }\n";
  (void)lay;
}

// The three backward sweeps of the double backward in one (per edge and
// channel, every path through V = sum_M C dm, no A entry): with V[m1][m2],
//   B1 = sum_m1 xd V, B2 = sum_m1 x V, T1 = sum_m2 y V, T2 = sum_m2 y2 V,
//   gs = y . B1 + y2 . B2,  dy += s B1 + sd B2,  t += s T2 + sd T1,
// i.e. ds of (xd, y, s) plus ds of (x, y2, s), dy of (xd, y, s) plus dy of
// (x, y, sd), and the x cotangents of (x, y2, s) and (x, y, sd).
void emit_bwd3_group(std::ostream& o, const std::vector<PathInfo>& pis, const Group& g) {
  o << "  template <int CPL, class DS, class T>\n";
  o << "  __device__ __forceinline__ static void edge3(const T (&Y)[D_SH], const T (&Y2)[D_SH],\n"
       "      const T (&x)[NXR][CPL], const T (&xd)[NXR][CPL], const T (&s)[NPATH][CPL],\n"
       "      const T (&sd)[NPATH][CPL], const T (&dm)[NROW][CPL], T (&t)[NXR][CPL],\n"
       "      T (&dy)[D_SH], DS& st_ds) {\n";
  // Per path and x row m1, with V[m2] = sum_M C dm[M], T1 = y . V and T2 = y2 . V:
  //   gs += xd[m1] T1 + x[m1] T2          (= y . B1 + y2 . B2 summed over m1),
  //   dy[m2] += z[m1] V[m2], z = s xd + sd x  (= s B1 + sd B2),
  //   t[m1] += s T2 + sd T1.
  int orow0 = 0;
  for (size_t pl = 0; pl < g.paths.size(); ++pl) {
    const PathInfo& pi = pis[g.paths[pl]];
    const Path& p = pi.p;
    const int d1 = 2 * p.l1 + 1, d3 = 2 * p.l3 + 1;
    const std::string S = "s[" + std::to_string(pl) + "][c]", SD = "sd[" + std::to_string(pl) + "][c]";
    auto DM = [&](int M) { return "dm[" + std::to_string(orow0 + M) + "][c]"; };
    auto xi = [&](int m1) { return std::to_string(index_of(g.xrows, p.x_off + m1)); };
    o << "    {  // path " << p.k << " (" << p.l1 << "," << p.l2 << "," << p.l3 << ")\n";
    o << "      T gsv[CPL];\n";
    o << "#pragma unroll\n      for (int c = 0; c < CPL; ++c) {\n";
    o << "        T gs = T(0);\n";
    for (int m1 = 0; m1 < d1; ++m1) {
      std::map<int, std::vector<std::pair<int, double>>> v;  // m2 -> (M, c)
      for (const Entry& en : pi.entries)
        if (en.m1 == m1)
          for (const Rec& r : en.recs) v[r.m2 - p.y_off].push_back({en.M, r.c});
      if (v.empty()) continue;
      o << "        {\n";
      o << "          const T z = e3fma(" << SD << ", x[" << xi(m1) << "][c], " << S << " * xd[" << xi(m1) << "][c]);\n";
      std::string t1, t2;
      for (const auto& [b, lst] : v) {
        const std::string vn = "v" + std::to_string(b);
        o << "          T " << vn << " = " << flit(lst[0].second) << " * " << DM(lst[0].first) << ";\n";
        for (size_t j = 1; j < lst.size(); ++j)
          o << "          " << vn << " = e3fma(" << flit(lst[j].second) << ", " << DM(lst[j].first) << ", " << vn
            << ");\n";
        const std::string dyi = "dy[" + std::to_string(p.y_off + b) + "]";
        o << "          " << dyi << " = e3fma(z, " << vn << ", " << dyi << ");\n";
        const std::string yb = "Y[" + std::to_string(p.y_off + b) + "]", y2b = "Y2[" + std::to_string(p.y_off + b) + "]";
        t1 = t1.empty() ? yb + " * " + vn : "e3fma(" + yb + ", " + vn + ", " + t1 + ")";
        t2 = t2.empty() ? y2b + " * " + vn : "e3fma(" + y2b + ", " + vn + ", " + t2 + ")";
      }
      o << "          const T t1 = " << t1 << ", t2 = " << t2 << ";\n";
      o << "          t[" << xi(m1) << "][c] = e3fma(" << S << ", t2, e3fma(" << SD << ", t1, t[" << xi(m1) << "][c]));\n";
      o << "          gs = e3fma(xd[" << xi(m1) << "][c], t1, e3fma(x[" << xi(m1) << "][c], t2, gs));\n";
      o << "        }\n";
    }
    o << "        gsv[c] = gs;\n";
    o << "      }\n";
    o << "      st_ds(" << pl << ", gsv);\n";
    o << "    }\n";
    orow0 += d3;
  }
  o << "  }\n";
}

void emit_tp_group(std::ostream& o, const Layout& lay, const std::vector<PathInfo>& pis, const Group& g) {
  o << "  // Weighted tensor product rows: z[i0] = w[i3(i0)] * sum A x; each row handed to st.\n";
  o << "  template <int CPL, class ST, class T>\n";
  o << "  __device__ __forceinline__ static void rows(const T* __restrict__ A, const T (&x)[NXR][CPL],\n"
       "      const T (&w)[NPATH][CPL], ST& st) {\n";
  o << "    using T4 = typename Vec4<T>::type;\n";
  o << "    const T4* __restrict__ A4 = reinterpret_cast<const T4*>(A);\n";
  std::vector<bool> loaded(g.na_pad / 4, false);
  int ei = 0;
  for (size_t pl = 0; pl < g.paths.size(); ++pl) {
    const PathInfo& pi = pis[g.paths[pl]];
    const int d3 = 2 * pi.p.l3 + 1;
    for (int M = 0; M < d3; ++M) {
      int lo = ei;
      while (ei < (int)g.entries.size() && g.entries[ei].k == pi.p.k && g.entries[ei].M == M) ++ei;
      if (ei > lo) emit_A_loads(o, lo, ei, loaded, "    ");
      o << "    {  // path " << pi.p.k << " row " << M << "\n";
      o << "      T v[CPL];\n";
      o << "#pragma unroll\n      for (int c = 0; c < CPL; ++c) {\n";
      if (ei == lo) {
        o << "        v[c] = T(0);\n";
      } else {
        for (int i = lo; i < ei; ++i) {
          int xl = index_of(g.xrows, pi.p.x_off + g.entries[i].m1);
          if (i == lo)
            o << "        T z = " << aval(i) << " * x[" << xl << "][c];\n";
          else
            o << "        z = e3fma(" << aval(i) << ", x[" << xl << "][c], z);\n";
        }
        o << "        v[c] = w[" << pl << "][c] * z;\n";
      }
      o << "      }\n";
      o << "      st(" << pi.p.out_off + M << ", v);\n";
      o << "    }\n";
    }
  }
  o << "  }\n";
  (void)lay;
}

void emit_group_meta(std::ostream& o, const Group& g) {
  o << "  static constexpr int NA = " << g.na_pad << ";\n";
  o << "  static constexpr int NXR = " << g.xrows.size() << ";\n";
  o << "  static constexpr int NPATH = " << g.paths.size() << ";\n";
  o << "  static constexpr int NROW = " << g.orows.size() << ";\n";
  o << "  static constexpr int XROW[" << std::max<size_t>(1, g.xrows.size()) << "] = " << int_list(g.xrows) << ";\n";
  o << "  static constexpr int PATH[" << std::max<size_t>(1, g.paths.size()) << "] = " << int_list(g.paths) << ";\n";
  o << "  static constexpr int OROW[" << std::max<size_t>(1, g.orows.size()) << "] = " << int_list(g.orows) << ";\n";
}

// Degrees of the blocks, with their parities when they select paths.
std::string tag_of(const VariantSpec& v) {
  std::string t = "V_x";
  for (char c : v.blocks)
    if (std::isdigit((unsigned char)c) || (v.natural && (c == 'e' || c == 'o'))) t += c;
  t += "_s" + std::to_string(v.lmax_sh) + "_o" + std::to_string(v.lmax_out);
  if (v.natural) t += "_n";
  return t;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc < 2) {
    std::fprintf(stderr,
                 "usage: gen <out_dir> [irreps/lmax_sh/lmax_out/parity ...]\n"
                 "writes <out_dir>/variants.inc (the code of every variant), variant_table.inc and one\n"
                 "v_<tag>.hip unit per variant; the listed layouts are compiled besides the defaults\n");
    return 2;
  }
  const std::string out_dir = argv[1];
  // Compiled variants: x blocks (all paths kept, or the natural-parity ones),
  // harmonics up to lmax_sh, outputs up to lmax_out.  Layouts with the same
  // kernels (same path signature and harmonics) are compiled once.
  std::vector<VariantSpec> specs = {
      {"0e+1o", 2, 2, false},
      {"0e+1o+2e", 3, 3, false},
      {"0e+1o", 3, 3, false},
      {"0e+1o+2e+3o", 3, 3, false},
      {"0e+1o+2e", 2, 2, false},
      {"0e+1o", 2, 2, true},
      {"0e+1o", 3, 3, true},
      {"0e+1o+2e", 3, 3, true},
      {"0e+1o+2e+3o", 3, 3, true},
      {"1o+0e+3o+2e", 3, 3, false},
  };
  for (int i = 2; i < argc; ++i) {
    VariantSpec v;
    if (!parse_spec(argv[i], v)) {
      std::fprintf(stderr, "gen: bad layout '%s' (want irreps/lmax_sh/lmax_out/all|natural, l <= 3)\n", argv[i]);
      return 2;
    }
    specs.push_back(v);
  }
  // Forward groups: contiguous paths balanced on per-channel FMA work, each
  // within a register budget (per channel of a lane: accumulators + two
  // buffered copies of its x rows and path weights).  Tuning knobs from the
  // environment (experiments only).
  auto knob = [](const char* name, int def) {
    const char* e = std::getenv(name);
    return e ? std::atoi(e) : def;
  };
  const int FWD_TARGET = knob("E3GEN_FWD_TARGET", 200);
  const int FWD_REGS = knob("E3GEN_FWD_REGS", 1000);
  const int FWD_RMAX = knob("E3GEN_FWD_RMAX", 56);
  kFwdLead = knob("E3GEN_FWD_LEAD", kFwdLead);
  kBwdLead = knob("E3GEN_BWD_LEAD", kBwdLead);
  const int BWD_TARGET = 640;
  const int BWD_RMAX = 56;

  std::ostringstream o;
  o << "// GENERATED by gen.cpp from the host table builder -- do not edit.\n";
  o << "#pragma once\n\nnamespace e3gen {\n\n";
  // the code below is generic in the scalar type T (float or double)
  o << "template <class T> struct Vec4;\n"
       "template <> struct Vec4<float> { using type = float4; };\n"
       "template <> struct Vec4<double> { using type = double4; };\n"
       "__device__ __forceinline__ float e3fma(float a, float b, float c) { return fmaf(a, b, c); }\n"
       "__device__ __forceinline__ double e3fma(double a, double b, double c) { return fma(a, b, c); }\n\n";
  for (int l = 0; l <= 3; ++l) emit_sh(o, l);

  // One layout's struct: its constants, forward groups, backward groups and
  // the tensor product's single group.  rt: strides and group offsets come at
  // run time (a single-block kind composed into larger layouts).
  auto emit_layout = [&](std::ostream& os, const std::string& tag, const Layout& lay, int lmax_sh, bool rt) {
    std::vector<PathInfo> pis = path_infos(lay);
    const int np = (int)pis.size();
    std::vector<int> fc(np), bc(np), rows(np);
    int total_f = 0;
    for (int k = 0; k < np; ++k) {
      fc[k] = fwd_cost(pis[k]);
      bc[k] = bwd_cost(pis[k]);
      rows[k] = 2 * pis[k].p.l3 + 1;
      total_f += fc[k];
    }
    // forward groups: contiguous paths, balanced cost
    auto fwd_regs = [&](int s, int e) {  // rows + 2 x rows + 2 path weights, per lane channel
      std::set<int> xs;
      int r = 0;
      for (int k = s; k < e; ++k) {
        r += rows[k];
        for (int a = 0; a < 2 * pis[k].p.l1 + 1; ++a) xs.insert(pis[k].p.x_off + a);
      }
      return r + 2 * (int)xs.size() + 2 * (e - s);
    };
    int gf = std::max(1, (int)std::lround((double)total_f / FWD_TARGET));
    std::vector<std::pair<int, int>> fparts;
    for (;; ++gf) {
      fparts = partition(fc, gf, [&](int s, int e) {
        int r = 0;
        for (int k = s; k < e; ++k) r += rows[k];
        return r <= FWD_RMAX && fwd_regs(s, e) <= FWD_REGS;
      });
      if (!fparts.empty()) break;
    }
    // backward groups: whole x blocks (so the x cotangent rows of different
    // groups never overlap), merged while small
    std::vector<std::pair<int, int>> bparts;
    {
      int s = 0;
      while (s < np) {
        int e = s, cost = 0, r = 0;
        while (e < np) {
          // extent of the x block starting at path e
          int xb = pis[e].p.xb, f = e, c2 = 0, r2 = 0;
          while (f < np && pis[f].p.xb == xb) c2 += bc[f], r2 += rows[f], ++f;
          if (e > s && (cost + c2 > BWD_TARGET || r + r2 > BWD_RMAX)) break;
          cost += c2, r += r2, e = f;
        }
        bparts.push_back({s, e});
        s = e;
      }
    }
    std::vector<Group> fg, bg;
    for (auto [b, e] : fparts) fg.push_back(make_group(lay, pis, b, e));
    for (auto [b, e] : bparts)
      bg.push_back(make_group(lay, pis, b, e, [&](int k) {
        const Route r = bwd_route(pis[k]).r;
        return r == kRouteA || r == kRouteB;
      }));
    Group tpg = make_group(lay, pis, 0, np);

    int maxf = 0, maxb = 0;
    for (auto& g : fg) maxf = std::max(maxf, g.na_pad);
    for (auto& g : bg) maxb = std::max(maxb, g.na_pad);
    os << "// ============================================================ " << tag << "\n";
    os << "// " << np << " paths, D_in " << lay.d_in << ", D_sh " << lay.d_sh << ", D_out " << lay.d_out << "\n";
    os << "struct " << tag << " {\n";
    os << "  static constexpr int D_IN = " << lay.d_in << ", D_SH = " << lay.d_sh << ", D_OUT = " << lay.d_out
       << ", NP = " << np << ", LSH = " << lmax_sh << ";\n";
    os << "  static constexpr bool RT = " << (rt ? "true" : "false") << ";\n";
    os << "  static constexpr const char* SIG = \"" << path_signature(lay) << "\";\n";
    os << "  static constexpr int NFG = " << fg.size() << ", NBG = " << bg.size() << ";\n";
    os << "  static constexpr int MAX_NA_F = " << maxf << ", MAX_NA_B = " << maxb << ", NA_TP = " << tpg.na_pad
       << ";\n";
    os << "  template <class T>\n  __device__ __forceinline__ static void sh(T x, T y, T z, T* Y) { sh_l" << lmax_sh
       << "(x, y, z, Y); }\n";
    os << "  template <class T>\n  __device__ __forceinline__ static void sh_grad(T x, T y, T z, const T* dY, T& gx, T& gy, T& gz) { sh_grad_l"
       << lmax_sh << "(x, y, z, dY, gx, gy, gz); }\n";
    os << "  template <int G> struct FG;\n  template <int G> struct BG;\n  struct TP;\n};\n\n";
    for (size_t gi = 0; gi < fg.size(); ++gi) {
      os << "template <> struct " << tag << "::FG<" << gi << "> {\n";
      os << "  static constexpr int D_SH = " << lay.d_sh << ";\n";
      emit_group_meta(os, fg[gi]);
      emit_make_A(os, fg[gi]);
      emit_fwd_group(os, lay, pis, fg[gi]);
      emit_fwd3_group(os, pis, fg[gi]);
      os << "};\n\n";
    }
    for (size_t gi = 0; gi < bg.size(); ++gi) {
      os << "template <> struct " << tag << "::BG<" << gi << "> {\n";
      os << "  static constexpr int D_SH = " << lay.d_sh << ";\n";
      emit_group_meta(os, bg[gi]);
      emit_make_A(os, bg[gi]);
      emit_bwd_group(os, lay, pis, bg[gi]);
      emit_bwd3_group(os, pis, bg[gi]);
      os << "};\n\n";
    }
    os << "struct " << tag << "::TP {\n";
    os << "  static constexpr int D_SH = " << lay.d_sh << ";\n";
    emit_group_meta(os, tpg);
    emit_make_A(os, tpg);
    emit_tp_group(os, lay, pis, tpg);
    os << "};\n\n";
  };

  std::vector<std::string> tags;
  std::set<std::string> seen;
  for (const auto& v : specs) {
    Layout lay;
    std::string err;
    if (!make_layout(irreps_of(v.blocks), v.lmax_sh, v.lmax_out, v.natural, lay, err)) {
      std::fprintf(stderr, "gen: %s\n", err.c_str());
      return 1;
    }
    if (lay.paths.empty()) {
      std::fprintf(stderr, "gen: layout %s has no paths\n", v.blocks.c_str());
      return 1;
    }
    if (!seen.insert(path_signature(lay) + "/" + std::to_string(lay.d_sh)).second) continue;
    const std::string tag = tag_of(v);
    tags.push_back(tag);
    emit_layout(o, tag, lay, v.lmax_sh, false);
  }
  o << "#define E3GEN_FOR_EACH_VARIANT(X)";
  for (const auto& t : tags) o << " X(" << t << ")";
  o << "\n\n}  // namespace e3gen\n";

  auto write = [&](const std::string& name, const std::string& text) {
    const std::string path = out_dir + "/" + name;
    FILE* f = std::fopen(path.c_str(), "w");
    if (!f) {
      std::perror(path.c_str());
      return false;
    }
    std::fwrite(text.data(), 1, text.size(), f);
    std::fclose(f);
    return true;
  };
  if (!write("variants.inc", o.str())) return 1;
  // the core unit's table of the variant units' entries
  std::ostringstream t;
  t << "// GENERATED by gen.cpp -- do not edit.\n";
  for (const auto& tag : tags) t << "const VariantOps* e3_variant_" << tag << "();\n";
  t << "namespace {\nconst VariantOps* (*const kVariants[])() = {";
  for (size_t i = 0; i < tags.size(); ++i) t << (i ? ", " : "") << "&e3_variant_" << tags[i];
  t << "};\nconstexpr int kNumVariants = " << tags.size() << ";\n}  // namespace\n";
  if (!write("variant_table.inc", t.str())) return 1;
  // one unit per variant: its launchers and kernels
  for (const auto& tag : tags) {
    std::ostringstream u;
    u << "// GENERATED by gen.cpp -- do not edit.  Kernels and launchers of variant " << tag << ".\n";
    u << "#include \"../e3mi_impl.h\"\n\n";
    u << "const VariantOps* e3_variant_" << tag << "() {\n  static const VariantOps ops = E3_VARIANT_OPS(" << tag
      << ");\n  return &ops;\n}\n";
    if (!write("v_" + tag + ".hip", u.str())) return 1;
  }
  // Kinds: every single x block (degree l1 <= 3, with all paths or with the
  // natural-parity ones of either block parity) under every harmonics and
  // output degree up to 3.  A layout without a compiled variant runs block by
  // block on these, with its strides and offsets given at run time.  Blocks
  // with the same path list and harmonics share one kind.
  std::ostringstream ko, kt;
  ko << "// GENERATED by gen.cpp from the host table builder -- do not edit.\n";
  ko << "// Single-block kinds, composed at run time into layouts without a compiled variant.\n";
  ko << "#pragma once\n\nnamespace e3gen {\n\n";
  std::vector<std::vector<std::string>> unit_kinds;
  std::vector<std::string> ktags;
  std::set<std::string> kseen;
  for (int l1 = 0; l1 <= 3; ++l1) {
    for (int lsh = 0; lsh <= 3; ++lsh) {
      std::vector<std::string> in_unit;
      for (int lout = 0; lout <= 3; ++lout) {
        for (int cls = 0; cls < 3; ++cls) {  // all paths; natural, block parity (-1)^l1; natural, the other
          const bool natural = cls != 0;
          const bool even = ((l1 % 2 == 0) == (cls != 2));
          const std::string blk = std::to_string(l1) + (even ? "e" : "o");
          Layout lay;
          std::string err;
          if (!make_layout("1x" + blk, lsh, lout, natural, lay, err)) {
            std::fprintf(stderr, "gen: kind %s: %s\n", blk.c_str(), err.c_str());
            return 1;
          }
          if (lay.paths.empty()) continue;
          if (!kseen.insert(path_signature(lay) + "/" + std::to_string(lay.d_sh)).second) continue;
          const std::string tag = "K_l" + std::to_string(l1) + "_s" + std::to_string(lsh) + "_o" +
                                  std::to_string(lout) + (cls == 0 ? "_a" : cls == 1 ? "_n" : "_p");
          emit_layout(ko, tag, lay, lsh, true);
          ktags.push_back(tag);
          in_unit.push_back(tag);
        }
      }
      if (!in_unit.empty()) unit_kinds.push_back(in_unit);
    }
  }
  ko << "#define E3GEN_FOR_EACH_KIND(X)";
  for (const auto& t : ktags) ko << " X(" << t << ")";
  ko << "\n\n}  // namespace e3gen\n";
  if (!write("kinds.inc", ko.str())) return 1;
  kt << "// GENERATED by gen.cpp -- do not edit.\n";
  for (const auto& tag : ktags) kt << "const KindOps* e3_kind_" << tag << "();\n";
  kt << "namespace {\nconst KindOps* (*const kKinds[])() = {";
  for (size_t i = 0; i < ktags.size(); ++i) kt << (i ? ", " : "") << "&e3_kind_" << ktags[i];
  kt << "};\nconstexpr int kNumKinds = " << ktags.size() << ";\n}  // namespace\n";
  if (!write("kind_table.inc", kt.str())) return 1;
  std::vector<std::string> kunits;
  for (size_t u = 0; u < unit_kinds.size(); ++u) {
    std::ostringstream k;
    k << "// GENERATED by gen.cpp -- do not edit.  Kernels and launchers of single-block kinds.\n";
    k << "#include \"../e3mi_impl.h\"\n#include \"kinds.inc\"\n\n";
    for (const auto& tag : unit_kinds[u])
      k << "const KindOps* e3_kind_" << tag << "() {\n  static const KindOps ops = E3_KIND_OPS(" << tag
        << ");\n  return &ops;\n}\n";
    const std::string name = "k_" + std::to_string(u) + ".hip";
    if (!write(name, k.str())) return 1;
    kunits.push_back(name);
  }
  // the unit list, one per line, for the build
  std::string units;
  for (const auto& tag : tags) units += "v_" + tag + ".hip\n";
  for (const auto& name : kunits) units += name + "\n";
  return write("units.txt", units) ? 0 : 1;
}
