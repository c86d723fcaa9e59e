// Host-side table builder: irreps, coupling paths, real Clebsch-Gordan tables
// and real spherical-harmonic polynomial tables, all in float64.
//
// Follows App. G of the paper: harmonics are built as polynomials from the
// top state (x+iy)^l lowered by the ladder operator, Clebsch-Gordan
// coefficients from the top-spin eigenvector of J^2 in the M = L subspace,
// lowered by J_-.  Conventions (normalisation, real basis, axes, canonical
// sign, path order) are fixed here and restated in each function.
#pragma once

#include <array>
#include <complex>
#include <cstdint>
#include <string>
#include <vector>

namespace e3b {

struct Block {
  int mul, l, p;  // p = +1 even, -1 odd
};

struct Path {
  int k;        // path index == index of its scalar block (the map i3)
  int xb;       // x block index
  int l1, p1, l2, l3, p3;
  int x_off;    // first row of the x block on the D_in axis
  int y_off;    // l2*l2: first row of the harmonic block on the D_sh axis
  int out_off;  // first row of the output block on the D_out axis
};

struct Layout {
  std::vector<Block> blocks;
  int C = 0, lmax_sh = 0, lmax_out = 0;
  int d_in = 0, d_sh = 0, d_out = 0;
  bool natural = false;
  std::vector<Path> paths;
};

// Parses "8x0e+8x1o" (multiplicity defaults to 1).  Returns false and sets err
// on a malformed string.
bool parse_irreps(const std::string& s, std::vector<Block>& out, std::string& err);

// Paths: x block (given order), then l2 = 0..lmax_sh, then l3 ascending from
// |l1-l2| to min(l1+l2, lmax_out).  Output parity p3 = p1 * (-1)^l2 (App. B.1);
// with natural == true only paths with p3 == (-1)^l3 are kept.  Every block must
// have the same multiplicity (channelwise coupling).
bool make_layout(const std::string& irreps, int lmax_sh, int lmax_out, bool natural,
                 Layout& out, std::string& err);

// Real coupling tensor of the path (l1, l2, l3), row-major [2l3+1][2l1+1][2l2+1],
// in the basis of the real harmonics below.  Unitary normalisation; an imaginary
// block is multiplied by -i; the first entry with |c| > 1e-12 is positive; exact
// zeros of the coupling are returned as 0.
std::vector<double> real_cg_block(int l1, int l2, int l3);

// Complex Clebsch-Gordan block C[M][m1][m2] (Condon-Shortley), row-major.
std::vector<double> complex_cg_block(int l1, int l2, int L);

// Real spherical harmonics as polynomials of the unit vector u = (ux, uy, uz):
// Y_l(u) = S_l(uz, ux, uy) with S_l the textbook real solid harmonics (no
// Condon-Shortley sign in the real functions), normalised so that
// sum_m Y_lm(u)^2 = 2l+1 on the unit sphere.  Rows are l-major, m = -l..l.
struct ShTable {
  int lmax = 0;
  std::vector<std::array<int, 3>> mono;  // exponents of (ux, uy, uz), degree <= lmax
  std::vector<double> coef;              // [(lmax+1)^2][mono.size()]
};
ShTable sh_table(int lmax);

// Evaluates the table at a unit vector (host reference, float64).
void sh_eval(const ShTable& t, const double u[3], double* y);

// Complex-to-real change of basis U_l (real = U_l . complex) of the harmonics
// above, row-major [2l+1][2l+1].
std::vector<std::complex<double>> real_basis(int l);

struct Record {
  int i0, i1, i2;
  double v;
};
// All non-zero coupling records of a layout, unfolded to (i0, i1, i2) on the
// D_out, D_in, D_sh axes (App. E.2), sorted by (i0, i1, i2).
std::vector<Record> coo(const Layout& lay);

// A short string naming the path list, used to match a layout with a compiled
// kernel variant: "l1.l2.l3,..." over all paths.
std::string path_signature(const Layout& lay);

}  // namespace e3b
