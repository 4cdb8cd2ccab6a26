// Host-side builder of the sparse combined coupling table (C++17, no GPU).
//
// The paper stores the combined tensor of Wigner 3-j coefficients of all
// tensor-product paths in a compressed sparse format (arxiv 2504.16068, §II.D).
// This builder obtains each real coupling tensor as the one-dimensional null
// space of the so(3) intertwiner equations
//     T(A1 u, v) + T(u, A2 v) = A3 T(u, v)   for the three generators,
// with the generators A_l of the real spherical-harmonic basis.  It uses no
// closed formula for the coefficients; normalisation and sign follow the
// library's documented rule (orthonormal in (m1, m2) for every m3; first
// non-zero entry in row-major (m1, m2, m3) order positive).
#pragma once

#include <vector>

namespace allegro {

struct Irrep {
  int l;
  int p;  // +1 even, -1 odd
};

struct Path {
  int a, b, c;  // indices into x irreps, env irreps, out (= x) irreps
};

struct CGEntry {
  int path, i, j, k;  // i: x component, j: env component, k: out component
  double value;
};

struct TPTable {
  int lmax = 0;
  bool full_parity = false;
  std::vector<Irrep> x_irreps, env_irreps;
  std::vector<int> x_off, env_off;
  int d1 = 0, d2 = 0;
  std::vector<Path> paths;
  std::vector<CGEntry> entries;  // grouped by path, then row-major (m1, m2, m3)
};

// Real coupling tensor of (l1, l2 -> l3), dense row-major [2l1+1][2l2+1][2l3+1].
// Throws std::runtime_error if the triangle rule fails or the solve is not clean.
std::vector<double> real_coupling_tensor(int l1, int l2, int l3);

// Irreps, paths and the sparse table for one (lmax, parity mode).
TPTable build_table(int lmax, bool full_parity);

}  // namespace allegro
