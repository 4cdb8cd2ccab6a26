// Sparse combined coupling table from the so(3) intertwiner null space.
// See cg_builder.hpp for what is computed and the normalisation / sign rule.
#include "cg_builder.hpp"

#include <cmath>
#include <complex>
#include <map>
#include <mutex>
#include <stdexcept>
#include <string>
#include <tuple>

namespace allegro {
namespace {

using ld = long double;
using cld = std::complex<long double>;

// Dense complex matrix helper, row-major.
struct CMat {
  int n = 0;
  std::vector<cld> v;
  explicit CMat(int n_) : n(n_), v(size_t(n_) * n_) {}
  cld &operator()(int r, int c) { return v[size_t(r) * n + c]; }
  cld operator()(int r, int c) const { return v[size_t(r) * n + c]; }
};

CMat matmul(const CMat &a, const CMat &b) {
  CMat r(a.n);
  for (int i = 0; i < a.n; ++i)
    for (int k = 0; k < a.n; ++k) {
      const cld aik = a(i, k);
      if (aik == cld(0)) continue;
      for (int j = 0; j < a.n; ++j) r(i, j) += aik * b(k, j);
    }
  return r;
}

CMat dagger(const CMat &a) {
  CMat r(a.n);
  for (int i = 0; i < a.n; ++i)
    for (int j = 0; j < a.n; ++j) r(i, j) = std::conj(a(j, i));
  return r;
}

// Angular-momentum matrices in the complex basis |l m>, m = -l..l (index m + l),
// with the standard ladder phases: J+ |m> = sqrt(l(l+1) - m(m+1)) |m+1>.
void angular_momentum(int l, CMat &jx, CMat &jy, CMat &jz) {
  const int d = 2 * l + 1;
  CMat jp(d), jm(d);
  for (int m = -l; m <= l; ++m) {
    jz(m + l, m + l) = cld(m);
    if (m < l) jp(m + 1 + l, m + l) = cld(std::sqrt(ld(l * (l + 1) - m * (m + 1))));
    if (m > -l) jm(m - 1 + l, m + l) = cld(std::sqrt(ld(l * (l + 1) - m * (m - 1))));
  }
  const cld half(0.5L), i2(0.0L, 2.0L);
  for (size_t t = 0; t < jp.v.size(); ++t) {
    jx.v[t] = (jp.v[t] + jm.v[t]) * half;
    jy.v[t] = (jp.v[t] - jm.v[t]) / i2;
  }
}

// Change of basis from complex to real harmonic components (row: real m,
// column: complex m'):  m > 0: Q[m,m] = (-1)^m/sqrt2, Q[m,-m] = 1/sqrt2;
// m = 0: 1;  m < 0: Q[m,m] = i/sqrt2, Q[m,-m] = -i (-1)^m/sqrt2.
CMat real_basis(int l) {
  const int d = 2 * l + 1;
  CMat q(d);
  const ld r = 1.0L / std::sqrt(2.0L);
  for (int m = -l; m <= l; ++m) {
    const ld sgn = (m % 2 == 0) ? 1.0L : -1.0L;
    if (m > 0) {
      q(m + l, m + l) = cld(sgn * r);
      q(m + l, -m + l) = cld(r);
    } else if (m == 0) {
      q(l, l) = cld(1.0L);
    } else {
      q(m + l, m + l) = cld(0.0L, r);
      q(m + l, -m + l) = cld(0.0L, -sgn * r);
    }
  }
  return q;
}

// Real generators G_alpha = Q (i J_alpha) Q^dagger of order l (real antisymmetric).
std::vector<std::vector<ld>> real_generators(int l) {
  const int d = 2 * l + 1;
  CMat jx(d), jy(d), jz(d);
  angular_momentum(l, jx, jy, jz);
  const CMat q = real_basis(l), qd = dagger(q);
  std::vector<std::vector<ld>> out;
  for (const CMat *j : {&jx, &jy, &jz}) {
    CMat ij(d);
    for (size_t t = 0; t < ij.v.size(); ++t) ij.v[t] = cld(0.0L, 1.0L) * j->v[t];
    const CMat g = matmul(matmul(q, ij), qd);
    std::vector<ld> re(size_t(d) * d);
    for (size_t t = 0; t < re.size(); ++t) {
      if (std::fabs(g.v[t].imag()) > 1e-15L) throw std::runtime_error("real generator has an imaginary part");
      re[t] = g.v[t].real();
    }
    out.push_back(std::move(re));
  }
  return out;
}

// One row of the intertwiner system, stored sparsely.
struct SparseRow {
  std::vector<int> col;
  std::vector<ld> val;
  void add(int c, ld v) {
    if (v == 0.0L) return;
    for (size_t t = 0; t < col.size(); ++t)
      if (col[t] == c) {
        val[t] += v;
        return;
      }
    col.push_back(c);
    val.push_back(v);
  }
};

std::vector<double> solve_null_space(int l1, int l2, int l3) {
  const int d1 = 2 * l1 + 1, d2 = 2 * l2 + 1, d3 = 2 * l3 + 1;
  const int n = d1 * d2 * d3;
  auto idx = [&](int a, int b, int c) { return (a * d2 + b) * d3 + c; };
  const auto g1 = real_generators(l1), g2 = real_generators(l2), g3 = real_generators(l3);

  // Equation (alpha, p, q, c):  sum_a T[a,q,c] G1[a,p] + sum_b T[p,b,c] G2[b,q]
  //                            - sum_r G3[c,r] T[p,q,r] = 0
  std::vector<SparseRow> rows;
  rows.reserve(size_t(3) * n);
  for (int al = 0; al < 3; ++al)
    for (int p = 0; p < d1; ++p)
      for (int q = 0; q < d2; ++q)
        for (int c = 0; c < d3; ++c) {
          SparseRow row;
          for (int a = 0; a < d1; ++a) row.add(idx(a, q, c), g1[al][size_t(a) * d1 + p]);
          for (int b = 0; b < d2; ++b) row.add(idx(p, b, c), g2[al][size_t(b) * d2 + q]);
          for (int r = 0; r < d3; ++r) row.add(idx(p, q, r), -g3[al][size_t(c) * d3 + r]);
          rows.push_back(std::move(row));
        }

  // Normal matrix A = M^T M (dense), shifted: A + sigma I is positive definite.
  std::vector<ld> a(size_t(n) * n, 0.0L);
  for (const SparseRow &row : rows)
    for (size_t s = 0; s < row.col.size(); ++s)
      for (size_t t = 0; t < row.col.size(); ++t)
        a[size_t(row.col[s]) * n + row.col[t]] += row.val[s] * row.val[t];
  const ld sigma = 1e-9L;
  for (int i = 0; i < n; ++i) a[size_t(i) * n + i] += sigma;

  // Cholesky factor L (lower), in place.
  for (int j = 0; j < n; ++j) {
    ld s = a[size_t(j) * n + j];
    for (int k = 0; k < j; ++k) s -= a[size_t(j) * n + k] * a[size_t(j) * n + k];
    if (!(s > 0.0L)) throw std::runtime_error("intertwiner normal matrix is not positive definite");
    const ld ljj = std::sqrt(s);
    a[size_t(j) * n + j] = ljj;
    for (int i = j + 1; i < n; ++i) {
      ld t = a[size_t(i) * n + j];
      for (int k = 0; k < j; ++k) t -= a[size_t(i) * n + k] * a[size_t(j) * n + k];
      a[size_t(i) * n + j] = t / ljj;
    }
  }

  // Inverse iteration towards the smallest eigenvector (the null vector).
  std::vector<ld> v(n), y(n);
  for (int i = 0; i < n; ++i) v[i] = 1.0L + 0.25L * std::sin(ld(1.0L + 0.7L * i));
  for (int it = 0; it < 5; ++it) {
    for (int i = 0; i < n; ++i) {  // L y = v
      ld t = v[i];
      for (int k = 0; k < i; ++k) t -= a[size_t(i) * n + k] * y[k];
      y[i] = t / a[size_t(i) * n + i];
    }
    for (int i = n - 1; i >= 0; --i) {  // L^T v = y
      ld t = y[i];
      for (int k = i + 1; k < n; ++k) t -= a[size_t(k) * n + i] * v[k];
      v[i] = t / a[size_t(i) * n + i];
    }
    ld norm = 0.0L;
    for (ld e : v) norm += e * e;
    norm = std::sqrt(norm);
    for (ld &e : v) e /= norm;
  }

  // Residual of the unshifted system.
  ld res = 0.0L;
  for (const SparseRow &row : rows) {
    ld t = 0.0L;
    for (size_t s = 0; s < row.col.size(); ++s) t += row.val[s] * v[row.col[s]];
    res = std::max(res, std::fabs(t));
  }
  if (res > 1e-14L) throw std::runtime_error("coupling tensor null space is not clean");

  // Normalisation: total sum of squares 2 l3 + 1; exact zeros; sign rule.
  ld vmax = 0.0L;
  for (ld e : v) vmax = std::max(vmax, std::fabs(e));
  for (ld &e : v)
    if (std::fabs(e) < 1e-12L * vmax) e = 0.0L;
  ld ss = 0.0L;
  for (ld e : v) ss += e * e;
  const ld scale = std::sqrt(ld(2 * l3 + 1) / ss);
  ld first = 0.0L;
  for (ld e : v)
    if (e != 0.0L) {
      first = e;
      break;
    }
  const ld sgn = first < 0.0L ? -1.0L : 1.0L;
  std::vector<double> out(n);
  for (int i = 0; i < n; ++i) out[i] = v[i] == 0.0L ? 0.0 : double(sgn * scale * v[i]);

  // Check orthonormality in (m1, m2) for every pair (m3, m3').
  for (int c = 0; c < d3; ++c)
    for (int c2 = 0; c2 < d3; ++c2) {
      double s = 0.0;
      for (int p = 0; p < d1; ++p)
        for (int q = 0; q < d2; ++q) s += out[idx(p, q, c)] * out[idx(p, q, c2)];
      if (std::fabs(s - (c == c2 ? 1.0 : 0.0)) > 1e-12) throw std::runtime_error("coupling tensor not orthonormal");
    }
  return out;
}

}  // namespace

std::vector<double> real_coupling_tensor(int l1, int l2, int l3) {
  if (l1 < 0 || l2 < 0 || l3 < std::abs(l1 - l2) || l3 > l1 + l2)
    throw std::runtime_error("triangle rule violated");
  static std::mutex mu;
  static std::map<std::tuple<int, int, int>, std::vector<double>> cache;
  const auto key = std::make_tuple(l1, l2, l3);
  {
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find(key);
    if (it != cache.end()) return it->second;
  }
  std::vector<double> t = solve_null_space(l1, l2, l3);
  std::lock_guard<std::mutex> lock(mu);
  cache.emplace(key, t);
  return t;
}

TPTable build_table(int lmax, bool full_parity) {
  TPTable t;
  t.lmax = lmax;
  t.full_parity = full_parity;
  for (int l = 0; l <= lmax; ++l) {
    const int natural = (l % 2 == 0) ? 1 : -1;
    t.x_irreps.push_back({l, natural});
    if (full_parity) t.x_irreps.push_back({l, -natural});
    t.env_irreps.push_back({l, natural});
  }
  for (const Irrep &ir : t.x_irreps) {
    t.x_off.push_back(t.d1);
    t.d1 += 2 * ir.l + 1;
  }
  for (const Irrep &ir : t.env_irreps) {
    t.env_off.push_back(t.d2);
    t.d2 += 2 * ir.l + 1;
  }
  const int nx = int(t.x_irreps.size()), ne = int(t.env_irreps.size());
  for (int a = 0; a < nx; ++a)
    for (int b = 0; b < ne; ++b)
      for (int c = 0; c < nx; ++c) {
        const Irrep &xa = t.x_irreps[a], &eb = t.env_irreps[b], &xc = t.x_irreps[c];
        if (std::abs(xa.l - eb.l) <= xc.l && xc.l <= xa.l + eb.l && xc.p == xa.p * eb.p)
          t.paths.push_back({a, b, c});
      }
  for (int p = 0; p < int(t.paths.size()); ++p) {
    const Path &ph = t.paths[p];
    const int l1 = t.x_irreps[ph.a].l, l2 = t.env_irreps[ph.b].l, l3 = t.x_irreps[ph.c].l;
    const std::vector<double> blk = real_coupling_tensor(l1, l2, l3);
    const int d2b = 2 * l2 + 1, d3b = 2 * l3 + 1;
    for (int m1 = 0; m1 < 2 * l1 + 1; ++m1)
      for (int m2 = 0; m2 < d2b; ++m2)
        for (int m3 = 0; m3 < d3b; ++m3) {
          const double v = blk[(size_t(m1) * d2b + m2) * d3b + m3];
          if (v != 0.0)
            t.entries.push_back({p, t.x_off[ph.a] + m1, t.env_off[ph.b] + m2, t.x_off[ph.c] + m3, v});
        }
  }
  return t;
}

}  // namespace allegro
