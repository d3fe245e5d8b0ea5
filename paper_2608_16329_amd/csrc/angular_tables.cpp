// Host construction of the irreducible harmonic projections Q_l (Section 3.3,
// "Irreducible Harmonic Projection").
//
// For each order l the rows of Q_l are coefficient vectors, over the degree-l
// Cartesian monomials u_x^a u_y^b u_z^c (lexicographic, x first), of harmonic
// polynomials: L_l Q_l^T = 0 with L_l the Laplacian on coefficient vectors.
// They are orthonormal in the D_l^{-1} inner product, Q_l D_l^{-1} Q_l^T = I,
// D_l = diag(l!/(a!b!c!)).  Here a basis of ker(L_l) is read off the reduced
// row-echelon form of L_l and orthonormalised by Gram-Schmidt in that inner
// product.  Any two valid Q_l differ by an orthogonal factor, which leaves
// the descriptor's squared norms unchanged; the l = 0 row is fixed to +1.
//
// The output table has one row per angular feature (l-major) and one column
// per Cartesian monomial, degree by degree and lexicographic with x first
// within a degree,
//   1 | x y z | x2 xy xz y2 yz z2 | x3 x2y x2z xy2 xyz xz2 y3 y2z yz2 z3 | ...
// so feature m of direction u is sum_q table[m][q] * monomial_q(u); it is
// followed by one weight per row, the diagonal of the block metric C_l of
// the descriptor (Eq. 5): 1 for the irreducible basis, the multinomial
// coefficients for the Cartesian basis (whose rows are the monomials).
#include <cmath>
#include <string>
#include <vector>

#include "mlip_internal.h"

namespace mlip {
namespace {

struct Exp3 {
  int a, b, c;
};

std::vector<Exp3> exponents(int l) {
  std::vector<Exp3> e;
  for (int a = l; a >= 0; --a)
    for (int b = l - a; b >= 0; --b) e.push_back({a, b, l - a - b});
  return e;
}

double factorial(int n) {
  double f = 1.0;
  for (int i = 2; i <= n; ++i) f *= i;
  return f;
}

int find_exp(const std::vector<Exp3>& e, int a, int b, int c) {
  for (size_t i = 0; i < e.size(); ++i)
    if (e[i].a == a && e[i].b == b && e[i].c == c) return int(i);
  return -1;
}

// Rows of Q_l, each of length (l+1)(l+2)/2.
bool harmonic_rows(int l, std::vector<std::vector<double>>* rows, std::string* err) {
  const std::vector<Exp3> cols = exponents(l);
  const int n = int(cols.size());
  std::vector<double> dinv(n);
  for (int c = 0; c < n; ++c)
    dinv[c] = factorial(cols[c].a) * factorial(cols[c].b) * factorial(cols[c].c) / factorial(l);
  rows->clear();
  if (l == 0) {
    rows->push_back({1.0});
    return true;
  }
  // Laplacian matrix, degree l -> degree l-2.
  std::vector<std::vector<double>> L;
  if (l >= 2) {
    const std::vector<Exp3> lo = exponents(l - 2);
    L.assign(lo.size(), std::vector<double>(n, 0.0));
    for (int c = 0; c < n; ++c) {
      const Exp3 e = cols[c];
      if (e.a >= 2) L[find_exp(lo, e.a - 2, e.b, e.c)][c] += e.a * (e.a - 1);
      if (e.b >= 2) L[find_exp(lo, e.a, e.b - 2, e.c)][c] += e.b * (e.b - 1);
      if (e.c >= 2) L[find_exp(lo, e.a, e.b, e.c - 2)][c] += e.c * (e.c - 1);
    }
  }
  // Reduced row-echelon form with partial pivoting.
  std::vector<int> pivot_col;
  int r = 0;
  for (int c = 0; c < n && r < int(L.size()); ++c) {
    int best = r;
    for (int i = r + 1; i < int(L.size()); ++i)
      if (std::fabs(L[i][c]) > std::fabs(L[best][c])) best = i;
    if (std::fabs(L[best][c]) < 1e-12) continue;
    std::swap(L[r], L[best]);
    const double p = L[r][c];
    for (int j = 0; j < n; ++j) L[r][j] /= p;
    for (int i = 0; i < int(L.size()); ++i) {
      if (i == r || L[i][c] == 0.0) continue;
      const double f = L[i][c];
      for (int j = 0; j < n; ++j) L[i][j] -= f * L[r][j];
    }
    pivot_col.push_back(c);
    ++r;
  }
  // Kernel basis: one vector per free column.
  std::vector<std::vector<double>> basis;
  for (int f = 0; f < n; ++f) {
    bool is_pivot = false;
    for (int pc : pivot_col) is_pivot |= (pc == f);
    if (is_pivot) continue;
    std::vector<double> v(n, 0.0);
    v[f] = 1.0;
    for (size_t i = 0; i < pivot_col.size(); ++i) v[pivot_col[i]] = -L[i][f];
    basis.push_back(v);
  }
  if (int(basis.size()) != 2 * l + 1) {
    *err = "harmonic kernel has unexpected dimension";
    return false;
  }
  // Gram-Schmidt (two passes) in <p, q> = sum_c p_c q_c / D_c.
  auto dot = [&](const std::vector<double>& p, const std::vector<double>& q) {
    double s = 0.0;
    for (int c = 0; c < n; ++c) s += p[c] * q[c] * dinv[c];
    return s;
  };
  for (size_t i = 0; i < basis.size(); ++i) {
    for (int pass = 0; pass < 2; ++pass)
      for (size_t j = 0; j < i; ++j) {
        const double pr = dot(basis[i], basis[j]);
        for (int c = 0; c < n; ++c) basis[i][c] -= pr * basis[j][c];
      }
    const double nrm = std::sqrt(dot(basis[i], basis[i]));
    for (int c = 0; c < n; ++c) basis[i][c] /= nrm;
  }
  *rows = basis;
  return true;
}

}  // namespace

bool build_angular_table(int lmax, int angular, int rows, int cols, std::vector<double>* out, int lrow[8],
                         std::string* err) {
  const int ncols_needed = (lmax + 1) * (lmax + 2) * (lmax + 3) / 6;  // monomials of degree <= lmax
  const int nrows_needed = angular == 0 ? (lmax + 1) * (lmax + 1) : ncols_needed;
  if (lmax < 0 || lmax > 5 || ncols_needed > cols || nrows_needed > rows || (angular != 0 && angular != 1)) {
    *err = "angular basis does not fit the kernel's table";
    return false;
  }
  out->assign(size_t(rows) * cols + rows, 0.0);
  double* w = out->data() + size_t(rows) * cols;  // per-row descriptor weights
  int row = 0, col0 = 0;
  for (int l = 0; l <= lmax; ++l) {
    lrow[l] = row;
    const std::vector<Exp3> ex = exponents(l);
    if (angular == 0) {
      std::vector<std::vector<double>> q;
      if (!harmonic_rows(l, &q, err)) return false;
      for (const auto& v : q) {
        for (size_t c = 0; c < v.size(); ++c) (*out)[size_t(row) * cols + col0 + int(c)] = v[c];
        w[row] = 1.0;
        ++row;
      }
    } else {
      // Cartesian basis: the monomials themselves, with the multinomial
      // coefficients l!/(a!b!c!) as the metric of the block
      for (size_t c = 0; c < ex.size(); ++c) {
        (*out)[size_t(row) * cols + col0 + int(c)] = 1.0;
        w[row] = factorial(l) / (factorial(ex[c].a) * factorial(ex[c].b) * factorial(ex[c].c));
        ++row;
      }
    }
    col0 += int(ex.size());
  }
  for (int l = lmax + 1; l < 8; ++l) lrow[l] = row;
  return true;
}

}  // namespace mlip
