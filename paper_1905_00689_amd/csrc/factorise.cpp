// Host-side float64 factorisation of one gate group (Sec. III and Eq. (1) of
// arXiv 1905.00689): repeated top-singular-triplet extraction from the
// residual, magnitude pruning of v, and residual update.
//
// The top triplet comes from the smaller Gram matrix (R R^T when R has no
// more rows than columns, else R^T R): Lanczos with full
// reorthogonalisation finds its top eigenvector, and sigma and the other
// singular vector follow from one product with R.  The Gram matrix is updated
// incrementally after each step (R' = R - s u v'^T changes it by a rank-2
// term) and recomputed exactly every few steps to keep rounding drift small.
#include "factorise.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>

namespace alstm {
namespace {

inline double dot(const double* a, const double* b, int n) {
  double s0 = 0, s1 = 0, s2 = 0, s3 = 0;
  int i = 0;
  for (; i + 4 <= n; i += 4) {
    s0 += a[i] * b[i];
    s1 += a[i + 1] * b[i + 1];
    s2 += a[i + 2] * b[i + 2];
    s3 += a[i + 3] * b[i + 3];
  }
  for (; i < n; ++i) s0 += a[i] * b[i];
  return (s0 + s1) + (s2 + s3);
}

inline void axpy(double a, const double* x, double* y, int n) {
  for (int i = 0; i < n; ++i) y[i] += a * x[i];
}

inline double norm2(const double* a, int n) { return std::sqrt(dot(a, a, n)); }

// Fixed start vector: the splitmix64 sequence (Steele, Lea and Flood, 2014)
// mapped to [-1, 1).  Any fixed vector with a component along the top
// eigenvector works; a pseudo-random one has one with probability 1.
void start_vector(double* q, int n) {
  uint64_t s = 0;
  for (int i = 0; i < n; ++i) {
    s += 0x9E3779B97F4A7C15ull;
    uint64_t z = s;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    q[i] = (double)(z >> 11) * (2.0 / 9007199254740992.0) - 1.0;
  }
}

// Number of eigenvalues of the symmetric tridiagonal (a, b) below x, from the
// signs of the pivots of the LDL^T factorisation of T - xI (Sturm count).
int sturm_count(const double* a, const double* b, int m, double x, double pivmin) {
  int cnt = 0;
  double d = a[0] - x;
  if (std::fabs(d) < pivmin) d = -pivmin;
  if (d < 0) ++cnt;
  for (int i = 1; i < m; ++i) {
    d = (a[i] - x) - b[i - 1] * b[i - 1] / d;
    if (std::fabs(d) < pivmin) d = -pivmin;
    if (d < 0) ++cnt;
  }
  return cnt;
}

// Solve (T - lam I) x = r for tridiagonal T (diag a, off-diagonal b) by
// Gaussian elimination with partial pivoting; tiny pivots are replaced by
// `tiny` (inverse iteration wants the near-singular solve).
void tri_solve_shifted(const double* a, const double* b, int m, double lam, double tiny, double* r,
                       double* x, std::vector<double>& U0, std::vector<double>& U1,
                       std::vector<double>& U2) {
  U0.assign(m, 0.0);
  U1.assign(m, 0.0);
  U2.assign(m, 0.0);
  // current row, columns (i, i+1, i+2), and its right-hand side
  double p0 = a[0] - lam, p1 = m > 1 ? b[0] : 0.0, p2 = 0.0, rp = r[0];
  for (int i = 0; i + 1 < m; ++i) {
    double q0 = b[i], q1 = a[i + 1] - lam, q2 = (i + 2 < m) ? b[i + 1] : 0.0, rq = r[i + 1];
    if (std::fabs(q0) > std::fabs(p0)) {
      std::swap(p0, q0);
      std::swap(p1, q1);
      std::swap(p2, q2);
      std::swap(rp, rq);
    }
    if (std::fabs(p0) < tiny) p0 = p0 < 0 ? -tiny : tiny;
    double l = q0 / p0;
    q1 -= l * p1;
    q2 -= l * p2;
    rq -= l * rp;
    U0[i] = p0;
    U1[i] = p1;
    U2[i] = p2;
    r[i] = rp;
    p0 = q1;
    p1 = q2;
    p2 = 0.0;
    rp = rq;
  }
  if (std::fabs(p0) < tiny) p0 = p0 < 0 ? -tiny : tiny;
  U0[m - 1] = p0;
  r[m - 1] = rp;
  for (int i = m - 1; i >= 0; --i) {
    double s = r[i];
    if (i + 1 < m) s -= U1[i] * x[i + 1];
    if (i + 2 < m) s -= U2[i] * x[i + 2];
    x[i] = s / U0[i];
  }
}

// Eigenpair idx (0: the largest, 1: the second largest, ...) of the m x m
// symmetric tridiagonal matrix: Sturm-count bisection for the eigenvalue
// (count(x) = eigenvalues below x; lambda_idx is the least x with
// count(x) >= m - idx), then inverse iteration for the unit vector s.
double tri_eigen_from_top(const double* a, const double* b, int m, int idx, std::vector<double>& s) {
  s.assign(m, 0.0);
  if (m == 1) {
    s[0] = 1.0;
    return a[0];
  }
  double lo = a[0], hi = a[0], scale = 0.0, bmax2 = 0.0;
  for (int i = 0; i < m; ++i) {
    double r = (i > 0 ? std::fabs(b[i - 1]) : 0.0) + (i + 1 < m ? std::fabs(b[i]) : 0.0);
    lo = std::min(lo, a[i] - r);
    hi = std::max(hi, a[i] + r);
    scale = std::max(scale, std::fabs(a[i]) + r);
    if (i + 1 < m) bmax2 = std::max(bmax2, b[i] * b[i]);
  }
  const double eps = 2.220446049250313e-16;
  double pivmin = std::max(1e-290, 1e-290 * bmax2);
  // invariant: count(lo) < m-idx (lambda_idx >= lo), count(hi) >= m-idx (lambda_idx < hi)
  hi += eps * scale + 1e-300;
  lo -= eps * scale + 1e-300;
  for (int it = 0; it < 200; ++it) {
    double mid = 0.5 * (lo + hi);
    if (mid <= lo || mid >= hi) break;
    if (hi - lo <= 2.0 * eps * std::max(std::fabs(lo), std::fabs(hi))) break;
    if (sturm_count(a, b, m, mid, pivmin) >= m - idx)
      hi = mid;
    else
      lo = mid;
  }
  double lam = 0.5 * (lo + hi);
  std::vector<double> r(m, 1.0), x(m), U0, U1, U2;
  double tiny = std::max(eps * scale, 1e-300);
  for (int it = 0; it < 3; ++it) {
    tri_solve_shifted(a, b, m, lam, tiny, r.data(), x.data(), U0, U1, U2);
    double nx = norm2(x.data(), m);
    if (!(nx > 0)) {
      x.assign(m, 0.0);
      x[m - 1] = 1.0;
      nx = 1.0;
    }
    for (int i = 0; i < m; ++i) r[i] = x[i] / nx;
  }
  s = r;
  return lam;
}

double tri_top_eigen(const double* a, const double* b, int m, std::vector<double>& s) {
  return tri_eigen_from_top(a, b, m, 0, s);
}

}  // namespace

double tridiag_top(const double* a, const double* b, int m, std::vector<double>& s) {
  return tri_top_eigen(a, b, m, s);
}

double tridiag_second(const double* a, const double* b, int m, std::vector<double>& s) {
  return tri_eigen_from_top(a, b, m, 1, s);
}

void lanczos_start(double* q, int n) {
  start_vector(q, n);
  const double nq = norm2(q, n);
  for (int i = 0; i < n; ++i) q[i] /= nq;
}

double lanczos_top(const double* G, int n, double tol, int max_iter, double* y, bool* converged,
                   int* iterations, int threads) {
  const int kmax = (max_iter > 0) ? std::min(max_iter, n) : n;
  std::vector<double> Q((size_t)(kmax + 1) * n), w(n), c(kmax + 1), alpha, beta, s;
  start_vector(Q.data(), n);
  {
    double nq = norm2(Q.data(), n);
    for (int i = 0; i < n; ++i) Q[i] /= nq;
  }
  double theta = 0.0, resid = 0.0;
  int m = 0;
  bool done = false;
  for (int k = 0; k < kmax && !done; ++k) {
    const double* q = &Q[(size_t)k * n];
    double* wp = w.data();
#pragma omp parallel for num_threads(threads) schedule(static) if (threads > 1 && n >= 256)
    for (int i = 0; i < n; ++i) wp[i] = dot(G + (size_t)i * n, q, n);
    double al = dot(q, w.data(), n);
    axpy(-al, q, w.data(), n);
    if (k > 0) axpy(-beta[k - 1], &Q[(size_t)(k - 1) * n], w.data(), n);
    for (int pass = 0; pass < 2; ++pass) {   // full reorthogonalisation, twice
      for (int j = 0; j <= k; ++j) c[j] = dot(&Q[(size_t)j * n], w.data(), n);
      for (int j = 0; j <= k; ++j) axpy(-c[j], &Q[(size_t)j * n], w.data(), n);
    }
    alpha.push_back(al);
    double be = norm2(w.data(), n);
    m = k + 1;
    bool last = (m == kmax);
    if ((m % 2) == 0 || last || be == 0.0) {
      theta = tri_top_eigen(alpha.data(), beta.data(), m, s);
      resid = be * std::fabs(s[m - 1]);
      if (resid <= tol * std::fabs(theta) || be == 0.0 || last) done = true;
    }
    if (!done) {
      beta.push_back(be);
      double* qn = &Q[(size_t)(k + 1) * n];
      for (int i = 0; i < n; ++i) qn[i] = w[i] / be;
    }
  }
  std::fill(y, y + n, 0.0);
  for (int j = 0; j < m; ++j) axpy(s[j], &Q[(size_t)j * n], y, n);
  double ny = norm2(y, n);
  if (ny > 0)
    for (int i = 0; i < n; ++i) y[i] /= ny;
  if (converged) *converged = (resid <= tol * std::fabs(theta)) || m == n;
  if (iterations) *iterations = m;
  return theta;
}

namespace {

void gram_exact(const std::vector<double>& R, int rows, int cols, bool left, std::vector<double>& G, int threads) {
  if (left) {
    // row i of the upper triangle, rows dealt cyclically to balance the triangle
#pragma omp parallel for num_threads(threads) schedule(static, 1) if (threads > 1)
    for (int i = 0; i < rows; ++i)
      for (int j = i; j < rows; ++j) {
        double v = dot(&R[(size_t)i * cols], &R[(size_t)j * cols], cols);
        G[(size_t)i * rows + j] = v;
        G[(size_t)j * rows + i] = v;
      }
  } else {
    std::fill(G.begin(), G.end(), 0.0);
    for (int r = 0; r < rows; ++r) {
      const double* rr = &R[(size_t)r * cols];
      for (int i = 0; i < cols; ++i) {
        double a = rr[i];
        if (a == 0.0) continue;
        double* gi = &G[(size_t)i * cols];
        for (int j = i; j < cols; ++j) gi[j] += a * rr[j];
      }
    }
    for (int i = 0; i < cols; ++i)
      for (int j = 0; j < i; ++j) G[(size_t)i * cols + j] = G[(size_t)j * cols + i];
  }
}

}  // namespace

void init_group(GroupFactors& out, int rows, int cols, int rank, int nz, bool keep_unpruned) {
  out.rows = rows;
  out.cols = cols;
  out.rank = rank;
  out.nz = nz;
  out.sigma.assign(rank, 0.0);
  out.u.assign((size_t)rank * rows, 0.0);
  out.v.assign(keep_unpruned ? (size_t)rank * cols : 0, 0.0);
  out.mask.resize((size_t)rank * nz);
  for (int t = 0; t < rank; ++t)
    for (int e = 0; e < nz; ++e) out.mask[(size_t)t * nz + e] = e;   // terminated-term default
  out.vals.assign((size_t)rank * nz, 0.0);
  out.eff_rank = 0;
  out.unconverged = 0;
}

void store_term(GroupFactors& out, int t, double s, std::vector<double>& uu, std::vector<double>& vv,
                bool keep_unpruned, std::vector<int32_t>& idx) {
  const int cols = out.cols, nz = out.nz;
  // sign: largest-magnitude entry of v (lowest index on ties) positive
  int kstar = 0;
  for (int k = 1; k < cols; ++k)
    if (std::fabs(vv[k]) > std::fabs(vv[kstar])) kstar = k;
  if (vv[kstar] < 0) {
    for (auto& a : uu) a = -a;
    for (auto& a : vv) a = -a;
  }
  // mask: nz largest |v|, ties to the lower index, kept ascending
  idx.resize(cols);
  std::iota(idx.begin(), idx.end(), 0);
  auto before = [&](int32_t a, int32_t b) {
    double fa = std::fabs(vv[a]), fb = std::fabs(vv[b]);
    return fa > fb || (fa == fb && a < b);
  };
  if (nz < cols) std::nth_element(idx.begin(), idx.begin() + (nz - 1), idx.end(), before);
  std::sort(idx.begin(), idx.begin() + nz, before);
  std::sort(idx.begin(), idx.begin() + nz);
  int32_t* mk = &out.mask[(size_t)t * nz];
  double* vl = &out.vals[(size_t)t * nz];
  for (int e = 0; e < nz; ++e) {
    mk[e] = idx[e];
    vl[e] = vv[idx[e]];
  }
  out.sigma[t] = s;
  std::copy(uu.begin(), uu.end(), out.u.begin() + (size_t)t * out.rows);
  if (keep_unpruned) std::copy(vv.begin(), vv.end(), out.v.begin() + (size_t)t * cols);
}

int factorise_group(const double* W, int rows, int cols, int rank, int nz,
                    const FactoriseOptions& opt, GroupFactors& out) {
  init_group(out, rows, cols, rank, nz, opt.keep_unpruned);

  std::vector<double> R(W, W + (size_t)rows * cols);
  const bool left = rows <= cols;
  const int n = left ? rows : cols;
  std::vector<double> G((size_t)n * n);
  gram_exact(R, rows, cols, left, G, opt.threads);

  std::vector<double> y(n), uu(rows), vv(cols), w(left ? rows : cols);
  std::vector<int32_t> idx(cols), all_cols(cols);
  std::iota(all_cols.begin(), all_cols.end(), 0);
  double tau = 0.0;
  for (int t = 0; t < rank; ++t) {
    if (t > 0 && opt.gram_refresh > 0 && t % opt.gram_refresh == 0) gram_exact(R, rows, cols, left, G, opt.threads);
    bool conv = false;
    int iters = 0;
    lanczos_top(G.data(), n, opt.lanczos_tol, opt.max_lanczos, y.data(), &conv, &iters, opt.threads);
    double s;
    if (left) {
      uu.assign(y.begin(), y.end());
      for (int k = 0; k < cols; ++k) vv[k] = 0.0;
      for (int r = 0; r < rows; ++r) axpy(uu[r], &R[(size_t)r * cols], vv.data(), cols);
      s = norm2(vv.data(), cols);
      if (s > 0)
        for (int k = 0; k < cols; ++k) vv[k] /= s;
    } else {
      vv.assign(y.begin(), y.end());
      for (int r = 0; r < rows; ++r) uu[r] = dot(&R[(size_t)r * cols], vv.data(), cols);
      s = norm2(uu.data(), rows);
      if (s > 0)
        for (int r = 0; r < rows; ++r) uu[r] /= s;
    }
    if (t == 0) tau = opt.stop_rel * s;
    if (!(s > tau)) break;   // this and every later term stay terminated
    if (!conv) ++out.unconverged;
    store_term(out, t, s, uu, vv, opt.keep_unpruned, idx);
    // the factor the residual loses: sigma u v'^T with the pruned v' (the
    // residual scheme), or sigma u v^T with the whole v (the alternative of
    // successive approximations of the original matrix)
    const int nzu = opt.residual ? nz : cols;
    const int32_t* mk = opt.residual ? &out.mask[(size_t)t * nz] : all_cols.data();
    const double* vl = opt.residual ? &out.vals[(size_t)t * nz] : vv.data();

    // Gram update for R' = R - s u v'^T, from the pre-update R
    double vp2 = 0.0;
    for (int e = 0; e < nzu; ++e) vp2 += vl[e] * vl[e];
    if (left) {
      for (int r = 0; r < rows; ++r) {   // w = R v'
        const double* rr = &R[(size_t)r * cols];
        double acc = 0.0;
        for (int e = 0; e < nzu; ++e) acc += rr[mk[e]] * vl[e];
        w[r] = acc;
      }
      for (int i = 0; i < rows; ++i) {
        double* gi = &G[(size_t)i * rows];
        const double ui = uu[i], wi = w[i];
        for (int j = 0; j < rows; ++j) gi[j] += -s * (wi * uu[j] + ui * w[j]) + s * s * vp2 * ui * uu[j];
      }
    } else {
      for (int k = 0; k < cols; ++k) w[k] = 0.0;   // p = R^T u
      for (int r = 0; r < rows; ++r) axpy(uu[r], &R[(size_t)r * cols], w.data(), cols);
      double usq = dot(uu.data(), uu.data(), rows);
      for (int e = 0; e < nzu; ++e) {
        const int i = mk[e];
        const double vi = vl[e];
        double* gi = &G[(size_t)i * cols];
        for (int j = 0; j < cols; ++j) gi[j] -= s * vi * w[j];
        for (int j = 0; j < cols; ++j) G[(size_t)j * cols + i] -= s * w[j] * vi;
      }
      for (int e = 0; e < nzu; ++e)
        for (int f = 0; f < nzu; ++f) G[(size_t)mk[e] * cols + mk[f]] += s * s * usq * vl[e] * vl[f];
    }
    // residual update
    for (int r = 0; r < rows; ++r) {
      double* rr = &R[(size_t)r * cols];
      const double a = s * uu[r];
      for (int e = 0; e < nzu; ++e) rr[mk[e]] -= a * vl[e];
    }
    out.eff_rank = t + 1;
  }
  return out.unconverged ? 1 : 0;
}

}  // namespace alstm
