// Host-side float64 factorisation of one gate group into pruned rank-1
// refinement terms (Sec. III, Eq. (1) of arXiv 1905.00689).  Plain C++17,
// no HIP.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace alstm {

struct GroupFactors {
  int rows = 0, cols = 0, rank = 0, nz = 0;
  std::vector<double> sigma;    // [rank]
  std::vector<double> u;        // [rank][rows]
  std::vector<double> v;        // [rank][cols] unpruned (only if keep_unpruned)
  std::vector<int32_t> mask;    // [rank][nz] ascending column indices
  std::vector<double> vals;     // [rank][nz] entries of v on the mask
  int eff_rank = 0;             // live terms; terms >= eff_rank are zero
  int unconverged = 0;          // solves that missed the Lanczos tolerance
};

struct FactoriseOptions {
  bool keep_unpruned = false;
  int gram_refresh = 32;        // recompute the Gram matrix exactly every this many steps
  int threads = 1;              // threads for the row loops of one group (results do not depend on it)
  double lanczos_tol = 4e-14;   // Ritz residual / Ritz value at which a solve stops
  double stop_rel = 1e-12;      // sigma <= stop_rel * sigma_1 ends the term list
  int max_lanczos = 0;          // 0: up to the Gram size
  bool residual = true;         // false: each term is deflated with its whole v (successive
                                // approximations of the original matrix), not its pruned v
};

// Factorise W (rows x cols, row-major, float64) into `rank` terms keeping
// `nz` entries of each v.  Returns 0, or 1 if a solve did not converge (the
// result is still complete).
int factorise_group(const double* W, int rows, int cols, int rank, int nz,
                    const FactoriseOptions& opt, GroupFactors& out);

// Pieces shared by the host and the device factorisations.
// init_group: size `out` for `rank` terms, every term terminated (zero).
void init_group(GroupFactors& out, int rows, int cols, int rank, int nz, bool keep_unpruned);
// store_term: term t from its singular value s and unit vectors uu (rows) and
// vv (cols): the sign rule (v's largest-magnitude entry, lowest index on
// ties, made positive; uu and vv are flipped in place), the mask (the nz
// largest |v|, ties to the lower index, stored ascending) and the values.
void store_term(GroupFactors& out, int t, double s, std::vector<double>& uu, std::vector<double>& vv,
                bool keep_unpruned, std::vector<int32_t>& idx);
// tridiag_top: largest eigenvalue and unit eigenvector s of the m x m
// symmetric tridiagonal matrix with diagonal a and off-diagonal b.
double tridiag_top(const double* a, const double* b, int m, std::vector<double>& s);
// tridiag_second: the second largest eigenvalue and a unit eigenvector.
double tridiag_second(const double* a, const double* b, int m, std::vector<double>& s);
// lanczos_start: the fixed unit start vector of every host Lanczos solve
// (and of each group's first device solve).
void lanczos_start(double* q, int n);

// Factorise the G groups of W ([G*rows][cols] row-major, float64; group g is
// rows g*rows .. g*rows+rows-1) on the current HIP device, on hip_stream,
// with the same scheme and options as factorise_group (threads unused).
// Returns 0, 1 if a solve did not converge (the result is still complete),
// or -1 on a HIP error (text in *err).  Synchronises hip_stream.
int factorise_groups_device(const double* W, int G, int rows, int cols, int rank, int nz,
                            const FactoriseOptions& opt, std::vector<GroupFactors>& out, void* hip_stream,
                            std::string* err);

// Top eigenpair of the symmetric n x n matrix G (row-major) by Lanczos with
// full reorthogonalisation from a fixed pseudo-random start.  Writes the unit
// eigenvector to y and returns the eigenvalue; *converged tells whether the
// Ritz residual met tol (relative to the eigenvalue).
double lanczos_top(const double* G, int n, double tol, int max_iter, double* y, bool* converged,
                   int* iterations, int threads = 1);

}  // namespace alstm
