// Factorisation of the gate groups on the GPU, in float64 (Sec. III and
// Eq. (1) of arXiv 1905.00689): the same greedy scheme as the host
// factorisation -- the top singular triplet of the residual, magnitude
// pruning of v, the residual update -- with the bulk of every step on the
// device and all groups advancing together (blockIdx.z = group).
//
// Each group's residual is held as M [n][m] with n <= m: M = R when R has no
// more rows than columns (u is the top eigenvector of M M^T), else M = R^T
// (v is).  Per step:
//   * the Gram matrix M M^T is kept up to date by the rank-2 change that the
//     residual update makes, and recomputed exactly every few steps;
//   * Lanczos with full reorthogonalisation (two classical Gram-Schmidt
//     passes) runs on it, the first solve of each group from the host
//     factorisation's fixed start and each later one from the previous
//     solve's top and second Ritz vectors plus that fixed vector (a warm
//     start: fewer iterations to the same tolerance), in blocks of 8 iterations
//     captured once as a HIP graph; the host reads the tridiagonal
//     coefficients after each block (one block behind the device) and solves
//     the small tridiagonal eigenproblem for the convergence test and the
//     Ritz vector.  The test runs every 8 iterations where the host
//     factorisation runs it every 2, so a solve may stop up to 6 iterations
//     later, converged at least as far;
//   * y = sum_j s_j q_j is the unit top eigenvector, x = M^T y the other
//     singular vector times sigma;
//   * the host takes sigma = |x|, the sign rule and the mask (the code the
//     host factorisation uses), and the device applies
//     M' = M - sigma a b^T (a, b the pruned outer-product factors) and the
//     matching Gram update.
// Every reduction has one fixed order, so the result does not depend on the
// launch; it differs from the host factorisation's only by rounding (the
// order of the sums), which the chain may amplify over many steps.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "factorise.hpp"

namespace alstm {

namespace {

constexpr int kFT = 512;          // threads per workgroup
constexpr int kFW = kFT / 64;     // waves per workgroup
constexpr int kGramTile = 64;     // Gram output tile (rows and columns)
constexpr int kGramK = 16;        // k slice of the Gram tile
constexpr int kRowBlock = 64;     // rows per partial sum of M^T y
constexpr int kIterBlock = 8;     // Lanczos iterations per graph replay (between convergence checks)
constexpr int kDotGroups = 32;    // workgroups of the reorthogonalisation dot products

__device__ inline double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum of one value per thread of the workgroup, in a fixed order; every
// thread receives it.
__device__ inline double block_sum_f64(double v, double* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum_f64(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < kFW; ++i) s += red[i];
  return s;
}

// G = M M^T for every group: 64 x 64 output tiles, k in slices of 16 staged
// in LDS.  G[i][j] and G[j][i] take the same products in the same order, so
// the result is exactly symmetric.
__global__ void __launch_bounds__(kFT) gram_kernel(const double* __restrict__ M, double* __restrict__ G, int n,
                                                    int m, size_t sM, size_t sG) {
  __shared__ double As[kGramTile][kGramK + 1];
  __shared__ double Bs[kGramTile][kGramK + 1];
  const int g = blockIdx.z;
  const double* Mg = M + g * sM;
  const int i0 = blockIdx.y * kGramTile, j0 = blockIdx.x * kGramTile;
  const int r = threadIdx.x >> 3, c8 = threadIdx.x & 7;
  double acc[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) acc[q] = 0.0;
  for (int k0 = 0; k0 < m; k0 += kGramK) {
    __syncthreads();
    for (int e = threadIdx.x; e < kGramTile * kGramK; e += kFT) {
      const int rr = e / kGramK, kk = e % kGramK;
      const int k = k0 + kk;
      As[rr][kk] = (i0 + rr < n && k < m) ? Mg[(size_t)(i0 + rr) * m + k] : 0.0;
      Bs[rr][kk] = (j0 + rr < n && k < m) ? Mg[(size_t)(j0 + rr) * m + k] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kGramK; ++kk) {
      const double a = As[r][kk];
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] = fma(a, Bs[c8 + 8 * q][kk], acc[q]);
    }
  }
  const int i = i0 + r;
  if (i < n) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int j = j0 + c8 + 8 * q;
      if (j < n) G[g * sG + (size_t)i * n + j] = acc[q];
    }
  }
}

// out[i] = sum_j A[i][j] v[j] (A [rows][cols] row-major), one wave per row.
__global__ void __launch_bounds__(kFT) rowdot_kernel(const double* __restrict__ A, const double* __restrict__ v,
                                                      double* __restrict__ out, int rows, int cols, size_t sA,
                                                      size_t sv, size_t so, const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int lane = threadIdx.x & 63, i = blockIdx.x * kFW + (threadIdx.x >> 6);
  if (i >= rows) return;
  const double* a = A + g * sA + (size_t)i * cols;
  const double* x = v + g * sv;
  double acc = 0.0;
  for (int j = lane; j < cols; j += 64) acc = fma(a[j], x[j], acc);
  acc = wave_sum_f64(acc);
  if (lane == 0) out[g * so + i] = acc;
}

// The Lanczos iteration kernels take the iteration index k of each group from
// kk[g] (advanced by lanczos_next_kernel), so that one captured sequence of
// launches serves every iteration; a group at k >= kmax does nothing.

// w = G q_k, one wave per row.
__global__ void __launch_bounds__(kFT) symv_kernel(const double* __restrict__ G, const double* __restrict__ Q,
                                                    const int* __restrict__ kk, double* __restrict__ w, int n,
                                                    int kmax, size_t sG, size_t sQ, const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int k = kk[g];
  if (k >= kmax) return;
  const int lane = threadIdx.x & 63, i = blockIdx.x * kFW + (threadIdx.x >> 6);
  if (i >= n) return;
  const double* a = G + g * sG + (size_t)i * n;
  const double* q = Q + g * sQ + (size_t)k * n;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
  int j = lane;
  for (; j + 192 < n; j += 256) {
    a0 = fma(a[j], q[j], a0);
    a1 = fma(a[j + 64], q[j + 64], a1);
    a2 = fma(a[j + 128], q[j + 128], a2);
    a3 = fma(a[j + 192], q[j + 192], a3);
  }
  for (; j < n; j += 64) a0 = fma(a[j], q[j], a0);
  const double acc = wave_sum_f64((a0 + a1) + (a2 + a3));
  if (lane == 0) w[(size_t)g * n + i] = acc;
}

// c[j] = q_j . w for j <= k, one wave per j (waves stride over j).
__global__ void __launch_bounds__(kFT) dots_kernel(const double* __restrict__ Q, const double* __restrict__ w,
                                                    const int* __restrict__ kk, double* __restrict__ c, int n,
                                                    int kmax, size_t sQ, size_t sc, const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int k = kk[g];
  if (k >= kmax) return;
  const int lane = threadIdx.x & 63;
  const double* wg = w + (size_t)g * n;
  for (int j = blockIdx.x * kFW + (threadIdx.x >> 6); j <= k; j += gridDim.x * kFW) {
    const double* q = Q + g * sQ + (size_t)j * n;
    // four independent partial sums per lane (more loads in flight), added
    // in a fixed order
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
    int i = lane;
    for (; i + 192 < n; i += 256) {
      a0 = fma(q[i], wg[i], a0);
      a1 = fma(q[i + 64], wg[i + 64], a1);
      a2 = fma(q[i + 128], wg[i + 128], a2);
      a3 = fma(q[i + 192], wg[i + 192], a3);
    }
    for (; i < n; i += 64) a0 = fma(q[i], wg[i], a0);
    const double acc = wave_sum_f64((a0 + a1) + (a2 + a3));
    if (lane == 0) c[g * sc + j] = acc;
  }
}

// Combination of the first cnt basis vectors, 64 elements per workgroup with
// the vectors dealt over the 8 waves and the wave partials added in order:
//   mode 0: w[i] -= sum_j c[j] Q[j][i]      mode 1: w[i] = sum_j c[j] Q[j][i]
// with cnt = cnts[g] + add_one per group (the Lanczos passes: cnts = the
// iteration index, add_one = 1, and nothing once it reaches kmax; the Ritz
// vector: cnts = the basis size, add_one = 0).
__global__ void __launch_bounds__(kFT) combine_kernel(const double* __restrict__ Q, const double* __restrict__ c,
                                                       double* __restrict__ w, const int* __restrict__ cnts,
                                                       int add_one, int kmax, int n, size_t sQ, size_t sc,
                                                       size_t sw, int mode, const int* __restrict__ act) {
  __shared__ double part[kFW][64];
  const int g = blockIdx.z;
  if (!act[g]) return;
  if (add_one && cnts[g] >= kmax) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = blockIdx.x * 64 + lane;
  const int nv = cnts[g] + add_one;
  const double* Qg = Q + g * sQ;
  const double* cg = c + g * sc;
  // two independent partial sums per lane, added in a fixed order
  double a0 = 0.0, a1 = 0.0;
  if (i < n) {
    int j = wave;
    for (; j + kFW < nv; j += 2 * kFW) {
      a0 = fma(cg[j], Qg[(size_t)j * n + i], a0);
      a1 = fma(cg[j + kFW], Qg[(size_t)(j + kFW) * n + i], a1);
    }
    if (j < nv) a0 = fma(cg[j], Qg[(size_t)j * n + i], a0);
  }
  part[wave][lane] = a0 + a1;
  __syncthreads();
  if (wave == 0 && i < n) {
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < kFW; ++q) s += part[q][lane];
    double* wg = w + g * sw;
    wg[i] = mode == 0 ? wg[i] - s : s;
  }
}

// After the reorthogonalisation of w: beta_k = |w|, q_{k+1} = w / beta_k (0
// when beta_k is 0), alpha_k = q_k . (G q_k) (the first pass's coefficient
// of q_k), and k advances.  One workgroup per group.
__global__ void __launch_bounds__(kFT) lanczos_next_kernel(const double* __restrict__ w, double* __restrict__ Q,
                                                            const double* __restrict__ c1, double* __restrict__ alpha,
                                                            double* __restrict__ beta, int* __restrict__ kk, int kmax,
                                                            int n, size_t sw, size_t sQ, size_t sc,
                                                            const int* __restrict__ act) {
  __shared__ double red[kFW];
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int k = kk[g];
  if (k >= kmax) return;
  const double* wg = w + g * sw;
  double ss = 0.0;
  for (int i = threadIdx.x; i < n; i += kFT) ss = fma(wg[i], wg[i], ss);
  const double b = sqrt(block_sum_f64(ss, red));
  double* qn = Q + g * sQ + (size_t)(k + 1) * n;
  for (int i = threadIdx.x; i < n; i += kFT) qn[i] = b > 0.0 ? wg[i] / b : 0.0;
  if (threadIdx.x == 0) {
    alpha[g * sc + k] = c1[g * sc + k];
    beta[g * sc + k] = b;
    kk[g] = k + 1;
  }
}

// y /= |y| (unchanged when |y| = 0).  One workgroup per group.
__global__ void __launch_bounds__(kFT) normalise_kernel(double* __restrict__ y, int n, size_t sy,
                                                         const int* __restrict__ act) {
  __shared__ double red[kFW];
  const int g = blockIdx.z;
  if (!act[g]) return;
  double* yg = y + g * sy;
  double ss = 0.0;
  for (int i = threadIdx.x; i < n; i += kFT) ss = fma(yg[i], yg[i], ss);
  const double ny = sqrt(block_sum_f64(ss, red));
  if (ny > 0.0)
    for (int i = threadIdx.x; i < n; i += kFT) yg[i] /= ny;
}

// part[rb][j] = sum over rows i of block rb of y[i] M[i][j] (thread per column).
__global__ void __launch_bounds__(kFT) mty_partial_kernel(const double* __restrict__ M, const double* __restrict__ y,
                                                           double* __restrict__ part, int n, int m, size_t sM,
                                                           size_t sy, size_t sp, const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int j = blockIdx.x * kFT + threadIdx.x;
  if (j >= m) return;
  const int r0 = blockIdx.y * kRowBlock, r1 = min(n, r0 + kRowBlock);
  const double* Mg = M + g * sM;
  const double* yg = y + g * sy;
  double acc = 0.0;
  for (int i = r0; i < r1; ++i) acc = fma(yg[i], Mg[(size_t)i * m + j], acc);
  part[g * sp + (size_t)blockIdx.y * m + j] = acc;
}

// x[j] = sum over row blocks of part[rb][j], in block order.
__global__ void __launch_bounds__(kFT) mty_reduce_kernel(const double* __restrict__ part, double* __restrict__ x,
                                                          int nrb, int m, size_t sp, size_t sx,
                                                          const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int j = blockIdx.x * kFT + threadIdx.x;
  if (j >= m) return;
  double s = 0.0;
  for (int rb = 0; rb < nrb; ++rb) s += part[g * sp + (size_t)rb * m + j];
  x[g * sx + j] = s;
}

// The Gram change of M' = M - s a b^T: G' = G - s (a w^T + w a^T) + s^2 |b|^2 a a^T
// with w = M b taken before the update (sb = {s, |b|^2} per group).
__global__ void __launch_bounds__(kFT) gram_update_kernel(double* __restrict__ G, const double* __restrict__ a,
                                                           const double* __restrict__ w, const double* __restrict__ sb,
                                                           int n, size_t sG, size_t sa, const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const size_t e = blockIdx.x * (size_t)kFT + threadIdx.x;
  if (e >= (size_t)n * n) return;
  const int i = (int)(e / n), j = (int)(e % n);
  const double s = sb[2 * g], bb = sb[2 * g + 1];
  const double* ag = a + g * sa;
  const double* wg = w + g * sa;
  double* Gg = G + g * sG;
  Gg[e] += -s * (wg[i] * ag[j] + ag[i] * wg[j]) + s * s * bb * ag[i] * ag[j];
}

// M' = M - s a b^T, written so that each entry takes the product the host
// factorisation takes: (s u_r) v_k, u the left and v the pruned right vector
// (left: a = u, b = v'; right, M = R^T: a = v', b = u).
__global__ void __launch_bounds__(kFT) residual_update_kernel(double* __restrict__ M, const double* __restrict__ a,
                                                               const double* __restrict__ b,
                                                               const double* __restrict__ sb, int n, int m, size_t sM,
                                                               size_t sa, size_t sbv, int left,
                                                               const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const size_t e = blockIdx.x * (size_t)kFT + threadIdx.x;
  if (e >= (size_t)n * m) return;
  const int i = (int)(e / m), j = (int)(e % m);
  const double s = sb[2 * g];
  const double ai = a[g * sa + i], bj = b[g * sbv + j];
  const double d = left ? (s * ai) * bj : (s * bj) * ai;
  if (d != 0.0) M[g * sM + e] -= d;
}

// q0[g] += qf (the fixed start vector) for the flagged groups.
__global__ void __launch_bounds__(kFT) add_start_kernel(double* __restrict__ q0, const double* __restrict__ qf, int n,
                                                         const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int i = blockIdx.x * kFT + threadIdx.x;
  if (i < n) q0[(size_t)g * n + i] += qf[i];
}

// Q[0] = q0 (the group's start vector, q0 + g*n) and k = 0 for every group.
__global__ void __launch_bounds__(kFT) start_kernel(double* __restrict__ Q, const double* __restrict__ q0,
                                                     int* __restrict__ kk, int n, size_t sQ,
                                                     const int* __restrict__ act) {
  const int g = blockIdx.z;
  if (!act[g]) return;
  const int i = blockIdx.x * kFT + threadIdx.x;
  if (i < n) Q[g * sQ + i] = q0[(size_t)g * n + i];
  if (blockIdx.x == 0 && threadIdx.x == 0) kk[g] = 0;
}

inline unsigned cdiv(size_t a, size_t b) { return (unsigned)((a + b - 1) / b); }

struct DevBuf {
  std::vector<void*> ptrs;
  ~DevBuf() {
    for (void* p : ptrs) (void)hipFree(p);
  }
  template <typename T>
  hipError_t alloc(T*& p, size_t count) {
    void* q = nullptr;
    hipError_t e = hipMalloc(&q, std::max<size_t>(count, 1) * sizeof(T));
    if (e == hipSuccess) ptrs.push_back(q);
    p = static_cast<T*>(q);
    return e;
  }
};

// Everything one factorisation holds on the device; released in reverse
// order after the stream has drained.
struct Resources {
  hipStream_t stream = nullptr;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  hipEvent_t ev[2] = {nullptr, nullptr};
  double* coef = nullptr;   // pinned host: two slots of [alpha | beta] for every group
  void* stage = nullptr;    // pinned host: the per-term uploads and reads (see factorise_groups_device)
  DevBuf buf;
  ~Resources() {
    if (stream) (void)hipStreamSynchronize(stream);
    if (coef) (void)hipHostFree(coef);
    if (stage) (void)hipHostFree(stage);
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
    if (exec) (void)hipGraphExecDestroy(exec);
    if (graph) (void)hipGraphDestroy(graph);
    for (void* p : buf.ptrs) (void)hipFree(p);
    buf.ptrs.clear();
    if (stream) (void)hipStreamDestroy(stream);
  }
};

}  // namespace

#define FD_TRY(expr, what)                        \
  do {                                            \
    hipError_t e_ = (expr);                       \
    if (e_ != hipSuccess) {                       \
      if (err) *err = std::string(what) + ": " + hipGetErrorString(e_); \
      return -1;                                  \
    }                                             \
  } while (0)

int factorise_groups_device(const double* W, int G, int rows, int cols, int rank, int nz,
                            const FactoriseOptions& opt, std::vector<GroupFactors>& out, void* hip_stream,
                            std::string* err) {
  out.assign(G, GroupFactors());
  for (int g = 0; g < G; ++g) init_group(out[g], rows, cols, rank, nz, opt.keep_unpruned);
  const bool left = rows <= cols;
  const int n = left ? rows : cols, m = left ? cols : rows;
  const int kmax = (opt.max_lanczos > 0) ? std::min(opt.max_lanczos, n) : n;
  const int nrb = (n + kRowBlock - 1) / kRowBlock;
  const size_t sM = (size_t)n * m, sG = (size_t)n * n, sQ = (size_t)(kmax + 1) * n;
  const size_t sc = (size_t)kmax + 1, sp = (size_t)nrb * m;

  // the work runs on a stream of its own (default priority), after the
  // caller's stream has drained
  FD_TRY(hipStreamSynchronize((hipStream_t)hip_stream), "hipStreamSynchronize");
  Resources res;
  FD_TRY(hipStreamCreateWithFlags(&res.stream, hipStreamNonBlocking), "hipStreamCreate");
  hipStream_t stream = res.stream;
  DevBuf& buf = res.buf;
  double *dM, *dG, *dQ, *dw, *dc1, *dc2, *dal, *dbe, *dy, *dx, *dpart, *da, *db, *dw2, *dsb, *dq0, *dqf, *dritz, *dritz2;
  int *dact, *dact2, *dcnt, *dk;
  FD_TRY(buf.alloc(dM, G * sM), "hipMalloc(residual)");
  FD_TRY(buf.alloc(dG, G * sG), "hipMalloc(Gram)");
  FD_TRY(buf.alloc(dQ, G * sQ), "hipMalloc(Lanczos basis)");
  FD_TRY(buf.alloc(dw, (size_t)G * n), "hipMalloc");
  FD_TRY(buf.alloc(dc1, G * sc), "hipMalloc");
  FD_TRY(buf.alloc(dc2, G * sc), "hipMalloc");
  FD_TRY(buf.alloc(dal, G * sc), "hipMalloc");
  FD_TRY(buf.alloc(dbe, G * sc), "hipMalloc");
  FD_TRY(buf.alloc(dritz, G * sc), "hipMalloc");
  FD_TRY(buf.alloc(dy, (size_t)G * n), "hipMalloc");
  FD_TRY(buf.alloc(dx, (size_t)G * m), "hipMalloc");
  FD_TRY(buf.alloc(dpart, G * sp), "hipMalloc");
  FD_TRY(buf.alloc(da, (size_t)G * n), "hipMalloc");
  FD_TRY(buf.alloc(db, (size_t)G * m), "hipMalloc");
  FD_TRY(buf.alloc(dw2, (size_t)G * n), "hipMalloc");
  FD_TRY(buf.alloc(dsb, (size_t)2 * G), "hipMalloc");
  FD_TRY(buf.alloc(dq0, (size_t)G * n), "hipMalloc");
  FD_TRY(buf.alloc(dqf, (size_t)n), "hipMalloc");
  FD_TRY(buf.alloc(dritz2, G * sc), "hipMalloc");
  FD_TRY(buf.alloc(dact2, (size_t)G), "hipMalloc");
  FD_TRY(buf.alloc(dact, (size_t)G), "hipMalloc");
  FD_TRY(buf.alloc(dcnt, (size_t)G), "hipMalloc");
  FD_TRY(buf.alloc(dk, (size_t)G), "hipMalloc");
  FD_TRY(hipHostMalloc((void**)&res.coef, (size_t)4 * G * sc * sizeof(double), hipHostMallocDefault),
         "hipHostMalloc");
  for (hipEvent_t& e : res.ev) FD_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreate");

  {  // residual M of every group, and the fixed Lanczos start
    std::vector<double> hM(sM);
    for (int g = 0; g < G; ++g) {
      const double* Wg = W + (size_t)g * rows * cols;
      if (left) {
        std::copy(Wg, Wg + sM, hM.begin());
      } else {
        for (int r = 0; r < rows; ++r)
          for (int k = 0; k < cols; ++k) hM[(size_t)k * m + r] = Wg[(size_t)r * cols + k];
      }
      FD_TRY(hipMemcpy(dM + g * sM, hM.data(), sM * 8, hipMemcpyHostToDevice), "upload residual");
    }
    // every group's first solve starts from the fixed vector of the host
    // factorisation
    std::vector<double> q0(n);
    lanczos_start(q0.data(), n);
    for (int g = 0; g < G; ++g)
      FD_TRY(hipMemcpy(dq0 + (size_t)g * n, q0.data(), (size_t)n * 8, hipMemcpyHostToDevice), "upload start vector");
    FD_TRY(hipMemcpy(dqf, q0.data(), (size_t)n * 8, hipMemcpyHostToDevice), "upload start vector");
  }

  // kIterBlock Lanczos iterations as one graph: w = G q_k, two classical
  // Gram-Schmidt passes against q_0 .. q_k, then beta_k, q_{k+1}, k + 1
  {
    FD_TRY(hipStreamBeginCapture(stream, hipStreamCaptureModeRelaxed), "hipStreamBeginCapture");
    const unsigned dgx = (unsigned)std::min<size_t>(cdiv(kmax, kFW), kDotGroups);
    for (int it = 0; it < kIterBlock; ++it) {
      symv_kernel<<<dim3(cdiv(n, kFW), 1, G), dim3(kFT), 0, stream>>>(dG, dQ, dk, dw, n, kmax, sG, sQ, dact);
      dots_kernel<<<dim3(dgx, 1, G), dim3(kFT), 0, stream>>>(dQ, dw, dk, dc1, n, kmax, sQ, sc, dact);
      combine_kernel<<<dim3(cdiv(n, 64), 1, G), dim3(kFT), 0, stream>>>(dQ, dc1, dw, dk, 1, kmax, n, sQ, sc, n, 0,
                                                                        dact);
      dots_kernel<<<dim3(dgx, 1, G), dim3(kFT), 0, stream>>>(dQ, dw, dk, dc2, n, kmax, sQ, sc, dact);
      combine_kernel<<<dim3(cdiv(n, 64), 1, G), dim3(kFT), 0, stream>>>(dQ, dc2, dw, dk, 1, kmax, n, sQ, sc, n, 0,
                                                                        dact);
      lanczos_next_kernel<<<dim3(1, 1, G), dim3(kFT), 0, stream>>>(dw, dQ, dc1, dal, dbe, dk, kmax, n, n, sQ, sc,
                                                                   dact);
    }
    hipError_t e = hipStreamEndCapture(stream, &res.graph);
    if (e == hipSuccess) e = hipGetLastError();
    FD_TRY(e, "capture of the Lanczos iterations");
    FD_TRY(hipGraphInstantiate(&res.exec, res.graph, nullptr, nullptr, 0), "hipGraphInstantiate");
  }

  // Pinned staging for the per-term transfers, one region per purpose, so
  // that the copies run asynchronously and no extra synchronisation is
  // needed: every region is rewritten only on the next term, after a stream
  // synchronisation that its previous copy precedes (the read of y and x,
  // which follows the flag, Ritz and start-vector uploads of a term; the
  // update uploads of a term come after it and before the next term's).
  enum { kActStart, kActLive, kActUpd, kActNum };
  const size_t st_doubles = 2 * (size_t)G * sc + 2 * (size_t)G * n + 2 * (size_t)G * m + 2 * (size_t)G;
  const size_t st_ints = (size_t)(kActNum + 2) * G;
  FD_TRY(hipHostMalloc(&res.stage, st_doubles * 8 + st_ints * 4, hipHostMallocDefault), "hipHostMalloc");
  double* st_ritz = static_cast<double*>(res.stage);   // [G][sc]
  double* st_ritz2 = st_ritz + (size_t)G * sc;          // [G][sc]
  double* st_a = st_ritz2 + (size_t)G * sc;             // [G][n]
  double* st_y = st_a + (size_t)G * n;                  // [G][n]
  double* st_b = st_y + (size_t)G * n;                  // [G][m]
  double* st_x = st_b + (size_t)G * m;                  // [G][m]
  double* st_sb = st_x + (size_t)G * m;                 // [2G]
  int* st_act = reinterpret_cast<int*>(st_sb + 2 * (size_t)G);   // [kActNum][G]
  int* st_cnt = st_act + (size_t)kActNum * G;                      // [G]
  int* st_has2 = st_cnt + G;                                       // [G]

  std::vector<int> live(G, 1);   // group still producing terms
  // group flags for the next kernels, from staging region `which`
  auto set_act = [&](const std::vector<int>& v, int which) -> hipError_t {
    int* dst = st_act + (size_t)which * G;
    std::copy(v.begin(), v.end(), dst);
    return hipMemcpyAsync(dact, dst, G * sizeof(int), hipMemcpyHostToDevice, stream);
  };
  auto gram = [&]() -> hipError_t {
    gram_kernel<<<dim3(cdiv(n, kGramTile), cdiv(n, kGramTile), G), dim3(kFT), 0, stream>>>(dM, dG, n, m, sM, sG);
    return hipGetLastError();
  };
  FD_TRY(set_act(live, kActLive), "upload flags");
  FD_TRY(gram(), "gram_kernel");

  std::vector<double> tau(G, 0.0), hy((size_t)G * n), hx((size_t)G * m);
  std::vector<double> ha((size_t)G * n), hb((size_t)G * m), hsb(2 * G), hritz(G * sc, 0.0), hritz2(G * sc, 0.0);
  std::vector<int> hcnt(G), idx(cols), has2(G, 0);
  std::vector<double> uu(rows), vv(cols), s, s2;

  for (int t = 0; t < rank; ++t) {
    if (std::none_of(live.begin(), live.end(), [](int v) { return v != 0; })) break;
    if (t > 0 && opt.gram_refresh > 0 && t % opt.gram_refresh == 0) FD_TRY(gram(), "gram_kernel");
    // ---- Lanczos on every live group's Gram matrix.  Blocks of kIterBlock
    // iterations run ahead of the host's convergence test by one block while
    // a solve is far from converged (a group that has converged keeps
    // iterating until all have; its later basis vectors are not used).  The
    // test runs at the end of each block (and where beta vanishes), on the
    // tridiagonal matrix of that size.
    std::vector<int> lz = live;           // groups still iterating
    std::vector<int> mdone(G, 0), conv(G, 0);
    FD_TRY(set_act(lz, kActStart), "upload flags");
    start_kernel<<<dim3(cdiv(n, kFT), 1, G), dim3(kFT), 0, stream>>>(dQ, dq0, dk, n, sQ, dact);
    FD_TRY(hipGetLastError(), "start_kernel");
    const int nblk = (kmax + kIterBlock - 1) / kIterBlock;
    auto enqueue_block = [&](int b) -> hipError_t {
      hipError_t e = hipGraphLaunch(res.exec, stream);
      double* slot = res.coef + (size_t)(b & 1) * 2 * G * sc;
      if (e == hipSuccess) e = hipMemcpyAsync(slot, dal, G * sc * 8, hipMemcpyDeviceToHost, stream);
      if (e == hipSuccess) e = hipMemcpyAsync(slot + G * sc, dbe, G * sc * 8, hipMemcpyDeviceToHost, stream);
      if (e == hipSuccess) e = hipEventRecord(res.ev[b & 1], stream);
      return e;
    };
    // Block b + 1 is queued before block b is examined unless every group
    // still iterating is expected to converge within block b (its relative
    // Ritz residual after block b - 1 times the factor of its last block at
    // or below the tolerance): then the host examines block b first and
    // queues b + 1 only if it is needed, instead of running a block whose
    // result is discarded.  Which iterations the solves stop at does not
    // depend on this.
    std::vector<double> rel(G, HUGE_VAL), rate(G, 1.0);
    int queued = 0;
    FD_TRY(enqueue_block(0), "Lanczos block");
    for (int b = 0; b < nblk; ++b) {
      if (b + 1 < nblk && queued < b + 1) {
        bool ahead = false;
        for (int g = 0; g < G; ++g)
          if (lz[g] && !(rel[g] * rate[g] <= opt.lanczos_tol)) ahead = true;
        if (ahead) {
          FD_TRY(enqueue_block(b + 1), "Lanczos block");
          queued = b + 1;
        }
      }
      FD_TRY(hipEventSynchronize(res.ev[b & 1]), "hipEventSynchronize");
      const double* slot = res.coef + (size_t)(b & 1) * 2 * G * sc;
      const int prev = b * kIterBlock, done_k = std::min(kmax, prev + kIterBlock);
      bool any = false;
      for (int g = 0; g < G; ++g) {
        if (!lz[g]) continue;
        const double* al = slot + g * sc;
        const double* be = slot + G * sc + g * sc;
        for (int mm = prev + 1; mm <= done_k; ++mm) {
          const bool last = mm == done_k;
          const double bt = be[mm - 1];
          if (!last && bt != 0.0) continue;
          const double theta = tridiag_top(al, be, mm, s);
          const double resid = bt * std::fabs(s[mm - 1]);
          {  // the relative residual and its factor over the last block
            const double r = theta != 0.0 ? resid / std::fabs(theta) : HUGE_VAL;
            rate[g] = (rel[g] < HUGE_VAL && rel[g] > 0.0) ? r / rel[g] : 1.0;
            rel[g] = r;
          }
          if (resid <= opt.lanczos_tol * std::fabs(theta) || bt == 0.0 || mm == kmax) {
            lz[g] = 0;
            mdone[g] = mm;
            conv[g] = (resid <= opt.lanczos_tol * std::fabs(theta)) || mm == n;
            std::copy(s.begin(), s.end(), hritz.begin() + g * sc);
            // the group's next solve starts from y1 + y2 + q_fixed (top and
            // second Ritz vectors of this solve, and the fixed start): the
            // next top direction lies close to y2 when the residual update
            // removed the top one, and close to y1 when pruning left much
            // of it behind; the fixed vector keeps a component along every
            // direction, so that the solve cannot settle on a lower pair
            has2[g] = mm >= 2 ? 1 : 0;
            if (has2[g]) {
              tridiag_second(al, be, mm, s2);
              for (int i = 0; i < mm; ++i) hritz2[g * sc + i] = s[i] + s2[i];
            }
          }
          break;
        }
        any = any || lz[g];
      }
      if (!any) break;
      if (b + 1 < nblk && queued < b + 1) {   // not queued ahead, and still needed
        FD_TRY(enqueue_block(b + 1), "Lanczos block");
        queued = b + 1;
      }
    }
    // ---- Ritz vector y and x = M^T y
    for (int g = 0; g < G; ++g) st_cnt[g] = mdone[g];
    std::copy(hritz.begin(), hritz.end(), st_ritz);
    FD_TRY(set_act(live, kActLive), "upload flags");
    FD_TRY(hipMemcpyAsync(dritz, st_ritz, G * sc * 8, hipMemcpyHostToDevice, stream), "upload Ritz");
    FD_TRY(hipMemcpyAsync(dcnt, st_cnt, G * sizeof(int), hipMemcpyHostToDevice, stream), "upload counts");
    combine_kernel<<<dim3(cdiv(n, 64), 1, G), dim3(kFT), 0, stream>>>(dQ, dritz, dy, dcnt, 0, kmax, n, sQ, sc, n, 1,
                                                                      dact);
    normalise_kernel<<<dim3(1, 1, G), dim3(kFT), 0, stream>>>(dy, n, n, dact);
    // the next start vectors (groups whose solve had a second Ritz vector;
    // the others keep theirs); the host arrays are read back by the stream
    // synchronisation below before they can change
    for (int g = 0; g < G; ++g) has2[g] = has2[g] && live[g];
    std::copy(hritz2.begin(), hritz2.end(), st_ritz2);
    std::copy(has2.begin(), has2.end(), st_has2);
    FD_TRY(hipMemcpyAsync(dritz2, st_ritz2, G * sc * 8, hipMemcpyHostToDevice, stream), "upload Ritz 2");
    FD_TRY(hipMemcpyAsync(dact2, st_has2, G * sizeof(int), hipMemcpyHostToDevice, stream), "upload flags 2");
    combine_kernel<<<dim3(cdiv(n, 64), 1, G), dim3(kFT), 0, stream>>>(dQ, dritz2, dq0, dcnt, 0, kmax, n, sQ, sc, n, 1,
                                                                      dact2);
    add_start_kernel<<<dim3(cdiv(n, kFT), 1, G), dim3(kFT), 0, stream>>>(dq0, dqf, n, dact2);
    normalise_kernel<<<dim3(1, 1, G), dim3(kFT), 0, stream>>>(dq0, n, n, dact2);
    mty_partial_kernel<<<dim3(cdiv(m, kFT), nrb, G), dim3(kFT), 0, stream>>>(dM, dy, dpart, n, m, sM, n, sp, dact);
    mty_reduce_kernel<<<dim3(cdiv(m, kFT), 1, G), dim3(kFT), 0, stream>>>(dpart, dx, nrb, m, sp, m, dact);
    FD_TRY(hipGetLastError(), "Ritz vector");
    FD_TRY(hipMemcpyAsync(st_y, dy, (size_t)G * n * 8, hipMemcpyDeviceToHost, stream), "read y");
    FD_TRY(hipMemcpyAsync(st_x, dx, (size_t)G * m * 8, hipMemcpyDeviceToHost, stream), "read x");
    FD_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
    std::copy(st_y, st_y + (size_t)G * n, hy.begin());
    std::copy(st_x, st_x + (size_t)G * m, hx.begin());
    // ---- sigma, sign, mask (host), and the update operands
    std::vector<int> upd(G, 0);
    for (int g = 0; g < G; ++g) {
      if (!live[g]) continue;
      const double* y = &hy[(size_t)g * n];
      const double* x = &hx[(size_t)g * m];
      double sg = 0.0;
      for (int j = 0; j < m; ++j) sg += x[j] * x[j];
      sg = std::sqrt(sg);
      if (left) {
        uu.assign(y, y + n);
        vv.assign(x, x + m);
        if (sg > 0)
          for (auto& a : vv) a /= sg;
      } else {
        vv.assign(y, y + n);
        uu.assign(x, x + m);
        if (sg > 0)
          for (auto& a : uu) a /= sg;
      }
      if (t == 0) tau[g] = opt.stop_rel * sg;
      if (!(sg > tau[g])) {   // this and every later term of the group stay terminated
        live[g] = 0;
        continue;
      }
      if (!conv[g]) ++out[g].unconverged;
      store_term(out[g], t, sg, uu, vv, opt.keep_unpruned, idx);
      out[g].eff_rank = t + 1;
      // the v the residual loses: pruned v' as a dense vector (zeros off the
      // mask), or the whole v for the non-residual alternative
      std::vector<double> vp(cols, 0.0);
      double vp2 = 0.0;
      if (opt.residual) {
        for (int e = 0; e < nz; ++e) {
          const double val = out[g].vals[(size_t)t * nz + e];
          vp[out[g].mask[(size_t)t * nz + e]] = val;
          vp2 += val * val;
        }
      } else {
        vp = vv;
        for (double a : vp) vp2 += a * a;
      }
      double* ag = &ha[(size_t)g * n];
      double* bg = &hb[(size_t)g * m];
      if (left) {
        std::copy(uu.begin(), uu.end(), ag);
        std::copy(vp.begin(), vp.end(), bg);
        hsb[2 * g + 1] = vp2;
      } else {
        std::copy(vp.begin(), vp.end(), ag);
        std::copy(uu.begin(), uu.end(), bg);
        double usq = 0.0;
        for (double a : uu) usq += a * a;
        hsb[2 * g + 1] = usq;
      }
      hsb[2 * g] = sg;
      upd[g] = 1;
    }
    if (std::none_of(upd.begin(), upd.end(), [](int v) { return v != 0; })) continue;
    // ---- residual and Gram updates on the device
    std::copy(ha.begin(), ha.end(), st_a);
    std::copy(hb.begin(), hb.end(), st_b);
    std::copy(hsb.begin(), hsb.end(), st_sb);
    FD_TRY(set_act(upd, kActUpd), "upload flags");
    FD_TRY(hipMemcpyAsync(da, st_a, (size_t)G * n * 8, hipMemcpyHostToDevice, stream), "upload a");
    FD_TRY(hipMemcpyAsync(db, st_b, (size_t)G * m * 8, hipMemcpyHostToDevice, stream), "upload b");
    FD_TRY(hipMemcpyAsync(dsb, st_sb, (size_t)2 * G * 8, hipMemcpyHostToDevice, stream), "upload scales");
    rowdot_kernel<<<dim3(cdiv(n, kFW), 1, G), dim3(kFT), 0, stream>>>(dM, db, dw2, n, m, sM, m, n, dact);
    gram_update_kernel<<<dim3(cdiv((size_t)n * n, kFT), 1, G), dim3(kFT), 0, stream>>>(dG, da, dw2, dsb, n, sG, n,
                                                                                       dact);
    residual_update_kernel<<<dim3(cdiv((size_t)n * m, kFT), 1, G), dim3(kFT), 0, stream>>>(dM, da, db, dsb, n, m, sM,
                                                                                           n, m, left ? 1 : 0, dact);
    FD_TRY(hipGetLastError(), "residual update");
  }
  FD_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
  int unconv = 0;
  for (int g = 0; g < G; ++g) unconv += out[g].unconverged;
  return unconv ? 1 : 0;
}

#undef FD_TRY

}  // namespace alstm
