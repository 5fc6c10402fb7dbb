// gfx950 bf16 MFMA path for many independent sequences (arXiv 1905.00689,
// Eq. (1) per gate, then the Sec. II cell update).
//
// With a batch of sequences every refinement step becomes a real dense
// contraction, so the factors are kept as zero-filled bf16 panels and the
// three products run on v_mfma_f32_16x16x32_bf16 with fp32 accumulation:
//   x-projection (once per run)  P[tau][t,b] = Vx[tau][:] . x_t[b][:]
//   per timestep, h-projection   z[tau][b]   = sigma_tau (P[tau][t,b] + Vh[tau][:] . h_{t-1}[b][:])
//   per timestep, accumulation   y[o][b]     = bias[o] + U[o][:] . z_g(o)[:][b],  then gates, c, h.
// Pruned entries are stored as zeros, so the MFMA executes the dense work
// (about 1/(1-p) times the method's own count); the results are those of
// Eq. (1) with bf16 operands (x~, the factor values and z) and fp32 sums.
//
// MFMA operand layout (v_mfma_f32_16x16x32_bf16, wave64): lane l holds
// A[l%16][8*(l/16) .. +7], B[8*(l/16) .. +7][l%16], and the result rows
// 4*(l/16) .. +3 of column l%16.  Every operand below is stored with the
// contraction index contiguous, so a lane reads its 8 values as one 16-byte
// load.
#include "kernels.hpp"

#include <algorithm>

namespace alstm {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 load8(const uint16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ uint16_t bf16_bits(float v) { return __builtin_bit_cast(uint16_t, (__bf16)v); }

// x[k .. k+7] of one sequence row as bf16 (nearest even); zeros past D
__device__ __forceinline__ bf16x8 load_x8(const float* row, int k, int D, bool vec) {
  bf16x8 r;
  if (vec && k + 8 <= D) {
    const float4 a = *reinterpret_cast<const float4*>(row + k);
    const float4 b = *reinterpret_cast<const float4*>(row + k + 4);
    r[0] = (__bf16)a.x; r[1] = (__bf16)a.y; r[2] = (__bf16)a.z; r[3] = (__bf16)a.w;
    r[4] = (__bf16)b.x; r[5] = (__bf16)b.y; r[6] = (__bf16)b.z; r[7] = (__bf16)b.w;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (__bf16)(k + i < D ? row[k + i] : 0.0f);
  }
  return r;
}

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)0.0f;
  return r;
}

__device__ __forceinline__ float sigmoid_b(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }
__device__ __forceinline__ float tanh_b(float x) { return 2.0f * sigmoid_b(2.0f * x) - 1.0f; }

}  // namespace

// P[tau][cb] = sum_k Vx[tau][k] * x[t][b][k] for tau < a.rows, cb = t*Bp + b.
// Workgroup: 4 waves over a 64 x 64 tile, each wave 32 x 32 (2 x 2 MFMA
// blocks).  Grid: (T*Bp/64, ceil(rows/64)).
__global__ void __launch_bounds__(256) batched_xproj_kernel(BatchedArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m0 = blockIdx.y * 64 + (wave & 1) * 32;
  const int n0 = blockIdx.x * 64 + (wave >> 1) * 32;
  const int li = lane & 15, lk = (lane >> 4) * 8;
  const int NB = a.T * a.Bp;
  const float* xrow[2];
  bool live[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int cb = n0 + 16 * j + li;
    const int t = cb / a.Bp, b = cb - t * a.Bp;
    live[j] = b < a.B;                                   // cb < NB by the grid
    xrow[j] = a.x + ((size_t)t * a.B + (live[j] ? b : 0)) * a.D;
  }
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < a.Dp; k += 32) {
    bf16x8 A[2], Bv[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) A[i] = load8(a.Vx + (size_t)(m0 + 16 * i + li) * a.Dp + k + lk);
#pragma unroll
    for (int j = 0; j < 2; ++j) Bv[j] = live[j] ? load_x8(xrow[j], k + lk, a.D, a.xvec != 0) : zero8();
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma(A[i], Bv[j], acc[i][j]);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + 16 * j + li;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + 16 * i + (lane >> 4) * 4 + r;
        if (row < a.rows) a.P[(size_t)row * NB + col] = acc[i][j][r];
      }
    }
}

// z of timestep t for panel rows tau < a.rows and sequences b < Bp:
// z[tau][b] = sigma_tau (P[tau][t*Bp+b] + sum_r Vh[tau][r] h[b][r]) for
// tau < GKl (the level's terms), 0 for the padding rows; stored as bf16 in
// Z[g][b][n] (tau = n*G + g), the contiguous-K operand of the accumulation.
// Grid: (ceil(rows/64), Bp/64).
__global__ void __launch_bounds__(256) batched_hproj_kernel(BatchedArgs a, int t, int GKl) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m0 = blockIdx.x * 64 + (wave & 1) * 32;
  const int n0 = blockIdx.y * 64 + (wave >> 1) * 32;
  const int li = lane & 15, lk = (lane >> 4) * 8;
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < a.Hp; k += 32) {
    bf16x8 A[2], Bv[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) A[i] = load8(a.Vh + (size_t)(m0 + 16 * i + li) * a.Hp + k + lk);
#pragma unroll
    for (int j = 0; j < 2; ++j) Bv[j] = load8(a.hb + (size_t)(n0 + 16 * j + li) * a.Hp + k + lk);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma(A[i], Bv[j], acc[i][j]);
  }
  const int NB = a.T * a.Bp;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int b = n0 + 16 * j + li;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int tau = m0 + 16 * i + (lane >> 4) * 4 + r;
        if (tau >= a.rows) continue;
        float z = 0.0f;
        if (tau < GKl) z = a.sigma[tau] * (a.P[(size_t)tau * NB + t * a.Bp + b] + acc[i][j][r]);
        const int g = tau % a.G, n = tau / a.G;
        a.Z[((size_t)g * a.Bp + b) * a.Kp + n] = bf16_bits(z);
      }
    }
}

// y of timestep t and the cell update.  Workgroup: hidden units
// [32*blockIdx.x, +32) x sequences [32*blockIdx.y, +32); wave q computes
// gate q's 32 x 32 block (rows q*H + r of U); the four gate values of each
// (unit, sequence) meet in LDS for the c/h update.  Grid: (ceil(H/32), Bp/32).
__global__ void __launch_bounds__(256) batched_accum_kernel(BatchedArgs a, int t, int Kl32, int level) {
  __shared__ float ys[4][32][33];
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int r0 = blockIdx.x * 32, b0 = blockIdx.y * 32;
  const int li = lane & 15, lk = (lane >> 4) * 8;
  const int g = (a.G == 4) ? q : 0;
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const uint16_t* urow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = r0 + 16 * i + li;
    urow[i] = a.Ut + (size_t)(q * a.H + (r < a.H ? r : 0)) * a.Kp;
  }
  for (int k = 0; k < Kl32; k += 32) {
    bf16x8 A[2], Bv[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) A[i] = load8(urow[i] + k + lk);
#pragma unroll
    for (int j = 0; j < 2; ++j) Bv[j] = load8(a.Z + ((size_t)g * a.Bp + b0 + 16 * j + li) * a.Kp + k + lk);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma(A[i], Bv[j], acc[i][j]);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) ys[q][16 * i + (lane >> 4) * 4 + r][16 * j + li] = acc[i][j][r];
  __syncthreads();
  for (int e = threadIdx.x; e < 32 * 32; e += 256) {
    const int rr = e & 31, bb = e >> 5;
    const int r = r0 + rr, b = b0 + bb;
    if (r >= a.H) continue;
    const float yi = ys[0][rr][bb] + a.bias[0 * a.H + r];
    const float yf = ys[1][rr][bb] + a.bias[1 * a.H + r];
    const float yg = ys[2][rr][bb] + a.bias[2 * a.H + r];
    const float yo = ys[3][rr][bb] + a.bias[3 * a.H + r];
    const float c = sigmoid_b(yf) * a.c[(size_t)b * a.H + r] + sigmoid_b(yi) * tanh_b(yg);
    const float h = sigmoid_b(yo) * tanh_b(c);
    a.c[(size_t)b * a.H + r] = c;
    a.hb[(size_t)b * a.Hp + r] = bf16_bits(h);
    if (b < a.B) a.h_out[(((size_t)level * a.T + t) * a.B + b) * a.H + r] = h;
  }
}

// initial state: hb = bf16(h0), c = c0 (zeros when null; padding rows and
// sequences zero)
__global__ void batched_init_kernel(BatchedArgs a) {
  const size_t n = (size_t)a.Bp * a.Hp;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int b = (int)(i / a.Hp), r = (int)(i % a.Hp);
    const bool live = b < a.B && r < a.H;
    a.hb[i] = bf16_bits((live && a.h0) ? a.h0[(size_t)b * a.H + r] : 0.0f);
    if (r < a.H) a.c[(size_t)b * a.H + r] = (live && a.c0) ? a.c0[(size_t)b * a.H + r] : 0.0f;
  }
}

__global__ void batched_cout_kernel(BatchedArgs a, int level) {
  const size_t n = (size_t)a.B * a.H;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    a.c_out[(size_t)level * n + i] = a.c[i];
}

hipError_t launch_batched(const BatchedArgs& a, const int* levels, int n_levels, hipStream_t stream) {
  if (a.Bp % 64 != 0 || a.Bp < a.B || a.Bp > (1 << 20)) return hipErrorInvalidValue;
  int kmax = 0;
  for (int l = 0; l < n_levels; ++l) kmax = std::max(kmax, levels[l]);
  if (kmax > a.Kp) return hipErrorInvalidValue;
  hipError_t e;
  if (kmax > 0) {
    BatchedArgs p = a;
    p.rows = a.G * ((kmax + 31) / 32) * 32;               // every term a level may use, padded
    batched_xproj_kernel<<<dim3(a.T * a.Bp / 64, (p.rows + 63) / 64), dim3(256), 0, stream>>>(p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  for (int l = 0; l < n_levels; ++l) {
    const int K = levels[l];
    const int Kl32 = ((K + 31) / 32) * 32;
    BatchedArgs p = a;
    p.rows = a.G * Kl32;
    batched_init_kernel<<<dim3(128), dim3(256), 0, stream>>>(p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    for (int t = 0; t < a.T; ++t) {
      if (K > 0) {
        batched_hproj_kernel<<<dim3((p.rows + 63) / 64, a.Bp / 64), dim3(256), 0, stream>>>(p, t, a.G * K);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      batched_accum_kernel<<<dim3((a.H + 31) / 32, a.Bp / 32), dim3(256), 0, stream>>>(p, t, Kl32, l);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (a.c_out) {
      batched_cout_kernel<<<dim3(64), dim3(256), 0, stream>>>(p, l);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace alstm
