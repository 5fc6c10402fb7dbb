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
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4 mfma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 load8(const uint16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ uint16_t bf16_bits(float v) { return __builtin_bit_cast(uint16_t, (__bf16)v); }

// Workgroup barrier that orders LDS traffic only: global loads still in
// flight (prefetches) are not waited for, unlike __syncthreads, whose
// workgroup-scope release fence waits for every outstanding memory operation.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float sigmoid_b(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }
__device__ __forceinline__ float tanh_b(float x) { return 2.0f * sigmoid_b(2.0f * x) - 1.0f; }

}  // namespace

// ---------------------------------------------------------------- x-projection
// P[t*Bp + b][tau] = sum_k Vx[tau][k] * x[t][b][k] for tau < a.rows.
// One 128 (tau) x 128 (t, b) tile per workgroup of 4 waves, each wave a
// 64 x 64 quadrant (4 x 4 MFMA blocks); the contraction runs in slices of 32
// staged through LDS, double-buffered: slice s+1 is fetched into registers
// (x converted to bf16 on the way) while slice s is multiplied.  Tiles are
// numbered so that each XCD (workgroups are dealt to the 8 XCDs round robin)
// takes whole columns of tiles: the x slice of a column is fetched into that
// XCD's L2 once and shared by every row tile.
constexpr int kXBM = kPanelRowAlign, kXBN = 128, kXBK = 32;
static_assert(kPanelDAlign == 2 * kXBK, "D is padded to a pair of x-projection slices");
constexpr int kXLD = kXBK + 8;   // LDS row stride (bf16): 80 bytes, conflict-free 16-byte reads

// VEC: x rows are 16-byte aligned and D is a multiple of the D padding (so
// Dp == D): every slice of a live row is whole float4s (no bounds tests in
// the fetch).
template <bool VEC>
__global__ void __launch_bounds__(256) batched_xproj_kernel(BatchedArgs a, int nM, int nN) {
  __shared__ __align__(16) uint16_t As[2][kXBM * kXLD];
  __shared__ __align__(16) uint16_t Bs[2][kXBN * kXLD];
  const int nt = nM * nN;
  int tile = blockIdx.x;
  if (nt % 8 == 0) tile = (blockIdx.x % 8) * (nt / 8) + blockIdx.x / 8;
  const int row0 = (tile % nM) * kXBM, col0 = (tile / nM) * kXBN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int li = lane & 15, lk = (lane >> 4) * 8;
  const int NB = a.T * a.Bp;

  // global -> register staging: A 2 x 16 bytes, B 4 x float4 per thread
  const int ar = tid >> 2, ac = tid & 3;       // A chunk: rows ar + 64j, bf16 8*ac
  const int bc = tid & 7, bcl = tid >> 3;      // B chunk: columns bcl + 32j, floats 4*bc
  // x offsets: row 0 stands in for padding columns, whose values are
  // replaced by zeros at the stash (so that no use of a fetched value precedes
  // it); the host guarantees T*B*D < 2^31 and rows*Dp < 2^31
  // 32-bit lane offsets (elements): the fetches below address a uniform base
  // plus these, so no per-fetch 64-bit address arithmetic is needed
  unsigned aoff[2], xoff[4];
#pragma unroll
  for (int j = 0; j < 2; ++j) aoff[j] = (unsigned)(row0 + ar + 64 * j) * (unsigned)a.Dp + 8u * ac;
  unsigned live = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = col0 + bcl + 32 * j;
    const int t = col / a.Bp, b = col - t * a.Bp;
    const bool l = col < NB && b < a.B;
    live |= (l ? 1u : 0u) << j;
    xoff[j] = (l ? (unsigned)((t * a.B + b) * a.D) : 0u) + 4u * bc;
  }
  u32x4 ra[2][2];
  f32x4 rb[2][4];
  const int nS = a.Dp / kXBK;
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // slice s lives in register set s & 1 from its fetch (issued before the
  // multiplication of slice s-2) until its stash into LDS buffer s & 1 (after
  // the multiplication of slice s-1): two multiplications hide each fetch.
  // A slice is one MFMA contraction step (32).
#define XPROJ_FETCH(R, S)                                                                              \
  do {                                                                                                 \
    const int k0 = (S) * kXBK;                                                                         \
    const uint16_t* va_ = a.Vx + k0;                                                                   \
    _Pragma("unroll") for (int j = 0; j < 2; ++j) ra[R][j] =                                           \
        *reinterpret_cast<const u32x4*>(va_ + aoff[j]);                                                \
    if constexpr (VEC) {                                                                               \
      const float* xa_ = a.x + k0;                                                                     \
      _Pragma("unroll") for (int j = 0; j < 4; ++j)                                                    \
          rb[R][j] = *reinterpret_cast<const f32x4*>(xa_ + xoff[j]);                                   \
    } else {                                                                                           \
      const int k = k0 + 4 * bc;                                                                       \
      _Pragma("unroll") for (int j = 0; j < 4; ++j) {                                                  \
        const float* q = a.x + (xoff[j] - 4u * bc);                                                    \
        const bool l = ((live >> j) & 1u) != 0;                                                        \
        rb[R][j] = f32x4{l && k < a.D ? q[k] : 0.f, l && k + 1 < a.D ? q[k + 1] : 0.f,                 \
                         l && k + 2 < a.D ? q[k + 2] : 0.f, l && k + 3 < a.D ? q[k + 3] : 0.f};        \
      }                                                                                                \
    }                                                                                                  \
  } while (0)
#define XPROJ_STASH(R)                                                                                 \
  do {                                                                                                 \
    _Pragma("unroll") for (int j = 0; j < 2; ++j)                                                      \
        *reinterpret_cast<u32x4*>(&As[R][(ar + 64 * j) * kXLD + 8 * ac]) = ra[R][j];                   \
    _Pragma("unroll") for (int j = 0; j < 4; ++j) {                                                    \
      const f32x4 v = ((live >> j) & 1u) ? rb[R][j] : f32x4{0.f, 0.f, 0.f, 0.f};                       \
      const uint32_t lo = bf16_bits(v[0]) | ((uint32_t)bf16_bits(v[1]) << 16);                         \
      const uint32_t hi = bf16_bits(v[2]) | ((uint32_t)bf16_bits(v[3]) << 16);                         \
      *reinterpret_cast<u32x2*>(&Bs[R][(bcl + 32 * j) * kXLD + 4 * bc]) = u32x2{lo, hi};               \
    }                                                                                                  \
  } while (0)

#define XPROJ_MUL(BUF)                                                                                 \
  do {                                                                                                 \
    bf16x8 A[4], Bv[4];                                                                                \
    _Pragma("unroll") for (int i = 0; i < 4; ++i)                                                      \
        A[i] = *reinterpret_cast<const bf16x8*>(&As[BUF][(wm * 64 + 16 * i + li) * kXLD + lk]);        \
    _Pragma("unroll") for (int j = 0; j < 4; ++j)                                                      \
        Bv[j] = *reinterpret_cast<const bf16x8*>(&Bs[BUF][(wn * 64 + 16 * j + li) * kXLD + lk]);       \
    _Pragma("unroll") for (int i = 0; i < 4; ++i)                                                      \
        _Pragma("unroll") for (int j = 0; j < 4; ++j) acc[i][j] = mfma(A[i], Bv[j], acc[i][j]);        \
  } while (0)

  // nS is even (Dp is a multiple of 2 slices): the steady-state loop handles
  // a pair of slices with no conditions, the last pair is peeled
  XPROJ_FETCH(0, 0);
  XPROJ_FETCH(1, 1);
  XPROJ_STASH(0);
  lds_barrier();
  // sched_barrier keeps the compiler from hoisting a stash (which must wait
  // for its fetch) above the multiplication it is meant to overlap
  for (int ss = 0; ss + 2 < nS; ss += 2) {
    XPROJ_FETCH(0, ss + 2);   // set 0 was stashed before the last barrier
    __builtin_amdgcn_sched_barrier(0);
    XPROJ_MUL(0);             // slice ss
    __builtin_amdgcn_sched_barrier(0);
    XPROJ_STASH(1);           // slice ss+1; buffer 1's readers passed the last barrier
    lds_barrier();
    XPROJ_FETCH(1, ss + 3);
    __builtin_amdgcn_sched_barrier(0);
    XPROJ_MUL(1);             // slice ss+1
    __builtin_amdgcn_sched_barrier(0);
    XPROJ_STASH(0);           // slice ss+2
    lds_barrier();
  }
  XPROJ_MUL(0);               // slice nS-2
  XPROJ_STASH(1);             // slice nS-1
  lds_barrier();
  XPROJ_MUL(1);
#undef XPROJ_MUL
#undef XPROJ_FETCH
#undef XPROJ_STASH
  // P is column-major in tau: the 4 result rows a lane holds are adjacent
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = row0 + wm * 64 + 16 * i + (lane >> 4) * 4;
    if (row >= a.rows) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = col0 + wn * 64 + 16 * j + li;
      if (col < NB)
        *reinterpret_cast<f32x4*>(a.P + (size_t)col * a.pld + row) = acc[i][j];
    }
  }
}

// ---------------------------------------------------------------- h-projection
// z of timestep t for panel rows [32*blockIdx.x, +32) and sequences
// [32*blockIdx.y, +32): z[tau][b] = sigma_tau (P[t*Bp+b][tau] + Vh[tau][:] .
// h[b][:]) for tau < GKl, 0 for the padding rows; stored as bf16 in
// Z[g][b][n] (tau = n*G + g).  The contraction over H is split over the 4
// waves (k-steps w, w+4, ...), each issuing the loads of up to 4 k-steps
// before its MFMAs; the partial tiles are summed in LDS.
__global__ void __launch_bounds__(256) batched_hproj_kernel(BatchedArgs a, int t, int GKl, int first) {
  __shared__ float red[4][32][33];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tau0 = blockIdx.x * 32, b0 = blockIdx.y * 32;
  const int li = lane & 15, lk = (lane >> 4) * 8;
  // epilogue mapping: thread -> one sequence b and 4 terms with consecutive n
  // of one group g; its P and sigma values are fetched first so that their
  // latency overlaps the contraction
  const int b = tid >> 3, jj = tid & 7;
  int g, nl0;
  if (a.G == 4) { g = jj >> 1; nl0 = (jj & 1) * 4; } else { g = 0; nl0 = jj * 4; }
  const float* prow = a.P + (size_t)(t * a.Bp + b0 + b) * a.pld;
  float pv[4], sg[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tau = tau0 + (nl0 + i) * a.G + g;
    const bool live = tau < GKl;
    pv[i] = live ? prow[tau] : 0.0f;
    sg[i] = live ? a.sigma[tau] : 0.0f;
  }
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nks = first ? 0 : (a.Hp >> 5);            // h_{-1} = 0: nothing to contract
  const uint16_t* va = a.Vh + (size_t)(tau0 + li) * a.Hp + lk;
  const uint16_t* hbp = a.hb + (size_t)(b0 + li) * a.Hp + lk;
  for (int base = wave; base < nks; base += 16) {
    bf16x8 A[4][2], Bv[4][2];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int ks = base + 4 * c;
      if (ks < nks) {
#pragma unroll
        for (int i = 0; i < 2; ++i) A[c][i] = load8(va + (size_t)16 * i * a.Hp + 32 * ks);
#pragma unroll
        for (int j = 0; j < 2; ++j) Bv[c][j] = load8(hbp + (size_t)16 * j * a.Hp + 32 * ks);
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (base + 4 * c < nks)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma(A[c][i], Bv[c][j], acc[i][j]);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][16 * i + (lane >> 4) * 4 + r][16 * j + li] = acc[i][j][r];
  lds_barrier();
  uint16_t zb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tl = (nl0 + i) * a.G + g;                 // tau within the tile
    const float s = red[0][tl][b] + red[1][tl][b] + red[2][tl][b] + red[3][tl][b];
    zb[i] = bf16_bits(sg[i] * (pv[i] + s));             // 0 for tau >= GKl
  }
  const int n0 = tau0 / a.G + nl0;
  *reinterpret_cast<u32x2*>(a.Z + ((size_t)g * a.Bp + b0 + b) * a.Kp + n0) =
      u32x2{zb[0] | ((uint32_t)zb[1] << 16), zb[2] | ((uint32_t)zb[3] << 16)};
}

// ---------------------------------------------------------------- accumulation
// y of timestep t and the cell update for hidden units [16*blockIdx.x, +16)
// and sequences [32*blockIdx.y, +32).  8 waves: wave w takes gate q = w & 3
// (rows q*H + r of U, z of group g(q)) and the k-steps of parity w >> 2,
// issuing the loads of up to 8 k-steps before its MFMAs; the halves and the
// four gates meet in LDS for the c/h update.
__global__ void __launch_bounds__(512) batched_accum_kernel(BatchedArgs a, int t, int Kl32, int level, int first) {
  __shared__ float red[8][16][33];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = wave & 3, half = wave >> 2;
  const int r0 = blockIdx.x * 16, b0 = blockIdx.y * 32;
  const int li = lane & 15, lk = (lane >> 4) * 8;
  const int g = (a.G == 4) ? q : 0;
  // epilogue operands first (their latency overlaps the contraction)
  const int rr = tid & 15, bb = tid >> 4;
  const int r = r0 + rr, b = b0 + bb;
  const bool unit = r < a.H;
  const int rs = unit ? r : 0;
  const float bi = a.bias[0 * a.H + rs], bf = a.bias[1 * a.H + rs];
  const float bg = a.bias[2 * a.H + rs], bo = a.bias[3 * a.H + rs];
  const float cprev = first ? 0.0f : a.c[(size_t)b * a.H + rs];
  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  const int ru = r0 + li;
  const uint16_t* ua = a.Ut + (size_t)(q * a.H + (ru < a.H ? ru : 0)) * a.Kp + lk;
  const uint16_t* zp = a.Z + ((size_t)g * a.Bp + b0 + li) * a.Kp + lk;
  const int nks = Kl32 >> 5;
  for (int base = half; base < nks; base += 16) {
    bf16x8 A[8], Bv[8][2];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int ks = base + 2 * c;
      if (ks < nks) {
        A[c] = load8(ua + 32 * ks);
#pragma unroll
        for (int j = 0; j < 2; ++j) Bv[c][j] = load8(zp + (size_t)16 * j * a.Kp + 32 * ks);
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
      if (base + 2 * c < nks)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[j] = mfma(A[c], Bv[c][j], acc[j]);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int k = 0; k < 4; ++k) red[wave][(lane >> 4) * 4 + k][16 * j + li] = acc[j][k];
  lds_barrier();
  if (!unit) return;
  const float yi = red[0][rr][bb] + red[4][rr][bb] + bi;
  const float yf = red[1][rr][bb] + red[5][rr][bb] + bf;
  const float yg = red[2][rr][bb] + red[6][rr][bb] + bg;
  const float yo = red[3][rr][bb] + red[7][rr][bb] + bo;
  const float c = sigmoid_b(yf) * cprev + sigmoid_b(yi) * tanh_b(yg);
  const float h = sigmoid_b(yo) * tanh_b(c);
  a.c[(size_t)b * a.H + r] = c;
  a.hb[(size_t)b * a.Hp + r] = bf16_bits(h);
  if (b < a.B) {
    a.h_out[(((size_t)level * a.T + t) * a.B + b) * a.H + r] = h;
    if (a.c_out && t == a.T - 1) a.c_out[((size_t)level * a.B + b) * a.H + r] = c;
  }
}

// initial state given by the caller: hb = bf16(h0), c = c0 (zeros where one
// of them is null; padding sequences zero; padding columns of hb untouched,
// they stay zero from allocation)
__global__ void batched_init_kernel(BatchedArgs a) {
  const int n = a.Bp * a.H;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const int b = i / a.H, r = i - b * a.H;
    const bool live = b < a.B;
    a.hb[(size_t)b * a.Hp + r] = bf16_bits((live && a.h0) ? a.h0[(size_t)b * a.H + r] : 0.0f);
    a.c[(size_t)b * a.H + r] = (live && a.c0) ? a.c0[(size_t)b * a.H + r] : 0.0f;
  }
}

hipError_t launch_batched(const BatchedArgs& a, const int* levels, int n_levels, hipStream_t stream) {
  if (a.Bp % kBatchAlign != 0 || a.Bp < a.B || a.Bp > (1 << 20) || a.Dp % kPanelDAlign != 0 || a.Dp < a.D ||
      a.Hp % 32 != 0 || a.Hp < a.H || a.Kp % 32 != 0)
    return hipErrorInvalidValue;
  int kmax = 0;
  for (int l = 0; l < n_levels; ++l) kmax = std::max(kmax, levels[l]);
  if (kmax > a.Kp) return hipErrorInvalidValue;
  BatchedArgs p = a;
  p.pld = a.G * ((kmax + 31) / 32) * 32;                  // every term a level may use, padded
  hipError_t e;
  if (kmax > 0) {
    p.rows = p.pld;
    const int nM = (p.rows + kXBM - 1) / kXBM, nN = (a.T * a.Bp + kXBN - 1) / kXBN;
    if (a.xvec && a.D % kPanelDAlign == 0)
      batched_xproj_kernel<true><<<dim3(nM * nN), dim3(256), 0, stream>>>(p, nM, nN);
    else
      batched_xproj_kernel<false><<<dim3(nM * nN), dim3(256), 0, stream>>>(p, nM, nN);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const bool init = a.h0 != nullptr || a.c0 != nullptr;
  for (int l = 0; l < n_levels; ++l) {
    const int K = levels[l];
    const int Kl32 = ((K + 31) / 32) * 32;
    p.rows = a.G * Kl32;
    if (init) {
      batched_init_kernel<<<dim3(128), dim3(256), 0, stream>>>(p);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    for (int t = 0; t < a.T; ++t) {
      const int first = (t == 0 && !init) ? 1 : 0;
      if (K > 0) {
        batched_hproj_kernel<<<dim3(p.rows / 32, a.Bp / 32), dim3(256), 0, stream>>>(p, t, a.G * K, first);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      batched_accum_kernel<<<dim3((a.H + 15) / 16, a.Bp / 32), dim3(512), 0, stream>>>(p, t, Kl32, l, first);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace alstm
