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
#include "device_common.hpp"

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
// With a.xsplit > 1 workgroup blockIdx.x takes part blockIdx.x / (nM * nN)
// of the contraction (a.Dp / a.xsplit columns) for its tile and writes the
// partial tile to Ppart[part]; batched_xproj_sum_kernel adds the parts.
template <bool VEC>
__global__ void __launch_bounds__(256) batched_xproj_kernel(BatchedArgs a, int nM, int nN) {
  __shared__ __align__(16) uint16_t As[2][kXBM * kXLD];
  __shared__ __align__(16) uint16_t Bs[2][kXBN * kXLD];
  const int nt = nM * nN;
  const int part = blockIdx.x / nt, bid = blockIdx.x - part * nt;
  int tile = bid;
  if (nt % 8 == 0) tile = (bid % 8) * (nt / 8) + bid / 8;
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
  const int nsplit = a.xsplit > 1 ? a.xsplit : 1;
  const int nS = a.Dp / kXBK / nsplit;   // slices of this part (even)
  const int kbase = part * nS * kXBK;
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
    const int k0 = kbase + (S) * kXBK;                                                                 \
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
  float* dst = nsplit > 1 ? a.Ppart + (size_t)part * NB * a.pld : a.P;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = row0 + wm * 64 + 16 * i + (lane >> 4) * 4;
    if (row >= a.rows) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = col0 + wn * 64 + 16 * j + li;
      if (col < NB)
        *reinterpret_cast<f32x4*>(dst + (size_t)col * a.pld + row) = acc[i][j];
    }
  }
}

// P = Ppart[0] + Ppart[1] + ... in part order, over the [T*Bp][pld] entries
// (pld is a multiple of 32: whole float4s).
__global__ void __launch_bounds__(256) batched_xproj_sum_kernel(BatchedArgs a) {
  const size_t stride = (size_t)a.T * a.Bp * a.pld;
  const size_t n4 = stride / 4;
  const f32x4* src = reinterpret_cast<const f32x4*>(a.Ppart);
  f32x4* out = reinterpret_cast<f32x4*>(a.P);
  for (size_t i = blockIdx.x * (size_t)256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
    f32x4 v = src[i];
    for (int k = 1; k < a.xsplit; ++k) v += src[k * (stride / 4) + i];
    out[i] = v;
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

// ---------------------------------------------------------------- persistent recurrence
// The whole recurrence of one level in one launch.  Sequences go in cohorts
// of 16 (one MFMA tile wide); a cohort is run by W workgroups of 8 waves,
// workgroup w owning hidden units [32w, 32w+32) of all four gates.  Every
// wave keeps two operand slices in registers for the whole launch:
//   * one h-projection tile: the 16 terms (g, n0 .. n0+15) of tile w*8 + wave
//     (tiles numbered group-major, so the 4 results a lane holds are
//     consecutive n of one group), their Vh rows over all of H;
//   * one accumulation tile: U rows q*H + 32w + 16*(wave>>2) + (0..15) of gate
//     q = wave & 3 over the K terms of group g(q).
// Per timestep: z tile = sigma (P + Vh . h_{t-1}) -> bf16, published to the
// cohort; every workgroup gathers all z of the cohort into LDS; y = U . z +
// bias on MFMA; the cell update (one thread per (unit, sequence), c in a
// register); h to h_out and, as bf16, published to the cohort; every
// workgroup gathers h_t into LDS.  P of the next timestep is fetched while
// the exchanges wait.
// Exchanges go through device memory with agent-scope (sc1) stores and loads,
// coherent across XCDs.  h, and z when the cohort's z are few, travel as
// tagged 64-bit words (two bf16 values | tag << 32) that readers poll
// directly; many z travel as plain bf16 behind one flag word per workgroup
// (half the bytes, one more round trip).  The exchange buffers are single: a
// workgroup writes z of step t+1 only after every workgroup has published
// h_t, which each does after it has read all of z_t (and likewise for h).
// Results equal the per-timestep kernels' up to the fp32 summation order of
// each product.
constexpr int kMaxKs = 16;   // register-resident contraction steps of 32 (H and K up to 512)

// dst (LDS, row stride dld) <- src (global, row stride sld), `rows` rows of
// 8*c8 bf16, with agent-scope (sc1) 16-byte loads, four in flight per thread
__device__ __forceinline__ void copy_rows_coherent(uint16_t* dst, int dld, const uint16_t* src, int sld, int rows,
                                                   int c8, int tid, int nthr) {
  const unsigned long long addr = reinterpret_cast<unsigned long long>(src);
  const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)addr);
  const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(addr >> 32));
  const int nbytes = __builtin_amdgcn_readfirstlane(rows * sld * 2);
  uint16_t* base = reinterpret_cast<uint16_t*>(((unsigned long long)hi << 32) | lo);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(base, (short)0, nbytes, 0x00020000);
  const int n = rows * c8;
  for (int i0 = 0; i0 < n; i0 += 4 * nthr) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * nthr + tid;
      const int r = i < n ? i / c8 : 0, c = i < n ? i - r * c8 : 0;
      v[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (r * sld + 8 * c) * 2, 0, 16 /* sc1 */));
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * nthr + tid;
      if (i < n) {
        const int r = i / c8, c = i - r * c8;
        *reinterpret_cast<u32x4*>(dst + r * dld + 8 * c) = v[u];
      }
    }
  }
}

// Tagged pairs: word p of row r of src (row stride swr words) holds bf16
// values 2p and 2p+1 of that row and the tag in its upper half.  dst (LDS, row
// stride dld bf16) <- the values of pairs p < npairs of `rows` rows, each once
// its word carries `tag`; up to 8 words in flight per thread, polled until
// they arrive.  Bounded: past the spin limit, or once another wait has failed,
// it records the failure and stores zeros.
__device__ void gather_pairs_tagged(uint16_t* dst, int dld, const unsigned long long* src, int swr, int rows,
                                    int npairs, unsigned tag, unsigned* err, int tid, int nthr) {
  const int n = rows * npairs;
  for (int base = 0; base < n; base += 8 * nthr) {
    const unsigned long long* sp[8];
    int dp[8];
    unsigned pending = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = base + k * nthr + tid;
      const int r = i < n ? i / npairs : 0, pr = i < n ? i - r * npairs : 0;
      sp[k] = src + (size_t)r * swr + pr;
      dp[k] = r * dld + 2 * pr;
      if (i < n) pending |= 1u << k;
    }
    unsigned long long wv[8];
    unsigned spins = 0;
    while (pending) {
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if ((pending >> k) & 1u) wv[k] = load_tagged(sp[k]);
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (((pending >> k) & 1u) && (unsigned)(wv[k] >> 32) == tag) {
          *reinterpret_cast<unsigned*>(dst + dp[k]) = (unsigned)wv[k];
          pending &= ~(1u << k);
        }
      if (pending && (++spins & 255u) == 0u &&
          (spins >= kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
        __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if ((pending >> k) & 1u) *reinterpret_cast<unsigned*>(dst + dp[k]) = 0u;
        pending = 0;
      }
    }
  }
}

__device__ __forceinline__ void store_coherent_u32(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void store_pair_tagged(unsigned long long* p, unsigned pair, unsigned tag) {
  __hip_atomic_store(p, ((unsigned long long)tag << 32) | pair, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// LDS bytes of a persistent launch at Kl32 (h and z tiles, y staging)
__host__ __device__ inline size_t persistent_lds(int G, int Hp, int Kl32) {
  return (size_t)2 * kCohort * ((Hp + 8) + (size_t)G * (Kl32 + 8)) + sizeof(float) * 4 * 32 * 17;
}

__global__ void __launch_bounds__(512) batched_persistent_kernel(BatchedArgs a, int K, int Kl32, int level,
                                                                 int W, int slots, int ztag) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int slot = blockIdx.x / W, w = blockIdx.x - slot * W;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, lq = lane >> 4, lk = lq * 8;
  const int G = a.G, H = a.H, Hp = a.Hp, Kp = a.Kp;
  const int hld = Hp + 8, zld = Kl32 + 8;
  uint16_t* hs = reinterpret_cast<uint16_t*>(lds_raw);                      // [16][hld]
  uint16_t* zs = hs + kCohort * hld;                                        // [G][16][zld]
  float* ys = reinterpret_cast<float*>(zs + (size_t)G * kCohort * zld);     // [4][32][17]
  // a slot's exchange: z as [G*16][Kp] bf16 (flagged) or [G*16][Kp/2] tagged
  // words; h as [16][Hp/2] tagged words
  uint16_t* zx = a.zx + (size_t)slot * G * kCohort * Kp * 2;
  unsigned long long* zxw = reinterpret_cast<unsigned long long*>(zx);
  unsigned long long* hxw = reinterpret_cast<unsigned long long*>(a.hx + (size_t)slot * kCohort * Hp * 2);
  unsigned* zflag = a.zflag + slot * W;
  const int nkh = Hp >> 5, nku = Kl32 >> 5;
  const int u0 = w * 32;
  const bool exch = K > 0;   // without terms no workgroup reads another's z or h

  // h-projection tile of this wave and its operands
  const int ntn = Kl32 >> 4;
  const int tile = w * 8 + wave;
  const bool has_tile = tile < G * ntn;
  const int tg = has_tile ? tile / ntn : 0, tn0 = has_tile ? (tile - tg * ntn) * 16 : 0;
  bf16x8 va[kMaxKs];
#pragma unroll
  for (int ks = 0; ks < kMaxKs; ++ks) {
    va[ks] = bf16x8{};
    if (has_tile && ks < nkh) va[ks] = load8(a.Vh + (size_t)((tn0 + li) * G + tg) * Hp + 32 * ks + lk);
  }
  float sg[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int n = tn0 + 4 * lq + r;
    sg[r] = (has_tile && n < K) ? a.sigma[n * G + tg] : 0.0f;
  }
  // accumulation tile of this wave
  const int q = wave & 3, half = wave >> 2;
  const int urow = u0 + 16 * half + li;
  bf16x8 ua[kMaxKs];
#pragma unroll
  for (int ks = 0; ks < kMaxKs; ++ks) {
    ua[ks] = bf16x8{};
    if (urow < H && ks < nku) ua[ks] = load8(a.Ut + (size_t)(q * H + urow) * Kp + 32 * ks + lk);
  }
  const int zg = (G == 4) ? q : 0;
  // cell-update role: unit u0 + (tid >> 4), sequence tid & 15 of the cohort
  const int ul = tid >> 4, gs = tid & 15;
  const int gu = u0 + ul;
  const bool gu_live = gu < H;
  const int gur = gu_live ? gu : 0;
  const float bi = a.bias[gur], bfg = a.bias[H + gur], bgg = a.bias[2 * H + gur], bo = a.bias[3 * H + gur];

  int iter = 0;
  for (int coh = slot; coh < (a.B + kCohort - 1) / kCohort; coh += slots, ++iter) {
    const int b0 = coh * kCohort;
    // h_{-1}; columns past H stay zero (the h gather writes units < H only)
    for (int i = tid; i < kCohort * Hp; i += 512) {
      const int sq = i / Hp, k = i - sq * Hp;
      const int b = b0 + sq;
      const float v = (a.h0 && b < a.B && k < H) ? a.h0[(size_t)b * H + k] : 0.0f;
      hs[sq * hld + k] = bf16_bits(v);
    }
    float c = 0.0f;
    if (a.c0 && b0 + gs < a.B && gu_live) c = a.c0[(size_t)(b0 + gs) * H + gu];
    // P of the lane's 4 result terms (sequence li), one timestep ahead
    float pv[4] = {0.f, 0.f, 0.f, 0.f};
    auto fetch_p = [&](int t) {
      const float* prow = a.P + (size_t)(t * a.Bp + b0 + li) * a.pld;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = tn0 + 4 * lq + r;
        pv[r] = (has_tile && n < K) ? prow[n * G + tg] : 0.0f;
      }
    };
    fetch_p(0);
    lds_barrier();
    for (int t = 0; t < a.T; ++t) {
      const unsigned tag = a.tag_base | (unsigned)(iter * a.T + t + 1);
      // ---- h-projection of the wave's tile, published as bf16
      if (has_tile) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < kMaxKs; ++ks)
          if (ks < nkh) acc = mfma(va[ks], *reinterpret_cast<const bf16x8*>(hs + li * hld + 32 * ks + lk), acc);
        unsigned zb[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) zb[r] = bf16_bits(sg[r] * (pv[r] + acc[r]));
        const size_t zoff = (size_t)(tg * kCohort + li) * Kp + tn0 + 4 * lq;   // even
        if (ztag) {
          store_pair_tagged(zxw + zoff / 2, zb[0] | (zb[1] << 16), tag);
          store_pair_tagged(zxw + zoff / 2 + 1, zb[2] | (zb[3] << 16), tag);
        } else {
          unsigned* zp = reinterpret_cast<unsigned*>(zx + zoff);
          store_coherent_u32(zp, zb[0] | (zb[1] << 16));
          store_coherent_u32(zp + 1, zb[2] | (zb[3] << 16));
        }
      }
      if (exch) {
        if (ztag) {
          if (t + 1 < a.T) fetch_p(t + 1);
          gather_pairs_tagged(zs, zld, zxw, Kp / 2, G * kCohort, Kl32 / 2, tag, a.err, tid, 512);
        } else {
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's z stores acknowledged
          lds_barrier();
          if (tid == 0) __hip_atomic_store(zflag + w, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (t + 1 < a.T) fetch_p(t + 1);
          await_flags(zflag, W, tag, a.err, tid, 512);
          lds_barrier();
          copy_rows_coherent(zs, zld, zx, Kp, G * kCohort, Kl32 >> 3, tid, 512);
        }
      } else if (t + 1 < a.T) {
        fetch_p(t + 1);
      }
      lds_barrier();
      // ---- y = U . z for the wave's rows
      {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < kMaxKs; ++ks)
          if (ks < nku)
            acc = mfma(ua[ks], *reinterpret_cast<const bf16x8*>(zs + (zg * kCohort + li) * zld + 32 * ks + lk), acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) ys[(q * 32 + 16 * half + 4 * lq + r) * 17 + li] = acc[r];
      }
      lds_barrier();
      // ---- gates and cell update
      const float yi = ys[(0 * 32 + ul) * 17 + gs] + bi;
      const float yf = ys[(1 * 32 + ul) * 17 + gs] + bfg;
      const float yg = ys[(2 * 32 + ul) * 17 + gs] + bgg;
      const float yo = ys[(3 * 32 + ul) * 17 + gs] + bo;
      c = sigmoid_b(yf) * c + sigmoid_b(yi) * tanh_b(yg);
      const float h = sigmoid_b(yo) * tanh_b(c);
      const int b = b0 + gs;
      if (gu_live && b < a.B) {
        a.h_out[(((size_t)level * a.T + t) * a.B + b) * H + gu] = h;
        if (a.c_out && t == a.T - 1) a.c_out[((size_t)level * a.B + b) * H + gu] = c;
      }
      if (exch) {
        // units in pairs (lanes l and l+16 hold units 2m and 2m+1 of one
        // sequence); a unit past H travels as zero
        const unsigned hb = gu_live ? (unsigned)bf16_bits(h) : 0u;
        const unsigned hn = (unsigned)__shfl_down((int)hb, 16, 64);
        if ((lq & 1) == 0 && gu_live) store_pair_tagged(hxw + ((size_t)gs * Hp + gu) / 2, hb | (hn << 16), tag);
        gather_pairs_tagged(hs, hld, hxw, Hp / 2, kCohort, (H + 1) / 2, tag, a.err, tid, 512);
      }
      lds_barrier();
    }
  }
}

int batched_xproj_split(int tiles, int ncu, int nslices) {
  int s = 1;
  while (2 * s <= 8 && (long long)tiles * 2 * s <= ncu && nslices % (4 * s) == 0) s *= 2;
  return s;
}

size_t batched_ppart_floats(int ncu) { return (size_t)std::max(1, ncu) * kXBM * kXBN; }

int plan_batched_persistent(const BatchedArgs& a, int K, int* W, int* slots) {
  const int Kl32 = ((K + 31) / 32) * 32;
  const int w = (a.H + 31) / 32;
  const int ncoh = (a.B + kCohort - 1) / kCohort;
  if (a.Hp > 32 * kMaxKs || Kl32 > 32 * kMaxKs || a.G * (Kl32 / 16) > 8 * w) return 0;
  if (w > a.max_wg || a.Bp % kCohort != 0) return 0;
  if (persistent_lds(a.G, a.Hp, Kl32) > kLdsCap) return 0;
  const int s = std::max(1, std::min(ncoh, a.max_wg / w));
  const long long iters = (ncoh + s - 1) / s;
  if (iters * a.T >= 65535) return 0;
  *W = w;
  *slots = s;
  return 1;
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
    p.xsplit = a.Ppart ? batched_xproj_split(nM * nN, a.ncu, a.Dp / kXBK) : 1;
    if (p.xsplit > 1 && (size_t)p.xsplit * a.T * a.Bp * p.pld > a.ppart_cap) p.xsplit = 1;
    const unsigned gx = (unsigned)(nM * nN * p.xsplit);
    if (a.xvec && a.D % kPanelDAlign == 0)
      batched_xproj_kernel<true><<<dim3(gx), dim3(256), 0, stream>>>(p, nM, nN);
    else
      batched_xproj_kernel<false><<<dim3(gx), dim3(256), 0, stream>>>(p, nM, nN);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (p.xsplit > 1) {
      const size_t n4 = (size_t)a.T * a.Bp * p.pld / 4;
      const unsigned gs = (unsigned)std::min<size_t>((n4 + 255) / 256, 2048);
      batched_xproj_sum_kernel<<<dim3(gs), dim3(256), 0, stream>>>(p);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  const bool init = a.h0 != nullptr || a.c0 != nullptr;
  for (int l = 0; l < n_levels; ++l) {
    const int K = levels[l];
    const int Kl32 = ((K + 31) / 32) * 32;
    p.rows = a.G * Kl32;
    int W = 0, slots = 0;
    if (a.zx && a.hx && a.zflag && a.err && plan_batched_persistent(p, K, &W, &slots)) {
      // one launch sequence number per level: its tags differ from every earlier launch's
      p.tag_base = a.tag_base + ((unsigned)l << 16);
      const int ztag = (a.G * Kl32 <= a.ztag_terms) ? 1 : 0;
      batched_persistent_kernel<<<dim3(W * slots), dim3(512), persistent_lds(a.G, a.Hp, Kl32), stream>>>(
          p, K, Kl32, l, W, slots, ztag);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      continue;
    }
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
