// The exact LSTM on gfx950: the dense baseline the progressive approximation
// is measured against.  Gate pre-activations y = W_x x_t + W_h h_{t-1} + b
// with the full weight matrices (Sec. II, Fig. 1; the augmented matrix of
// Sec. III without any factorisation), then the same cell update.
//
// Two launches per run.  exact_xproj_kernel computes the x part of every
// gate row for every timestep at once (it does not depend on h).  The
// persistent exact_lstm_kernel then runs the recurrence: workgroup j owns a
// slice of hidden units and the four W_h rows of each, held in registers for
// the whole sequence, so one timestep needs a single exchange between
// workgroups (the h all-gather), where the progressive scheme needs two
// (z, then h).
//
// A row budget (a.rows < H) gives the paper's anytime baseline (Sec. VI-B):
// the dense products stopped after that many rows of every gate, the rows
// not reached holding the bias alone.  Only the computed rows are projected
// and multiplied.
#include <type_traits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace alstm {

namespace {

constexpr int kExactLanes = 16;   // lanes per W_h row
constexpr int kExactRows = kThreads / kExactLanes;   // rows per pass (32)
constexpr int kExactWpl = 32;     // W_h entries per lane held in registers (H <= 512)
constexpr int kExactCols = 16;    // x columns per staging pass of the x projection
constexpr int kExactXprojRegs = 32;   // weights per lane of the x projection held in registers (D <= 2048)
constexpr int kExactSeq = 8;      // sequences sharing one read of a W_h row in the recurrence

}  // namespace

// px[tb][o] = b[o] + W_x[o] . x[tb] for every computed gate row o = q*H + r
// (r < rows) and column tb = t*B + b; the px entries of the other rows are
// not written.  One wave per row; the workgroup stages up to `cols` x
// columns (contiguous in x) in LDS, read by the lanes at consecutive k.  The
// lane's first 32 weights of its row are loaded into registers before the
// staging, so that their latency overlaps it; the staging keeps 8 16-byte
// loads in flight per thread when x rows are 16-byte aligned.  The column
// chunks are dealt over gridDim.y workgroups per row group.
__global__ void __launch_bounds__(kThreads) exact_xproj_kernel(ExactArgs a, int cols) {
  extern __shared__ __align__(16) float xs[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ol = blockIdx.x * kWaves + wave;     // index among the 4*rows computed rows
  const int TB = a.T * a.B, D = a.D, R = 4 * a.H;
  const bool live = ol < 4 * a.rows;
  const int q = live ? ol / a.rows : 0;
  const int o = live ? q * a.H + (ol - q * a.rows) : 0;
  const float* w = a.Wx + (size_t)o * D;
  float wv[kExactXprojRegs];
#pragma unroll
  for (int i = 0; i < kExactXprojRegs; ++i) wv[i] = w[min(lane + 64 * i, D - 1)];   // masked at use
  for (int c0 = blockIdx.y * cols; c0 < TB; c0 += gridDim.y * cols) {
    const int cn = min(cols, TB - c0);
    __syncthreads();
    const float* xsrc = a.x + (size_t)c0 * D;
    const int n = cn * D;
    if (a.xvec) {
      typedef float f4 __attribute__((ext_vector_type(4)));
      const int n4 = n >> 2;
      for (int base = 0; base < n4; base += 8 * kThreads) {
        f4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = base + u * kThreads + (int)threadIdx.x;
          v[u] = reinterpret_cast<const f4*>(xsrc)[i < n4 ? i : 0];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = base + u * kThreads + (int)threadIdx.x;
          if (i < n4) reinterpret_cast<f4*>(xs)[i] = v[u];
        }
      }
    } else {
      for (int i = threadIdx.x; i < n; i += kThreads) xs[i] = xsrc[i];
    }
    __syncthreads();
    if (live) {
      float acc[kExactCols];
#pragma unroll
      for (int c = 0; c < kExactCols; ++c) acc[c] = 0.0f;
#pragma unroll
      for (int i = 0; i < kExactXprojRegs; ++i) {
        const int k = lane + 64 * i;
        if (k < D) {
#pragma unroll
          for (int c = 0; c < kExactCols; ++c)
            if (c < cn) acc[c] += wv[i] * xs[c * D + k];
        }
      }
      for (int k = lane + 64 * kExactXprojRegs; k < D; k += 64) {
        const float wk = w[k];
#pragma unroll
        for (int c = 0; c < kExactCols; ++c)
          if (c < cn) acc[c] += wk * xs[c * D + k];
      }
#pragma unroll
      for (int c = 0; c < kExactCols; ++c) {
        if (c < cn) {
          const float s = wave_sum(acc[c]);
          if (lane == 0) a.px[(size_t)(c0 + c) * R + o] = s + a.bias[o];
        }
      }
    }
  }
}

// The recurrence.  Workgroup j owns hidden units [j*RP, j*RP + rc) and the
// gate rows q*H + r of each (q = i, f, g, o); 16 lanes per row, rows in
// passes of 32.  Per timestep and sequence: y = px + W_h . h_{t-1} (lane
// partial sums, fixed-order reduction), the cell update, h published as
// tagged words, then the full h_t gathered by every workgroup.
__global__ void __launch_bounds__(kThreads) exact_lstm_kernel(ExactArgs a) {
  extern __shared__ __align__(16) float lds[];
  const int P = gridDim.x, j = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int H = a.H, B = a.B, T = a.T, RP = a.rows_per, R4 = 4 * H;
  const int r0 = j * RP;
  const int rc = max(0, min(RP, H - r0));
  const int outs = 4 * rc;
  float* hs = lds;                         // [B][H]  h_{t-1}
  float* ys = hs + (size_t)B * H;          // [B][4*RP] y of the owned rows
  float* cs = ys + (size_t)B * 4 * RP;     // [B][RP]   c of the owned units
  float* hown = cs + (size_t)B * RP;       // [B][RP]   new h of the owned units
  float* pxs = hown + (size_t)B * RP;      // [T*B][4*RP] x part of the owned rows (px_lds)

  const int sl = threadIdx.x % kExactLanes, ob = threadIdx.x / kExactLanes;
  const int passes = (outs + kExactRows - 1) / kExactRows;
  const int rlive = max(0, min(rc, a.rows - r0));   // owned units whose rows are computed
  // pass 0's row entries in registers when H fits (the common case); zero for
  // rows not computed, so their sums are 0
  float wr[kExactWpl];
  const bool wreg = a.wreg != 0;
  {
    const int ol = ob;
    const int q = ol < outs ? ol / rc : 0, rr = ol < outs ? ol - q * rc : 0;
    const bool live = ol < outs && rr < rlive;
    const float* wrow = a.Wh + (size_t)(q * H + r0 + rr) * H;
#pragma unroll
    for (int i = 0; i < kExactWpl; ++i) {
      const int k = sl + kExactLanes * i;
      wr[i] = (wreg && live && k < H) ? wrow[k] : 0.0f;
    }
  }
  for (int i = threadIdx.x; i < B * H; i += kThreads) {
    const int b = i / H, r = i - b * H;
    hs[i] = a.h0 ? a.h0[(size_t)b * H + r] : 0.0f;
  }
  for (int i = threadIdx.x; i < B * RP; i += kThreads) {
    const int b = i / RP, rr = i - b * RP;
    cs[i] = (a.c0 && rr < rc) ? a.c0[(size_t)b * H + r0 + rr] : 0.0f;
  }
  if (a.px_lds) {
    for (int i = threadIdx.x; i < T * B * outs; i += kThreads) {
      const int tb = i / outs, ol = i - tb * outs;
      const int q = ol / rc, rr = ol - q * rc;
      const int o = q * H + r0 + rr;
      pxs[tb * 4 * RP + ol] = rr < rlive ? a.px[(size_t)tb * R4 + o] : a.bias[o];
    }
  }
  __syncthreads();

  const bool local = P == 1;
  const bool publisher = wave == kWaves - 1;
  const int gthr = kThreads - 64;
  // y of owned row ol for sequence b: the W_h sum plus the x part and bias
  auto store_y = [&](int t, int b, int ol, float sum) {
    const int q = ol / rc, rr = ol - q * rc;
    const int o = q * H + r0 + rr;
    const float px = a.px_lds ? pxs[(t * B + b) * 4 * RP + ol]
                              : (rr < rlive ? a.px[(size_t)(t * B + b) * R4 + o] : a.bias[o]);
    ys[b * 4 * RP + ol] = sum + px;
  };
  for (int t = 0; t < T; ++t) {
    const unsigned tag = a.tag_base | (unsigned)(t + 1);
    if (wreg) {
      // pass 0's entries are in registers; later passes read their rows
      for (int b = 0; b < B; ++b) {
        const float* h = hs + (size_t)b * H;
        for (int ps = 0; ps < passes; ++ps) {
          const int ol = ob + ps * kExactRows;
          float acc = 0.0f;
          if (ol < outs) {
            if (ps == 0) {
#pragma unroll
              for (int i = 0; i < kExactWpl; ++i) acc += wr[i] * h[min(sl + kExactLanes * i, H - 1)];
            } else {
              const int q = ol / rc, rr = ol - q * rc;
              const float* wrow = a.Wh + (size_t)(q * H + r0 + rr) * H;
              if (rr < rlive) {
#pragma unroll 4
                for (int k = sl; k < H; k += kExactLanes) acc += wrow[k] * h[k];
              }
            }
          }
          acc = group_sum<kExactLanes>(acc);
          if (sl == 0 && ol < outs) store_y(t, b, ol, acc);
        }
      }
    } else {
      // rows are read once per group of up to kExactSeq sequences, each entry
      // applied to every sequence of the group (NB a compile-time group size,
      // so the inner loop carries no predicates); every (row, sequence) sum
      // keeps the per-sequence order
      auto group = [&](auto nbc, int b0) {
        constexpr int NB = decltype(nbc)::value;
        for (int ps = 0; ps < passes; ++ps) {
          const int ol = ob + ps * kExactRows;
          float acc[NB];
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[j] = 0.0f;
          if (ol < outs) {
            const int q = ol / rc, rr = ol - q * rc;
            const float* wrow = a.Wh + (size_t)(q * H + r0 + rr) * H;
            if (rr < rlive && NB == 1) {
#pragma unroll 4
              for (int k = sl; k < H; k += kExactLanes) acc[0] += wrow[k] * hs[(size_t)b0 * H + k];
            } else if (rr < rlive) {
              // 8 entries of the row in flight, then each applied to the group
              for (int k0 = sl; k0 < H; k0 += 8 * kExactLanes) {
                float wk[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                  const int k = k0 + i * kExactLanes;
                  wk[i] = wrow[k < H ? k : sl];
                }
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                  const int k = k0 + i * kExactLanes;
                  if (k < H) {
#pragma unroll
                    for (int j = 0; j < NB; ++j) acc[j] += wk[i] * hs[(size_t)(b0 + j) * H + k];
                  }
                }
              }
            }
          }
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const float sum = group_sum<kExactLanes>(acc[j]);
            if (sl == 0 && ol < outs) store_y(t, b0 + j, ol, sum);
          }
        }
      };
      for (int b0 = 0; b0 < B; b0 += kExactSeq) {
        switch (min(kExactSeq, B - b0)) {
          case 1: group(std::integral_constant<int, 1>{}, b0); break;
          case 2: group(std::integral_constant<int, 2>{}, b0); break;
          case 3: group(std::integral_constant<int, 3>{}, b0); break;
          case 4: group(std::integral_constant<int, 4>{}, b0); break;
          case 5: group(std::integral_constant<int, 5>{}, b0); break;
          case 6: group(std::integral_constant<int, 6>{}, b0); break;
          case 7: group(std::integral_constant<int, 7>{}, b0); break;
          default: group(std::integral_constant<int, 8>{}, b0); break;
        }
      }
    }
    lds_barrier();
    for (int i = threadIdx.x; i < B * rc; i += kThreads) {
      const int b = i / rc, rr = i - b * rc;
      const float* y = ys + b * 4 * RP;
      float c = cs[b * RP + rr], hv;
      cell_update(y[0 * rc + rr], y[1 * rc + rr], y[2 * rc + rr], y[3 * rc + rr], c, hv);
      cs[b * RP + rr] = c;
      hown[b * RP + rr] = hv;
      if (local) hs[(size_t)b * H + r0 + rr] = hv;
    }
    lds_barrier();
    if (publisher) {
      for (int i = lane; i < B * rc; i += 64) {
        const int b = i / rc, rr = i - b * rc;
        const float hv = hown[b * RP + rr];
        a.h_out[((size_t)t * B + b) * H + r0 + rr] = hv;
        if (!local) publish(a.hx + (size_t)b * H + r0 + rr, hv, tag);
      }
    }
    if (!local && !publisher) gather_tagged<2>(hs, nullptr, a.hx, B * H, tag, a.err, threadIdx.x, gthr);
    lds_barrier();
  }
  if (a.c_out)
    for (int i = threadIdx.x; i < B * rc; i += kThreads) {
      const int b = i / rc, rr = i - b * rc;
      a.c_out[(size_t)b * H + r0 + rr] = cs[b * RP + rr];
    }
}

size_t plan_exact(ExactArgs& a, int P) {
  a.rows_per = (a.H + P - 1) / P;
  a.wreg = (a.H <= kExactLanes * kExactWpl) ? 1 : 0;
  const size_t base = 4 * ((size_t)a.B * a.H + (size_t)a.B * 4 * a.rows_per + 2 * (size_t)a.B * a.rows_per);
  const size_t pxb = 4 * (size_t)a.T * a.B * 4 * a.rows_per;
  a.px_lds = (base + pxb <= kLdsCap) ? 1 : 0;
  return base + (a.px_lds ? pxb : 0);
}

hipError_t launch_exact(const ExactArgs& a, int blocks, hipStream_t stream) {
  const int TB = a.T * a.B;
  const int cols = std::max(1, std::min(kExactCols, (int)(kLdsCap / (4 * (size_t)a.D))));
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)exact_xproj_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)kLdsCap);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute((const void*)exact_lstm_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsCap);
    if (e != hipSuccess) return e;
    attr = true;
  }
  if (a.rows > 0) {
    const size_t xl = 4 * (size_t)std::min(cols, TB) * a.D;
    const int gx = (4 * a.rows + kWaves - 1) / kWaves;
    const int gy = column_slices(gx, (TB + cols - 1) / cols);
    exact_xproj_kernel<<<dim3(gx, gy), dim3(kThreads), xl, stream>>>(a, cols);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  ExactArgs c = a;
  const size_t lds = plan_exact(c, blocks);
  if (lds > kLdsCap) return hipErrorInvalidValue;
  exact_lstm_kernel<<<dim3(blocks), dim3(kThreads), lds, stream>>>(c);
  return hipGetLastError();
}

}  // namespace alstm
