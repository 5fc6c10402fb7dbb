// Internal interface between the C-ABI host code and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace alstm {

constexpr int kMaxLevels = 16;
constexpr int kThreads = 512;          // 8 wave64 per workgroup
constexpr int kMaxXChunk = 16;         // (t, b) pairs staged per prologue pass

// Everything one launch of the progressive-LSTM kernel needs.  Device
// pointers unless noted.  Layouts (row-major):
//   x      [T][B][D]            h0, c0 [B][H] or null
//   h_out  [L][T][B][H]         c_out  [L][B][H] or null
//   sigma  [N*G]                term tau = n*G + g (refinement order)
//   Ut     [4H][N]              Ut[o][n] = u of term (n, g(o)) at row o within its group
//   vidx   [N*G][NZ] uint16     ascending column indices into [x; h]
//   vval   [N*G][NZ]            entries of prune(v) on vidx
//   nx     [N*G] uint16         number of vidx entries < D (the x/h split)
//   bias   [4H]
//   px     [GK][T*B]            x-part projections (workspace)
//   zx     [L*B][GK] u64        tagged z exchange (value | tag << 32)
//   hx     [L*B][H] u64         tagged h exchange
struct RunArgs {
  const float* x;
  const float* h0;
  const float* c0;
  float* h_out;
  float* c_out;
  const float* sigma;
  const float* Ut;
  const uint16_t* vidx;
  const float* vval;
  const uint16_t* nx;
  const float* bias;
  float* px;
  unsigned long long* zx;
  unsigned long long* hx;
  unsigned* err;
  int D, H, G, N, NZ, T, B, L;
  int GK;          // G * max level: terms in use
  int rows_per;    // hidden units owned per workgroup
  int xchunk;      // (t, b) pairs staged per prologue pass (<= kMaxXChunk)
  unsigned tag_base;
  int levels[kMaxLevels];
};

// LDS bytes the kernel needs for these sizes.
size_t progressive_lds_bytes(const RunArgs& a);

// Cooperative launch of `blocks` workgroups on `stream`.
hipError_t launch_progressive(const RunArgs& a, int blocks, hipStream_t stream);

// Zero `n` 64-bit words (exchange-buffer reset) with a plain kernel.
hipError_t launch_clear_u64(unsigned long long* p, size_t n, hipStream_t stream);

}  // namespace alstm
