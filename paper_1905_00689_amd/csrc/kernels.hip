// gfx950 kernels for progressive approximate-LSTM inference
// (arXiv 1905.00689, Sec. III Eq. (1) per gate, then the Sec. II cell update).
//
// One cooperative, persistent launch runs a whole sequence.  Workgroup j of P
// owns the refinement terms tau = j, j+P, j+2P, ... (round-robin, so every
// prefix K is spread over all workgroups) and a contiguous slice of hidden
// units.  Per timestep:
//   phase A  for each owned term: s = P_x + prune(v)_h . h_{t-1};  z = sigma*s
//            (the x-part P_x was computed for all timesteps in the prologue);
//            z is published as a tagged 64-bit word;
//   phase B  gather every z of the level, accumulate y = b + sum_n z_n u_n for
//            the owned rows of all four gates, apply the gate nonlinearities
//            and the c/h update, publish h as tagged words;
//   phase C  gather the full h_t for the next timestep.
// The exchanges use relaxed agent-scope 64-bit atomics whose upper half is a
// per-launch, per-timestep tag: a reader spins until the tag it expects
// appears, so no counter barrier and no cache-flushing fence is needed.
#include "kernels.hpp"

namespace alstm {

namespace {

constexpr int kWaves = kThreads / 64;
constexpr unsigned kSpinLimit = 1u << 21;   // ~1 s at the polling interval below

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ void publish(unsigned long long* p, float v, unsigned tag) {
  unsigned long long w = ((unsigned long long)tag << 32) | (unsigned long long)__float_as_uint(v);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Spin until *p carries `tag`, then return its value.  Every wait is bounded:
// past the limit (or once another wait has failed) it records the failure in
// *err and returns 0 so that the grid drains.
__device__ __forceinline__ float await_tagged(const unsigned long long* p, unsigned tag, unsigned* err) {
  unsigned long long w = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  unsigned spins = 0;
  while ((unsigned)(w >> 32) != tag) {
    __builtin_amdgcn_s_sleep(1);
    ++spins;
    if ((spins & 255u) == 0u) {
      if (spins >= kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) {
        __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return 0.0f;
      }
    }
    w = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return __uint_as_float((unsigned)w);
}

__device__ __forceinline__ float sigmoidf_(float z) {
  // 1/(1+e^-z), written so that the exponential never overflows
  if (z >= 0.0f) return 1.0f / (1.0f + expf(-z));
  float e = expf(z);
  return e / (1.0f + e);
}

}  // namespace

__global__ void __launch_bounds__(kThreads) progressive_lstm_kernel(RunArgs a) {
  extern __shared__ float lds[];
  const int P = gridDim.x, j = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int D = a.D, H = a.H, G = a.G, N = a.N, NZ = a.NZ, T = a.T, B = a.B;
  const int LB = a.L * B, TB = T * B, GK = a.GK, RP = a.rows_per;
  const int r0 = j * RP;
  const int rc = max(0, min(RP, H - r0));               // hidden units owned here
  const int n_owned = (GK > j) ? (GK - j + P - 1) / P : 0;

  // LDS carve-up: [shared: x staging | z of one level] [h per (level, b)] [y] [c]
  const int shared_floats = max(a.xchunk * D, GK);
  float* xs = lds;
  float* zs = lds;
  float* hs = lds + shared_floats;
  float* ys = hs + LB * H;
  float* cs = ys + 4 * RP;

  // ---- prologue: x-part projections P_x[tau][t*B+b] of the owned terms ----
  for (int cb = 0; cb < TB; cb += a.xchunk) {
    const int cnt = min(a.xchunk, TB - cb);
    for (int i = threadIdx.x; i < cnt * D; i += kThreads) xs[i] = a.x[(size_t)cb * D + i];
    __syncthreads();
    for (int i = wave; i < n_owned; i += kWaves) {
      const int tau = j + i * P;
      const int ne = a.nx[tau];
      const uint16_t* vi = a.vidx + (size_t)tau * NZ;
      const float* vv = a.vval + (size_t)tau * NZ;
      float acc[kMaxXChunk];
#pragma unroll
      for (int c = 0; c < kMaxXChunk; ++c) acc[c] = 0.0f;
      for (int e = lane; e < ne; e += 64) {
        const float v = vv[e];
        const int k = vi[e];
#pragma unroll
        for (int c = 0; c < kMaxXChunk; ++c)
          if (c < cnt) acc[c] += v * xs[c * D + k];
      }
#pragma unroll
      for (int c = 0; c < kMaxXChunk; ++c) {
        if (c < cnt) {
          const float s = wave_sum(acc[c]);
          if (lane == 0) a.px[(size_t)tau * TB + cb + c] = s;
        }
      }
    }
    __syncthreads();
  }

  // ---- initial state ----
  for (int i = threadIdx.x; i < LB * H; i += kThreads) {
    const int b = (i / H) % B, r = i % H;
    hs[i] = a.h0 ? a.h0[(size_t)b * H + r] : 0.0f;
  }
  for (int i = threadIdx.x; i < LB * RP; i += kThreads) {
    const int lb = i / RP, rr = i % RP, b = lb % B;
    cs[i] = (a.c0 && rr < rc) ? a.c0[(size_t)b * H + r0 + rr] : 0.0f;
  }
  __syncthreads();

  for (int t = 0; t < T; ++t) {
    const unsigned tag = a.tag_base | (unsigned)(t + 1);

    // ---- phase A: z for the owned terms of every (level, sequence) ----
    for (int lb = 0; lb < LB; ++lb) {
      const int l = lb / B, b = lb % B;
      const int GKl = G * a.levels[l];
      const float* h = hs + lb * H;
      for (int i = wave; i < n_owned; i += kWaves) {
        const int tau = j + i * P;
        if (tau >= GKl) break;
        const int e0 = a.nx[tau];
        const uint16_t* vi = a.vidx + (size_t)tau * NZ;
        const float* vv = a.vval + (size_t)tau * NZ;
        float acc = 0.0f;
        for (int e = e0 + lane; e < NZ; e += 64) acc += vv[e] * h[vi[e] - D];
        acc = wave_sum(acc);
        if (lane == 0) {
          const float z = a.sigma[tau] * (a.px[(size_t)tau * TB + t * B + b] + acc);
          publish(a.zx + (size_t)lb * GK + tau, z, tag);
        }
      }
    }

    // ---- phase B: y for the owned rows, gates, c and h ----
    for (int lb = 0; lb < LB; ++lb) {
      const int l = lb / B, b = lb % B;
      const int Kl = a.levels[l];
      const int GKl = G * Kl;
      for (int i = threadIdx.x; i < GKl; i += kThreads)
        zs[i] = await_tagged(a.zx + (size_t)lb * GK + i, tag, a.err);
      __syncthreads();
      for (int ol = wave; ol < 4 * rc; ol += kWaves) {
        const int q = ol / rc, rr = ol % rc;
        const int o = q * H + r0 + rr;                  // row of the 4H gate stack
        const int g = (G == 4) ? q : 0;
        const float* urow = a.Ut + (size_t)o * N;
        float acc = 0.0f;
        for (int n = lane; n < Kl; n += 64) acc += zs[n * G + g] * urow[n];
        acc = wave_sum(acc);
        if (lane == 0) ys[q * RP + rr] = acc + a.bias[o];
      }
      __syncthreads();
      for (int rr = threadIdx.x; rr < rc; rr += kThreads) {
        const float gi = sigmoidf_(ys[0 * RP + rr]);
        const float gf = sigmoidf_(ys[1 * RP + rr]);
        const float gg = tanhf(ys[2 * RP + rr]);
        const float go = sigmoidf_(ys[3 * RP + rr]);
        const float c = gf * cs[lb * RP + rr] + gi * gg;
        const float hv = go * tanhf(c);
        cs[lb * RP + rr] = c;
        const int r = r0 + rr;
        a.h_out[(((size_t)l * T + t) * B + b) * H + r] = hv;
        publish(a.hx + (size_t)lb * H + r, hv, tag);
      }
      __syncthreads();
    }

    // ---- phase C: gather h_t ----
    for (int i = threadIdx.x; i < LB * H; i += kThreads) hs[i] = await_tagged(a.hx + i, tag, a.err);
    __syncthreads();
  }

  if (a.c_out) {
    for (int i = threadIdx.x; i < LB * rc; i += kThreads) {
      const int lb = i / rc, rr = i % rc;
      a.c_out[(size_t)lb * H + r0 + rr] = cs[lb * RP + rr];
    }
  }
}

__global__ void clear_u64_kernel(unsigned long long* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0ull;
}

size_t progressive_lds_bytes(const RunArgs& a) {
  const size_t shared_floats = (size_t)std::max(a.xchunk * a.D, a.GK);
  const size_t LB = (size_t)a.L * a.B;
  return sizeof(float) * (shared_floats + LB * a.H + 4 * (size_t)a.rows_per + LB * a.rows_per);
}

hipError_t launch_progressive(const RunArgs& a, int blocks, hipStream_t stream) {
  const size_t lds = progressive_lds_bytes(a);
  hipError_t e = hipFuncSetAttribute((const void*)progressive_lstm_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  RunArgs copy = a;
  void* args[] = {&copy};
  return hipLaunchCooperativeKernel((const void*)progressive_lstm_kernel, dim3(blocks), dim3(kThreads),
                                    args, (unsigned)lds, stream);
}

hipError_t launch_clear_u64(unsigned long long* p, size_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  int blocks = (int)std::min<size_t>((n + 255) / 256, 1024);
  clear_u64_kernel<<<blocks, 256, 0, stream>>>(p, n);
  return hipGetLastError();
}

}  // namespace alstm
