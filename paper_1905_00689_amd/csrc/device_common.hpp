// Device helpers shared by the gfx950 kernels: fixed-order lane reductions,
// the tagged-word and bulk exchanges between workgroups of a persistent
// launch, an LDS-only workgroup barrier and the gate nonlinearities.
#pragma once

#include "kernels.hpp"

namespace alstm {

namespace {

constexpr int kWaves = kThreads / 64;
constexpr unsigned kSpinLimit = 1u << 21;   // about a second at the polling interval below
constexpr int kGatherSlots = 8;             // tagged words per thread per gather pass

// Sum over aligned groups of S lanes (S = 1, 2, 4, 8, 16) with DPP lane
// moves: quad swaps (xor 1, xor 2), then half-row and row mirrors.  Every
// lane of a group ends with the group's sum; the association order is fixed.
template <int S>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (S >= 2)
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
  if constexpr (S >= 4)
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
  if constexpr (S >= 8)
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
  if constexpr (S >= 16)
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));
  return v;
}

__device__ __forceinline__ float group_sum_rt(float v, int S) {
  switch (S) {
    case 1: return v;
    case 2: return group_sum<2>(v);
    case 4: return group_sum<4>(v);
    case 8: return group_sum<8>(v);
    default: return group_sum<16>(v);
  }
}

// Full-wave sum (input projection): 16-lane rows, then (r0 + r1) + (r2 + r3)
// over the four row sums, read into scalar registers (v_readlane: no LDS
// round trip, unlike a cross-row lane shuffle).  The result is uniform.
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum<16>(v);
  const int b = __builtin_bit_cast(int, v);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 48));
  return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ void publish(unsigned long long* p, float v, unsigned tag) {
  unsigned long long w = ((unsigned long long)tag << 32) | (unsigned long long)__float_as_uint(v);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned long long load_tagged(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Gather of tagged exchange words by threads tid < nthr: word i (< n) lands
// at dst[map ? map[i] : i] once it carries `tag`.  Each thread keeps two
// generations of loads of its words in flight (re-issued unconditionally, so
// the in-order completion counter lets one generation be consumed while the
// next travels), which halves the delay between a word's arrival and its
// detection.  Bounded: past the spin limit, or once another wait has failed,
// it records the failure and stores 0.
template <int NS>
__device__ void gather_tagged(float* dst, const uint16_t* map, const unsigned long long* src, int n, unsigned tag,
                              unsigned* err, int tid, int nthr) {
  for (int base = 0; base < n; base += nthr * NS) {
    const unsigned long long* sp[NS];
    unsigned pending = 0;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int i = base + k * nthr + tid;
      sp[k] = src + (i < n ? i : 0);
      if (i < n) pending |= 1u << k;
    }
    unsigned long long wa[NS], wb[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) wa[k] = load_tagged(sp[k]);
    __builtin_amdgcn_s_sleep(4);
#pragma unroll
    for (int k = 0; k < NS; ++k) wb[k] = load_tagged(sp[k]);
    unsigned spins = 0;
    while (true) {
#pragma unroll
      for (int k = 0; k < NS; ++k) {
        if (((pending >> k) & 1u) && (unsigned)(wa[k] >> 32) == tag) {
          const int i = base + k * nthr + tid;
          dst[map ? map[i] : i] = __uint_as_float((unsigned)wa[k]);
          pending &= ~(1u << k);
        }
      }
      if (!pending) break;
#pragma unroll
      for (int k = 0; k < NS; ++k) wa[k] = load_tagged(sp[k]);
#pragma unroll
      for (int k = 0; k < NS; ++k) {
        if (((pending >> k) & 1u) && (unsigned)(wb[k] >> 32) == tag) {
          const int i = base + k * nthr + tid;
          dst[map ? map[i] : i] = __uint_as_float((unsigned)wb[k]);
          pending &= ~(1u << k);
        }
      }
      if (!pending) break;
#pragma unroll
      for (int k = 0; k < NS; ++k) wb[k] = load_tagged(sp[k]);
      spins += 2;
      if ((spins & 254u) == 0u &&
          (spins >= kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
        __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int k = 0; k < NS; ++k)
          if ((pending >> k) & 1u) {
            const int i = base + k * nthr + tid;
            dst[map ? map[i] : i] = 0.0f;
          }
        break;
      }
    }
  }
}

// Bulk h exchange.  The publisher wave stores its h values with agent-scope
// (sc1, write-through) stores, waits until the wave's stores are acknowledged
// (vmcnt 0), then stores its tag in its flag word.  Readers poll every workgroup's flag, then
// read the whole h_t with agent-scope 16-byte loads; coherent across XCDs
// without any cache writeback or invalidation.
__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<unsigned*>(p), __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 1 when flag word w carries `tag` or a later timestep's tag of the same
// launch (tag = launch sequence << 16 | timestep + 1)
__device__ __forceinline__ bool flag_reached(unsigned w, unsigned tag) {
  return (w >> 16) == (tag >> 16) && (w & 0xFFFFu) >= (tag & 0xFFFFu);
}

// threads tid < nthr poll flags [0, P) until each has reached `tag` (bounded)
__device__ __forceinline__ void await_flags(const unsigned* flag, int P, unsigned tag, unsigned* err, int tid,
                                            int nthr) {
  for (int f = tid; f < P; f += nthr) {
    unsigned spins = 0;
    while (!flag_reached(__hip_atomic_load(flag + f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), tag)) {
      __builtin_amdgcn_s_sleep(2);
      if ((++spins & 255u) == 0u &&
          (spins >= kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
        __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
}

// dst[i] = src[i] for i < n (src 16-byte aligned, readable up to n rounded up
// to 4), agent-scope loads, 4 in flight per thread
__device__ __forceinline__ void read_coherent(float* dst, const float* src, int n, int tid, int nthr) {
  typedef float f32x4_t __attribute__((ext_vector_type(4)));
  // the buffer descriptor must be wave-uniform (scalar registers)
  const unsigned long long addr = reinterpret_cast<unsigned long long>(src);
  const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)addr);
  const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(addr >> 32));
  const int n4 = __builtin_amdgcn_readfirstlane((n + 3) >> 2);
  float* base = reinterpret_cast<float*>(((unsigned long long)hi << 32) | lo);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(base, (short)0, n4 * 16, 0x00020000);
  for (int base = 0; base < n4; base += 4 * nthr) {
    f32x4_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i4 = base + u * nthr + tid;
      v[u] = __builtin_amdgcn_raw_buffer_load_b128(rs, (i4 < n4 ? i4 : 0) * 16, 0, 16 /* sc1 */);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i4 = base + u * nthr + tid;
      if (i4 < n4)
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (4 * i4 + c < n) dst[4 * i4 + c] = v[u][c];
    }
  }
}

// Workgroup barrier that orders LDS only.  __syncthreads() would also wait
// for every outstanding global store of the wave (gfx9 counts stores in
// vmcnt), i.e. for the agent-scope exchange stores to reach memory.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Gate nonlinearities from the exponential: sigmoid(z) = 1/(1+e^-z) and
// tanh(x) = 2 sigmoid(2x) - 1, with the hardware exp2 and reciprocal
// (relative error ~1e-6 for |z| < 20, exact limits 0 and 1 beyond).
__device__ __forceinline__ float sigmoid_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

__device__ __forceinline__ float tanh_fast(float x) {
  return __builtin_fmaf(2.0f, sigmoid_fast(2.0f * x), -1.0f);
}

// The cell update of Sec. II from the four gate pre-activations (rows i, f,
// g, o): c' = sigmoid(y_f) c + sigmoid(y_i) tanh(y_g), h = sigmoid(y_o)
// tanh(c').  Every kernel takes it from here, with its one fused
// multiply-add written out, so that the rounding never depends on how a
// kernel's surrounding code lets the compiler contract the expression.
__device__ __forceinline__ void cell_update(float yi, float yf, float yg, float yo, float& c, float& h) {
  const float gi = sigmoid_fast(yi);
  const float gf = sigmoid_fast(yf);
  const float gg = tanh_fast(yg);
  const float go = sigmoid_fast(yo);
  c = __builtin_fmaf(gf, c, gi * gg);
  h = go * tanh_fast(c);
}

}  // namespace

}  // namespace alstm
