// gfx950 kernels for progressive approximate-LSTM inference
// (arXiv 1905.00689, Sec. III Eq. (1) per gate, then the Sec. II cell update).
//
// input_proj_kernel computes, before the recurrence and over the whole GPU,
// the x-part projections P_x = prune(v)_x . x_t of every term in use and
// every timestep (they do not depend on h).  Then one persistent launch runs
// the whole sequence.  Workgroup j of P owns the refinement terms tau = j,
// j+P, j+2P, ... (round-robin, so every prefix K is spread over all
// workgroups) and a contiguous slice of hidden units (all four gates of
// each).  The prologue loads the owned terms' h-part entries and the owned
// rows of U into registers (HPL / UPT instances; LDS, or for U global memory,
// where they do not fit) and sigma, the bias and P_x into LDS, where they
// stay for the whole sequence.  Per timestep:
//   phase A  for each owned term: s = P_x + prune(v)_h . h_{t-1};  z = sigma*s;
//            z is published as a tagged 64-bit word;
//   phase B  gather every z of the level, accumulate y = b + sum_n z_n u_n for
//            the owned rows of all four gates, apply the gate nonlinearities
//            and the c/h update, publish h (tagged words, or in bulk behind
//            one flag word per workgroup);
//   phase C  gather the full h_t for the next timestep.
// The exchanges use relaxed agent-scope 64-bit atomics whose upper half is a
// per-launch, per-timestep tag: a reader spins until the tag it expects
// appears, so there is no counter barrier and no cache-flushing fence.  Every
// wait is bounded; on expiry the kernel records an error and drains.
#include "kernels.hpp"
#include "device_common.hpp"

#include <algorithm>

namespace alstm {

namespace {

// z gather of one (level, sequence): exchange slot s carries term
// tau = slot_term[s]; slots with tau >= GKl are not part of this level (not
// written this timestep) and are skipped.  z of tau = n*G + g lands at
// zs[g*Kmax + n].  Same two-generation polling as gather_tagged.
template <int NS>
__device__ void gather_level(float* zs, const uint16_t* slot_term, const unsigned long long* src, int nslots,
                             int GKl, int G, int Kmax, unsigned tag, unsigned* err, int tid, int nthr) {
  for (int base = 0; base < nslots; base += nthr * NS) {
    const unsigned long long* sp[NS];
    int dst[NS];
    unsigned pending = 0;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int s = base + k * nthr + tid;
      const int tau = s < nslots ? (int)slot_term[s] : GKl;
      sp[k] = src + (s < nslots ? s : 0);
      dst[k] = (G == 4) ? ((tau & 3) * Kmax + (tau >> 2)) : tau;
      if (tau < GKl) pending |= 1u << k;
    }
    if (!pending) continue;
    unsigned long long wa[NS], wb[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) wa[k] = load_tagged(sp[k]);
    __builtin_amdgcn_s_sleep(4);
#pragma unroll
    for (int k = 0; k < NS; ++k) wb[k] = load_tagged(sp[k]);
    unsigned spins = 0;
    while (true) {
#pragma unroll
      for (int k = 0; k < NS; ++k)
        if (((pending >> k) & 1u) && (unsigned)(wa[k] >> 32) == tag) {
          zs[dst[k]] = __uint_as_float((unsigned)wa[k]);
          pending &= ~(1u << k);
        }
      if (!pending) break;
#pragma unroll
      for (int k = 0; k < NS; ++k) wa[k] = load_tagged(sp[k]);
#pragma unroll
      for (int k = 0; k < NS; ++k)
        if (((pending >> k) & 1u) && (unsigned)(wb[k] >> 32) == tag) {
          zs[dst[k]] = __uint_as_float((unsigned)wb[k]);
          pending &= ~(1u << k);
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
          if ((pending >> k) & 1u) zs[dst[k]] = 0.0f;
        break;
      }
    }
  }
}

__device__ __forceinline__ void gather_level_any(float* zs, const uint16_t* slot_term, const unsigned long long* src,
                                                 int nslots, int GKl, int G, int Kmax, unsigned tag, unsigned* err,
                                                 int tid, int nthr) {
  const int per = (nslots + nthr - 1) / nthr;     // slots per thread for a single pass
  if (per <= 1) gather_level<1>(zs, slot_term, src, nslots, GKl, G, Kmax, tag, err, tid, nthr);
  else if (per <= 2) gather_level<2>(zs, slot_term, src, nslots, GKl, G, Kmax, tag, err, tid, nthr);
  else if (per <= 3) gather_level<3>(zs, slot_term, src, nslots, GKl, G, Kmax, tag, err, tid, nthr);
  else if (per <= 5) gather_level<5>(zs, slot_term, src, nslots, GKl, G, Kmax, tag, err, tid, nthr);
  else gather_level<8>(zs, slot_term, src, nslots, GKl, G, Kmax, tag, err, tid, nthr);
}

// z gather of every (level, sequence) pair at once: word i of the LB x nslots
// exchange words belongs to pair lb = i / nslots, slot s = i % nslots, which
// carries term tau = slot_term[s]; it lands at zs[lb*GK + g*Kmax + n] (tau =
// n*G + g) when tau is inside the budget of the pair's level (lane l of vlev
// holds level l's budget; kcur >= 0 overrides it).  One polling pipeline for
// all pairs, the same two-generation polling as gather_level.
template <int NS>
__device__ void gather_every_pair(float* zs, const uint16_t* slot_term, const unsigned long long* src, int nslots,
                                  int LB, int B, int GK, int G, int Kmax, int vlev, int kcur, unsigned tag,
                                  unsigned* err, int tid, int nthr) {
  const int n = LB * nslots;
  for (int base = 0; base < n; base += nthr * NS) {
    const unsigned long long* sp[NS];
    int dst[NS];
    unsigned pending = 0;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int i = base + k * nthr + tid;
      const int lb = i < n ? i / nslots : 0, s = i < n ? i - lb * nslots : 0;
      const int lev = __shfl(vlev, lb / B, 64);
      const int GKl = G * (kcur >= 0 ? kcur : lev);
      const int tau = i < n ? (int)slot_term[s] : GKl;
      sp[k] = src + (i < n ? i : 0);
      dst[k] = lb * GK + ((G == 4) ? ((tau & 3) * Kmax + (tau >> 2)) : tau);
      if (tau < GKl) pending |= 1u << k;
    }
    if (!pending) continue;
    unsigned long long wa[NS], wb[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) wa[k] = load_tagged(sp[k]);
    __builtin_amdgcn_s_sleep(4);
#pragma unroll
    for (int k = 0; k < NS; ++k) wb[k] = load_tagged(sp[k]);
    unsigned spins = 0;
    while (true) {
#pragma unroll
      for (int k = 0; k < NS; ++k)
        if (((pending >> k) & 1u) && (unsigned)(wa[k] >> 32) == tag) {
          zs[dst[k]] = __uint_as_float((unsigned)wa[k]);
          pending &= ~(1u << k);
        }
      if (!pending) break;
#pragma unroll
      for (int k = 0; k < NS; ++k) wa[k] = load_tagged(sp[k]);
#pragma unroll
      for (int k = 0; k < NS; ++k)
        if (((pending >> k) & 1u) && (unsigned)(wb[k] >> 32) == tag) {
          zs[dst[k]] = __uint_as_float((unsigned)wb[k]);
          pending &= ~(1u << k);
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
          if ((pending >> k) & 1u) zs[dst[k]] = 0.0f;
        break;
      }
    }
  }
}

// z gather of one tile of one group's terms, n in [k0, k0 + kn) of group g,
// for every (level, sequence) pair of a one-level launch.  The K-tiled
// launch publishes z group-major (word g*Kmax + n of the pair's block of
// P*OM words), so a tile's words are contiguous from goff = g*Kmax + k0.
// The nthr gathering threads split into LB groups of tpp = nthr / LB, one
// per pair; thread t of pair lb's group takes words r = t + tpp*k (k < NS),
// whose z land at zt[lb*zpl + (r % S)*zrow + r / S]: phase-B lane sl's
// terms k0 + sl + S*e, e ascending, are consecutive (zrow = KT/S + 4, a
// multiple of 4 that spreads the lanes' 16-byte reads over the banks;
// zpl = S * zrow).  Every load is issued at once and
// only the words still missing are loaded again (after the first tile every
// word has usually arrived: one load round trip per tile).  Bounded like
// gather_level.
template <int NS>
__device__ void gather_tile(float* zt, const unsigned long long* src, size_t pstride, int LB, int goff, int kn, int lgS,
                            int zrow, unsigned tag, unsigned* err, int tid, int nthr) {
  const int tpp = nthr / LB, lb = tid / tpp, t = tid - lb * tpp;
  if (lb >= LB) return;
  const unsigned long long* sp = src + (size_t)lb * pstride + goff + t;
  float* zl = zt + (size_t)lb * (zrow << lgS);
  const int sm = (1 << lgS) - 1;
  unsigned pending = 0;
#pragma unroll
  for (int k = 0; k < NS; ++k)
    if (t + tpp * k < kn) pending |= 1u << k;
  unsigned spins = 0;
  while (pending) {
    unsigned long long w[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k)
      if ((pending >> k) & 1u) w[k] = load_tagged(sp + tpp * k);
#pragma unroll
    for (int k = 0; k < NS; ++k)
      if (((pending >> k) & 1u) && (unsigned)(w[k] >> 32) == tag) {
        const int r = t + tpp * k;
        zl[(r & sm) * zrow + (r >> lgS)] = __uint_as_float((unsigned)w[k]);
        pending &= ~(1u << k);
      }
    if (pending && (++spins & 255u) == 0u &&
        (spins >= kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
      __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
      for (int k = 0; k < NS; ++k)
        if ((pending >> k) & 1u) {
          const int r = t + tpp * k;
          zl[(r & sm) * zrow + (r >> lgS)] = 0.0f;
        }
      break;
    }
  }
}

// words per thread: the planner keeps a tile within kTileWords words per
// thread of a pair's group
__device__ __forceinline__ void gather_tile_any(float* zt, const unsigned long long* src, size_t pstride, int LB,
                                                int goff, int kn, int lgS, int zrow, unsigned tag, unsigned* err,
                                                int tid, int nthr) {
  const int tpp = nthr / LB;
  const int per = (kn + tpp - 1) / tpp;
  if (per <= 4) gather_tile<4>(zt, src, pstride, LB, goff, kn, lgS, zrow, tag, err, tid, nthr);
  else if (per <= 8) gather_tile<8>(zt, src, pstride, LB, goff, kn, lgS, zrow, tag, err, tid, nthr);
  else gather_tile<kTileWords>(zt, src, pstride, LB, goff, kn, lgS, zrow, tag, err, tid, nthr);
}

// LDS carve-up shared by the host planner and the kernel (byte offsets).
struct Layout {
  size_t zs, hs, ys, bs, cs, zown, hown, sig, pxb, zmap, hval, hidx, us, total;
};

__host__ __device__ inline size_t align16(size_t b) { return (b + 15) & ~(size_t)15; }

__host__ __device__ inline Layout layout_of(const RunArgs& a, int online) {
  Layout l;
  const size_t LB = (size_t)a.L * a.B;
  const size_t kmax = a.G > 0 ? (size_t)a.GK / a.G : 0;
  size_t o = 0;
  // z of one (level, seq), [g][Kmax]; a single workgroup keeps every pair's
  // (a K-tiled phase B holds one tile of every pair's z instead)
  const size_t zfl = ((a.P == 1 || a.allpairs) ? LB : 1) * (a.GK > 1 ? (size_t)a.GK : 1);
  const size_t ztl = a.ktile > 0 ? LB * (size_t)(a.ktile + 4 * a.lanes_b[0]) : 0;   // [pair][S][KT/S + 4]
  l.zs = o;     o = align16(o + 4 * (zfl > ztl ? zfl : ztl));
  // h_{t-1} per (level, seq); an online run receives K_t in one more slot
  l.hs = o;     o = align16(o + 4 * (LB * a.H + (online ? 1 : 0)));
  l.ys = o;     o = align16(o + 4 * 4 * (size_t)a.rows_per * ((a.allpairs || a.ktile > 0) ? LB : 1));   // y of the owned rows
  l.bs = o;     o = align16(o + 4 * 4 * (size_t)a.rows_per);          // bias of the owned rows
  l.cs = o;     o = align16(o + 4 * LB * a.rows_per);                 // c of the owned rows
  l.zown = o;   o = align16(o + 4 * LB * (size_t)a.owned_max);        // z of the owned terms
  l.hown = o;   o = align16(o + 4 * LB * a.rows_per);                 // new h of the owned rows
  l.sig = o;    o = align16(o + 4 * (size_t)a.owned_max);
  l.pxb = o;    // P_x of every timestep (px_all) or of this and the next one
  o = align16(o + 4 * (a.px_all ? (size_t)a.T : 2) * a.B * a.owned_max);
  l.zmap = o;   o = align16(o + 2 * (size_t)a.owned_max * a.P);        // exchange slot -> term
  l.hval = o;   o = align16(o + (a.vh_lds ? 4 * (size_t)a.owned_max * a.hcap : 0));
  l.hidx = o;   o = align16(o + (a.vh_lds ? 2 * (size_t)a.owned_max * a.hcap : 0));
  l.us = o;     o = align16(o + 4 * 4 * (size_t)a.rows_per * a.ustride);
  (void)kmax;
  l.total = o;
  return l;
}

}  // namespace

// HPL > 0: each phase-A lane keeps HPL h-part entries of its term in
// registers (requires <= 32 owned terms and hcap <= 16*HPL); 0: entries in
// LDS.  UPT > 0: each phase-B thread keeps UPT entries of each of OPT output
// rows in registers (requires one budget K for all levels, S*UPT >= K and
// 4*rows_per*S <= 512*OPT); 0: U rows in LDS (ustride > 0) or from global.
// ONLINE: one level whose budget is chosen per timestep (RunArgs::online);
// the fixed-budget kernels carry none of its code.
template <int HPL, int OPT, int UPT, bool ONLINE, bool AP, bool TILE>
__global__ void __launch_bounds__(kThreads) progressive_lstm_kernel(RunArgs a) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const Layout L = layout_of(a, ONLINE ? 1 : 0);
  const int P = gridDim.x, j = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int D = a.D, H = a.H, G = a.G, N = a.N, NZ = a.NZ, T = a.T, B = a.B;
  const int LB = a.L * B, GK = a.GK, RP = a.rows_per, OM = a.owned_max;
  const int Kmax = GK / G;
  const int r0 = j * RP;
  const int rc = max(0, min(RP, H - r0));               // hidden units owned here
  const int n_owned = (GK > j) ? (GK - j + P - 1) / P : 0;
  const int outs = 4 * rc;

  float* zs = reinterpret_cast<float*>(lds_raw + L.zs);
  float* hs = reinterpret_cast<float*>(lds_raw + L.hs);
  float* ys = reinterpret_cast<float*>(lds_raw + L.ys);
  float* bs = reinterpret_cast<float*>(lds_raw + L.bs);
  float* cs = reinterpret_cast<float*>(lds_raw + L.cs);
  float* zown = reinterpret_cast<float*>(lds_raw + L.zown);
  float* hown = reinterpret_cast<float*>(lds_raw + L.hown);
  float* sig = reinterpret_cast<float*>(lds_raw + L.sig);
  float* pxb = reinterpret_cast<float*>(lds_raw + L.pxb);
  uint16_t* zmap = reinterpret_cast<uint16_t*>(lds_raw + L.zmap);
  float* hval = reinterpret_cast<float*>(lds_raw + L.hval);
  uint16_t* hidx = reinterpret_cast<uint16_t*>(lds_raw + L.hidx);
  float* us = reinterpret_cast<float*>(lds_raw + L.us);

  // phase-A lane roles: 16 lanes per term, 4 terms per wave per pass
  const int sub = lane >> 4, sla = lane & 15;
  // per-level budget and phase-B lane count, level l in lane l of one
  // register each, read with v_readlane: opaque to the compiler, so that it
  // keeps them instead of reloading them from the kernel arguments (a scalar
  // memory round trip) in every pass over the (level, sequence) pairs
  int vlev = lane < kMaxLevels ? a.levels[lane] : 0;
  int vlanes = lane < kMaxLevels ? a.lanes_b[lane] : 1;
  asm volatile("" : "+v"(vlev), "+v"(vlanes));
  // phase-B thread roles (register path: one output row per S threads)
  const int S0 = a.lanes_b[0];
  const int ob = threadIdx.x / S0, slb = threadIdx.x % S0;

  // ---- prologue: owned slices into LDS / registers ----
  for (int i = threadIdx.x; i < n_owned; i += kThreads) sig[i] = a.sigma[j + i * P];
  for (int i = threadIdx.x; i < outs; i += kThreads) {
    const int q = i / rc, rr = i - q * rc;
    bs[q * RP + rr] = a.bias[q * H + r0 + rr];
  }
  for (int i = threadIdx.x; i < LB * H; i += kThreads) {
    const int b = (i / H) % B, r = i % H;
    hs[i] = a.h0 ? a.h0[(size_t)b * H + r] : 0.0f;
  }
  for (int i = threadIdx.x; i < LB * RP; i += kThreads) {
    const int lb = i / RP, rr = i % RP, b = lb % B;
    cs[i] = (a.c0 && rr < rc) ? a.c0[(size_t)b * H + r0 + rr] : 0.0f;
  }
  // P_x: every timestep if it fits, else timestep 0 (later ones are prefetched)
  const int px_steps = a.px_all ? T : 1;
  for (int i = threadIdx.x; i < px_steps * B * n_owned; i += kThreads) {
    const int tb = i / n_owned, io = i - tb * n_owned;
    pxb[tb * OM + io] = a.px[(size_t)(j + io * P) * (T * B) + tb];
  }
  // z of every pair held here start at zero: a level at K = 0 never writes
  // its z, and the register accumulation multiplies them by zero
  for (int i = threadIdx.x; i < ((P == 1 || a.allpairs) ? LB : 1) * GK; i += kThreads) zs[i] = 0.0f;
  // exchange slot s = j'*OM + i' carries term tau = j' + i'*P
  for (int sl = threadIdx.x; sl < P * OM; sl += kThreads) {
    const int jj = sl / OM, ii = sl - jj * OM;
    zmap[sl] = (uint16_t)(jj + ii * P);
  }
  float hv[HPL > 0 ? HPL : 1];
  int hi[HPL > 0 ? HPL : 1];
  const int ia = wave * 4 + sub;                          // register path: this lane's term
  if constexpr (HPL > 0) {
#pragma unroll
    for (int k = 0; k < HPL; ++k) { hv[k] = 0.0f; hi[k] = 0; }
    if (ia < n_owned) {
      const int tau = j + ia * P;
      const int e0 = a.nx[tau], cnt = NZ - e0;
      const size_t src = (size_t)tau * NZ + e0;
#pragma unroll
      for (int k = 0; k < HPL; ++k) {
        const int e = sla + 16 * k;
        if (e < cnt) {
          hv[k] = a.vval[src + e];
          hi[k] = (int)a.vidx[src + e] - D;
        }
      }
    }
  } else if (a.vh_lds) {
    const int tot = n_owned * a.hcap;
#pragma unroll 4
    for (int idx = threadIdx.x; idx < tot; idx += kThreads) {
      const int i = idx / a.hcap, e = idx - i * a.hcap;
      const int tau = j + i * P;
      const int e0 = a.nx[tau];
      const bool live = e < NZ - e0;
      const size_t src = (size_t)tau * NZ + e0 + e;
      hval[idx] = live ? a.vval[src] : 0.0f;
      hidx[idx] = live ? (uint16_t)(a.vidx[src] - D) : (uint16_t)0;
    }
  }
  // register path: output rows ob + o*(512/S0), o < OPT; for each, the
  // LDS offsets of its y slot and of its group's z, and UPT entries of u
  float uv[UPT > 0 ? OPT * UPT : 1];
  int yslot[OPT > 0 ? OPT : 1], zbase[OPT > 0 ? OPT : 1];
  if constexpr (UPT > 0) {
    const int stride_o = kThreads / S0;
#pragma unroll
    for (int o = 0; o < OPT; ++o) {
      const int ol = ob + o * stride_o;
      yslot[o] = -1;
      zbase[o] = 0;
#pragma unroll
      for (int k = 0; k < UPT; ++k) uv[o * UPT + k] = 0.0f;
      if (ol < outs) {
        const int q = ol / rc, rr = ol - q * rc;
        yslot[o] = q * RP + rr;
        zbase[o] = ((G == 4) ? q : 0) * Kmax;
        const float* urow = a.Ut + (size_t)(q * H + r0 + rr) * N;
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
          const int n = slb + S0 * k;
          if (n < Kmax) uv[o * UPT + k] = urow[n];
        }
      }
    }
  } else if (a.ustride) {
    const int tot = outs * Kmax;
#pragma unroll 4
    for (int idx = threadIdx.x; idx < tot; idx += kThreads) {
      const int row = idx / Kmax, n = idx - row * Kmax;
      const int q = row / rc, rr = row - q * rc;
      us[(size_t)(q * RP + rr) * a.ustride + n] = a.Ut[(size_t)(q * H + r0 + rr) * N + n];
    }
  }
  __syncthreads();

  // A single workgroup keeps z and h in LDS: nothing is exchanged.
  const bool local = (P == 1);
  // The last wave does every global store of the recurrence (exchange words
  // and h_out); the other waves do the gathers, so no wave waits on its own
  // stores before its loads.
  const bool publisher = wave == kWaves - 1;
  const int gthr = kThreads - 64;

  // stamps come from the publisher wave, which does the stores anyway
  const bool stamp = a.stamps && j == 0 && (int)threadIdx.x == kThreads - 64;
  if (stamp) {
    a.stamps[0] = wall_clock64();
    a.stamps[1] = clock64();
  }
  // online run: the same thread of workgroup 0 keeps the clock and chooses;
  // K_0 is the choice for one budget, the same in every workgroup
  const bool chooser = ONLINE && j == 0 && (int)threadIdx.x == kThreads - 64;
  unsigned long long t_begin = 0ull, t_decide = 0ull;
  // the part of a timestep after the chooser's decision (its h publication
  // and exchange), measured on the previous timestep: step t+1 starts that
  // long after the decision for it
  long long t_rest = 0;
  int kcur = 0;
  if constexpr (ONLINE) {
    kcur = a.sched ? a.sched[0] : online_pick(a, (long long)a.budget);
    if (chooser) {
      t_begin = wall_clock64();
      if (!a.sched) a.kt[0] = kcur;
    }
  }
  for (int t = 0; t < T; ++t) {
    const unsigned tag = a.tag_base | (unsigned)(t + 1);
    const float* pxc = pxb + (a.px_all ? t : (t & 1)) * B * OM;
    if (stamp) a.stamps[2 + 4 * t] = clock64();

    // ---- phase A: z = sigma * (P_x + prune(v)_h . h_{t-1}) for the owned terms ----
    for (int lb = 0; lb < LB; ++lb) {
      const int l = lb / B, b = lb % B;
      const int GKl = G * (ONLINE ? kcur : __builtin_amdgcn_readlane(vlev, l));
      const int nl = (GKl > j) ? (GKl - j + P - 1) / P : 0;
      const float* h = hs + lb * H;
      if constexpr (HPL > 0) {
        if (wave * 4 < nl) {
          float hg[HPL];
#pragma unroll
          for (int k = 0; k < HPL; ++k) hg[k] = h[hi[k]];
          float acc = 0.0f;
#pragma unroll
          for (int k = 0; k < HPL; ++k) acc += hv[k] * hg[k];
          acc = group_sum<16>(acc);
          if (sla == 0 && ia < nl) {
            const float z = sig[ia] * (pxc[b * OM + ia] + acc);
            const int tau = j + ia * P;
            if (local) zs[lb * GK + (tau % G) * Kmax + tau / G] = z;
            else zown[lb * OM + ia] = z;
          }
        }
      } else {
        for (int base = wave * 4; base < nl; base += kWaves * 4) {
          const int i = base + sub;
          float acc = 0.0f;
          if (i < nl) {
            const float* hvp = hval + i * a.hcap;
            const uint16_t* hip = hidx + i * a.hcap;
#pragma unroll 4
            for (int e = sla; e < a.hcap; e += 16) acc += hvp[e] * h[hip[e]];
          }
          acc = group_sum<16>(acc);
          if (sla == 0 && i < nl) {
            const float z = sig[i] * (pxc[b * OM + i] + acc);
            const int tau = j + i * P;
            if (local) zs[lb * GK + (tau % G) * Kmax + tau / G] = z;
            else zown[lb * OM + i] = z;
          }
        }
      }
    }
    lds_barrier();
    if (stamp) a.stamps[3 + 4 * t] = clock64();
    // P_x of the next timestep (when not all resident) travels while this
    // timestep's z are exchanged.  Its slot (t+1)&1 was last read by phase A
    // of timestep t-1; every branch below (K_t = 0 included) and a single
    // workgroup take it here, so timestep t+1 never reads a stale slot.
    if (!a.px_all && t + 1 < T && !publisher) {
      float* pxn = pxb + ((t + 1) & 1) * B * OM;
      for (int i = threadIdx.x; i < B * n_owned; i += gthr) {
        const int b = i / n_owned, io = i - b * n_owned;
        pxn[b * OM + io] = a.px[(size_t)(j + io * P) * (T * B) + (t + 1) * B + b];
      }
    }
    if (publisher && !local) {
      for (int lb = 0; lb < LB; ++lb) {
        const int GKl = G * (ONLINE ? kcur : __builtin_amdgcn_readlane(vlev, lb / B));
        const int nl = (GKl > j) ? (GKl - j + P - 1) / P : 0;
        for (int i = lane; i < nl; i += 64) {
          // slot j*OM + i, or (K-tiled phase B) word g*Kmax + n of term
          // tau = j + i*P = n*G + g: a tile's terms of one group are then
          // contiguous words
          const int tau = j + i * P;
          const size_t wd = TILE ? (size_t)(tau & 3) * Kmax + (tau >> 2) : (size_t)(j * OM + i);   // TILE: G = 4
          publish(a.zx + (size_t)lb * P * OM + wd, zown[lb * OM + i], tag);
        }
      }
    }

    // ---- phase B: y = b + sum_n z_n u_n for the owned rows, gates, c and h ----
    if ((ONLINE ? kcur == 0 : GK == 0) && rc > 0) {
      // every level at K = 0 (an online run: this timestep's K_t = 0): y is
      // the bias alone (the same values as 0 + b below), so all (level,
      // sequence) pairs take one pass and one barrier
      if (stamp) a.stamps[4 + 4 * t] = clock64();
      for (int i = threadIdx.x; i < LB * rc; i += kThreads) {
        const int lb = i / rc, rr = i - lb * rc;
        float c = cs[lb * RP + rr], hv2;
        cell_update(bs[0 * RP + rr], bs[1 * RP + rr], bs[2 * RP + rr], bs[3 * RP + rr], c, hv2);
        cs[lb * RP + rr] = c;
        hown[lb * RP + rr] = hv2;
        if (local) hs[lb * H + r0 + rr] = hv2;
      }
      lds_barrier();
    } else if (rc > 0) {
      if constexpr (AP) {
        // every pair at once: one gather of all their z, one accumulation
        // pass, one cell-update pass.
        // y of the owned rows of one pair: yl[q*RP + rr] = b + sum_{n<Kl} u z
        auto accumulate = [&](const float* zl, float* yl, int Kl, int l) {
          if constexpr (UPT > 0) {
            // branch-free: entries past the budget multiply a valid z by 0
#pragma unroll
            for (int o = 0; o < OPT; ++o) {
              // all z reads first (independent LDS loads in flight), then the FMAs
              float zv[UPT];
#pragma unroll
              for (int k = 0; k < UPT; ++k) {
                const int n = slb + S0 * k;
                zv[k] = zl[zbase[o] + (n < Kl ? n : 0)];
              }
              float acc = 0.0f;
#pragma unroll
              for (int k = 0; k < UPT; ++k) {
                const int n = slb + S0 * k;
                acc += (n < Kl ? uv[o * UPT + k] : 0.0f) * zv[k];
              }
              acc = group_sum_rt(acc, S0);
              if (yslot[o] >= 0 && slb == 0) yl[yslot[o]] = acc + bs[yslot[o]];
            }
          } else {
            // S is a power of two (1 .. 16)
            const int S = __builtin_amdgcn_readlane(vlanes, l), lgS = 31 - __builtin_clz(S);
            const int OPP = kThreads >> lgS, os = (int)threadIdx.x >> lgS, sl = (int)threadIdx.x & (S - 1);
            for (int base = 0; base < outs; base += OPP) {
              const int ol = base + os;
              float acc = 0.0f;
              int q = 0, rr = 0;
              if (ol < outs) {
                q = ol / rc;
                rr = ol - q * rc;
                const float* zg = zl + ((G == 4) ? q : 0) * Kmax;
                if (a.ustride) {
                  const float* urow = us + (size_t)(q * RP + rr) * a.ustride;
#pragma unroll 8
                  for (int n = sl; n < Kl; n += S) acc += urow[n] * zg[n];
                } else {
                  const float* urow = a.Ut + (size_t)(q * H + r0 + rr) * N;
#pragma unroll 8
                  for (int n = sl; n < Kl; n += S) acc += urow[n] * zg[n];
                }
              }
              acc = group_sum_rt(acc, S);
              if (sl == 0 && ol < outs) yl[q * RP + rr] = acc + bs[q * RP + rr];
            }
          }
        };
        // gates and the c/h update of owned unit rr of pair lb
        auto cell = [&](const float* yl, int lb, int rr) {
          float c = cs[lb * RP + rr], hv2;
          cell_update(yl[0 * RP + rr], yl[1 * RP + rr], yl[2 * RP + rr], yl[3 * RP + rr], c, hv2);
          cs[lb * RP + rr] = c;
          hown[lb * RP + rr] = hv2;
          if (local) hs[lb * H + r0 + rr] = hv2;
        };
        if (!local && !publisher) {
          const int nslots = P * OM, n = LB * nslots, per = (n + gthr - 1) / gthr;
          const int kc = ONLINE ? kcur : -1;
          if (per <= 1)
            gather_every_pair<1>(zs, zmap, a.zx, nslots, LB, B, GK, G, Kmax, vlev, kc, tag, a.err, threadIdx.x, gthr);
          else if (per <= 2)
            gather_every_pair<2>(zs, zmap, a.zx, nslots, LB, B, GK, G, Kmax, vlev, kc, tag, a.err, threadIdx.x, gthr);
          else if (per <= 3)
            gather_every_pair<3>(zs, zmap, a.zx, nslots, LB, B, GK, G, Kmax, vlev, kc, tag, a.err, threadIdx.x, gthr);
          else if (per <= 5)
            gather_every_pair<5>(zs, zmap, a.zx, nslots, LB, B, GK, G, Kmax, vlev, kc, tag, a.err, threadIdx.x, gthr);
          else
            gather_every_pair<8>(zs, zmap, a.zx, nslots, LB, B, GK, G, Kmax, vlev, kc, tag, a.err, threadIdx.x, gthr);
        }
        lds_barrier();
        if (stamp) a.stamps[4 + 4 * t] = clock64();
        for (int lb = 0; lb < LB; ++lb)
          accumulate(zs + lb * GK, ys + lb * 4 * RP, ONLINE ? kcur : __builtin_amdgcn_readlane(vlev, lb / B), lb / B);
        lds_barrier();
        for (int i = threadIdx.x; i < LB * rc; i += kThreads) {
          const int lb = i / rc, rr = i - lb * rc;
          cell(ys + lb * 4 * RP, lb, rr);
        }
        lds_barrier();
      } else {
        if constexpr (TILE) {
          {
            // One level over several sequences, U read from memory, G = 4,
            // P a multiple of 4.  Workgroup j keeps the cell update of its
            // units [r0, r0 + rc) but accumulates the rows of gate gq = j % 4
            // for the 4*RP units of its block (workgroups 4*(j/4) .. +3,
            // whose cell units those are): it needs only group gq's z.  Each
            // lane reads each of its U entries once per timestep and applies
            // it to every sequence (one accumulator per sequence), K in tiles
            // of KT terms whose group-gq z of every sequence are gathered
            // into LDS (zs[lb*KT + n - k0]).  y = sum + bias goes to the cell
            // owners as tagged words (y words after the pairs' z blocks:
            // [lb][gate][H]).  Per (row, sequence) the sums run in the
            // per-pair pass's order (entries sl, sl + S, ... ascending, then
            // the S-lane reduction, then the bias).
            const int KT = a.ktile;
            const int Kl = ONLINE ? kcur : __builtin_amdgcn_readlane(vlev, 0);
            const int S = __builtin_amdgcn_readlane(vlanes, 0), lgS = 31 - __builtin_clz(S);
            const int os = (int)threadIdx.x >> lgS, sl = (int)threadIdx.x & (S - 1);
            const int gq = j & 3;
            const int ub0 = (j >> 2) * 4 * RP;                 // first unit of the block
            const int zrow = (KT >> lgS) + 4, zpl = zrow << lgS;   // LDS row of a lane, block of a pair
            unsigned long long* yx = a.zx + (size_t)LB * P * OM;
            // one output row per thread (the planner's condition): gate gq,
            // unit ub0 + os
            float acc[kTilePairs];
            const int u = ub0 + os;
            const bool rv = os < 4 * RP && u < H;
            const float* urow = a.Ut + (size_t)(gq * H + (rv ? u : 0)) * N;
            const float brow = rv ? a.bias[gq * H + u] : 0.0f;
#pragma unroll
            for (int lb = 0; lb < kTilePairs; ++lb) acc[lb] = 0.0f;
            for (int k0 = 0; k0 < Kl; k0 += KT) {
              const int kn = min(KT, Kl - k0);
              // the lane's U entries of the tile (KT <= kTileEntries * S), in
              // registers before the gather so that their latency overlaps it
              float ut[kTileEntries];
              if (rv) {
#pragma unroll
                for (int e = 0; e < kTileEntries; ++e) ut[e] = urow[min(k0 + sl + S * e, Kl - 1)];
              }
              if (k0 > 0) lds_barrier();   // every read of the previous tile is done
              if (!publisher)
                gather_tile_any(zs, a.zx, (size_t)P * OM, LB, gq * Kmax + k0, kn, lgS, zrow, tag, a.err,
                                threadIdx.x, gthr);
              lds_barrier();
              if (stamp && k0 == 0) a.stamps[4 + 4 * t] = clock64();
              if (rv) {
                // lane sl's z of the tile: zs[lb*zpl + sl*zrow + e], e ascending
                const float* zl = zs + sl * zrow;
#pragma unroll
                for (int e4 = 0; e4 < kTileEntries / 4; ++e4) {
                  if (4 * e4 >= (KT >> lgS)) break;   // the lane's row holds KT / S values
#pragma unroll
                  for (int lb = 0; lb < kTilePairs; ++lb) {
                    if (lb >= LB) break;
                    const float4 z4 = *reinterpret_cast<const float4*>(zl + lb * zpl + 4 * e4);
                    const int e = 4 * e4;
                    if (sl + S * e < kn) acc[lb] += ut[e] * z4.x;
                    if (sl + S * (e + 1) < kn) acc[lb] += ut[e + 1] * z4.y;
                    if (sl + S * (e + 2) < kn) acc[lb] += ut[e + 2] * z4.z;
                    if (sl + S * (e + 3) < kn) acc[lb] += ut[e + 3] * z4.w;
                  }
                }
              }
            }
#pragma unroll
            for (int lb = 0; lb < kTilePairs; ++lb)
              if (lb < LB) {
                const float v = group_sum_rt(acc[lb], S);
                if (sl == 0 && rv) publish(yx + ((size_t)lb * 4 + gq) * H + u, v + brow, tag);
              }
            // the owned units' four gate rows from the block's workgroups
            // (bounded polls), then the cell update
            for (int i = threadIdx.x; i < LB * rc; i += kThreads) {
              const int lb = i / rc, rr = i - lb * rc;
              const unsigned long long* yw = yx + (size_t)lb * 4 * H + r0 + rr;
              float yv[4] = {0.f, 0.f, 0.f, 0.f};
              unsigned pending = 0xFu, spins = 0;
              while (pending) {
                unsigned long long w4[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                  if ((pending >> q) & 1u) w4[q] = load_tagged(yw + (size_t)q * H);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                  if (((pending >> q) & 1u) && (unsigned)(w4[q] >> 32) == tag) {
                    yv[q] = __uint_as_float((unsigned)w4[q]);
                    pending &= ~(1u << q);
                  }
                if (pending && (++spins & 255u) == 0u &&
                    (spins >= kSpinLimit ||
                     __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
                  __hip_atomic_fetch_or(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                  pending = 0;
                }
              }
              float c = cs[lb * RP + rr], hv2;
              cell_update(yv[0], yv[1], yv[2], yv[3], c, hv2);
              cs[lb * RP + rr] = c;
              hown[lb * RP + rr] = hv2;
            }
            lds_barrier();
          }
        } else {
          for (int lb = 0; lb < LB; ++lb) {
            const int l = lb / B;
            const int Kl = ONLINE ? kcur : __builtin_amdgcn_readlane(vlev, l);
            if (!local && !publisher) {
              // every slot of the exchange whose term is in this level (slots of
              // workgroups that own fewer terms are skipped by the map check)
              const int nslots = P * OM;
              const int GKl = G * Kl;
              gather_level_any(zs, zmap, a.zx + (size_t)lb * P * OM, nslots, GKl, G, Kmax, tag, a.err, threadIdx.x, gthr);
            }
            lds_barrier();
            if (stamp && lb == 0) a.stamps[4 + 4 * t] = clock64();
            const float* zl = zs + (local ? lb * GK : 0);
            if constexpr (UPT > 0) {
              // branch-free: entries past the budget multiply a valid z by 0
  #pragma unroll
              for (int o = 0; o < OPT; ++o) {
                // all z reads first (independent LDS loads in flight), then the FMAs
                float zv[UPT];
  #pragma unroll
                for (int k = 0; k < UPT; ++k) {
                  const int n = slb + S0 * k;
                  zv[k] = zl[zbase[o] + (n < Kl ? n : 0)];
                }
                float acc = 0.0f;
  #pragma unroll
                for (int k = 0; k < UPT; ++k) {
                  const int n = slb + S0 * k;
                  acc += (n < Kl ? uv[o * UPT + k] : 0.0f) * zv[k];
                }
                acc = group_sum_rt(acc, S0);
                if (yslot[o] >= 0 && slb == 0) ys[yslot[o]] = acc + bs[yslot[o]];
              }
            } else {
              // S is a power of two (1 .. 16)
              const int S = __builtin_amdgcn_readlane(vlanes, l), lgS = 31 - __builtin_clz(S);
              const int OPP = kThreads >> lgS, os = (int)threadIdx.x >> lgS, sl = (int)threadIdx.x & (S - 1);
              for (int base = 0; base < outs; base += OPP) {
                const int ol = base + os;
                float acc = 0.0f;
                int q = 0, rr = 0;
                if (ol < outs) {
                  q = ol / rc;
                  rr = ol - q * rc;
                  const float* zg = zl + ((G == 4) ? q : 0) * Kmax;
                  if (a.ustride) {
                    const float* urow = us + (size_t)(q * RP + rr) * a.ustride;
  #pragma unroll 8
                    for (int n = sl; n < Kl; n += S) acc += urow[n] * zg[n];
                  } else {
                    const float* urow = a.Ut + (size_t)(q * H + r0 + rr) * N;
  #pragma unroll 8
                    for (int n = sl; n < Kl; n += S) acc += urow[n] * zg[n];
                  }
                }
                acc = group_sum_rt(acc, S);
                if (sl == 0 && ol < outs) ys[q * RP + rr] = acc + bs[q * RP + rr];
              }
            }
            lds_barrier();
            for (int rr = threadIdx.x; rr < rc; rr += kThreads) {
              float c = cs[lb * RP + rr], hv2;
              cell_update(ys[0 * RP + rr], ys[1 * RP + rr], ys[2 * RP + rr], ys[3 * RP + rr], c, hv2);
              cs[lb * RP + rr] = c;
              hown[lb * RP + rr] = hv2;
              if (local) hs[lb * H + r0 + rr] = hv2;
            }
            lds_barrier();
          }

        }
      }
    }
    if (stamp) a.stamps[5 + 4 * t] = clock64();
    // without terms (every level K = 0) no workgroup reads another's h
    const bool exch = !local && GK > 0;
    // h_t (and an online run's K_{t+1}) travel in the half of the exchange
    // selected by step parity, tagged words and bulk alike
    float* hbt = a.bulk_h ? a.hbx + (size_t)(t & 1) * a.hb_stride : nullptr;
    unsigned long long* hxt = a.hx + (size_t)(t & 1) * a.hb_stride;
    if (ONLINE && chooser && t + 1 < T) {
      // K_{t+1}: timestep t+1 must end by (t+2) * budget after the start
      // time banked by the end of step t (negative: behind the schedule);
      // a surplus is spread evenly over the remaining steps (even budgets
      // rather than a large K after a K = 0), a deficit recovered at once,
      // so step t+1 still ends by (t+2) * budget
      t_decide = wall_clock64();
      const long long used = (long long)(t_decide - t_begin);
      const long long banked = (long long)(t + 1) * (long long)a.budget - used - t_rest;
      const long long share = banked > 0 ? banked / (long long)(T - t - 1) : banked;
      const int knext = a.sched ? a.sched[t + 1] : online_pick(a, (long long)a.budget + share);
      if (!a.sched) a.kt[t + 1] = knext;
      const float kbits = __int_as_float(knext);
      if (local) hs[LB * H] = kbits;
      else if (a.bulk_h) store_coherent(hbt + (size_t)LB * H, kbits);
      else publish(hxt + (size_t)LB * H, kbits, tag);
    }
    if (publisher) {
      for (int lb = 0; lb < LB; ++lb) {
        const int l = lb / B, b = lb % B;
        for (int rr = lane; rr < rc; rr += 64) {
          const float h2 = hown[lb * RP + rr];
          const int r = r0 + rr;
          a.h_out[(((size_t)l * T + t) * B + b) * H + r] = h2;
          if (exch) {
            if (a.bulk_h) store_coherent(hbt + (size_t)lb * H + r, h2);
            else publish(hxt + (size_t)lb * H + r, h2, tag);
          }
        }
      }
      if (exch && a.bulk_h) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's h stores acknowledged
        if (lane == 0) __hip_atomic_store(a.hflag + j, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }

    // ---- phase C: gather h_t (and K_{t+1} of an online run) ----
    const int online_word = (ONLINE && t + 1 < T) ? 1 : 0;
    if (exch) {
      if (a.bulk_h) {
        // h_t is double-buffered by step parity.  A workgroup publishes
        // h_{t+2} (into this half again) only after it has gathered h_{t+1}
        // from every workgroup, and each publishes h_{t+1} only after
        // reading h_t: so no half is overwritten while it is still read,
        // even at online timesteps with K_t = 0, which exchange no z.  A
        // flag may then already carry tag t+2 (its owner one step ahead,
        // writing the other half), which await_flags accepts.
        if (!publisher) await_flags(a.hflag, P, tag, a.err, threadIdx.x, gthr);
        lds_barrier();
        if (!publisher) read_coherent(hs, hbt, LB * H + online_word, threadIdx.x, gthr);
      } else if (!publisher) {
        gather_tagged<2>(hs, nullptr, hxt, LB * H + online_word, tag, a.err, threadIdx.x, gthr);
      }
    }
    lds_barrier();
    if (ONLINE && t + 1 < T) kcur = __float_as_int(hs[LB * H]);
    if (ONLINE && chooser && t + 1 < T) t_rest = (long long)(wall_clock64() - t_decide);
  }
  if (stamp) {
    a.stamps[2 + 4 * T] = clock64();
    a.stamps[3 + 4 * T] = wall_clock64();
  }

  if (a.c_out) {
    for (int i = threadIdx.x; i < LB * rc; i += kThreads) {
      const int lb = i / rc, rr = i % rc;
      a.c_out[(size_t)lb * H + r0 + rr] = cs[lb * RP + rr];
    }
  }
}

// x-part projections P_x[tau][t*B+b] = prune(v_tau)[k<D] . x_t[b] for every
// term in use and every (t, b).  They do not depend on h, so they are taken
// off the recurrence (the x part holds most of each term's non-zeros) and
// spread over the GPU: each wave takes one term and each workgroup stages a
// chunk of x transposed in LDS, xt[k][c] with a padded
// row of xrow floats, so that one entry's values for every (t, b) of the
// chunk are adjacent.  The term's entries are read once from HBM.  The
// chunks are dealt over gridDim.y workgroups per term group, so that few
// terms with long sequences (or wide x, hence small chunks) still fill the
// device.  XC is the widest chunk: xchunk == XC with 16-byte x rows takes
// the vector path (xrow a multiple of 4), anything else the scalar one.  The
// per-(t, b) sums run in the same order at every XC.
// PT terms per wave (consecutive terms of the workgroup's PT*8): with many
// terms, several share each staged chunk of x.
template <int XC, int PT>
__global__ void __launch_bounds__(kThreads) input_proj_kernel(RunArgs a, int xchunk, int xrow) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  float* xt = reinterpret_cast<float*>(lds_raw);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int TB = a.T * a.B, D = a.D, NZ = a.NZ;
  // the wave's term's first 64*kProjEntries x-part entries sit in registers,
  // loaded (unconditionally, masked afterwards) before x is staged so that
  // their HBM latency overlaps the staging
  constexpr int kProjTerms = PT, kProjEntries = 16 / PT;
  int ne[kProjTerms];
  float ev[kProjTerms][kProjEntries];
  int ek[kProjTerms][kProjEntries];
#pragma unroll
  for (int w = 0; w < kProjTerms; ++w) {
    const int tau = (blockIdx.x * kWaves + wave) * kProjTerms + w;
    const int tc = tau < a.GK ? tau : 0;
    const uint16_t* vi = a.vidx + (size_t)tc * NZ;
    const float* vv = a.vval + (size_t)tc * NZ;
#pragma unroll
    for (int q = 0; q < kProjEntries; ++q) {
      const int e = min(lane + 64 * q, NZ - 1);
      ev[w][q] = vv[e];
      ek[w][q] = vi[e];
    }
    ne[w] = tau < a.GK ? (int)a.nx[tau] : 0;
  }
#pragma unroll
  for (int w = 0; w < kProjTerms; ++w)
#pragma unroll
    for (int q = 0; q < kProjEntries; ++q)
      if (lane + 64 * q >= ne[w]) {
        ev[w][q] = 0.0f;
        ek[w][q] = 0;
      }
  for (int cb = blockIdx.y * xchunk; cb < TB; cb += gridDim.y * xchunk) {
    const int cnt = min(xchunk, TB - cb);
    __syncthreads();
    if (a.xvec && xchunk == XC) {
      // lane (c, k4) loads x[cb+c][4k4 .. 4k4+3] and writes it down column c
      const int n = XC * (D >> 2);
      constexpr int kStage = 8;                            // float4 loads in flight per thread
      for (int base = 0; base < n; base += kThreads * kStage) {
        float4 v[kStage];
#pragma unroll
        for (int u = 0; u < kStage; ++u) {
          const int i = base + u * kThreads + (int)threadIdx.x;
          const int c = i % XC, k4 = i / XC;
          v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (i < n && c < cnt) v[u] = reinterpret_cast<const float4*>(a.x + (size_t)(cb + c) * D)[k4];
        }
#pragma unroll
        for (int u = 0; u < kStage; ++u) {
          const int i = base + u * kThreads + (int)threadIdx.x;
          if (i < n) {
            const int c = i % XC, k4 = i / XC;
            float* d = xt + (4 * k4) * xrow + c;
            d[0] = v[u].x;
            d[xrow] = v[u].y;
            d[2 * xrow] = v[u].z;
            d[3 * xrow] = v[u].w;
          }
        }
      }
    } else {
      for (int c = 0; c < xchunk; ++c)
        for (int k = threadIdx.x; k < D; k += kThreads)
          xt[k * xrow + c] = c < cnt ? a.x[(size_t)(cb + c) * D + k] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kProjTerms; ++w) {
      const int tau = (blockIdx.x * kWaves + wave) * kProjTerms + w;
      if (tau >= a.GK) break;
      const uint16_t* vi = a.vidx + (size_t)tau * NZ;
      const float* vv = a.vval + (size_t)tau * NZ;
      float acc[XC];
#pragma unroll
      for (int c = 0; c < XC; ++c) acc[c] = 0.0f;
      if ((xrow & 3) == 0 && xchunk == XC) {
#pragma unroll
        for (int q = 0; q < kProjEntries; ++q) {
          if (64 * q < ne[w]) {
            const float v = ev[w][q];
            const float4* xk = reinterpret_cast<const float4*>(xt + ek[w][q] * xrow);
#pragma unroll
            for (int r = 0; r < XC / 4; ++r) {
              const float4 x4 = xk[r];
              acc[4 * r + 0] += v * x4.x;
              acc[4 * r + 1] += v * x4.y;
              acc[4 * r + 2] += v * x4.z;
              acc[4 * r + 3] += v * x4.w;
            }
          }
        }
        for (int e = lane + 64 * kProjEntries; e < ne[w]; e += 64) {
          const float v = vv[e];
          const float4* xk = reinterpret_cast<const float4*>(xt + (int)vi[e] * xrow);
#pragma unroll
          for (int r = 0; r < XC / 4; ++r) {
            const float4 x4 = xk[r];
            acc[4 * r + 0] += v * x4.x;
            acc[4 * r + 1] += v * x4.y;
            acc[4 * r + 2] += v * x4.z;
            acc[4 * r + 3] += v * x4.w;
          }
        }
      } else {
#pragma unroll
        for (int q = 0; q < kProjEntries; ++q) {
          if (64 * q < ne[w]) {
            const float v = ev[w][q];
            const float* xk = xt + ek[w][q] * xrow;
#pragma unroll
            for (int c = 0; c < XC; ++c)
              if (c < xchunk) acc[c] += v * xk[c];
          }
        }
        for (int e = lane + 64 * kProjEntries; e < ne[w]; e += 64) {
          const float v = vv[e];
          const float* xk = xt + (int)vi[e] * xrow;
#pragma unroll
          for (int c = 0; c < XC; ++c)
            if (c < xchunk) acc[c] += v * xk[c];
        }
      }
#pragma unroll
      for (int c = 0; c < XC; ++c) {
        if (c < cnt) {
          const float s = wave_sum(acc[c]);
          if (lane == 0) a.px[(size_t)tau * TB + cb + c] = s;
        }
      }
    }
  }
}

__global__ void clear_u64_kernel(unsigned long long* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0ull;
}

int lanes_for_terms(int nz, int D, int H) {
  (void)nz; (void)D; (void)H;
  return 16;   // phase A always reduces over 16 lanes per term
}

int lanes_for_level(int K) {
  // about 32 terms per lane, at most 16 lanes per output row
  int s = 1;
  while (s < 16 && 32 * s < K) s <<= 1;
  return s;
}

size_t plan_progressive(RunArgs& a, int P) {
  a.rows_per = (a.H + P - 1) / P;
  a.owned_max = a.GK > 0 ? (a.GK + P - 1) / P : 0;
  a.lanes_a = 16;
  int smax = 1;
  bool same_s = true;
  for (int l = 0; l < a.L; ++l) {
    smax = std::max(smax, a.lanes_b[l]);
    same_s = same_s && a.lanes_b[l] == a.lanes_b[0];
  }
  const int Kmax = a.G > 0 ? a.GK / a.G : 0;
  // register residency (no LDS needed for those slices)
  a.hpl = 0;
  if (a.owned_max <= 4 * kWaves) {
    const int need = (a.hcap + 15) / 16;
    for (int c : {4, 8, 12, 16, 24, 32})
      if (need <= c) { a.hpl = c; break; }
  }
  a.upt = 0;
  a.opt = 0;
  bool same_k = true;
  for (int l = 0; l < a.L; ++l) same_k = same_k && a.levels[l] == a.levels[0];
  if (same_k && same_s && Kmax > 0) {
    const int S = a.lanes_b[0];
    const int need_u = (Kmax + S - 1) / S;
    const int need_o = (4 * a.rows_per * S + kThreads - 1) / kThreads;
    if (need_o <= 1 && need_u <= 32) { a.opt = 1; a.upt = 32; }
    else if (need_o <= 1 && need_u <= 64) { a.opt = 1; a.upt = 64; }
    else if (need_o <= 2 && need_u <= 16) { a.opt = 2; a.upt = 16; }
    else if (need_o <= 4 && need_u <= 8) { a.opt = 4; a.upt = 8; }
    if (a.opt == 1 && need_u <= 8) a.upt = 8;
    else if (a.opt == 1 && need_u <= 16) a.upt = 16;
    // 64 U entries per thread only next to at most 8 h-part entries per
    // lane: beyond that the register file (256 per lane) spills
    if (a.upt == 64 && a.hpl > 8) { a.opt = 0; a.upt = 0; }
    // online runs are built for one output row per thread and up to 32 U
    // entries in registers only, 32 of them next to at most 12 h-part
    // entries per lane (more spills)
    if (a.online && (a.opt != 1 || a.upt > 32 || (a.upt == 32 && a.hpl > 12))) { a.opt = 0; a.upt = 0; }
  }
  a.P = P;
  a.vh_lds = 0;
  a.ustride = 0;
  a.px_all = 0;
  // several (level, sequence) pairs: one phase-B pass for all of them when
  // their z fit in LDS next to everything else
  a.allpairs = (a.L * a.B > 1 && a.GK > 0) ? 1 : 0;
  if (a.allpairs && layout_of(a, a.online).total > kLdsCap) a.allpairs = 0;
  size_t need = layout_of(a, a.online).total;
  if (need > kLdsCap) return need;
  if (a.hpl == 0) {
    a.vh_lds = 1;
    if (layout_of(a, a.online).total > kLdsCap) return layout_of(a, a.online).total;   // h-part entries must fit
  }
  if (a.upt == 0 && Kmax > 0) {
    // stride = smax * odd: the lanes of consecutive rows hit distinct banks
    a.ustride = smax * ((((Kmax + smax - 1) / smax)) | 1);
    if (layout_of(a, a.online).total > kLdsCap) a.ustride = 0;
  }
  // one level over several sequences with U read from memory: phase B reads
  // each U entry once per timestep for every sequence, K in the largest tile
  // (a multiple of 16 lanes, at most 1024 terms) whose z of every pair fit
  a.ktile = 0;
  if (a.upt == 0 && a.ustride == 0 && !a.allpairs && a.L == 1 && a.B > 1 && a.B <= kTilePairs && a.G == 4 &&
      P > 1 && P % 4 == 0 && Kmax > 0 && 4 * a.rows_per <= kThreads / a.lanes_b[0]) {
    // at most kTileEntries U entries per lane and row in a tile, and at
    // most kTileWords z words per gathering thread (448 of them)
    // (KT a multiple of 4 S: a lane's terms of a tile are read as 16-byte vectors)
    const int s4 = 4 * a.lanes_b[0];
    int ktmax = std::min(kTileEntries * a.lanes_b[0], (Kmax + s4 - 1) / s4 * s4);
    while (ktmax > s4 && ktmax > kTileWords * ((kThreads - 64) / a.B)) ktmax = ktmax / (2 * s4) * s4;
    for (int kt = ktmax; kt >= s4; kt = kt / (2 * s4) * s4) {
      a.ktile = kt;
      if (layout_of(a, a.online).total <= kLdsCap) break;
      a.ktile = 0;
    }
  }
  a.px_all = 1;
  if (layout_of(a, a.online).total > kLdsCap) a.px_all = 0;
  return layout_of(a, a.online).total;
}

template <int HPL, int OPT, int UPT, bool ONLINE, bool AP, bool TILE = false>
hipError_t launch_kernel(const RunArgs& a, int blocks, int cooperative, size_t lds, hipStream_t stream) {
  static bool attr_set = false;
  const void* fn = (const void*)progressive_lstm_kernel<HPL, OPT, UPT, ONLINE, AP, TILE>;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsCap);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  if (cooperative) {
    RunArgs copy = a;
    void* args[] = {&copy};
    return hipLaunchCooperativeKernel(fn, dim3(blocks), dim3(kThreads), args, (unsigned)lds, stream);
  }
  progressive_lstm_kernel<HPL, OPT, UPT, ONLINE, AP, TILE><<<dim3(blocks), dim3(kThreads), lds, stream>>>(a);
  return hipGetLastError();
}

// The all-pairs and the K-tiled phase B are compiled only into the
// instances that launches with several (level, sequence) pairs use: they
// cost the others registers.
template <int HPL, int OPT, int UPT, bool ONLINE = false>
hipError_t launch_one(const RunArgs& a, int blocks, int cooperative, size_t lds, hipStream_t stream) {
  if (a.allpairs) return launch_kernel<HPL, OPT, UPT, ONLINE, true>(a, blocks, cooperative, lds, stream);
  if constexpr (UPT == 0)
    if (a.ktile > 0) return launch_kernel<HPL, OPT, UPT, ONLINE, false, true>(a, blocks, cooperative, lds, stream);
  return launch_kernel<HPL, OPT, UPT, ONLINE, false>(a, blocks, cooperative, lds, stream);
}

template <int HPL>
hipError_t launch_u(const RunArgs& a, int blocks, int cooperative, size_t lds, hipStream_t stream) {
  if (a.online) {   // the planner keeps online runs to these shapes
    if (a.opt == 1 && a.upt == 8) return launch_one<HPL, 1, 8, true>(a, blocks, cooperative, lds, stream);
    if (a.opt == 1 && a.upt == 16) return launch_one<HPL, 1, 16, true>(a, blocks, cooperative, lds, stream);
    if constexpr (HPL <= 12)
      if (a.opt == 1 && a.upt == 32) return launch_one<HPL, 1, 32, true>(a, blocks, cooperative, lds, stream);
    return launch_one<HPL, 1, 0, true>(a, blocks, cooperative, lds, stream);
  }
  if (a.opt == 1 && a.upt == 8) return launch_one<HPL, 1, 8>(a, blocks, cooperative, lds, stream);
  if (a.opt == 1 && a.upt == 16) return launch_one<HPL, 1, 16>(a, blocks, cooperative, lds, stream);
  if (a.opt == 1 && a.upt == 32) return launch_one<HPL, 1, 32>(a, blocks, cooperative, lds, stream);
  if constexpr (HPL <= 8)
    if (a.opt == 1 && a.upt == 64) return launch_one<HPL, 1, 64>(a, blocks, cooperative, lds, stream);
  if (a.opt == 2) return launch_one<HPL, 2, 16>(a, blocks, cooperative, lds, stream);
  if (a.opt == 4) return launch_one<HPL, 4, 8>(a, blocks, cooperative, lds, stream);
  return launch_one<HPL, 1, 0>(a, blocks, cooperative, lds, stream);
}

template <int XC, int PT = 1>
hipError_t launch_input_proj_xc(const RunArgs& a, int gx, int gy, int xchunk, int xrow, size_t plds,
                                hipStream_t stream) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)input_proj_kernel<XC, PT>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsCap);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  input_proj_kernel<XC, PT><<<dim3(gx, gy), dim3(kThreads), plds, stream>>>(a, xchunk, xrow);
  return hipGetLastError();
}

hipError_t launch_input_proj(const RunArgs& a, hipStream_t stream) {
  if (a.GK <= 0) return hipSuccess;
  const int TB = a.T * a.B;
  const int gx = (a.GK + kWaves - 1) / kWaves;   // one term per wave
  // few terms over a short sequence: chunks of 4 (t, b) pairs, each its own
  // workgroup, so that the staging latency is spread over more workgroups
  // (driving shape, T = 16, up to 512 terms: 6 us against 11 with one
  // workgroup per term group); otherwise chunks of 16
  const int c4 = (TB + 3) / 4;
  if ((size_t)a.D * 4 * 4 <= kLdsCap && (long long)gx * c4 <= (long long)std::max(1, a.num_cu))
    return launch_input_proj_xc<4>(a, gx, c4, 4, 4, (size_t)a.D * 4 * 4, stream);
  // full chunks of 16 (t, b) pairs use a 16-byte aligned row of 20 floats
  // (a wave's 64 writes of one component land in distinct banks); x too
  // wide for that takes the largest smaller chunk that fits, with an odd row
  // (the lanes' rows then fall in different banks)
  int xchunk = kMaxXChunk, xrow = kMaxXChunk + 4;
  if ((size_t)a.D * xrow * 4 > kLdsCap) {
    xchunk = kMaxXChunk - 1;
    while (xchunk > 1 && (size_t)a.D * (xchunk | 1) * 4 > kLdsCap) --xchunk;
    xrow = xchunk | 1;
  }
  const size_t plds = (size_t)a.D * xrow * 4;
  // terms enough for every compute unit at 4 terms per wave: each staged
  // chunk of x then serves 32 terms instead of 8 (deadline shape, 8192
  // terms over 32 chunks: the staging was 4 GB over the device)
  if (gx >= 4 * std::max(1, a.num_cu)) {
    const int gx4 = (a.GK + 4 * kWaves - 1) / (4 * kWaves);
    const int gy4 = column_slices(gx4, (TB + xchunk - 1) / xchunk);
    return launch_input_proj_xc<kMaxXChunk, 4>(a, gx4, gy4, xchunk, xrow, plds, stream);
  }
  const int gy = column_slices(gx, (TB + xchunk - 1) / xchunk);
  return launch_input_proj_xc<kMaxXChunk>(a, gx, gy, xchunk, xrow, plds, stream);
}

hipError_t launch_progressive(const RunArgs& a, int blocks, int cooperative, hipStream_t stream) {
  hipError_t e = launch_input_proj(a, stream);
  if (e != hipSuccess) return e;
  const size_t lds = layout_of(a, a.online).total;
  switch (a.hpl) {
    case 4: return launch_u<4>(a, blocks, cooperative, lds, stream);
    case 8: return launch_u<8>(a, blocks, cooperative, lds, stream);
    case 12: return launch_u<12>(a, blocks, cooperative, lds, stream);
    case 16: return launch_u<16>(a, blocks, cooperative, lds, stream);
    case 24: return launch_u<24>(a, blocks, cooperative, lds, stream);
    case 32: return launch_u<32>(a, blocks, cooperative, lds, stream);
    default: return launch_u<0>(a, blocks, cooperative, lds, stream);
  }
}

hipError_t launch_clear_u64(unsigned long long* p, size_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  int blocks = (int)std::min<size_t>((n + 255) / 256, 1024);
  clear_u64_kernel<<<blocks, 256, 0, stream>>>(p, n);
  return hipGetLastError();
}

}  // namespace alstm
