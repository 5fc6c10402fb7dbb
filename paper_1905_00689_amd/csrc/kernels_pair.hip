// gfx950 recurrence for one (level, sequence) pair of the progressive
// approximate LSTM (arXiv 1905.00689: Sec. III Eq. (1) per gate, then the
// Sec. II cell update): the batch-1, single-budget run.
//
// P workgroups of 512 threads, all resident.  Workgroup j owns the terms
// tau = j + i*P (i < OM, round-robin over the refinement order, so every
// budget prefix is spread over all workgroups) and the hidden units
// [j*RU, j*RU + RU).  Every slice it needs stays in registers for the whole
// sequence: the h-part entries of its terms (16 lanes per term, hpl entries
// per lane, one or two passes) and the U entries of its 4*RU gate rows
// (S lanes per row, upt entries per lane, one, two or four rows per thread).
// P_x of every timestep (input_proj_kernel) is staged in LDS up front.
// Per timestep:
//   phase A  each term's lane group sums its h-part entries against h_{t-1}
//            (LDS), reduces over its 16 lanes and forms z = sigma * (P_x + s);
//   z        the last wave (the publisher) stores the workgroup's z as
//            tagged words; waves 0-6 poll every workgroup's words into LDS;
//   phase B  each row's lanes sum u * z over their terms and reduce; the four
//            gate rows of a unit lie in one wave (rows gate-minor), so the
//            unit's lane gathers them by lane shuffles and applies the gate
//            nonlinearities and the c/h update with c held in a register;
//   h        the publisher writes h to h_out and stores it as tagged words;
//            waves 0-6 poll every unit's h into LDS.
// The publisher only stores and the pollers only load: a wave's loads and
// stores retire through one in-order counter, so a wave that polled after
// storing would wait for its own stores' acknowledgements every round.
// With one workgroup (P = 1) nothing is exchanged: z and h go through LDS.
//
// The order of every sum is that of progressive_lstm_kernel (phase A: entry
// sla + 16k of the term's h part at lane sla, k ascending, then the 16-lane
// DPP reduction; phase B: term sl + S*k at lane sl, k ascending, then the
// S-lane reduction, then the bias), so the two kernels' outputs are bitwise
// equal; the launch shape never changes a result.
#include "kernels.hpp"
#include "device_common.hpp"

#include <algorithm>

namespace alstm {

namespace {

// Poll tagged words src[si[k]] (si[k] < 0: none) until each carries `tag`;
// the value goes to dst[di[k]] (LDS).  One generation of loads per round:
// every word of the thread is loaded, all are awaited, the arrived ones are
// kept and the rest loaded again.  Nothing is left in flight when it returns,
// so no later instruction waits on a stray poll (a second generation in
// flight would halve the detection delay, but its loads outlive the poll and
// the compiler's wait counts across the loop then stall every round anyway).
// Bounded: past the spin limit, or once another wait has failed, the
// failure is recorded and the missing values read 0.
template <int NW>
__device__ __forceinline__ void poll_words(float* dst, const unsigned long long* src, const int* si, const int* di,
                                           int nw, unsigned tag, unsigned* err) {
  unsigned pending = 0;
#pragma unroll
  for (int k = 0; k < NW; ++k)
    if (k < nw && si[k] >= 0) pending |= 1u << k;
  unsigned spins = 0;
  while (pending) {
    unsigned long long w[NW];
    // words k < nw (uniform): every one loaded, unused ones at src[0]
#pragma unroll
    for (int k = 0; k < NW; ++k)
      if (k < nw) w[k] = load_tagged(src + max(si[k], 0));
#pragma unroll
    for (int k = 0; k < NW; ++k)
      if (((pending >> k) & 1u) && (unsigned)(w[k] >> 32) == tag) {
        dst[di[k]] = __uint_as_float((unsigned)w[k]);
        pending &= ~(1u << k);
      }
    if ((++spins & 255u) == 0u && pending &&
        (spins >= kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
      __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
      for (int k = 0; k < NW; ++k)
        if ((pending >> k) & 1u) dst[di[k]] = 0.0f;
      break;
    }
  }
}

// The last wave publishes (z, h and h_out: every global store of the
// recurrence); the other waves poll.  A wave's stores and loads share one
// in-order completion counter, so a wave that polled after storing would
// wait for its own stores to be acknowledged at every poll round.
constexpr int kPollThreads = kThreads - 64;
// Words polled per thread and exchange (up to 8 * 448 = 3584 slots).
constexpr int kMaxWords = 8;

// Timestep stamps of workgroup 0 are kept in LDS (written out at the end) up
// to this many timesteps; beyond, they go straight to memory.
constexpr int kLdsStamps = 255;

// LDS carve-up (floats): stamps [2 * (4 + 4 * kLdsStamps)] (8-byte aligned
// at offset 0), P_x [T][OM], then h [hpad], z [G][zstride], z of the owned
// terms [OM], h of the owned units [RU], and per wave the gate
// pre-activations of its rows [opt][64 / S] (16-byte aligned).
constexpr int kStampFloats = 2 * (4 + 4 * kLdsStamps);
struct PairLayout {
  size_t px, hs, zs, zown, hown, ys, total;
};
__host__ __device__ inline PairLayout pair_layout(const PairArgs& a) {
  PairLayout l;
  l.px = kStampFloats;
  l.hs = l.px + (((size_t)a.T * a.OM + 3) & ~(size_t)3);
  l.zs = l.hs + a.hpad;
  l.zown = l.zs + (size_t)a.G * a.zstride;
  l.hown = l.zown + a.OM;
  l.ys = (l.hown + a.RU + 3) & ~(size_t)3;   // 16-byte aligned
  l.total = l.ys + (size_t)kWaves * a.opt * (64 / a.S);
  return l;
}
__host__ __device__ inline size_t pair_lds_floats(const PairArgs& a) { return pair_layout(a).total; }

// OPT output rows per thread with UMAX U entries each in registers, APASS
// phase-A passes with HMAX h-part entries per lane each.  Every loop runs to
// its compile-time bound: entries past a lane's share are zeros (a U entry
// past the budget, an h-part slot past the term's count), whose products add
// nothing, so the sums equal those over the live entries in the same order.
template <int OPT, int UMAX, int APASS, int HMAX>
__global__ void __launch_bounds__(kThreads) pair_lstm_kernel(PairArgs a) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  constexpr int kChunk = 16;   // LDS reads in flight per batch
  constexpr int NWMAX = kMaxWords;
  const int P = gridDim.x, j = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const bool publisher = tid >= kPollThreads;
  const int D = a.D, H = a.H, G = a.G, N = a.N, NZ = a.NZ, T = a.T, K = a.K, GK = a.GK;
  const int OM = a.OM, RU = a.RU, zst = a.zstride, kst = a.kstride;
  const bool local = P == 1;
  const PairLayout lay = pair_layout(a);
  float* ldsf = reinterpret_cast<float*>(lds_raw);
  unsigned long long* lstamp = reinterpret_cast<unsigned long long*>(lds_raw);
  float* pxs = ldsf + lay.px;      // P_x [T][OM]
  float* hs = ldsf + lay.hs;       // h_{t-1} [H]
  float* zs = ldsf + lay.zs;       // z of this timestep [G][zst]
  float* zown = ldsf + lay.zown;   // z of the owned terms [OM]
  float* hown = ldsf + lay.hown;   // h of the owned units [RU]
  const int r0 = j * RU, rc = max(0, min(RU, H - r0));
  const int n_owned = GK > j ? (GK - j + P - 1) / P : 0;
  // uniform plan values, kept in scalar registers
  const int S = __builtin_amdgcn_readfirstlane(a.S), lgS = __builtin_amdgcn_readfirstlane(a.lgS);
  // z of term (n, g) sits at zs[g*zst + (n % S)*kst + n / S]: lane sl of a row
  // reads its terms sl + S*k at consecutive addresses (immediate offsets)
  auto zpos = [&](int tau) { const int g = tau % G, n = tau / G; return g * zst + (n & (S - 1)) * kst + (n >> lgS); };

  // Prologue loads, ordered so that every independent load is in flight
  // before the first wait: the first share of P_x and h0, sigma and the
  // h/x split of the owned terms, the U entries, bias and c0; then the
  // h-part entries (their addresses need the split).
  const int npx = T * n_owned;
  float px0 = 0.0f, h00 = 0.0f;
  if (tid < npx) {
    const int t0 = tid / n_owned, io0 = tid - t0 * n_owned;
    px0 = a.px[(size_t)(j + io0 * P) * T + t0];
  }
  if (tid < H && a.h0) h00 = a.h0[tid];

  // ---- phase-A roles: lane group sub (16 lanes) takes owned terms sub + 32p
  const int sub = tid >> 4, sla = tid & 15;
  float hv[APASS][HMAX];
  int hi[APASS][HMAX];
  float sg[APASS];
  int slot[APASS], zdst[APASS], e0v[APASS];
#pragma unroll
  for (int p = 0; p < APASS; ++p) {
    const int ia = sub + 32 * p;
    const bool own = ia < n_owned;
    const int tau = j + ia * P;
    sg[p] = own ? a.sigma[tau] : 0.0f;
    slot[p] = own ? j * OM + ia : -1;
    zdst[p] = own ? zpos(tau) : 0;
    e0v[p] = own ? (int)a.nx[tau] : NZ;
  }

  // ---- phase-B roles: row slot rs = tid / S, rows rs + o * (512 / S); row ol
  // is gate q = ol & 3 of owned unit ol >> 2 (gate-minor: a unit's four rows
  // are four adjacent lane groups of one wave)
  const int rs = tid >> lgS, sl = tid & (S - 1);
  const int nslots = kThreads >> lgS;
  float uv[OPT][UMAX];
  float bq[OPT];
  // every row of a thread has gate q = rs & 3 (row slots per pass are a
  // multiple of 4): one z base for all of them
  const int zb = (G == 4 ? (rs & 3) : 0) * zst + sl * kst;
  // ---- cell roles: a wave holds the rows of 16 * OPT / S units (row slots
  // [w * 64/S, (w+1) * 64/S) in each of the OPT passes); its lane cl takes
  // unit cl, pass co = cl / (16/S), row slots 4 ck .. 4 ck + 3 (ck = cl %
  // (16/S)), and keeps that unit's c in a register.  The rows' sums reach
  // it through the wave's LDS block ysw[o][64/S] (no cross-wave traffic).
  const int wv = tid >> 6, rpw = 64 >> lgS, upw = (16 * OPT) >> lgS;
  const int co = lane / (16 >> lgS), ck = lane % (16 >> lgS);
  const int cunit = (wv * rpw + 4 * ck + co * nslots) >> 2;
  const bool cell_ok = lane < upw && cunit < rc;
  float cst = (cell_ok && a.c0) ? a.c0[r0 + cunit] : 0.0f;
  float* ysw = ldsf + lay.ys + (size_t)wv * OPT * rpw;
#pragma unroll
  for (int o = 0; o < OPT; ++o) {
    const int ol = rs + o * nslots, ul = ol >> 2, q = ol & 3;
    const bool rowv = ul < rc;
    const size_t row = (size_t)q * H + r0 + ul;
    bq[o] = rowv ? a.bias[row] : 0.0f;
    const float* urow = a.Ut + (rowv ? row : 0) * N;
#pragma unroll
    for (int k = 0; k < UMAX; ++k) uv[o][k] = urow[min(sl + S * k, K - 1)];
#pragma unroll
    for (int k = 0; k < UMAX; ++k) uv[o][k] = (rowv && sl + S * k < K) ? uv[o][k] : 0.0f;
  }

#pragma unroll
  for (int p = 0; p < APASS; ++p) {
    const int ia = sub + 32 * p;
    const int tau = ia < n_owned ? j + ia * P : 0;
    const int e0 = e0v[p], cnt = NZ - e0;
    const size_t src = (size_t)tau * NZ;
    // every load issued (index clamped into the term's entries), then masked
#pragma unroll
    for (int k = 0; k < HMAX; ++k) {
      const int e = min(e0 + sla + 16 * k, NZ - 1);
      hv[p][k] = a.vval[src + e];
      hi[p][k] = (int)a.vidx[src + e];
    }
#pragma unroll
    for (int k = 0; k < HMAX; ++k) {
      const bool live = sla + 16 * k < cnt;
      hv[p][k] = live ? hv[p][k] : 0.0f;
      hi[p][k] = 4 * (int)lay.hs + (live ? 4 * (hi[p][k] - D) : 0);   // byte offset of h[k - D] in LDS
    }
  }

  // ---- exchange roles: z slots tid + 512 r (slot s = j'*OM + i' carries
  // term j' + i'*P), h words tid + 512 r
  int zsi[NWMAX], zdi[NWMAX], hsi[NWMAX];
  const int nslot = P * OM;
  const int nwz = (nslot + kPollThreads - 1) / kPollThreads, nwh = (H + kPollThreads - 1) / kPollThreads;
#pragma unroll
  for (int r = 0; r < NWMAX; ++r) {
    const int s = tid + kPollThreads * r;
    const int jj = s / (OM > 0 ? OM : 1), ii = s - jj * OM;
    const int tau = jj + ii * P;
    const bool v = !local && !publisher && r < nwz && s < nslot && tau < GK;
    zsi[r] = v ? s : -1;
    zdi[r] = v ? zpos(tau) : 0;
    hsi[r] = (!local && !publisher && r < nwh && s < H) ? s : -1;
  }

  // ---- LDS: initial state, P_x of every timestep when it fits
  if (tid < H) hs[tid] = h00;
  for (int i = tid + kThreads; i < H; i += kThreads) hs[i] = a.h0 ? a.h0[i] : 0.0f;
  // z slots of terms past the budget (n >= K in a lane's last entry) are
  // never written and must read 0 (their u entries are 0 as well)
  for (int i = tid; i < G * zst; i += kThreads) zs[i] = 0.0f;
  if (tid < npx) pxs[(tid / n_owned) * OM + tid % n_owned] = px0;
  for (int i = tid + kThreads; i < npx; i += kThreads) {
    const int t = i / n_owned, io = i - t * n_owned;
    pxs[t * OM + io] = a.px[(size_t)(j + io * P) * T + t];
  }
  __syncthreads();

  const bool stamp = a.stamps && j == 0 && tid == 0;
  // stamps of short runs stay in LDS until the end (no stores on the way)
  unsigned long long* st = (T <= kLdsStamps) ? lstamp : a.stamps;
  if (stamp) {
    st[0] = wall_clock64();
    st[1] = clock64();
  }
  for (int t = 0; t < T; ++t) {
    const unsigned tag = a.tag_base | (unsigned)(t + 1);
    if (stamp) st[2 + 4 * t] = clock64();

    // ---- phase A: z = sigma * (P_x + prune(v)_h . h_{t-1}) ----
#pragma unroll
    for (int p = 0; p < APASS; ++p) {
      if (p * 32 >= n_owned) break;
      float acc = 0.0f;
#pragma unroll
      for (int k0 = 0; k0 < HMAX; k0 += kChunk) {
        // the bound k0 + k < HMAX is a constant once unrolled (a last chunk
        // may be partial: HMAX = 24)
        float hg[kChunk];
#pragma unroll
        for (int k = 0; k < kChunk; ++k)
          if (k0 + k < HMAX) hg[k] = *reinterpret_cast<const float*>(lds_raw + hi[p][k0 + k]);
#pragma unroll
        for (int k = 0; k < kChunk; ++k)
          if (k0 + k < HMAX) acc += hv[p][k0 + k] * hg[k];
      }
      acc = group_sum<16>(acc);
      if (sla == 0 && slot[p] >= 0) {
        const float pxv = pxs[t * OM + sub + 32 * p];
        const float z = sg[p] * (pxv + acc);
        if (local) zs[zdst[p]] = z;
        else zown[sub + 32 * p] = z;
      }
    }
    if (stamp) st[3 + 4 * t] = clock64();
    if (!local) {
      lds_barrier();
      if (publisher) {
        for (int i = lane; i < n_owned; i += 64) publish(a.zx + j * OM + i, zown[i], tag);
      } else {
        poll_words<NWMAX>(zs, a.zx, zsi, zdi, nwz, tag, a.err);
      }
    }
    lds_barrier();
    if (stamp) st[4 + 4 * t] = clock64();

    // ---- phase B: y = b + sum_n u_n z_n, then the cell update ----
    float y[OPT], acc[OPT];
#pragma unroll
    for (int o = 0; o < OPT; ++o) acc[o] = 0.0f;
#pragma unroll
    for (int k0 = 0; k0 < UMAX; k0 += kChunk) {
      float zv[kChunk];
#pragma unroll
      for (int k = 0; k < kChunk; ++k)
        if (k0 + k < UMAX) zv[k] = zs[zb + k0 + k];
#pragma unroll
      for (int o = 0; o < OPT; ++o)
#pragma unroll
        for (int k = 0; k < kChunk; ++k)
          if (k0 + k < UMAX) acc[o] += uv[o][k0 + k] * zv[k];
    }
#pragma unroll
    for (int o = 0; o < OPT; ++o) y[o] = group_sum_rt(acc[o], S) + bq[o];
    // the rows' sums go to the wave's block (lane sl == 0 of each row), then
    // each unit's lane reads its four gate rows at once and updates c and h
    if (sl == 0) {
#pragma unroll
      for (int o = 0; o < OPT; ++o) ysw[o * rpw + ((tid & 63) >> lgS)] = y[o];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < upw) {
      const float4 g4 = *reinterpret_cast<const float4*>(ysw + co * rpw + 4 * ck);
      float h2;
      cell_update(g4.x, g4.y, g4.z, g4.w, cst, h2);
      if (cell_ok) {
        if (local) {
          hs[r0 + cunit] = h2;
          a.h_out[(size_t)t * H + r0 + cunit] = h2;
        } else {
          hown[cunit] = h2;
        }
      }
    }
    if (stamp) st[5 + 4 * t] = clock64();
    if (!local) {
      lds_barrier();
      if (publisher) {
        for (int u = lane; u < rc; u += 64) {
          const float h2 = hown[u];
          a.h_out[(size_t)t * H + r0 + u] = h2;
          publish(a.hx + r0 + u, h2, tag);
        }
      } else {
        poll_words<NWMAX>(hs, a.hx, hsi, hsi, nwh, tag, a.err);
      }
    }
    lds_barrier();
  }
  if (stamp) {
    st[2 + 4 * T] = clock64();
    st[3 + 4 * T] = wall_clock64();
    if (st == lstamp)
      for (int i = 0; i < 4 + 4 * T; ++i) a.stamps[i] = lstamp[i];
  }
  if (a.c_out && cell_ok) a.c_out[r0 + cunit] = cst;
}

template <int OPT, int UMAX, int APASS, int HMAX>
hipError_t launch_pair_kernel(const PairArgs& a, int P, size_t lds, hipStream_t stream) {
  static bool attr_set = false;
  const void* fn = (const void*)pair_lstm_kernel<OPT, UMAX, APASS, HMAX>;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsCap);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  pair_lstm_kernel<OPT, UMAX, APASS, HMAX><<<dim3(P), dim3(kThreads), lds, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

int plan_pair(PairArgs& a, int num_cu, int want, size_t* lds) {
  *lds = 0;
  if (a.K < 1 || a.GK < 1 || a.G < 1) return 0;
  a.S = lanes_for_level(a.K);
  a.lgS = 31 - __builtin_clz((unsigned)a.S);
  a.upt = (a.K + a.S - 1) / a.S;
  const int need_h = (a.hcap + 15) / 16;   // h-part entries per lane
  const int cap = std::max(1, num_cu);
  auto fits = [&](int P) -> bool {
    const int OM = (a.GK + P - 1) / P;
    const int apass = OM <= 32 ? 1 : (OM <= 64 ? 2 : 0);
    if (!apass) return false;
    if (need_h > (apass == 1 ? 32 : 16)) return false;
    const int RU = (a.H + P - 1) / P;
    const int slots = kThreads / a.S;      // row slots per pass of the threads
    const int opt = (4 * RU + slots - 1) / slots;
    const int opt_b = opt <= 1 ? 1 : (opt <= 2 ? 2 : (opt <= 4 ? 4 : 0));
    if (!opt_b || a.upt > 32 / (opt_b == 4 ? 2 : 1)) return false;
    // register budget: two phase-A passes hold at most 16 h-part entries per
    // lane (every instance fits its registers without spilling)
    if (apass == 2 && need_h > 16) return false;
    // the four gate rows of a unit must be adjacent lane groups of one wave
    if (4 * a.S > 64) return false;
    if ((size_t)P * OM > (size_t)kMaxWords * kPollThreads || a.H > kMaxWords * kPollThreads) return false;
    a.OM = OM;
    a.RU = RU;
    a.apass = apass;
    a.opt = opt_b;
    return true;
  };
  int P = 0;
  if (want > 0) {
    if (want > cap || !fits(want)) return 0;
    P = want;
  } else if (fits(1)) {
    P = 1;   // one workgroup: nothing exchanged
  } else {
    // the exchanges cost about the same at any width (their latency is
    // that of device-scope visibility, not of the words moved), so take the
    // narrowest width at which each thread has one phase-A term group and one
    // output row (MI355X, driving shape, K = 512: 5.5 us per timestep on 64
    // workgroups against 6.3 on 32 and 5.7 on 128), else the narrowest that fits
    for (int p = 2; p <= cap && !P; ++p)
      if (fits(p) && a.apass == 1 && a.opt == 1) P = p;
    for (int p = 2; p <= cap && !P; ++p)
      if (fits(p)) P = p;
    if (!P) return 0;
    // below 64 terms per group that width leaves each workgroup hundreds of
    // output rows, and phase B then takes longer than the wider exchange
    // costs: at least 16 workgroups from 17 terms per group, 32 from 64
    // (each keeping 16 rows or more).  MI355X, driving shape, us per
    // timestep at P = 4 / 8 / 16 / 32 / 64: K = 32 5.70 / 5.12 / 4.80 / 4.84
    // / 5.42; K = 64 6.28 / 5.19 / 4.81 / 4.71 / 4.92; K = 128 - / 5.70 /
    // 4.94 / 4.79 / 4.91; K = 256 32 and 64 equal (5.28, 5.27), K = 512 best
    // at its own 64; outputs bitwise equal at every width.
    const int floor_p = std::min({a.K >= 64 ? 32 : (a.K > 16 ? 16 : 0), (4 * a.H) / 16, cap});
    if (P < floor_p && fits(floor_p)) P = floor_p;
    fits(P);
  }
  // register buckets: h-part entries per lane, U entries per row and lane
  a.hpl = need_h <= 4 ? 4 : need_h <= 8 ? 8 : need_h <= 12 ? 12 : need_h <= 16 ? 16 : need_h <= 24 ? 24 : 32;
  if (a.apass == 2 && a.hpl > 16) return 0;
  a.umax = a.opt == 4 ? (a.upt <= 8 ? 8 : 16) : a.opt == 2 ? (a.upt <= 16 ? 16 : 32)
                      : (a.upt <= 8 ? 8 : a.upt <= 16 ? 16 : 32);
  // lane sl's terms at stride kstride (odd, and covering the lane's whole
  // register bucket: every read stays in the lane's zero-filled slots); gates
  // at zstride = 16 (mod 64) apart (the four gate rows of a unit, in one
  // wave, read distinct banks)
  a.kstride = a.umax | 1;
  a.zstride = ((a.S * a.kstride + 63) / 64) * 64 + 16;
  a.hpad = (a.H + 3) & ~3;
  // P_x of every timestep in LDS (no loads inside the recurrence); longer
  // sequences take the general kernel
  a.px_lds = 1;
  const size_t bytes = 4 * pair_lds_floats(a);
  if (bytes > kLdsCap) return 0;
  *lds = bytes;
  return P;
}

template <int APASS, int HMAX>
hipError_t launch_pair_u(const PairArgs& a, int P, size_t lds, hipStream_t stream) {
  if (a.opt == 4) {
    if (a.umax == 8) return launch_pair_kernel<4, 8, APASS, HMAX>(a, P, lds, stream);
    return launch_pair_kernel<4, 16, APASS, HMAX>(a, P, lds, stream);
  } else if (a.opt == 2) {
    if (a.umax == 16) return launch_pair_kernel<2, 16, APASS, HMAX>(a, P, lds, stream);
    return launch_pair_kernel<2, 32, APASS, HMAX>(a, P, lds, stream);
  } else {
    if (a.umax == 8) return launch_pair_kernel<1, 8, APASS, HMAX>(a, P, lds, stream);
    if (a.umax == 16) return launch_pair_kernel<1, 16, APASS, HMAX>(a, P, lds, stream);
    if (a.umax == 32) return launch_pair_kernel<1, 32, APASS, HMAX>(a, P, lds, stream);
  }
  return hipErrorInvalidValue;   // the planner never asks for it
}

hipError_t launch_pair(const RunArgs& proj, const PairArgs& a, int P, hipStream_t stream) {
  hipError_t e = launch_input_proj(proj, stream);
  if (e != hipSuccess) return e;
  const size_t lds = 4 * pair_lds_floats(a);
  if (a.apass == 2) {
    switch (a.hpl) {
      case 4: return launch_pair_u<2, 4>(a, P, lds, stream);
      case 8: return launch_pair_u<2, 8>(a, P, lds, stream);
      case 12: return launch_pair_u<2, 12>(a, P, lds, stream);
      default: return launch_pair_u<2, 16>(a, P, lds, stream);
    }
  }
  switch (a.hpl) {
    case 4: return launch_pair_u<1, 4>(a, P, lds, stream);
    case 8: return launch_pair_u<1, 8>(a, P, lds, stream);
    case 12: return launch_pair_u<1, 12>(a, P, lds, stream);
    case 16: return launch_pair_u<1, 16>(a, P, lds, stream);
    case 24: return launch_pair_u<1, 24>(a, P, lds, stream);
    default: return launch_pair_u<1, 32>(a, P, lds, stream);
  }
}

}  // namespace alstm
