// C-ABI implementation: argument checking, host factorisation (float64),
// packing of the device factor store, run workspace and kernel launch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/approx_lstm.h"
#include "factorise.hpp"
#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;

approx_lstm_status fail(approx_lstm_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

approx_lstm_status hip_fail(hipError_t e, const char* what) {
  if (e == hipErrorOutOfMemory)
    return fail(APPROX_LSTM_ERR_OUT_OF_MEMORY, "%s: %s", what, hipGetErrorString(e));
  return fail(APPROX_LSTM_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                    \
  do {                                         \
    hipError_t _e = (expr);                    \
    if (_e != hipSuccess) return hip_fail(_e, what); \
  } while (0)

template <class T>
void dfree(T*& p) {
  if (p) (void)hipFree((void*)p);
  p = nullptr;
}

// Sets the model's device current for the scope and restores the caller's.
struct DeviceScope {
  int prev = -1;
  bool ok = true;
  explicit DeviceScope(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceScope() {
    int cur;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

}  // namespace

struct approx_lstm_model {
  int D = 0, H = 0, C = 0, G = 0, Rg = 0, N = 0, NZ = 0;
  uint64_t flags = 0;
  int eff_rank[4] = {0, 0, 0, 0};
  int unconverged = 0;
  // host copies, as stored (fp32) -- [G][N]..., per group
  std::vector<float> sigma, u, vval, bias;
  std::vector<int32_t> vidx;
  std::vector<double> sigma64, u64, v64;   // only with KEEP_UNPRUNED
  // device factor store
  int device = -1;
  bool has_dev = false;
  float* d_sigma = nullptr;
  float* d_Ut = nullptr;
  float* d_vval = nullptr;
  float* d_bias = nullptr;
  uint16_t* d_vidx = nullptr;
  uint16_t* d_nx = nullptr;
  uint64_t dev_bytes = 0;
  int num_cu = 0;
  // bf16 panel store (factor_dtype 1): Vx [prow][Dp], Vh [prow][Hp], Ut [4H][Kp];
  // Dp = D rounded up to 64, Hp, Kp = H, rank rounded up to 32 (the MFMA
  // contraction step), prow = G*Kp rounded up to 128 (the x-projection's row
  // tile)
  int dtype = 0;
  int Dp = 0, Hp = 0, Kp = 0, prow = 0;
  uint16_t* d_Vx = nullptr;
  uint16_t* d_Vh = nullptr;
  uint16_t* d_Ut16 = nullptr;
  uint16_t* d_bz = nullptr;          // batched workspace: Z [G][Bp][Kp]
  size_t bz_cap = 0;
  uint16_t* d_bh = nullptr;          // hb [Bp][Hp]
  size_t bh_cap = 0;
  float* d_bc = nullptr;             // c [Bp][H]
  size_t bc_cap = 0;
  std::vector<int> hpre;             // [N*G] max over terms 0..tau of the h-part entry count
  // run workspace
  float* d_px = nullptr;
  size_t px_cap = 0;                 // floats
  unsigned long long* d_zx = nullptr;
  size_t zx_cap = 0;                 // words
  unsigned long long* d_hx = nullptr;
  size_t hx_cap = 0;
  float* d_hbx = nullptr;            // bulk h exchange, [2][hb_stride]
  size_t hbx_cap = 0;                // floats
  unsigned* d_hflag = nullptr;       // bulk h exchange flags, one per workgroup
  size_t hflag_cap = 0;
  unsigned* d_err = nullptr;
  unsigned long long* d_stamps = nullptr;
  size_t stamps_cap = 0;             // words
  int timing = 0;                    // record per-timestep stamps
  int last_T = 0;                    // T of the last run that recorded stamps
  unsigned seq = 0;
  float* d_stack = nullptr;          // intermediate h of stacked runs (owned by the first layer)
  size_t stack_cap = 0;              // floats
  // deadline calibration: in-kernel microseconds per timestep against K, for
  // the (T, B, launch_blocks) it was measured at
  std::vector<std::pair<int, double>> calib;
  int calib_T = -1, calib_B = -1, calib_blocks = -1;
  // online (anytime) calibration: microseconds per timestep against K inside
  // the online launch (sized for the full rank), cached per (T, B, width)
  std::vector<std::pair<int, double>> ocalib;
  int ocalib_T = -1, ocalib_B = -1, ocalib_blocks = -1;
  int* d_kt = nullptr;               // [kt_cap] budgets chosen by an online run
  size_t kt_cap = 0;
  int launch_blocks = 0;             // 0 = automatic
  int cooperative = 0;               // 1: cooperative launch API
  int recurrence = 0;                // 0: one-pair kernel where it applies, 1: general kernel only
  // persistent batched recurrence (bf16 models): cohort exchange buffers
  int batched_persistent = 1;        // 0: per-timestep kernel pairs only; 1: persistent where it
                                     // fits; 2, 3: persistent with z always tagged / always flagged
  uint16_t* d_pzx = nullptr;         // [slots][G][16][Kp] bf16
  size_t pzx_cap = 0;                // elements
  uint16_t* d_phx = nullptr;         // [slots][16][Hp] bf16, padding columns zero
  size_t phx_cap = 0;
  unsigned* d_pflag = nullptr;       // [2][slots][W]
  size_t pflag_cap = 0;
  float* d_ppart = nullptr;          // partial x-projections of a split contraction
  size_t ppart_cap = 0;              // floats

  ~approx_lstm_model() {
    if (!has_dev && !d_px && !d_zx && !d_hx && !d_hbx && !d_hflag && !d_err && !d_stamps && !d_stack && !d_bz &&
        !d_bh && !d_bc && !d_kt && !d_pzx && !d_phx && !d_pflag && !d_ppart)
      return;
    DeviceScope ds(device);
    dfree(d_pzx);
    dfree(d_phx);
    dfree(d_pflag);
    dfree(d_ppart);
    dfree(d_Vx);
    dfree(d_Vh);
    dfree(d_Ut16);
    dfree(d_bz);
    dfree(d_bh);
    dfree(d_bc);
    dfree(d_sigma);
    dfree(d_Ut);
    dfree(d_vval);
    dfree(d_bias);
    dfree(d_vidx);
    dfree(d_nx);
    dfree(d_px);
    dfree(d_zx);
    dfree(d_hx);
    dfree(d_hbx);
    dfree(d_hflag);
    dfree(d_err);
    dfree(d_stamps);
    dfree(d_kt);
    dfree(d_stack);
  }
};

namespace {

approx_lstm_status ensure_workspace(approx_lstm_model* m, size_t px_floats, size_t zx_words, size_t hx_words,
                                    hipStream_t stream) {
  bool fresh = false;
  if (!m->d_err) {
    HIP_TRY(hipMalloc(&m->d_err, 64), "hipMalloc(err)");
    HIP_TRY(hipMemsetAsync(m->d_err, 0, 64, stream), "hipMemsetAsync(err)");
  }
  if (px_floats > m->px_cap) {
    HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
    dfree(m->d_px);
    m->px_cap = 0;
    HIP_TRY(hipMalloc(&m->d_px, px_floats * sizeof(float)), "hipMalloc(px)");
    m->px_cap = px_floats;
  }
  if (zx_words > m->zx_cap) {
    HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
    dfree(m->d_zx);
    m->zx_cap = 0;
    HIP_TRY(hipMalloc(&m->d_zx, zx_words * 8), "hipMalloc(zx)");
    m->zx_cap = zx_words;
    fresh = true;
  }
  if (hx_words > m->hx_cap) {
    HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
    dfree(m->d_hx);
    m->hx_cap = 0;
    HIP_TRY(hipMalloc(&m->d_hx, hx_words * 8), "hipMalloc(hx)");
    m->hx_cap = hx_words;
    fresh = true;
  }
  if (fresh) {
    // New exchange memory: clear every tag before its first use.
    if (m->d_zx) HIP_TRY(alstm::launch_clear_u64(m->d_zx, m->zx_cap, stream), "clear(zx)");
    if (m->d_hx) HIP_TRY(alstm::launch_clear_u64(m->d_hx, m->hx_cap, stream), "clear(hx)");
    m->seq = 0;
  }
  return APPROX_LSTM_OK;
}

// fp64 -> fp32 (nearest even) -> bf16 (nearest even), returned as the fp32
// value it represents; finite inputs.
float round_bf16(double v) {
  float f = (float)v;
  uint32_t bits;
  std::memcpy(&bits, &f, 4);
  bits = (bits + 0x7FFFu + ((bits >> 16) & 1u)) & 0xFFFF0000u;
  std::memcpy(&f, &bits, 4);
  return f;
}

uint16_t bf16_bits_of(float exact_bf16) {
  uint32_t bits;
  std::memcpy(&bits, &exact_bf16, 4);
  return (uint16_t)(bits >> 16);
}

size_t round_up(size_t v, size_t m) { return (v + m - 1) / m * m; }

template <class T>
approx_lstm_status grow(T*& p, size_t& cap, size_t want, hipStream_t stream, const char* what) {
  if (want <= cap) return APPROX_LSTM_OK;
  HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
  dfree(p);
  cap = 0;
  HIP_TRY(hipMalloc(&p, want * sizeof(T)), what);
  cap = want;
  return APPROX_LSTM_OK;
}

// Workspace of the batched path for T timesteps, Bp padded sequences and
// budgets up to kmax.
approx_lstm_status ensure_batched(approx_lstm_model* m, int T, size_t Bp, int kmax, hipStream_t stream) {
  const size_t prows = (size_t)m->G * round_up((size_t)kmax, 32);
  approx_lstm_status st = grow(m->d_px, m->px_cap, std::max<size_t>(1, prows * T * Bp), stream, "hipMalloc(P)");
  if (st == APPROX_LSTM_OK) st = grow(m->d_bz, m->bz_cap, (size_t)m->G * Bp * m->Kp, stream, "hipMalloc(Z)");
  if (st == APPROX_LSTM_OK && Bp * m->Hp > m->bh_cap) {
    // the padding columns of hb (units H..Hp-1) are never written by a run:
    // they must hold zeros (bf16 +0) from allocation on
    st = grow(m->d_bh, m->bh_cap, Bp * m->Hp, stream, "hipMalloc(hb)");
    if (st == APPROX_LSTM_OK)
      HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_bh), m->bh_cap / 4, stream),
              "clear(hb)");
  }
  if (st == APPROX_LSTM_OK) st = grow(m->d_bc, m->bc_cap, Bp * m->H, stream, "hipMalloc(c)");
  if (st == APPROX_LSTM_OK)
    st = grow(m->d_ppart, m->ppart_cap, alstm::batched_ppart_floats(m->num_cu), stream, "hipMalloc(partial P)");
  return st;
}

// Bulk h exchange buffers: `floats` for the two parities of h_t and one flag
// word per possible workgroup (cleared when new, so no stale tag can match).
approx_lstm_status ensure_bulk(approx_lstm_model* m, size_t floats, hipStream_t stream) {
  approx_lstm_status st = grow(m->d_hbx, m->hbx_cap, floats, stream, "hipMalloc(hbx)");
  if (st != APPROX_LSTM_OK) return st;
  const size_t flags = round_up((size_t)std::max(1, m->num_cu), 2);
  if (flags > m->hflag_cap) {
    st = grow(m->d_hflag, m->hflag_cap, flags, stream, "hipMalloc(hflag)");
    if (st != APPROX_LSTM_OK) return st;
    HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_hflag), m->hflag_cap / 2, stream),
            "clear(hflag)");
  }
  return APPROX_LSTM_OK;
}

// z of a persistent batched launch travel as tagged words (no flag round
// trip, twice the bytes) up to this many terms in use (G times K rounded up
// to 32), as plain bf16 behind flags beyond.  Measured on MI355X at the
// batched workload (H=512, 256 sequences), the flagged form is as fast or
// faster at every K from 32 to 512 (the tagged polls wait as long as the
// flag round trip), so the automatic choice is always flagged.
constexpr int kZtagTerms = 0;

// Exchange buffers of the persistent batched recurrence: z and h of every
// cohort in flight (zeroed when new, so that no stale tag can match) and the
// flag words (zeroed when new and when the launch sequence would wrap).
// Reserves n_levels launch sequence numbers: on return m->seq + n_levels <=
// 0xFFFF.
approx_lstm_status ensure_persistent(approx_lstm_model* m, size_t zx, size_t hx, size_t flags, int n_levels,
                                     hipStream_t stream) {
  if (!m->d_err) {
    HIP_TRY(hipMalloc(&m->d_err, 64), "hipMalloc(err)");
    HIP_TRY(hipMemsetAsync(m->d_err, 0, 64, stream), "hipMemsetAsync(err)");
  }
  approx_lstm_status st = APPROX_LSTM_OK;
  if (round_up(zx, 4) > m->pzx_cap) {
    st = grow(m->d_pzx, m->pzx_cap, round_up(zx, 4), stream, "hipMalloc(zx)");
    if (st == APPROX_LSTM_OK)
      HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_pzx), m->pzx_cap / 4, stream),
              "clear(zx)");
  }
  if (st == APPROX_LSTM_OK && round_up(hx, 4) > m->phx_cap) {
    st = grow(m->d_phx, m->phx_cap, round_up(hx, 4), stream, "hipMalloc(hx)");
    if (st == APPROX_LSTM_OK)
      HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_phx), m->phx_cap / 4, stream),
              "clear(hx)");
  }
  bool clear_flags = false;
  if (st == APPROX_LSTM_OK && round_up(flags, 2) > m->pflag_cap) {
    st = grow(m->d_pflag, m->pflag_cap, round_up(flags, 2), stream, "hipMalloc(flags)");
    clear_flags = true;
  }
  if (st != APPROX_LSTM_OK) return st;
  if (m->seq == 0 || m->seq + (unsigned)n_levels > 0xFFFFu) {
    clear_flags = true;
    m->seq = 1;
  }
  if (clear_flags) {
    HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_pflag), m->pflag_cap / 2, stream),
            "clear(flags)");
    HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_pzx), m->pzx_cap / 4, stream),
            "clear(zx)");
    HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_phx), m->phx_cap / 4, stream),
            "clear(hx)");
  }
  return APPROX_LSTM_OK;
}

// The batched bf16 run (factor_dtype 1): arguments already checked.
approx_lstm_status run_batched(approx_lstm_model* m, const float* x, int T, int B, const float* h0, const float* c0,
                               const int32_t* levels, int n_levels, float* h_out, float* c_out,
                               hipStream_t stream) {
  const size_t Bp = round_up((size_t)B, alstm::kBatchAlign);
  if (Bp > ((size_t)1 << 20)) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "B = %d exceeds 2^20 for a bf16 model", B);
  if ((size_t)T * Bp > (size_t)1 << 30)
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "T * padded B = %zu exceeds 2^30", (size_t)T * Bp);
  if ((size_t)T * B * m->D >= ((size_t)1 << 31))
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "T * B * D = %zu reaches 2^31", (size_t)T * B * m->D);
  int kmax = 0;
  for (int l = 0; l < n_levels; ++l) kmax = std::max(kmax, (int)levels[l]);
  approx_lstm_status st = ensure_batched(m, T, Bp, kmax, stream);
  if (st != APPROX_LSTM_OK) return st;
  alstm::BatchedArgs a{};
  a.x = x; a.h0 = h0; a.c0 = c0; a.h_out = h_out; a.c_out = c_out;
  a.sigma = m->d_sigma; a.Vx = m->d_Vx; a.Vh = m->d_Vh; a.Ut = m->d_Ut16; a.bias = m->d_bias;
  a.P = m->d_px; a.Z = m->d_bz; a.hb = m->d_bh; a.c = m->d_bc;
  a.D = m->D; a.Dp = m->Dp; a.H = m->H; a.Hp = m->Hp; a.G = m->G; a.Kp = m->Kp;
  a.T = T; a.B = B; a.Bp = (int)Bp;
  a.xvec = (m->D % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0) ? 1 : 0;
  a.max_wg = std::max(1, m->launch_blocks > 0 ? std::min(m->launch_blocks, m->num_cu) : m->num_cu);
  a.Ppart = m->d_ppart; a.ppart_cap = m->ppart_cap; a.ncu = m->num_cu;
  int W = 0, slots = 0;
  if (m->batched_persistent && alstm::plan_batched_persistent(a, kmax, &W, &slots)) {
    st = ensure_persistent(m, (size_t)slots * 2 * m->G * alstm::kCohort * m->Kp,
                           (size_t)slots * 2 * alstm::kCohort * m->Hp, (size_t)slots * W, n_levels, stream);
    if (st != APPROX_LSTM_OK) return st;
    a.zx = m->d_pzx; a.hx = m->d_phx; a.zflag = m->d_pflag;
    a.err = m->d_err;
    a.ztag_terms = m->batched_persistent == 2 ? (1 << 30) : m->batched_persistent == 3 ? 0 : kZtagTerms;
    a.tag_base = m->seq << 16;
    m->seq += (unsigned)n_levels;
  }
  std::vector<int> lv(levels, levels + n_levels);
  HIP_TRY(alstm::launch_batched(a, lv.data(), n_levels, stream), "launch batched kernels");
  return APPROX_LSTM_OK;
}

// Workgroups for a run: about one per 32 terms in use (so that every
// workgroup's terms and rows fit registers), at most 256.
int auto_blocks(const approx_lstm_model* m, int GK, int LB, int LB_seq, int num_cu) {
  int cap = std::max(1, std::min(num_cu, 256));
  // without terms the workgroups are independent (no exchange): spread the
  // cell updates, about 256 (unit, sequence) pairs per workgroup
  // with several sequences every workgroup's rows serve each of them: widen
  // by the sequence count (up to 8)
  int want = GK > 0 ? (GK + 31) / 32 * std::min(std::max(1, LB_seq), 8) : (int)(((long long)m->H * LB + 255) / 256);
  // wide enough that each thread of the accumulation holds one output row
  // with its U entries in registers (4 * units per workgroup * lanes per row
  // <= threads).  Below 5 terms per group a single workgroup, which
  // exchanges nothing, is faster (MI355X, driving shape: 4.1 against 4.3 us
  // per timestep at K = 1; at K = 8 four workgroups take 4.45 us, one 4.65).
  if (GK > 0 && m->G > 0 && (want > 1 || GK / m->G > 4)) {
    const int S = alstm::lanes_for_level(GK / m->G);
    const int rows_max = std::max(1, alstm::kThreads / (4 * S));
    want = std::max(want, (m->H + rows_max - 1) / rows_max);
  }
  // one sequence with 32 to 127 terms per group: 16 workgroups beat the 4 to
  // 15 above (MI355X, driving shape, one box: K = 32 5.62 against 5.72 us per
  // timestep, K = 64 5.74 against 6.06; K = 16 stays fastest on 4)
  if (LB_seq == 1 && m->G > 0 && GK / m->G >= 32 && GK / m->G < 128) want = std::max(want, 16);
  return std::max(1, std::min(cap, want));
}

// Budget options of an online run (see RunArgs::online).
struct OnlineCfg {
  int n = 0;
  int k[alstm::kMaxOptions];
  unsigned ticks[alstm::kMaxOptions];
  unsigned long long budget = 0;
  const int* sched = nullptr;   // device [T]: K_t given by the caller instead of the clock
};

// Launch plan of an fp32 progressive run: fills the shape fields of `a` and
// the workgroup count; returns the LDS bytes per workgroup (> kLdsCap: the
// run does not fit).  num_cu: compute units of the device.
size_t plan_run(const approx_lstm_model* m, alstm::RunArgs& a, int32_t T, int32_t B, const int32_t* levels,
                int32_t n_levels, int kmax, const OnlineCfg* on, int num_cu, int* blocks) {
  a = alstm::RunArgs{};
  a.D = m->D; a.H = m->H; a.G = m->G; a.N = m->N; a.NZ = m->NZ; a.T = T; a.B = B; a.L = n_levels;
  a.GK = m->G * kmax;
  a.num_cu = num_cu;
  for (int l = 0; l < n_levels; ++l) a.levels[l] = levels[l];
  if (on) {
    // one level sized for the largest budget; the kernel takes K_t per timestep
    a.online = 1;
    a.n_opts = on->n;
    for (int i = 0; i < on->n; ++i) {
      a.opt_k[i] = on->k[i];
      a.opt_ticks[i] = on->ticks[i];
    }
    a.budget = on->budget;
    a.sched = on->sched;
  }
  a.hcap = a.GK > 0 ? m->hpre[a.GK - 1] : 0;
  a.lanes_a = alstm::lanes_for_terms(m->NZ, m->D, m->H);
  for (int l = 0; l < n_levels; ++l) a.lanes_b[l] = alstm::lanes_for_level(levels[l]);
  const int maxP = std::max(1, num_cu);
  int P = m->launch_blocks > 0 ? std::min(m->launch_blocks, maxP) : auto_blocks(m, a.GK, n_levels * B, B, num_cu);
  size_t lds = alstm::plan_progressive(a, P);
  if (m->launch_blocks == 0)   // automatic: widen until the per-workgroup slices fit in LDS
    while (lds > alstm::kLdsCap && P < maxP) {
      P = std::min(maxP, 2 * P);
      lds = alstm::plan_progressive(a, P);
    }
  *blocks = P;
  return lds;
}

// Byte layout of a run's workspace carved from one caller-side region (the
// allocation-free entry point): P_x, z words, h words, bulk h, flags, each
// aligned to 256 bytes.
struct ScratchLayout {
  size_t px, zx, hx, hbx, hflag, total;
};

ScratchLayout scratch_layout(size_t px_floats, size_t zx_words, size_t hx_words, size_t hbx_floats, size_t flags) {
  ScratchLayout l{};
  size_t o = 0;
  l.px = o;    o = round_up(o + 4 * px_floats, 256);
  l.zx = o;    o = round_up(o + 8 * zx_words, 256);
  l.hx = o;    o = round_up(o + 8 * hx_words, 256);
  l.hbx = o;   o = round_up(o + 4 * hbx_floats, 256);
  l.hflag = o; o = round_up(o + 4 * flags, 256);
  l.total = o;
  return l;
}

// Workspace handed in by the allocation-free entry point: `base` (device,
// 256-byte aligned) holds `bytes`; launch tags come from `seq` (per device),
// and the exchange words of the region are cleared whenever it wraps.
struct CallerScratch {
  unsigned char* base;
  size_t bytes;
  unsigned* seq;
};

// Launch tag sequence of the next run: the model's own counter, or the
// caller workspace's; on wrap the exchange words are cleared (fill kernels)
// so that no stale tag can match.
approx_lstm_status next_tag(approx_lstm_model* m, const CallerScratch* ws, size_t ws_exchange_offset,
                            hipStream_t stream, unsigned* tag_seq) {
  if (ws) {
    *ws->seq = (*ws->seq + 1) & 0xFFFFu;
    if (*ws->seq == 0) {
      const size_t words = (ws->bytes - ws_exchange_offset) / 8;
      HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(ws->base + ws_exchange_offset), words,
                                      stream),
              "clear(scratch)");
      *ws->seq = 1;
    }
    *tag_seq = *ws->seq;
    return APPROX_LSTM_OK;
  }
  m->seq = (m->seq + 1) & 0xFFFFu;
  if (m->seq == 0) {
    HIP_TRY(alstm::launch_clear_u64(m->d_zx, m->zx_cap, stream), "clear(zx)");
    HIP_TRY(alstm::launch_clear_u64(m->d_hx, m->hx_cap, stream), "clear(hx)");
    if (m->d_hflag)
      HIP_TRY(alstm::launch_clear_u64(reinterpret_cast<unsigned long long*>(m->d_hflag), m->hflag_cap / 2, stream),
              "clear(hflag)");
    m->seq = 1;
  }
  *tag_seq = m->seq;
  return APPROX_LSTM_OK;
}

approx_lstm_status ensure_stamps(approx_lstm_model* m, int T, hipStream_t stream) {
  const size_t words = 4 + 4 * (size_t)T;
  if (words > m->stamps_cap) {
    HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
    dfree(m->d_stamps);
    m->stamps_cap = 0;
    HIP_TRY(hipMalloc(&m->d_stamps, words * 8), "hipMalloc(stamps)");
    m->stamps_cap = words;
  }
  m->last_T = T;
  return APPROX_LSTM_OK;
}

// Plan of a one-pair run (one level, one sequence, K >= 1): P > 0 when the
// one-pair kernel takes it.
int plan_pair_run(const approx_lstm_model* m, alstm::PairArgs& pa, int T, int K, int num_cu, size_t* lds) {
  pa = alstm::PairArgs{};
  pa.D = m->D; pa.H = m->H; pa.G = m->G; pa.N = m->N; pa.NZ = m->NZ; pa.T = T;
  pa.K = K; pa.GK = m->G * K;
  pa.hcap = m->hpre[pa.GK - 1];
  return alstm::plan_pair(pa, num_cu, m->launch_blocks, lds);
}

// One (level, sequence) pair on the one-pair kernel (P workgroups from
// plan_pair_run): input projection, then the recurrence.
approx_lstm_status run_pair(approx_lstm_model* m, alstm::PairArgs& pa, int P, const float* x, int32_t T,
                            const float* h0, const float* c0, float* h_out, float* c_out, hipStream_t stream,
                            const CallerScratch* ws) {
  const size_t px_floats = (size_t)pa.GK * T, zx_words = (size_t)P * pa.OM, hx_words = round_up(m->H, 4);
  size_t exch_off = 0;
  float* pxw = nullptr;   // x-part projections: written by the input projection, read by the recurrence
  if (ws) {
    const ScratchLayout sl = scratch_layout(px_floats, zx_words, hx_words, 0, 0);
    if (sl.total > ws->bytes)
      return fail(APPROX_LSTM_ERR_UNSUPPORTED,
                  "run needs %zu bytes of workspace, above the %zu-byte static scratch of the allocation-free entry "
                  "point (T=%d, B=1, G*K=%d)",
                  sl.total, ws->bytes, T, pa.GK);
    pa.zx = reinterpret_cast<unsigned long long*>(ws->base + sl.zx);
    pa.hx = reinterpret_cast<unsigned long long*>(ws->base + sl.hx);
    pxw = reinterpret_cast<float*>(ws->base + sl.px);
    exch_off = sl.zx;
  } else {
    approx_lstm_status st = ensure_workspace(m, px_floats, zx_words, hx_words, stream);
    if (st != APPROX_LSTM_OK) return st;
    pa.zx = m->d_zx; pa.hx = m->d_hx; pxw = m->d_px;
  }
  pa.px = pxw;
  unsigned tag_seq = 0;
  approx_lstm_status st = next_tag(m, ws, exch_off, stream, &tag_seq);
  if (st != APPROX_LSTM_OK) return st;
  pa.tag_base = tag_seq << 16;
  pa.stamps = nullptr;
  if (m->timing && !ws) {
    st = ensure_stamps(m, T, stream);
    if (st != APPROX_LSTM_OK) return st;
    pa.stamps = m->d_stamps;
  }
  pa.h0 = h0; pa.c0 = c0; pa.h_out = h_out; pa.c_out = c_out;
  pa.sigma = m->d_sigma; pa.Ut = m->d_Ut; pa.vidx = m->d_vidx; pa.vval = m->d_vval; pa.nx = m->d_nx;
  pa.bias = m->d_bias; pa.err = m->d_err;
  alstm::RunArgs proj{};
  proj.x = x; proj.D = m->D; proj.NZ = m->NZ; proj.T = T; proj.B = 1; proj.GK = pa.GK;
  proj.vidx = m->d_vidx; proj.vval = m->d_vval; proj.nx = m->d_nx; proj.px = pxw;
  proj.xvec = (m->D % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0) ? 1 : 0;
  proj.num_cu = m->num_cu;
  HIP_TRY(alstm::launch_pair(proj, pa, P, stream), "launch pair_lstm_kernel");
  return APPROX_LSTM_OK;
}

// The fp32 progressive run (argument checks done by the caller): fixed
// levels, or with `on` one online level sized for kmax.  With `ws` the
// workspace is carved from the caller's region (nothing is allocated; no
// timing stamps), otherwise it is the model's own, grown on demand.
approx_lstm_status run_progressive(approx_lstm_model* m, const float* x, int32_t T, int32_t B, const float* h0,
                                   const float* c0, const int32_t* levels, int32_t n_levels, int kmax, float* h_out,
                                   float* c_out, hipStream_t stream, const OnlineCfg* on,
                                   const CallerScratch* ws = nullptr) {
  if (on && ws) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "online runs need the model's own workspace");
  if (!on && n_levels == 1 && B == 1 && kmax > 0 && m->recurrence == 0 && !m->cooperative) {
    alstm::PairArgs pa{};
    size_t plds = 0;
    const int Pp = plan_pair_run(m, pa, T, kmax, m->num_cu, &plds);
    if (Pp > 0) return run_pair(m, pa, Pp, x, T, h0, c0, h_out, c_out, stream, ws);
  }
  alstm::RunArgs a{};
  int P = 1;
  const size_t lds = plan_run(m, a, T, B, levels, n_levels, kmax, on, m->num_cu, &P);
  const size_t LB = (size_t)n_levels * B;
  if (lds > alstm::kLdsCap)
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "LDS need %zu bytes exceeds 160 KiB (H=%d, levels*B=%zu, G*K=%d)",
                lds, m->H, LB, a.GK);

  const size_t kword = on ? 1 : 0;   // K_t of an online run rides with h
  // h words per step parity (tagged words in hx, floats in the bulk hbx)
  a.hb_stride = (int)round_up(LB * m->H + kword, 4);
  a.bulk_h = alstm::use_bulk_h(n_levels, B, m->H);
  const size_t px_floats = std::max<size_t>(1, (size_t)a.GK * T * B);
  // z words, then (K-tiled phase B) the y words of every pair's gate rows
  const size_t zx_words = std::max<size_t>(1, LB * P * a.owned_max + (a.ktile > 0 ? LB * 4 * (size_t)m->H : 0));
  const size_t hx_words = 2 * (size_t)a.hb_stride;
  unsigned tag_seq = 0;
  size_t exch_off = 0;
  if (ws) {
    const ScratchLayout sl = scratch_layout(px_floats, zx_words, hx_words, a.bulk_h ? hx_words : 0, (size_t)P);
    if (sl.total > ws->bytes)
      return fail(APPROX_LSTM_ERR_UNSUPPORTED,
                  "run needs %zu bytes of workspace, above the %zu-byte static scratch of the allocation-free entry "
                  "point (T=%d, B=%d, levels=%d, G*K=%d)",
                  sl.total, ws->bytes, T, B, n_levels, a.GK);
    a.px = reinterpret_cast<float*>(ws->base + sl.px);
    a.zx = reinterpret_cast<unsigned long long*>(ws->base + sl.zx);
    a.hx = reinterpret_cast<unsigned long long*>(ws->base + sl.hx);
    a.hbx = a.bulk_h ? reinterpret_cast<float*>(ws->base + sl.hbx) : nullptr;
    a.hflag = a.bulk_h ? reinterpret_cast<unsigned*>(ws->base + sl.hflag) : nullptr;
    exch_off = sl.zx;
  } else {
    approx_lstm_status st = ensure_workspace(m, px_floats, zx_words, hx_words, stream);
    if (st != APPROX_LSTM_OK) return st;
    if (a.bulk_h) {
      st = ensure_bulk(m, hx_words, stream);
      if (st != APPROX_LSTM_OK) return st;
    }
    a.px = m->d_px; a.zx = m->d_zx; a.hx = m->d_hx;
    a.hbx = a.bulk_h ? m->d_hbx : nullptr;
    a.hflag = a.bulk_h ? m->d_hflag : nullptr;
  }
  {
    approx_lstm_status st = next_tag(m, ws, exch_off, stream, &tag_seq);
    if (st != APPROX_LSTM_OK) return st;
  }
  a.tag_base = tag_seq << 16;
  a.x = x; a.h0 = h0; a.c0 = c0; a.h_out = h_out; a.c_out = c_out;
  a.xvec = (m->D % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0) ? 1 : 0;
  a.sigma = m->d_sigma; a.Ut = m->d_Ut; a.vidx = m->d_vidx; a.vval = m->d_vval; a.nx = m->d_nx;
  a.bias = m->d_bias; a.err = m->d_err;
  a.stamps = nullptr;
  if (m->timing && !ws) {
    approx_lstm_status st = ensure_stamps(m, T, stream);
    if (st != APPROX_LSTM_OK) return st;
    a.stamps = m->d_stamps;
  }
  if (on) {
    if ((size_t)T > m->kt_cap) {
      HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
      dfree(m->d_kt);
      m->kt_cap = 0;
      HIP_TRY(hipMalloc(&m->d_kt, (size_t)T * sizeof(int)), "hipMalloc(kt)");
      m->kt_cap = T;
    }
    a.kt = m->d_kt;
  }
  HIP_TRY(alstm::launch_progressive(a, P, m->cooperative, stream), "launch progressive_lstm_kernel");
  return APPROX_LSTM_OK;
}

}  // namespace

// Workspace of approx_lstm_run_noalloc (callers that cannot allocate): one
// array on every device the library runs on, held until the process ends.
// In host code this name is only a host-side stand-in: the array's device
// address is taken once per device with hipGetSymbolAddress and only that
// address is used (kernel arguments, fills).  Every call on a device shares
// its array, which keeps the last call's contents.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
struct ScratchSlot {
  unsigned char* ptr = nullptr;   // device address of `scratch` on this device
  unsigned seq = 0;               // launch tags of the calls using it
};
std::mutex g_scratch_mu;
ScratchSlot g_scratch_slot[kMaxScratchDevices];

}  // namespace

extern "C" {

const char* approx_lstm_last_error(void) { return g_last_error.c_str(); }

approx_lstm_status approx_lstm_prepare(const float* w_ih, const float* w_hh, const float* bias,
                                       const approx_lstm_prepare_params* p, void* hip_stream,
                                       approx_lstm_model** out) {
  g_last_error.clear();
  if (!w_ih || !w_hh || !p || !out) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null pointer argument");
  const int D = p->input_size, H = p->hidden_size;
  if (D < 1 || H < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "input_size and hidden_size must be >= 1");
  const long long Cll = (long long)D + H;
  if (Cll > 65535) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "D + H = %lld exceeds 65535", Cll);
  const int C = (int)Cll;
  if (p->groups != 1 && p->groups != 4) return fail(APPROX_LSTM_ERR_INVALID_ARG, "groups must be 1 or 4");
  if (p->rank < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "rank must be >= 1");
  if (p->factor_dtype != 0 && p->factor_dtype != 1)
    return fail(APPROX_LSTM_ERR_INVALID_ARG, "factor_dtype must be 0 (fp32) or 1 (bf16)");
  int nz = p->nz;
  if (nz == 0) {
    if (!(p->prune_ratio >= 0.0 && p->prune_ratio < 1.0))
      return fail(APPROX_LSTM_ERR_INVALID_ARG, "prune_ratio must be in [0, 1)");
    nz = C - (int)std::floor(p->prune_ratio * (double)C);
  }
  if (nz < 1 || nz > C) return fail(APPROX_LSTM_ERR_INVALID_ARG, "nz = %d not in [1, %d]", nz, C);
  const bool host_only = (p->flags & APPROX_LSTM_FLAG_HOST_ONLY) != 0;
  const bool keep = (p->flags & APPROX_LSTM_FLAG_KEEP_UNPRUNED) != 0;
  const bool on_device = (p->flags & APPROX_LSTM_FLAG_DEVICE_FACTORISE) != 0;
  if (host_only && on_device)
    return fail(APPROX_LSTM_ERR_INVALID_ARG, "DEVICE_FACTORISE and HOST_ONLY exclude each other");

  approx_lstm_model* m = new (std::nothrow) approx_lstm_model();
  if (!m) return fail(APPROX_LSTM_ERR_OUT_OF_MEMORY, "host allocation failed");
  const int G = p->groups, Rg = 4 * H / G, N = p->rank;
  m->D = D; m->H = H; m->C = C; m->G = G; m->Rg = Rg; m->N = N; m->NZ = nz; m->flags = p->flags;
  m->dtype = p->factor_dtype;

  std::vector<alstm::GroupFactors> gf(G);
  try {
    std::vector<double> W((size_t)4 * H * C);
    for (int o = 0; o < 4 * H; ++o) {
      for (int k = 0; k < D; ++k) W[(size_t)o * C + k] = w_ih[(size_t)o * D + k];
      for (int k = 0; k < H; ++k) W[(size_t)o * C + D + k] = w_hh[(size_t)o * H + k];
    }
    alstm::FactoriseOptions opt;
    opt.keep_unpruned = keep;
    opt.residual = (p->flags & APPROX_LSTM_FLAG_NON_RESIDUAL) == 0;
    // groups run on their own threads; the host's thread budget (OMP_NUM_THREADS
    // when set, else the hardware's) is split over the row loops of the groups
    unsigned hw = std::max(1u, std::thread::hardware_concurrency());
    if (const char* env = std::getenv("OMP_NUM_THREADS")) {
      const long v = std::strtol(env, nullptr, 10);
      if (v > 0) hw = std::min<unsigned>(hw, (unsigned)v);
    }
    opt.threads = std::max(1, (int)(hw / (unsigned)G));
    if (on_device) {
      std::string err;
      if (alstm::factorise_groups_device(W.data(), G, Rg, C, N, nz, opt, gf, hip_stream, &err) < 0) {
        delete m;
        return fail(APPROX_LSTM_ERR_DEVICE, "device factorisation: %s", err.c_str());
      }
    } else {
      std::vector<std::thread> th;
      for (int g = 0; g < G; ++g)
        th.emplace_back([&, g] { alstm::factorise_group(&W[(size_t)g * Rg * C], Rg, C, N, nz, opt, gf[g]); });
      for (auto& t : th) t.join();
    }

    m->sigma.assign((size_t)G * N, 0.f);
    m->u.assign((size_t)G * N * Rg, 0.f);
    m->vidx.assign((size_t)G * N * nz, 0);
    m->vval.assign((size_t)G * N * nz, 0.f);
    m->bias.assign((size_t)4 * H, 0.f);
    if (bias) std::copy(bias, bias + 4 * H, m->bias.begin());
    if (keep) {
      m->sigma64.assign((size_t)G * N, 0.0);
      m->u64.assign((size_t)G * N * Rg, 0.0);
      m->v64.assign((size_t)G * N * C, 0.0);
    }
    // stored values: fp32 (nearest even), or bf16 via fp32; sigma is fp32 in
    // both, and the masks were decided in fp64 before any rounding
    const bool bf = m->dtype == 1;
    auto store = [bf](double v) { return bf ? round_bf16(v) : (float)v; };
    for (int g = 0; g < G; ++g) {
      m->eff_rank[g] = gf[g].eff_rank;
      m->unconverged += gf[g].unconverged;
      for (int n = 0; n < N; ++n) {
        m->sigma[(size_t)g * N + n] = (float)gf[g].sigma[n];
        for (int r = 0; r < Rg; ++r) m->u[((size_t)g * N + n) * Rg + r] = store(gf[g].u[(size_t)n * Rg + r]);
        for (int e = 0; e < nz; ++e) {
          m->vidx[((size_t)g * N + n) * nz + e] = gf[g].mask[(size_t)n * nz + e];
          m->vval[((size_t)g * N + n) * nz + e] = store(gf[g].vals[(size_t)n * nz + e]);
        }
      }
      if (keep) {
        std::copy(gf[g].sigma.begin(), gf[g].sigma.end(), m->sigma64.begin() + (size_t)g * N);
        std::copy(gf[g].u.begin(), gf[g].u.end(), m->u64.begin() + (size_t)g * N * Rg);
        std::copy(gf[g].v.begin(), gf[g].v.end(), m->v64.begin() + (size_t)g * N * C);
      }
    }
  } catch (const std::bad_alloc&) {
    delete m;
    return fail(APPROX_LSTM_ERR_OUT_OF_MEMORY, "host allocation failed during factorisation");
  } catch (const std::exception& ex) {
    delete m;
    return fail(APPROX_LSTM_ERR_DEVICE, "factorisation failed: %s", ex.what());
  }

  {
    // h-part entry counts (entries of prune(v) at columns >= D), running
    // maximum over the terms in refinement order: sizes the launch plan
    const size_t NT = (size_t)N * G;
    m->hpre.resize(NT);
    for (size_t tau = 0; tau < NT; ++tau) {
      const size_t src = (tau % G) * N + tau / G;
      int h = 0;
      for (int e = 0; e < nz; ++e) h += m->vidx[src * nz + e] >= D ? 1 : 0;
      m->hpre[tau] = tau ? std::max(m->hpre[tau - 1], h) : h;
    }
  }
  if (!host_only) {
    // Pack the device store: term tau = n*G + g in refinement order.
    const size_t NT = (size_t)N * G;
    std::vector<float> s_h(NT), Ut_h((size_t)4 * H * N), vv_h(NT * nz);
    std::vector<uint16_t> vi_h(NT * nz), nx_h(NT);
    for (int n = 0; n < N; ++n)
      for (int g = 0; g < G; ++g) {
        const size_t tau = (size_t)n * G + g, src = (size_t)g * N + n;
        s_h[tau] = m->sigma[src];
        int cnt = 0;
        for (int e = 0; e < nz; ++e) {
          const int32_t k = m->vidx[src * nz + e];
          vi_h[tau * nz + e] = (uint16_t)k;
          vv_h[tau * nz + e] = m->vval[src * nz + e];
          cnt += (k < D) ? 1 : 0;
        }
        nx_h[tau] = (uint16_t)cnt;
      }
    for (int o = 0; o < 4 * H; ++o) {
      const int g = o / Rg, r = o % Rg;
      for (int n = 0; n < N; ++n) Ut_h[(size_t)o * N + n] = m->u[((size_t)g * N + n) * Rg + r];
    }
    // bf16 models: dense zero-filled panels (x-part and h-part of every v,
    // U with the term index contiguous), padded for the MFMA tiles
    std::vector<uint16_t> vx16, vh16, ut16;
    const bool bf = m->dtype == 1;
    if (bf) {
      m->Dp = (int)round_up(D, alstm::kPanelDAlign);
      m->Hp = (int)round_up(H, alstm::kPanelAlign);
      m->Kp = (int)round_up(N, alstm::kPanelAlign);
      m->prow = (int)round_up((size_t)G * m->Kp, alstm::kPanelRowAlign);
      vx16.assign((size_t)m->prow * m->Dp, 0);
      vh16.assign((size_t)m->prow * m->Hp, 0);
      ut16.assign((size_t)4 * H * m->Kp, 0);
      for (size_t tau = 0; tau < NT; ++tau)
        for (int e = 0; e < nz; ++e) {
          const int k = vi_h[tau * nz + e];
          const uint16_t bits = bf16_bits_of(vv_h[tau * nz + e]);
          if (k < D) vx16[tau * m->Dp + k] = bits;
          else vh16[tau * m->Hp + (k - D)] = bits;
        }
      for (int o = 0; o < 4 * H; ++o)
        for (int n = 0; n < N; ++n) ut16[(size_t)o * m->Kp + n] = bf16_bits_of(Ut_h[(size_t)o * N + n]);
    }
    approx_lstm_status st = APPROX_LSTM_OK;
    auto step = [&](hipError_t e, const char* what) {
      if (st == APPROX_LSTM_OK && e != hipSuccess) st = hip_fail(e, what);
    };
    hipStream_t stream = (hipStream_t)hip_stream;
    step(hipGetDevice(&m->device), "hipGetDevice");
    if (st == APPROX_LSTM_OK) {
      hipDeviceProp_t prop;
      step(hipGetDeviceProperties(&prop, m->device), "hipGetDeviceProperties");
      m->num_cu = prop.multiProcessorCount;
    }
    m->has_dev = true;
    auto up = [&](auto*& dst, const void* src, size_t bytes, const char* what) {
      step(hipMalloc(&dst, bytes), what);
      if (st == APPROX_LSTM_OK) step(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, stream), what);
      m->dev_bytes += bytes;
    };
    up(m->d_sigma, s_h.data(), NT * 4, "sigma");
    up(m->d_bias, m->bias.data(), (size_t)4 * H * 4, "bias");
    if (bf) {
      up(m->d_Vx, vx16.data(), vx16.size() * 2, "Vx panel");
      up(m->d_Vh, vh16.data(), vh16.size() * 2, "Vh panel");
      up(m->d_Ut16, ut16.data(), ut16.size() * 2, "U panel");
    } else {
      up(m->d_Ut, Ut_h.data(), Ut_h.size() * 4, "Ut");
      up(m->d_vval, vv_h.data(), vv_h.size() * 4, "vval");
      up(m->d_vidx, vi_h.data(), vi_h.size() * 2, "vidx");
      up(m->d_nx, nx_h.data(), NT * 2, "nx");
    }
    // the device-side error word, cleared once here: runs (including those
    // that may not allocate) only set it, approx_lstm_check reads and clears it
    if (st == APPROX_LSTM_OK) step(hipMalloc(&m->d_err, 64), "hipMalloc(err)");
    if (st == APPROX_LSTM_OK) step(hipMemsetAsync(m->d_err, 0, 64, stream), "clear(err)");
    if (st == APPROX_LSTM_OK) step(hipStreamSynchronize(stream), "hipStreamSynchronize");
    if (st != APPROX_LSTM_OK) {
      delete m;
      return st;
    }
  }
  *out = m;
  if (m->unconverged)
    return fail(APPROX_LSTM_ERR_NOT_CONVERGED, "%d top-triplet solves missed tolerance", m->unconverged);
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_reserve(approx_lstm_model* m, int32_t T_max, int32_t B_max, int32_t L_max) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (!m->has_dev) return fail(APPROX_LSTM_ERR_INVALID_ARG, "model has no device store (HOST_ONLY)");
  if (T_max < 1 || B_max < 1 || L_max < 1 || L_max > APPROX_LSTM_MAX_LEVELS)
    return fail(APPROX_LSTM_ERR_INVALID_ARG, "reserve sizes out of range");
  DeviceScope ds(m->device);
  if (!ds.ok) return fail(APPROX_LSTM_ERR_DEVICE, "cannot select the model's device");
  approx_lstm_status st;
  if (m->dtype == 1) {
    st = ensure_batched(m, T_max, round_up((size_t)B_max, alstm::kBatchAlign), m->N, nullptr);
    if (st != APPROX_LSTM_OK) return st;
    HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize");
    return APPROX_LSTM_OK;
  }
  const size_t GK = (size_t)m->G * m->N, LB = (size_t)L_max * B_max;
  const size_t P_max = std::max(1, m->num_cu);
  // h exchange: two step-parity halves of L*B*H words plus an online run's K word
  const size_t hhalf = round_up(LB * m->H + 1, 4);
  st = ensure_workspace(m, GK * T_max * B_max, LB * (GK + P_max), 2 * hhalf, nullptr);
  if (st == APPROX_LSTM_OK && alstm::use_bulk_h(L_max, B_max, m->H))
    st = ensure_bulk(m, 2 * hhalf, nullptr);
  if (st != APPROX_LSTM_OK) return st;
  HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize");
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_run(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                   const float* h0, const float* c0, const int32_t* levels,
                                   int32_t n_levels, float* h_out, float* c_out, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (!m->has_dev) return fail(APPROX_LSTM_ERR_INVALID_ARG, "model has no device store (HOST_ONLY)");
  if (T < 0 || B < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "need T >= 0 and B >= 1");
  if (T > 65534) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "T = %d exceeds 65534", T);
  if (!levels || n_levels < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "need at least one level");
  if (n_levels > APPROX_LSTM_MAX_LEVELS)
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "at most %d levels per run", APPROX_LSTM_MAX_LEVELS);
  int kmax = 0;
  for (int l = 0; l < n_levels; ++l) {
    if (levels[l] < 0 || levels[l] > m->N)
      return fail(APPROX_LSTM_ERR_INVALID_ARG, "level %d: K = %d not in [0, %d]", l, levels[l], m->N);
    kmax = std::max(kmax, (int)levels[l]);
  }
  if (T == 0) return APPROX_LSTM_OK;
  if (!x || !h_out) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null x or h_out");

  DeviceScope ds(m->device);
  if (!ds.ok) return fail(APPROX_LSTM_ERR_DEVICE, "cannot select the model's device");
  hipStream_t stream = (hipStream_t)hip_stream;
  if (m->dtype == 1) return run_batched(m, x, T, B, h0, c0, levels, n_levels, h_out, c_out, stream);

  return run_progressive(m, x, T, B, h0, c0, levels, n_levels, kmax, h_out, c_out, stream, nullptr);
}

approx_lstm_status approx_lstm_run_noalloc(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                           const float* h0, const float* c0, const int32_t* levels,
                                           int32_t n_levels, float* h_out, float* c_out, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (!m->has_dev) return fail(APPROX_LSTM_ERR_INVALID_ARG, "model has no device store (HOST_ONLY)");
  if (m->dtype != 0) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "the allocation-free run takes fp32 models only");
  if (T < 0 || B < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "need T >= 0 and B >= 1");
  if (T > 65534) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "T = %d exceeds 65534", T);
  if (!levels || n_levels < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "need at least one level");
  if (n_levels > APPROX_LSTM_MAX_LEVELS)
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "at most %d levels per run", APPROX_LSTM_MAX_LEVELS);
  int kmax = 0;
  for (int l = 0; l < n_levels; ++l) {
    if (levels[l] < 0 || levels[l] > m->N)
      return fail(APPROX_LSTM_ERR_INVALID_ARG, "level %d: K = %d not in [0, %d]", l, levels[l], m->N);
    kmax = std::max(kmax, (int)levels[l]);
  }
  if (T == 0) return APPROX_LSTM_OK;
  if (!x || !h_out) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null x or h_out");
  if (m->device < 0 || m->device >= kMaxScratchDevices)
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "device %d beyond the %d the scratch registry holds", m->device,
                kMaxScratchDevices);
  DeviceScope ds(m->device);
  if (!ds.ok) return fail(APPROX_LSTM_ERR_DEVICE, "cannot select the model's device");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  ScratchSlot& slot = g_scratch_slot[m->device];
  if (!slot.ptr) {
    // first call on this device (current): the array's address on it
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(APPROX_LSTM_ERR_DEVICE, "hipGetSymbolAddress(scratch) returned null");
    slot.ptr = static_cast<unsigned char*>(p);
  }
  const CallerScratch ws{slot.ptr, kScratchBytes, &slot.seq};
  return run_progressive(m, x, T, B, h0, c0, levels, n_levels, kmax, h_out, c_out, (hipStream_t)hip_stream,
                         nullptr, &ws);
}

approx_lstm_status approx_lstm_run_stack(approx_lstm_model* const* layers, int32_t n_layers, const float* x, int32_t T,
                                         int32_t B, const int32_t* levels, int32_t n_levels, float* h_out,
                                         void* hip_stream) {
  g_last_error.clear();
  if (!layers || n_layers < 1 || !levels || n_levels < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "bad arguments");
  if (n_levels > APPROX_LSTM_MAX_LEVELS)
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "at most %d levels per run", APPROX_LSTM_MAX_LEVELS);
  if (T < 0 || B < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "need T >= 0 and B >= 1");
  for (int l = 0; l < n_layers; ++l) {
    if (!layers[l] || !layers[l]->has_dev) return fail(APPROX_LSTM_ERR_INVALID_ARG, "layer %d has no device store", l);
    if (l > 0 && layers[l]->D != layers[l - 1]->H)
      return fail(APPROX_LSTM_ERR_INVALID_ARG, "layer %d input size %d != layer %d hidden size %d", l, layers[l]->D,
                  l - 1, layers[l - 1]->H);
    if (layers[l]->device != layers[0]->device) return fail(APPROX_LSTM_ERR_INVALID_ARG, "layers on different devices");
    for (int j = 0; j < n_levels; ++j) {
      const int K = levels[(size_t)j * n_layers + l];
      if (K < 0 || K > layers[l]->N)
        return fail(APPROX_LSTM_ERR_INVALID_ARG, "level %d layer %d: K = %d not in [0, %d]", j, l, K, layers[l]->N);
    }
  }
  if (T == 0) return APPROX_LSTM_OK;
  if (!x || !h_out) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null x or h_out");
  if (n_layers == 1) {
    std::vector<int32_t> lv(n_levels);
    for (int j = 0; j < n_levels; ++j) lv[j] = levels[j];
    return approx_lstm_run(layers[0], x, T, B, nullptr, nullptr, lv.data(), n_levels, h_out, nullptr, hip_stream);
  }
  approx_lstm_model* m0 = layers[0];
  DeviceScope ds(m0->device);
  if (!ds.ok) return fail(APPROX_LSTM_ERR_DEVICE, "cannot select the model's device");
  hipStream_t stream = (hipStream_t)hip_stream;
  // two ping-pong buffers of [n_levels][T][B][H] for the intermediate layers
  size_t hmax = 0;
  for (int l = 0; l + 1 < n_layers; ++l) hmax = std::max(hmax, (size_t)layers[l]->H);
  const size_t one = (size_t)n_levels * T * B * hmax;
  if (2 * one > m0->stack_cap) {
    HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
    dfree(m0->d_stack);
    m0->stack_cap = 0;
    HIP_TRY(hipMalloc(&m0->d_stack, 2 * one * sizeof(float)), "hipMalloc(stack)");
    m0->stack_cap = 2 * one;
  }
  // layer 0 runs every level at once (they share x); later layers run each
  // level on that level's output of the layer below
  std::vector<int32_t> lv(n_levels);
  for (int j = 0; j < n_levels; ++j) lv[j] = levels[(size_t)j * n_layers];
  float* cur = m0->d_stack;
  approx_lstm_status st = approx_lstm_run(layers[0], x, T, B, nullptr, nullptr, lv.data(), n_levels, cur, nullptr,
                                          hip_stream);
  if (st != APPROX_LSTM_OK) return st;
  for (int l = 1; l < n_layers; ++l) {
    const bool last = l + 1 == n_layers;
    float* nxt = last ? h_out : (cur == m0->d_stack ? m0->d_stack + one : m0->d_stack);
    const size_t in_sz = (size_t)T * B * layers[l - 1]->H, out_sz = (size_t)T * B * layers[l]->H;
    for (int j = 0; j < n_levels; ++j) {
      const int32_t K = levels[(size_t)j * n_layers + l];
      st = approx_lstm_run(layers[l], cur + j * in_sz, T, B, nullptr, nullptr, &K, 1, nxt + j * out_sz, nullptr,
                           hip_stream);
      if (st != APPROX_LSTM_OK) return st;
    }
    cur = nxt;
  }
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_check(approx_lstm_model* m, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (!m->has_dev) return APPROX_LSTM_OK;
  DeviceScope ds(m->device);
  hipStream_t stream = (hipStream_t)hip_stream;
  HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
  if (!m->d_err) return APPROX_LSTM_OK;
  unsigned flag = 0;
  HIP_TRY(hipMemcpy(&flag, m->d_err, sizeof flag, hipMemcpyDeviceToHost), "read error flag");
  if (flag) {
    HIP_TRY(hipMemset(m->d_err, 0, sizeof flag), "clear error flag");
    return fail(APPROX_LSTM_ERR_DEVICE, "a device-side exchange wait exceeded its spin limit");
  }
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_set_launch(approx_lstm_model* m, int32_t blocks, int32_t cooperative) {
  g_last_error.clear();
  if (!m || blocks < 0) return fail(APPROX_LSTM_ERR_INVALID_ARG, "bad arguments");
  m->launch_blocks = blocks;
  m->cooperative = cooperative ? 1 : 0;
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_set_recurrence(approx_lstm_model* m, int32_t kernel) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (kernel < 0 || kernel > 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "kernel must be 0 or 1");
  m->recurrence = kernel;
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_set_batched_path(approx_lstm_model* m, int32_t persistent) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (persistent < 0 || persistent > 3) return fail(APPROX_LSTM_ERR_INVALID_ARG, "persistent must be 0..3");
  m->batched_persistent = persistent;
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_set_timing(approx_lstm_model* m, int32_t enable) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  m->timing = enable ? 1 : 0;
  return APPROX_LSTM_OK;
}

namespace {

// Mean in-kernel microseconds per timestep of the last timed run, and the
// per-timestep values (stamp of one timestep's start to the next one's).
approx_lstm_status per_step_us(approx_lstm_model* m, void* hip_stream, int T, std::vector<double>& steps, double* mean) {
  std::vector<double> st(2 + 4 * (size_t)T);
  approx_lstm_status s = approx_lstm_get_timing(m, hip_stream, st.data(), (int32_t)st.size());
  if (s != APPROX_LSTM_OK) return s;
  steps.resize(T);
  double sum = 0.0;
  for (int t = 0; t < T; ++t) {
    const double next = (t + 1 < T) ? st[1 + 4 * (t + 1)] : st[1 + 4 * T];
    steps[t] = next - st[1 + 4 * t];
    sum += steps[t];
  }
  *mean = T > 0 ? sum / T : 0.0;
  return APPROX_LSTM_OK;
}

}  // namespace

approx_lstm_status approx_lstm_run_deadline(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                            const float* h0, const float* c0, double deadline_us_per_step,
                                            float* h_out, int32_t* k_achieved, float* step_us, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (!m->has_dev) return fail(APPROX_LSTM_ERR_INVALID_ARG, "model has no device store (HOST_ONLY)");
  if (T < 1 || B < 1 || !x || !h_out || !k_achieved) return fail(APPROX_LSTM_ERR_INVALID_ARG, "bad arguments");
  if (!(deadline_us_per_step > 0.0)) return fail(APPROX_LSTM_ERR_INVALID_ARG, "deadline must be > 0");
  if (m->dtype != 0) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "deadline mode needs an fp32 model");
  const int saved_timing = m->timing;
  m->timing = 1;
  auto measure = [&](int K, double* mean, std::vector<double>* steps) -> approx_lstm_status {
    approx_lstm_status s = approx_lstm_run(m, x, T, B, h0, c0, &K, 1, h_out, nullptr, hip_stream);
    if (s != APPROX_LSTM_OK) return s;
    std::vector<double> tmp;
    s = per_step_us(m, hip_stream, T, steps ? *steps : tmp, mean);
    if (s != APPROX_LSTM_OK) return s;
    return approx_lstm_check(m, hip_stream);
  };
  approx_lstm_status st = APPROX_LSTM_OK;
  // calibration: K = 0, 1, 2, 4, ..., rank (cached for this T, B and launch width)
  if (m->calib_T != T || m->calib_B != B || m->calib_blocks != m->launch_blocks || m->calib.empty()) {
    m->calib.clear();
    std::vector<int> ks{0};
    for (int k = 1; k < m->N; k *= 2) ks.push_back(k);
    ks.push_back(m->N);
    for (int k : ks) {
      double us = 0.0;
      st = measure(k, &us, nullptr);
      if (st != APPROX_LSTM_OK) break;
      m->calib.emplace_back(k, us);
    }
    if (st != APPROX_LSTM_OK) {
      m->calib.clear();
      m->timing = saved_timing;
      return st;
    }
    m->calib_T = T;
    m->calib_B = B;
    m->calib_blocks = m->launch_blocks;
  }
  // largest calibrated K within the deadline, then bisection towards the next
  // calibrated K with fresh measurements
  int lo = -1, hi = -1;
  for (size_t i = 0; i < m->calib.size(); ++i) {
    if (m->calib[i].second <= deadline_us_per_step) {
      lo = m->calib[i].first;
      hi = (i + 1 < m->calib.size()) ? m->calib[i + 1].first : lo;
    }
  }
  if (lo < 0) {
    m->timing = saved_timing;
    return fail(APPROX_LSTM_ERR_DEADLINE_INFEASIBLE, "K = 0 takes %.3f us per timestep, above %.3f",
                m->calib[0].second, deadline_us_per_step);
  }
  while (hi - lo > 1) {
    const int mid = lo + (hi - lo) / 2;
    double us = 0.0;
    st = measure(mid, &us, nullptr);
    if (st != APPROX_LSTM_OK) {
      m->timing = saved_timing;
      return st;
    }
    if (us <= deadline_us_per_step) lo = mid; else hi = mid;
  }
  std::vector<double> steps;
  double mean = 0.0;
  st = measure(lo, &mean, &steps);
  m->timing = saved_timing;
  if (st != APPROX_LSTM_OK) return st;
  for (int t = 0; t < T; ++t) {
    k_achieved[t] = lo;
    if (step_us) step_us[t] = (float)steps[t];
  }
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_run_anytime(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                           const float* h0, const float* c0, double deadline_us_per_step,
                                           float* h_out, int32_t* k_achieved, float* step_us, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (!m->has_dev) return fail(APPROX_LSTM_ERR_INVALID_ARG, "model has no device store (HOST_ONLY)");
  if (T < 1 || B < 1 || !x || !h_out || !k_achieved) return fail(APPROX_LSTM_ERR_INVALID_ARG, "bad arguments");
  if (T > 65534) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "T = %d exceeds 65534", T);
  if (!(deadline_us_per_step > 0.0)) return fail(APPROX_LSTM_ERR_INVALID_ARG, "deadline must be > 0");
  if (m->dtype != 0) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "anytime mode needs an fp32 model");
  DeviceScope ds(m->device);
  if (!ds.ok) return fail(APPROX_LSTM_ERR_DEVICE, "cannot select the model's device");
  hipStream_t stream = (hipStream_t)hip_stream;
  int khz = 0;
  HIP_TRY(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, m->device), "wall clock rate");
  if (khz <= 0) return fail(APPROX_LSTM_ERR_DEVICE, "device reports no wall clock rate");
  const int32_t full = m->N;
  const int saved_timing = m->timing;
  m->timing = 1;
  auto run_online = [&](const OnlineCfg& cfg, double* mean, std::vector<double>* steps) -> approx_lstm_status {
    approx_lstm_status s = run_progressive(m, x, T, B, h0, c0, &full, 1, full, h_out, nullptr, stream, &cfg);
    if (s != APPROX_LSTM_OK) return s;
    std::vector<double> tmp;
    s = per_step_us(m, hip_stream, T, steps ? *steps : tmp, mean);
    if (s != APPROX_LSTM_OK) return s;
    return approx_lstm_check(m, hip_stream);
  };
  approx_lstm_status st = APPROX_LSTM_OK;
  // calibration inside the online launch: each candidate K forced at every
  // timestep (cached for this T, B and launch width)
  if (m->ocalib_T != T || m->ocalib_B != B || m->ocalib_blocks != m->launch_blocks || m->ocalib.empty()) {
    m->ocalib.clear();
    std::vector<int> ks{0};
    for (int k = 1; k < m->N; k *= 2) ks.push_back(k);
    ks.push_back(m->N);
    while ((int)ks.size() > alstm::kMaxOptions) ks.erase(ks.begin() + 1);   // drop the smallest positive K
    for (int k : ks) {
      OnlineCfg cfg;
      cfg.n = 1;
      cfg.k[0] = k;
      cfg.ticks[0] = 0;
      cfg.budget = 1ull << 40;
      double us = 0.0;
      st = run_online(cfg, &us, nullptr);
      if (st != APPROX_LSTM_OK) break;
      m->ocalib.emplace_back(k, us);
    }
    if (st != APPROX_LSTM_OK) {
      m->ocalib.clear();
      m->timing = saved_timing;
      return st;
    }
    m->ocalib_T = T;
    m->ocalib_B = B;
    m->ocalib_blocks = m->launch_blocks;
  }
  if (m->ocalib[0].second > deadline_us_per_step) {
    m->timing = saved_timing;
    return fail(APPROX_LSTM_ERR_DEADLINE_INFEASIBLE, "K = 0 takes %.3f us per timestep, above %.3f",
                m->ocalib[0].second, deadline_us_per_step);
  }
  OnlineCfg cfg;
  cfg.n = (int)m->ocalib.size();
  for (int i = 0; i < cfg.n; ++i) {
    cfg.k[i] = m->ocalib[i].first;
    cfg.ticks[i] = (unsigned)std::ceil(m->ocalib[i].second * khz / 1000.0);
  }
  cfg.budget = (unsigned long long)std::floor(deadline_us_per_step * khz / 1000.0);
  std::vector<double> steps;
  double mean = 0.0;
  st = run_online(cfg, &mean, &steps);
  m->timing = saved_timing;
  if (st != APPROX_LSTM_OK) return st;
  HIP_TRY(hipMemcpy(k_achieved, m->d_kt, (size_t)T * sizeof(int32_t), hipMemcpyDeviceToHost), "read budgets");
  if (step_us)
    for (int t = 0; t < T; ++t) step_us[t] = (float)steps[t];
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_run_schedule(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                            const float* h0, const float* c0, const int32_t* k_sched, float* h_out,
                                            float* c_out, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (!m->has_dev) return fail(APPROX_LSTM_ERR_INVALID_ARG, "model has no device store (HOST_ONLY)");
  if (T < 1 || B < 1 || !x || !h_out || !k_sched) return fail(APPROX_LSTM_ERR_INVALID_ARG, "bad arguments");
  if (T > 65534) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "T = %d exceeds 65534", T);
  if (m->dtype != 0) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "scheduled runs need an fp32 model");
  int kmax = 0;
  for (int t = 0; t < T; ++t) {
    if (k_sched[t] < 0 || k_sched[t] > m->N)
      return fail(APPROX_LSTM_ERR_INVALID_ARG, "timestep %d: K = %d not in [0, %d]", t, k_sched[t], m->N);
    kmax = std::max(kmax, (int)k_sched[t]);
  }
  DeviceScope ds(m->device);
  if (!ds.ok) return fail(APPROX_LSTM_ERR_DEVICE, "cannot select the model's device");
  hipStream_t stream = (hipStream_t)hip_stream;
  // the schedule goes to the model's budget array (no run may still read it)
  HIP_TRY(hipStreamSynchronize(stream), "hipStreamSynchronize");
  if ((size_t)T > m->kt_cap) {
    dfree(m->d_kt);
    m->kt_cap = 0;
    HIP_TRY(hipMalloc(&m->d_kt, (size_t)T * sizeof(int)), "hipMalloc(kt)");
    m->kt_cap = T;
  }
  HIP_TRY(hipMemcpy(m->d_kt, k_sched, (size_t)T * sizeof(int32_t), hipMemcpyHostToDevice), "copy schedule");
  OnlineCfg cfg;
  cfg.n = 1;
  cfg.k[0] = kmax;
  cfg.ticks[0] = 0;
  cfg.budget = 1ull << 40;
  cfg.sched = m->d_kt;
  return run_progressive(m, x, T, B, h0, c0, &kmax, 1, kmax, h_out, c_out, stream, &cfg);
}

approx_lstm_status approx_lstm_plan(const approx_lstm_model* m, int32_t T, int32_t B, const int32_t* levels,
                                    int32_t n_levels, int32_t online, int32_t num_cu, int32_t* out) {
  g_last_error.clear();
  if (!m || !out || T < 1 || B < 1 || num_cu < 0) return fail(APPROX_LSTM_ERR_INVALID_ARG, "bad arguments");
  if (m->dtype != 0) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "launch plans describe fp32 models");
  int kmax = 0;
  std::vector<int32_t> lv;
  if (online) {
    kmax = m->N;
    lv.push_back(kmax);
  } else {
    if (!levels || n_levels < 1 || n_levels > APPROX_LSTM_MAX_LEVELS)
      return fail(APPROX_LSTM_ERR_INVALID_ARG, "need 1..%d levels", APPROX_LSTM_MAX_LEVELS);
    for (int l = 0; l < n_levels; ++l) {
      if (levels[l] < 0 || levels[l] > m->N)
        return fail(APPROX_LSTM_ERR_INVALID_ARG, "level %d: K = %d not in [0, %d]", l, levels[l], m->N);
      kmax = std::max(kmax, (int)levels[l]);
      lv.push_back(levels[l]);
    }
  }
  const int ncu = num_cu > 0 ? num_cu : m->num_cu;
  for (int i = 0; i < 10; ++i) out[i] = 0;
  if (!online && lv.size() == 1 && B == 1 && kmax > 0 && m->recurrence == 0 && !m->cooperative) {
    alstm::PairArgs pa{};
    size_t plds = 0;
    const int Pp = plan_pair_run(m, pa, T, kmax, ncu, &plds);
    if (Pp > 0) {
      out[0] = Pp;
      out[1] = pa.px_lds;
      out[3] = pa.hpl;
      out[4] = pa.upt;
      out[5] = pa.opt;
      out[7] = (int32_t)plds;
      out[8] = 1;
      return APPROX_LSTM_OK;
    }
  }
  OnlineCfg cfg;
  cfg.n = 1;
  cfg.k[0] = kmax;
  alstm::RunArgs a{};
  int P = 1;
  const size_t lds = plan_run(m, a, T, B, lv.data(), (int)lv.size(), kmax, online ? &cfg : nullptr, ncu, &P);
  out[0] = P;
  out[1] = a.px_all;
  out[2] = a.allpairs;
  out[3] = a.hpl;
  out[4] = a.upt;
  out[5] = a.opt;
  out[6] = alstm::use_bulk_h((int)lv.size(), B, m->H);
  out[7] = (int32_t)std::min<size_t>(lds, 0x7fffffff);
  out[9] = a.ktile;
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_get_timing(approx_lstm_model* m, void* hip_stream, double* stamps_us, int32_t n) {
  g_last_error.clear();
  if (!m || !stamps_us) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null pointer argument");
  if (!m->d_stamps || m->last_T <= 0) return fail(APPROX_LSTM_ERR_INVALID_ARG, "no run recorded timing");
  const int T = m->last_T;
  const int words = 4 + 4 * T;
  if (n < 2 + 4 * T) return fail(APPROX_LSTM_ERR_INVALID_ARG, "need %d slots", 2 + 4 * T);
  DeviceScope ds(m->device);
  HIP_TRY(hipStreamSynchronize((hipStream_t)hip_stream), "hipStreamSynchronize");
  std::vector<unsigned long long> raw(words);
  HIP_TRY(hipMemcpy(raw.data(), m->d_stamps, words * 8, hipMemcpyDeviceToHost), "read stamps");
  int khz = 0;
  HIP_TRY(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, m->device), "wall clock rate");
  if (khz <= 0) return fail(APPROX_LSTM_ERR_DEVICE, "device reports no wall clock rate");
  // shader-clock stamps, converted with the wall-clock span of the same run
  const double wall_us = (double)(long long)(raw[3 + 4 * T] - raw[0]) * 1e3 / khz;
  const double clk = (double)(long long)(raw[2 + 4 * T] - raw[1]);
  const double us_per_clk = clk > 0 ? wall_us / clk : 0.0;
  stamps_us[0] = 0.0;
  for (int i = 0; i < 4 * T; ++i) stamps_us[1 + i] = (double)(long long)(raw[2 + i] - raw[1]) * us_per_clk;
  stamps_us[1 + 4 * T] = (double)(long long)(raw[2 + 4 * T] - raw[1]) * us_per_clk;
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_model_info(const approx_lstm_model* m, approx_lstm_info* out) {
  g_last_error.clear();
  if (!m || !out) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null pointer argument");
  std::memset(out, 0, sizeof *out);
  out->input_size = m->D;
  out->hidden_size = m->H;
  out->aug_size = m->C;
  out->groups = m->G;
  out->rows_per_group = m->Rg;
  out->rank = m->N;
  out->nz = m->NZ;
  for (int g = 0; g < 4; ++g) out->eff_rank[g] = g < m->G ? m->eff_rank[g] : 0;
  out->unconverged_steps = m->unconverged;
  out->has_device_store = m->has_dev ? 1 : 0;
  out->device_bytes = m->dev_bytes;
  out->factor_dtype = m->dtype;
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_get_factors(const approx_lstm_model* m, int32_t group, float* sigma, float* u,
                                           int32_t* v_idx, float* v_val) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (group < 0 || group >= m->G) return fail(APPROX_LSTM_ERR_INVALID_ARG, "group %d out of range", group);
  const size_t N = m->N, Rg = m->Rg, nz = m->NZ;
  if (sigma) std::copy_n(m->sigma.begin() + group * N, N, sigma);
  if (u) std::copy_n(m->u.begin() + group * N * Rg, N * Rg, u);
  if (v_idx) std::copy_n(m->vidx.begin() + group * N * nz, N * nz, v_idx);
  if (v_val) std::copy_n(m->vval.begin() + group * N * nz, N * nz, v_val);
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_get_factors_f64(const approx_lstm_model* m, int32_t group, double* sigma,
                                               double* u, double* v_unpruned) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (group < 0 || group >= m->G) return fail(APPROX_LSTM_ERR_INVALID_ARG, "group %d out of range", group);
  if (m->sigma64.empty()) return fail(APPROX_LSTM_ERR_INVALID_ARG, "prepared without KEEP_UNPRUNED");
  const size_t N = m->N, Rg = m->Rg, C = m->C;
  if (sigma) std::copy_n(m->sigma64.begin() + group * N, N, sigma);
  if (u) std::copy_n(m->u64.begin() + group * N * Rg, N * Rg, u);
  if (v_unpruned) std::copy_n(m->v64.begin() + group * N * C, N * C, v_unpruned);
  return APPROX_LSTM_OK;
}

void approx_lstm_destroy(approx_lstm_model* m) { delete m; }

}  // extern "C"

struct approx_lstm_exact {
  int D = 0, H = 0;
  int device = -1, num_cu = 0;
  float* d_Wx = nullptr;
  float* d_Wh = nullptr;
  float* d_bias = nullptr;
  float* d_px = nullptr;
  size_t px_cap = 0;
  unsigned long long* d_hx = nullptr;
  size_t hx_cap = 0;
  unsigned* d_err = nullptr;
  unsigned seq = 0;
  int launch_blocks = 0;

  ~approx_lstm_exact() {
    if (device < 0) return;
    DeviceScope ds(device);
    dfree(d_Wx);
    dfree(d_Wh);
    dfree(d_bias);
    dfree(d_px);
    dfree(d_hx);
    dfree(d_err);
  }
};

extern "C" {

approx_lstm_status approx_lstm_exact_prepare(const float* w_ih, const float* w_hh, const float* bias,
                                             int32_t input_size, int32_t hidden_size, void* hip_stream,
                                             approx_lstm_exact** out) {
  g_last_error.clear();
  if (!w_ih || !w_hh || !out) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null pointer argument");
  if (input_size < 1 || hidden_size < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "sizes must be >= 1");
  approx_lstm_exact* m = new (std::nothrow) approx_lstm_exact();
  if (!m) return fail(APPROX_LSTM_ERR_OUT_OF_MEMORY, "host allocation failed");
  m->D = input_size;
  m->H = hidden_size;
  const size_t R = 4 * (size_t)m->H;
  std::vector<float> b(R, 0.0f);
  if (bias) std::copy(bias, bias + R, b.begin());
  hipStream_t stream = (hipStream_t)hip_stream;
  approx_lstm_status st = APPROX_LSTM_OK;
  auto step = [&](hipError_t e, const char* what) {
    if (st == APPROX_LSTM_OK && e != hipSuccess) st = hip_fail(e, what);
  };
  step(hipGetDevice(&m->device), "hipGetDevice");
  if (st == APPROX_LSTM_OK) {
    hipDeviceProp_t prop;
    step(hipGetDeviceProperties(&prop, m->device), "hipGetDeviceProperties");
    m->num_cu = prop.multiProcessorCount;
  }
  auto up = [&](float*& dst, const float* src, size_t n, const char* what) {
    step(hipMalloc(&dst, n * 4), what);
    if (st == APPROX_LSTM_OK) step(hipMemcpyAsync(dst, src, n * 4, hipMemcpyHostToDevice, stream), what);
  };
  up(m->d_Wx, w_ih, R * m->D, "W_ih");
  up(m->d_Wh, w_hh, R * m->H, "W_hh");
  up(m->d_bias, b.data(), R, "bias");
  step(hipMalloc(&m->d_err, 64), "hipMalloc(err)");
  if (st == APPROX_LSTM_OK) step(hipMemsetAsync(m->d_err, 0, 64, stream), "clear(err)");
  if (st == APPROX_LSTM_OK) step(hipStreamSynchronize(stream), "hipStreamSynchronize");
  if (st != APPROX_LSTM_OK) {
    delete m;
    return st;
  }
  *out = m;
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_exact_run_rows(approx_lstm_exact* m, const float* x, int32_t T, int32_t B,
                                              const float* h0, const float* c0, int32_t rows, float* h_out,
                                              float* c_out, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  if (T < 0 || B < 1) return fail(APPROX_LSTM_ERR_INVALID_ARG, "need T >= 0 and B >= 1");
  if (rows < 0 || rows > m->H) return fail(APPROX_LSTM_ERR_INVALID_ARG, "rows = %d not in [0, %d]", rows, m->H);
  if (T > 65534) return fail(APPROX_LSTM_ERR_UNSUPPORTED, "T = %d exceeds 65534", T);
  if (T == 0) return APPROX_LSTM_OK;
  if (!x || !h_out) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null x or h_out");
  DeviceScope ds(m->device);
  if (!ds.ok) return fail(APPROX_LSTM_ERR_DEVICE, "cannot select the model's device");
  hipStream_t stream = (hipStream_t)hip_stream;
  alstm::ExactArgs a{};
  a.x = x; a.h0 = h0; a.c0 = c0; a.h_out = h_out; a.c_out = c_out;
  a.Wx = m->d_Wx; a.Wh = m->d_Wh; a.bias = m->d_bias;
  a.D = m->D; a.H = m->H; a.T = T; a.B = B; a.rows = rows;
  a.xvec = (m->D % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0) ? 1 : 0;
  const int maxP = std::max(1, m->num_cu);
  int P = m->launch_blocks > 0 ? std::min(m->launch_blocks, maxP) : std::min(maxP, std::max(1, (m->H + 7) / 8));
  size_t lds = alstm::plan_exact(a, P);
  if (m->launch_blocks == 0)
    while (lds > alstm::kLdsCap && P < maxP) {
      P = std::min(maxP, 2 * P);
      lds = alstm::plan_exact(a, P);
    }
  if (lds > alstm::kLdsCap)
    return fail(APPROX_LSTM_ERR_UNSUPPORTED, "LDS need %zu bytes exceeds 160 KiB (H=%d, B=%d)", lds, m->H, B);
  approx_lstm_status st = grow(m->d_px, m->px_cap, (size_t)T * B * 4 * m->H, stream, "hipMalloc(px)");
  if (st != APPROX_LSTM_OK) return st;
  if ((size_t)B * m->H > m->hx_cap) {
    st = grow(m->d_hx, m->hx_cap, (size_t)B * m->H, stream, "hipMalloc(hx)");
    if (st != APPROX_LSTM_OK) return st;
    HIP_TRY(alstm::launch_clear_u64(m->d_hx, m->hx_cap, stream), "clear(hx)");
    m->seq = 0;
  }
  m->seq = (m->seq + 1) & 0xFFFFu;
  if (m->seq == 0) {
    HIP_TRY(alstm::launch_clear_u64(m->d_hx, m->hx_cap, stream), "clear(hx)");
    m->seq = 1;
  }
  a.tag_base = m->seq << 16;
  a.px = m->d_px; a.hx = m->d_hx; a.err = m->d_err;
  HIP_TRY(alstm::launch_exact(a, P, stream), "launch exact_lstm_kernel");
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_exact_run(approx_lstm_exact* m, const float* x, int32_t T, int32_t B,
                                         const float* h0, const float* c0, float* h_out, float* c_out,
                                         void* hip_stream) {
  if (!m) {
    g_last_error.clear();
    return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  }
  return approx_lstm_exact_run_rows(m, x, T, B, h0, c0, m->H, h_out, c_out, hip_stream);
}

approx_lstm_status approx_lstm_exact_check(approx_lstm_exact* m, void* hip_stream) {
  g_last_error.clear();
  if (!m) return fail(APPROX_LSTM_ERR_INVALID_ARG, "null model");
  DeviceScope ds(m->device);
  HIP_TRY(hipStreamSynchronize((hipStream_t)hip_stream), "hipStreamSynchronize");
  unsigned flag = 0;
  HIP_TRY(hipMemcpy(&flag, m->d_err, sizeof flag, hipMemcpyDeviceToHost), "read error flag");
  if (flag) {
    HIP_TRY(hipMemset(m->d_err, 0, sizeof flag), "clear error flag");
    return fail(APPROX_LSTM_ERR_DEVICE, "a device-side exchange wait exceeded its spin limit");
  }
  return APPROX_LSTM_OK;
}

approx_lstm_status approx_lstm_exact_set_launch(approx_lstm_exact* m, int32_t blocks) {
  g_last_error.clear();
  if (!m || blocks < 0) return fail(APPROX_LSTM_ERR_INVALID_ARG, "bad arguments");
  m->launch_blocks = blocks;
  return APPROX_LSTM_OK;
}

void approx_lstm_exact_destroy(approx_lstm_exact* m) { delete m; }

}  // extern "C"
