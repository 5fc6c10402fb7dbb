// Internal interface between the C-ABI host code and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace alstm {

constexpr int kMaxLevels = 16;
constexpr int kTilePairs = 8;           // sequences of a K-tiled phase B (RunArgs::ktile)
constexpr int kTileEntries = 16;        // U entries per lane and row in one tile of it
constexpr int kTileWords = 16;          // z words per gathering thread in one tile of it
constexpr int kMaxOptions = 24;        // candidate budgets of an online (anytime) run
constexpr int kThreads = 512;          // 8 wave64 per workgroup
constexpr int kMaxXChunk = 16;         // (t, b) pairs accumulated per pass of the input projection
constexpr size_t kLdsCap = 160 * 1024; // LDS per CU on gfx950

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
//   px     [GK][T*B]            x-part projections (workspace, written by input_proj_kernel)
//   zx     [L*B][P][owned_max] u64  tagged z exchange (value | tag << 32), slot
//                                   j*owned_max + i carries term j + i*P
//   hx     [2][hb_stride] u64   tagged h exchange (few values per workgroup): h_t of every
//                                (level, seq) and an online run's K_{t+1} in half t & 1
//   hbx, hflag                  bulk h exchange (many values: large L*B*H)
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
  float* hbx;      // bulk h exchange: [2][hb_stride] floats, h_t of every (level, seq) at
                   // parity t & 1 (agent-coherent stores and loads); null unless bulk_h
  unsigned* hflag; // bulk h exchange: [P] words, workgroup j's tag once its h_t is stored
  unsigned* err;
  unsigned long long* stamps;  // null, or [4 + 4T] stamps written by workgroup 0: [0] wall clock
                               // and [1] shader clock at the start of the recurrence; shader
                               // clock at [2+4t..5+4t], the starts of phase A, the z wait, the
                               // U accumulation and the h wait of timestep t; [2+4T] shader
                               // clock and [3+4T] wall clock at the end
  int D, H, G, N, NZ, T, B, L;
  int GK;          // G * max level: terms in use
  int rows_per;    // hidden units owned per workgroup
  int owned_max;   // max terms owned by one workgroup = ceil(GK / P)
  int hcap;        // slots per owned term for its h-part entries (max over terms of NZ - nx)
  int hpl;         // h-part entries per lane held in registers (0: in LDS, see vh_lds)
  int vh_lds;      // 1: owned terms' h-part entries resident in LDS
  int upt;         // U entries per output row and thread held in registers (0: LDS or global)
  int opt;         // output rows per thread in the register path
  int ustride;     // LDS row stride (floats) of the resident U slice; 0 = U read from global
  int px_all;      // 1: x-part projections of every timestep resident in LDS
  int xvec;        // 1: x rows may be read as 16-byte vectors (D % 4 == 0, x 16-byte aligned)
  int bulk_h;      // 1: h exchanged in bulk (hbx + hflag), 0: as tagged words (hx)
  int allpairs;    // 1: phase B takes every (level, sequence) pair in one pass (z of all
                   //    pairs resident in LDS); 0: one pass per pair
  int ktile;       // > 0 (one level, U read from memory, G = 4, P % 4 == 0): phase B
                   //    reads each U entry once per timestep for every sequence, K in
                   //    tiles of ktile terms of one group whose z of every pair sit in
                   //    LDS; workgroup j accumulates the gate j % 4 rows of its block of
                   //    four workgroups' units, and y travels to the cell owners in
                   //    LB * 4 * H tagged words after the LB * P * owned_max z words
  int hb_stride;   // words per step parity of hx and hbx: L*B*H (+1 online) rounded up to 4
  int P;           // workgroups of the launch
  int num_cu;      // compute units of the device (sizes the input projection's grid)
  int lanes_a;     // lanes per term in phase A (16)
  unsigned tag_base;
  int levels[kMaxLevels];
  int lanes_b[kMaxLevels];  // lanes per output row in phase B, per level (a function of K only)
  // online (anytime) run: one level of up to levels[0] terms whose budget K_t
  // is chosen per timestep on the device.  Workgroup 0 reads the wall clock
  // (100 MHz) at the end of timestep t's gate update and takes the largest
  // option whose predicted timestep still ends by (t+2) * budget ticks after
  // the recurrence began; the choice travels to every workgroup as one more
  // word of the h exchange (slot L*B*H), so all agree on K_{t+1}.
  int online;                       // 0: fixed levels
  int n_opts;                       // options, K ascending
  int opt_k[kMaxOptions];           // candidate budgets
  unsigned opt_ticks[kMaxOptions];  // predicted wall ticks of one timestep at that budget
  unsigned long long budget;        // wall ticks per timestep
  int* kt;                          // [T] chosen budgets (written by workgroup 0)
  const int* sched;                 // null, or device [T]: K_t given by the caller (read by
                                    // workgroup 0 in place of the clock-based choice; every
                                    // other step of an online run unchanged)
};

// Budget of an online run for `avail` wall ticks: the largest option that
// fits, else the smallest.
__host__ __device__ inline int online_pick(const RunArgs& a, long long avail) {
  int k = a.opt_k[0];
  for (int i = 0; i < a.n_opts; ++i)
    if ((long long)a.opt_ticks[i] <= avail) k = a.opt_k[i] > k ? a.opt_k[i] : k;
  return k;
}

// Reduction shapes.  They depend only on the model (phase A) and on each
// level's own budget (phase B), never on the launch width or on the other
// levels of a run, so every result has one fixed summation order.
int lanes_for_terms(int nz, int D, int H);
int lanes_for_level(int K);

// 1 when the h_t of a launch (L*B*H values) is exchanged in bulk: the
// tagged-word gather needs one polling round per 2 values per thread, the
// bulk one a flag round and one 16-byte load per 4 values.
inline int use_bulk_h(int L, int B, int H) { return (long long)L * B * H > 2048 ? 1 : 0; }

// Workgroups along the (t, b) columns of an input projection whose rows take
// `row_groups` workgroups and whose columns come in `chunks` chunks: enough
// for about two workgroups per compute unit, at most one per chunk.
inline int column_slices(int row_groups, int chunks) {
  const int want = (512 + row_groups - 1) / row_groups;
  return want < 1 ? 1 : (want < chunks ? want : (chunks < 1 ? 1 : chunks));
}

// Fills the launch-shape fields (rows_per .. lanes_a) for P workgroups and
// returns the LDS bytes the kernel then needs (> kLdsCap: does not fit).
size_t plan_progressive(RunArgs& a, int P);

// Launches, on `stream`, the x-part projections px[tau][t*B+b] of the first
// a.GK terms (input_proj_kernel over the whole device; nothing when GK = 0).
// Uses a.x, a.T, a.B, a.D, a.NZ, a.GK, a.vidx, a.vval, a.nx, a.px, a.xvec.
hipError_t launch_input_proj(const RunArgs& a, hipStream_t stream);

// One (level, sequence) pair: the recurrence of one budget K over one
// sequence, with every owned slice in registers (pair_lstm_kernel).  The
// summation order of every quantity is that of progressive_lstm_kernel (16
// lanes per term in phase A, lanes_for_level(K) lanes per U row in phase B),
// so both kernels give bitwise the same outputs.  Device pointers:
//   px     [GK][T]              x-part projections (input_proj_kernel, B = 1)
//   zx     [P*OM] u64           tagged z words, slot j*OM + i carries term j + i*P
//   hx     [H] u64              tagged h words
//   h_out  [T][H]               this level's outputs; c_out [H] or null
struct PairArgs {
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
  const float* px;
  unsigned long long* zx;
  unsigned long long* hx;
  unsigned* err;
  unsigned long long* stamps;   // as RunArgs::stamps (workgroup 0), or null
  int D, H, G, N, NZ, T;
  int K;         // budget (terms per group), >= 1
  int GK;        // G * K
  int hcap;      // largest h-part entry count of the terms in use
  // launch plan (plan_pair)
  int OM;        // terms owned per workgroup (at most 32 * apass)
  int RU;        // hidden units owned per workgroup
  int apass;     // phase-A passes of 32 terms (1 or 2)
  int hpl;       // h-part entries per lane held (register bucket: 4, 8, 12, 16, 24, 32)
  int S, lgS;    // lanes per U row (lanes_for_level(K)) and its log2
  int upt;       // U entries per row and lane in use: ceil(K / S)
  int umax;      // U entries per row and lane held (register bucket: 8, 16, 32)
  int opt;       // output rows per thread (1, 2, 4)
  int kstride;   // LDS floats between the terms of consecutive lanes of a row
  int zstride;   // LDS floats per group of z
  int hpad;      // LDS floats of h (H rounded up to 4)
  int px_lds;    // 1: P_x of every timestep staged in LDS (required)
  unsigned tag_base;
};

// Launch shape of a pair run: fills the plan fields and returns the
// workgroup count P (0: the shape does not fit this kernel) for `num_cu`
// compute units, or checks a requested width (`want` > 0).  *lds receives
// the LDS bytes per workgroup.
int plan_pair(PairArgs& a, int num_cu, int want, size_t* lds);

// Launches, on `stream`, the input projection (as launch_progressive) and the
// one-pair recurrence with P workgroups.
hipError_t launch_pair(const RunArgs& proj, const PairArgs& a, int P, hipStream_t stream);

// Launches, on `stream`, the input projection over the whole device and then
// the persistent recurrence kernel with `blocks` workgroups.  cooperative != 0
// uses the cooperative launch API for the latter (co-residency checked by the
// runtime).
hipError_t launch_progressive(const RunArgs& a, int blocks, int cooperative, hipStream_t stream);

// Zero `n` 64-bit words (exchange-buffer reset) with a plain kernel.
hipError_t launch_clear_u64(unsigned long long* p, size_t n, hipStream_t stream);

// Batched bf16 path (many sequences; the factors as zero-filled bf16 panels
// and every product on MFMA with fp32 accumulation).  bf16 arrays are raw
// 16-bit patterns.  Padded sizes: Dp a multiple of 64, Hp of 32, Bp of 64;
// Kp = rank rounded up to 32; panel rows = G*Kp rounded up to 128.
//   x      [T][B][D] fp32           h0, c0 [B][H] fp32 or null
//   h_out  [L][T][B][H]             c_out  [L][B][H] or null
//   sigma  [N*G] fp32               term tau = n*G + g
//   Vx     [rows][Dp] bf16          x-part of prune(v) of term tau (zeros off the mask)
//   Vh     [rows][Hp] bf16          h-part of prune(v) of term tau
//   Ut     [4H][Kp] bf16            Ut[o][n] = u of term (n, g(o)) at row o within its group
//   bias   [4H] fp32
//   P      [T*Bp][pld] fp32         x-part projections: P[t*Bp + b][tau] (workspace)
//   Z      [G][Bp][Kp] bf16         sigma * s of the current timestep (workspace)
//   hb     [Bp][Hp] bf16            h of the previous timestep (workspace)
//   c      [Bp][H] fp32             cell state (workspace)
constexpr int kPanelAlign = 32;      // Hp, Kp granularity (the MFMA contraction step)
constexpr int kPanelDAlign = 64;     // Dp granularity (two x-projection slices)
constexpr int kPanelRowAlign = 128;  // panel row granularity (the x-projection row tile)
constexpr int kBatchAlign = 64;      // Bp granularity

struct BatchedArgs {
  const float* x;
  const float* h0;
  const float* c0;
  float* h_out;
  float* c_out;
  const float* sigma;
  const uint16_t* Vx;
  const uint16_t* Vh;
  const uint16_t* Ut;
  const float* bias;
  float* P;
  uint16_t* Z;
  uint16_t* hb;
  float* c;
  int D, Dp, H, Hp, G, Kp, T, B, Bp;
  int rows;        // panel rows a launch covers (set per launch)
  int pld;         // row count of P: G * (largest level rounded up to 32)
  int xvec;        // 1: x rows may be read as 16-byte vectors (D % 4 == 0, x 16-byte aligned)
  // persistent recurrence (one launch per level instead of T kernel pairs);
  // null zx selects the per-timestep kernels
  uint16_t* zx;      // [slots][2*G*16*Kp] bf16 slots: z of a cohort's current timestep, as
                     // [G*16][Kp] bf16 behind flags or [G*16][Kp/2] tagged 64-bit words
  uint16_t* hx;      // [slots][2*16*Hp]: h of a cohort's current timestep, [16][Hp/2] tagged words
  unsigned* zflag;   // [slots][W]: workgroup w's tag once its (untagged) z tile is stored
  unsigned* err;     // set when a bounded wait expires
  unsigned tag_base; // launch sequence << 16 of level 0; level l uses tag_base + (l << 16)
  int max_wg;        // workgroups that may be resident at once (one per compute unit)
  int ztag_terms;    // z travel as tagged words when G * K (rounded up to 32) <= this
  // x-projection with its contraction over D split in xsplit parts when it
  // has fewer output tiles than the device has compute units: each part's
  // tile goes to Ppart[part] ([T*Bp][pld]), then the parts are added in part
  // order.  The split depends only on the tile count and ncu (not on the
  // launch width), so every result keeps one summation order per shape.
  float* Ppart;      // null: no split
  size_t ppart_cap;  // floats of Ppart
  int ncu;           // compute units of the device
  int xsplit;        // set by launch_batched
};

// Largest split (a power of two, at most 8) that keeps the x-projection's
// tiles times the split within `ncu` workgroups and gives every part an even
// number of contraction slices (of `nslices`).
int batched_xproj_split(int tiles, int ncu, int nslices);
// Floats of Ppart that cover every split batched_xproj_split can choose.
size_t batched_ppart_floats(int ncu);

// Sequences per cohort of the persistent batched recurrence (the MFMA tile width).
constexpr int kCohort = 16;


// Shape of a persistent batched launch at budget K: W workgroups per cohort
// (32 hidden units each), `slots` cohorts in flight.  Returns 0 when the
// shape does not fit (then the per-timestep kernels run): H and K each at
// most 512 (their contraction steps are held in registers), at most one
// h-projection tile of 16 terms per wave, a cohort's workgroups resident at
// once, and fewer than 2^16 tagged timesteps per launch.  Exchange sizes (in
// 16-bit elements): zx slots*2*G*16*Kp, hx slots*2*16*Hp; flags slots*W.
int plan_batched_persistent(const BatchedArgs& a, int K, int* W, int* slots);

// Exact (dense) LSTM: x [T][B][D], h0, c0 [B][H] or null, h_out [T][B][H],
// c_out [B][H] or null; Wx [4H][D], Wh [4H][H], bias [4H] (gate rows i, f,
// g, o); px [T*B][4H] (x part plus bias, workspace); hx [B][H] tagged words.
struct ExactArgs {
  const float* x;
  const float* h0;
  const float* c0;
  float* h_out;
  float* c_out;
  const float* Wx;
  const float* Wh;
  const float* bias;
  float* px;
  unsigned long long* hx;
  unsigned* err;
  int D, H, T, B;
  int rows;        // rows of every gate computed (0..H); later rows hold the bias alone
  int xvec;        // 1: x may be read as 16-byte vectors (x 16-byte aligned, D % 4 == 0)
  int rows_per;    // hidden units per workgroup (set by plan_exact)
  int wreg;        // 1: the first 32 rows of each workgroup keep their W_h entries in registers
  int px_lds;      // 1: x parts of the owned rows for every timestep in LDS
  unsigned tag_base;
};

// Fills rows_per / wreg / px_lds for P workgroups; returns the LDS bytes the
// recurrence kernel needs (> kLdsCap: does not fit).
size_t plan_exact(ExactArgs& a, int P);

// Launches the x projection and the persistent recurrence (`blocks`
// workgroups) on `stream`.
hipError_t launch_exact(const ExactArgs& a, int blocks, hipStream_t stream);

// Launches, on `stream`, the x-projection once and then, for every level,
// either the persistent recurrence (a.zx set and the shape fits) or T pairs
// of per-timestep kernels.  Requires Bp % 64 == 0 and every level K <= Kp.
hipError_t launch_batched(const BatchedArgs& a, const int* levels, int n_levels, hipStream_t stream);

}  // namespace alstm
