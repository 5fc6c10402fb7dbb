/*
 * approx_lstm.h -- C ABI of the MI355X (gfx950) progressive approximate-LSTM
 * library.
 *
 * Method: "Approximate LSTMs for Time-Constrained Inference" (Rizakis et al.,
 * arXiv 1905.00689).  Each LSTM gate's augmented matrix W = [W_x W_h]
 * (Sec. III, "information-maximising approximation") is replaced by an ordered
 * list of refinement terms sigma^(n) u^(n) prune(v^(n), NZ)^T, each the top
 * singular triplet of the residual left by the terms before it, with v pruned
 * to its NZ largest-magnitude entries (Sec. III, Eq. (1) and the residual
 * definition after it).  Running with a budget of K terms per gate gives a
 * usable approximation whose quality grows with K; the gate outputs then pass
 * through the usual sigmoid/tanh cell update (Sec. II, Fig. 1).
 *
 * Conventions shared by every call:
 *   - Every call returns approx_lstm_status; 0 means success.  On error the
 *     outputs are left untouched and approx_lstm_last_error() (thread-local)
 *     describes the failure.  No C++ exception crosses this boundary.
 *   - Host pointers are marked "host", device pointers "device".  The caller
 *     owns every pointer it passes; the library never frees them and keeps no
 *     reference after the call returns.
 *   - Arrays are dense, row-major, float32 unless stated otherwise.
 *   - Gate rows are stacked in the order i, f, g (cell candidate), o, each
 *     block H rows tall, as in torch.nn.LSTM.  A bias b = b_ih + b_hh is added
 *     to the gate pre-activations exactly (outside the approximation).
 *   - hip_stream is a hipStream_t (NULL = the default stream).  Device work is
 *     enqueued on it asynchronously unless stated otherwise.
 *   - A model is immutable after approx_lstm_prepare except for its run
 *     workspace; calls that use one model on several streams at once race on
 *     that workspace and must be serialised by the caller.
 */
#ifndef APPROX_LSTM_H
#define APPROX_LSTM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  APPROX_LSTM_OK = 0,
  APPROX_LSTM_ERR_INVALID_ARG = 1,         /* null pointer, size <= 0, nz not in [1,C], rank < 1,
                                              a level K outside [0,rank], groups not 1 or 4 */
  APPROX_LSTM_ERR_OUT_OF_MEMORY = 2,       /* host or device allocation failed */
  APPROX_LSTM_ERR_DEVICE = 3,              /* HIP runtime failure or a device-side wait that
                                              exceeded its spin limit */
  APPROX_LSTM_ERR_NOT_CONVERGED = 4,       /* prepare: a top-triplet solve missed its tolerance;
                                              the model is still returned, with the count in info */
  APPROX_LSTM_ERR_DEADLINE_INFEASIBLE = 5, /* even K = 0 misses the requested deadline */
  APPROX_LSTM_ERR_UNSUPPORTED = 6          /* a size or combination this build does not handle
                                              (e.g. C > 65535, more levels than APPROX_LSTM_MAX_LEVELS) */
} approx_lstm_status;

#define APPROX_LSTM_MAX_LEVELS 16

/* prepare flags */
#define APPROX_LSTM_FLAG_HOST_ONLY      (1ull << 0) /* factorise on the host only; no device store
                                                       (get_factors works, run returns INVALID_ARG) */
#define APPROX_LSTM_FLAG_KEEP_UNPRUNED  (1ull << 1) /* keep the fp64 sigma, u and unpruned v of every
                                                       term for approx_lstm_get_factors_f64 */
#define APPROX_LSTM_FLAG_DEVICE_FACTORISE (1ull << 2) /* run the factorisation on the current HIP device
                                                       (float64 kernels, same scheme and stop rules;
                                                       results agree with the host factorisation up to
                                                       rounding); not with HOST_ONLY */
#define APPROX_LSTM_FLAG_NON_RESIDUAL   (1ull << 3) /* ablation (Sec. III): deflate each term with its
                                                       whole v, so that the terms are the singular
                                                       triplets of the original gate matrix, each v
                                                       pruned on its own and the pruning error never
                                                       corrected by a later term */

typedef struct approx_lstm_model approx_lstm_model;   /* opaque */

typedef struct {
  int32_t input_size;   /* D >= 1 */
  int32_t hidden_size;  /* H >= 1; C = D + H must be <= 65535 */
  int32_t rank;         /* N >= 1: refinement terms stored per group (the paper's maximum N_steps) */
  int32_t nz;           /* NZ kept per v, 1..C; 0 means nz = C - floor(prune_ratio * C) with the
                           product taken as one IEEE double multiplication */
  double prune_ratio;   /* p in [0, 1); used only when nz == 0 */
  int32_t groups;       /* 4: each gate's H x C block is factorised separately (the paper's scheme);
                           1: the stacked 4H x C matrix is factorised as one */
  int32_t factor_dtype; /* 0 = fp32 factors (sparse store, persistent run kernel);
                           1 = bf16 factor values stored as dense zero-filled panels, run by
                           MFMA kernels with fp32 accumulation (for many sequences at once) */
  uint64_t flags;       /* APPROX_LSTM_FLAG_* */
} approx_lstm_prepare_params;

typedef struct {
  int32_t input_size, hidden_size, aug_size;  /* D, H, C */
  int32_t groups, rows_per_group;             /* G, R_g = 4H / G */
  int32_t rank, nz;                           /* N, NZ */
  int32_t eff_rank[4];                        /* live terms per group (later terms are zero) */
  int32_t unconverged_steps;                  /* solves that missed tolerance (0 normally) */
  int32_t has_device_store;
  uint64_t device_bytes;                      /* factor store on the device */
  int32_t factor_dtype;                       /* as prepared */
} approx_lstm_info;

/*
 * approx_lstm_prepare -- factorise and prune the gate weights (Sec. III,
 * Eq. (1)); upload the packed factor store to the current device.
 *
 *   w_ih  host [4H][D]   input weights   (W_x of every gate)
 *   w_hh  host [4H][H]   recurrent weights (W_h of every gate)
 *   bias  host [4H] or NULL (zeros)
 *   p     host, see approx_lstm_prepare_params
 *   out   host; receives the new model (destroy with approx_lstm_destroy)
 *
 * Per group, in float64 on the host: R <- W_g; for n = 1..rank: the top
 * singular triplet (sigma, u, v) of R (Lanczos on R R^T or R^T R with full
 * reorthogonalisation, then sigma and the other vector from one product with
 * R); sign fixed so that v's largest-magnitude entry (lowest index on ties) is
 * positive; mask = the NZ entries of largest |v| (ties to the lower index),
 * ascending; R <- R - sigma u prune(v)^T.  A step with sigma <= 1e-12 times
 * the first step's sigma ends the list: that and every later term are zero.
 * Values are then rounded to fp32 (nearest even); with factor_dtype 1, u and
 * the v values are further rounded fp32 -> bf16 (nearest even) while sigma
 * stays fp32; masks are decided in fp64 before any rounding.  Synchronises hip_stream
 * before returning.  Returns NOT_CONVERGED (with a usable model) if a solve
 * missed its tolerance.
 */
approx_lstm_status approx_lstm_prepare(const float* w_ih, const float* w_hh, const float* bias,
                                       const approx_lstm_prepare_params* p, void* hip_stream,
                                       approx_lstm_model** out);

/*
 * approx_lstm_run -- progressive LSTM over a sequence at one or more
 * refinement budgets (Eq. (1) per gate, then the Sec. II cell update).
 *
 *   x        device [T][B][D]
 *   T, B     sequence length (T >= 0; T == 0 does nothing) and batch (B >= 1)
 *   h0, c0   device [B][H] or NULL (zeros)
 *   levels   host [n_levels]; each K in [0, rank] is the number of refinement
 *            terms used per group at every timestep
 *   n_levels 1..APPROX_LSTM_MAX_LEVELS
 *   h_out    device [n_levels][T][B][H]: h_t of each level
 *   c_out    device [n_levels][B][H] or NULL: final cell state of each level
 *
 * Each level is its own recurrence (its h feeds only itself); the x-part of
 * the projections is shared.  With a bf16 model (factor_dtype 1) every
 * product takes bf16 operands -- x~ = [x_t; h_{t-1}], the factor values and
 * z = sigma * (prune(v)^T x~) -- with fp32 accumulation; h_out and c_out stay
 * fp32; sequences are padded to a multiple of 64 internally (B <= 2^20,
 * T * padded B <= 2^30 and T * B * D < 2^31, else UNSUPPORTED).  Asynchronous on hip_stream; the call blocks
 * only to allocate workspace on first use (see approx_lstm_reserve).  The
 * device-side waits of the kernel are bounded; if one expires the next
 * approx_lstm_check call reports APPROX_LSTM_ERR_DEVICE.
 */
approx_lstm_status approx_lstm_run(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                   const float* h0, const float* c0, const int32_t* levels,
                                   int32_t n_levels, float* h_out, float* c_out, void* hip_stream);

/*
 * approx_lstm_run_noalloc -- approx_lstm_run for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results and kernels as
 * approx_lstm_run for an fp32 model (bitwise the same outputs), but the run
 * workspace (x-part projections, exchange words, bulk h buffers and flags)
 * lives in one static device array of 32 MiB per device, held until the
 * process ends; the call itself calls no hipMalloc, hipFree or other
 * allocating routine (the model's factor store and error word were allocated
 * by approx_lstm_prepare).  The first call on a device looks up the array's
 * address there (hipGetSymbolAddress).
 *
 * Limits and errors: UNSUPPORTED when the run's workspace exceeds 32 MiB
 * (about G*K*T*B*4 bytes of x-part projections plus the exchange words; the
 * message gives the size), for bf16 models and for T > 65534; otherwise as
 * approx_lstm_run.  No timing stamps are recorded.
 *
 * Concurrency: every call on one device shares that device's array; calls
 * whose work overlaps on one device (different streams, or different host
 * threads without ordering) race on it and must be serialised by the caller.
 * Calls on one stream are ordered and safe.
 */
approx_lstm_status approx_lstm_run_noalloc(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                           const float* h0, const float* c0, const int32_t* levels,
                                           int32_t n_levels, float* h_out, float* c_out, void* hip_stream);

/*
 * approx_lstm_run_deadline -- progressive LSTM under a per-timestep time
 * budget (the paper's time-constrained setting: the best output reachable
 * within the budget, Sec. I, and computation cut when the budget is hit,
 * Sec. VI-B).  Picks the largest K whose measured in-kernel time per timestep
 * (from the start of one timestep to the start of the next, device clock)
 * meets deadline_us_per_step and runs the sequence at that K.
 *
 *   x, T, B, h0, c0  as for approx_lstm_run (T >= 1)
 *   h_out            device [T][B][H]
 *   k_achieved       host [T]: the K used at every timestep
 *   step_us          host [T] or NULL: measured microseconds of every timestep
 *
 * fp32 models only (UNSUPPORTED for factor_dtype 1).
 * On first use for a (T, B, launch width) the call calibrates time against K
 * by running the sequence at K = 0, 1, 2, 4, ..., rank (cached in the model),
 * then bisects between the two calibrated budgets around the deadline with
 * fresh runs.  Synchronises hip_stream.  Returns
 * APPROX_LSTM_ERR_DEADLINE_INFEASIBLE if even K = 0 misses the deadline;
 * individual timesteps of the final run may still exceed it (step_us tells).
 */
approx_lstm_status approx_lstm_run_deadline(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                            const float* h0, const float* c0, double deadline_us_per_step,
                                            float* h_out, int32_t* k_achieved, float* step_us, void* hip_stream);

/*
 * approx_lstm_run_anytime -- progressive LSTM whose budget K_t is chosen
 * online, on the device, at every timestep: the computation of each step is
 * cut to what its share of the time budget allows (Sec. VI-B: predictions
 * whose computation is cut short when the available time is used up; Sec. I:
 * the best estimate for the time available).  One launch runs the sequence
 * with room for every term of the model; at the end of timestep t workgroup
 * 0 reads the device's wall clock and picks, among the candidate budgets
 * K = 0, 1, 2, 4, ..., rank, the largest whose predicted step time fits
 * one deadline plus an even share, over the remaining steps, of the time
 * banked by the end of timestep t (the rest of timestep t, its h exchange,
 * taken as measured on the previous step); a deficit is recovered at once,
 * so timestep t+1 still ends by (t+2) * deadline_us_per_step after the
 * recurrence began.  The choice reaches every workgroup with the h
 * exchange, so all compute with the same K_{t+1}.  K_0 is the largest
 * candidate predicted to fit one deadline.
 *
 *   x, T, B, h0, c0  as for approx_lstm_run (T >= 1)
 *   h_out            device [T][B][H]
 *   k_achieved       host [T]: the K each timestep was computed with
 *   step_us          host [T] or NULL: measured microseconds of every timestep
 *
 * fp32 models only (UNSUPPORTED for factor_dtype 1).  The predicted step
 * times come from a calibration inside the same launch configuration (each
 * candidate forced at every timestep), run on first use for a (T, B, launch
 * width) and cached in the model.  Synchronises hip_stream.  Returns
 * APPROX_LSTM_ERR_DEADLINE_INFEASIBLE if K = 0 is predicted to miss the
 * deadline; otherwise the run completes (a step whose time ran out computes
 * K = 0, and step_us tells whether the deadline was met).  The result equals
 * a replay of the sequence with the reported k_achieved.
 */
approx_lstm_status approx_lstm_run_anytime(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                           const float* h0, const float* c0, double deadline_us_per_step,
                                           float* h_out, int32_t* k_achieved, float* step_us, void* hip_stream);

/*
 * approx_lstm_run_schedule -- progressive LSTM with a caller-given budget K_t
 * for every timestep (Sec. VI-B: the computation of each prediction cut to the
 * budget available for it).  Runs the same online launch as
 * approx_lstm_run_anytime (sized for the largest K_t), with K_t taken from
 * k_sched instead of the device clock: the result is the recurrence of Eq. (1)
 * with K_t terms per gate at timestep t, then the Sec. II cell update.
 *
 *   x, T, B, h0, c0  as for approx_lstm_run (1 <= T <= 65534)
 *   k_sched          host [T]: K_t, each in [0, rank]
 *   h_out            device [T][B][H]
 *   c_out            device [B][H] or NULL: c after the last timestep
 *
 * fp32 models only (UNSUPPORTED for factor_dtype 1).  Blocking: synchronises
 * hip_stream and copies k_sched to the device before the launch, which then
 * runs asynchronously.  Errors: INVALID_ARG for a null pointer, T or B below
 * 1, or a K_t outside [0, rank].
 */
approx_lstm_status approx_lstm_run_schedule(approx_lstm_model* m, const float* x, int32_t T, int32_t B,
                                            const float* h0, const float* c0, const int32_t* k_sched,
                                            float* h_out, float* c_out, void* hip_stream);

/*
 * approx_lstm_plan -- the launch plan an fp32 run would use, without any
 * device work (for tests and tuning; no part of the paper's method).
 *
 *   T, B               sequence length and count (>= 1)
 *   levels, n_levels   host [n_levels] budgets as for approx_lstm_run
 *                      (ignored when online != 0: the plan of an anytime or
 *                      scheduled run sized for the whole rank)
 *   num_cu             compute units to plan for (0 = the model's device)
 *   out                host [10]: workgroups, all-timestep P_x resident in LDS
 *                      (1/0), all (level, sequence) pairs in one phase-B pass
 *                      (1/0), h-part entries per lane in registers, U entries
 *                      per thread in registers, output rows per thread, bulk
 *                      h exchange (1/0), LDS bytes per workgroup (above
 *                      163840: the run returns UNSUPPORTED), 1 when the run
 *                      takes the one-pair recurrence kernel (see
 *                      approx_lstm_set_recurrence), else 0, and the K tile of
 *                      a phase B that reads each U entry once per timestep
 *                      for every sequence (0: one pass per sequence)
 *
 * Works on HOST_ONLY models.  Errors: INVALID_ARG for bad sizes or levels;
 * UNSUPPORTED for bf16 models.
 */
approx_lstm_status approx_lstm_plan(const approx_lstm_model* m, int32_t T, int32_t B, const int32_t* levels,
                                    int32_t n_levels, int32_t online, int32_t num_cu, int32_t* out);

/*
 * approx_lstm_run_stack -- stacked LSTM layers, each progressive: layer l
 * (l >= 1) takes as its input sequence the h_t of layer l-1 at the same level.
 *
 *   layers    host [n_layers]: prepared models; layers[l]->input_size must
 *             equal layers[l-1]->hidden_size; all on one device
 *   x         device [T][B][D_0]
 *   levels    host [n_levels][n_layers]: K of every layer at every level
 *   h_out     device [n_levels][T][B][H_last]
 *
 * Initial states are zero.  Intermediate sequences live in a buffer owned by
 * layers[0] (allocated on first use, which blocks).  Asynchronous on
 * hip_stream otherwise.  Layers are run one after another; layer 0 runs all
 * levels in one launch pair, each later layer one launch pair per level.
 */
approx_lstm_status approx_lstm_run_stack(approx_lstm_model* const* layers, int32_t n_layers, const float* x,
                                         int32_t T, int32_t B, const int32_t* levels, int32_t n_levels,
                                         float* h_out, void* hip_stream);

/*
 * approx_lstm_reserve -- preallocate the run workspace for up to T_max
 * timesteps, B_max sequences and L_max levels, so that later runs within
 * those sizes allocate nothing.  Blocking.
 */
approx_lstm_status approx_lstm_reserve(approx_lstm_model* m, int32_t T_max, int32_t B_max,
                                       int32_t L_max);

/*
 * approx_lstm_check -- synchronise hip_stream and report whether any device
 * wait of an earlier run on this model expired (APPROX_LSTM_ERR_DEVICE) or a
 * HIP error is pending.  Clears the recorded flag.
 */
approx_lstm_status approx_lstm_check(approx_lstm_model* m, void* hip_stream);

/*
 * approx_lstm_set_launch -- launch shape of the run kernel, from the next run
 * on.  blocks: workgroups (0 = automatic: about one per 32 terms in use, at
 * most 64, widened until the per-workgroup slices fit in LDS; at most the
 * device's compute units).  The results do not depend on it: every sum has a
 * fixed order.  cooperative != 0 launches through the cooperative-launch API,
 * which has the runtime guarantee that all workgroups are resident at once
 * (about 17 us more per launch); the default plain launch relies on the
 * device being otherwise idle enough to hold them, and if it is not, the
 * kernel's bounded waits expire and approx_lstm_check reports
 * APPROX_LSTM_ERR_DEVICE instead of hanging.  For bf16 models, blocks > 0
 * caps the workgroups of the persistent recurrence (fewer cohorts in flight;
 * below one cohort's workgroups the per-timestep kernels run); cooperative is
 * ignored there.
 */
approx_lstm_status approx_lstm_set_launch(approx_lstm_model* m, int32_t blocks, int32_t cooperative);

/*
 * approx_lstm_set_recurrence -- recurrence kernel of an fp32 model's fixed-
 * budget runs, from the next run on.  kernel = 0 (the default): a run of one
 * level over one sequence (approx_lstm_run with n_levels = 1 and B = 1, and
 * the runs approx_lstm_run_deadline and approx_lstm_run_stack make of that
 * form) takes the one-pair kernel where its launch plan fits (every owned
 * h-part entry and U entry in registers: at most 2048 terms per
 * sequence in use, K <= 1024, and the entries per lane it needs), every other
 * run the general persistent kernel; kernel = 1: the general kernel always.
 * Both compute every sum in the same order: the outputs are bitwise equal.
 * Errors: null model, kernel not 0 or 1.
 */
approx_lstm_status approx_lstm_set_recurrence(approx_lstm_model* m, int32_t kernel);

/*
 * approx_lstm_set_batched_path -- kernels of a bf16 model's recurrence (Eq. (1)
 * per gate with bf16 operands, then the Sec. II cell update), from the next
 * run on.  persistent = 1 (the default): one persistent launch per level
 * where the shape allows it (H and every K at most 512; sequences in cohorts
 * of 16, each run by ceil(H/32) workgroups that exchange z and h through
 * device memory every timestep); other shapes, and persistent = 0, run two
 * kernels per timestep.  2 and 3 force the persistent launch's z exchange to
 * tagged words or to flagged plain bf16 (tuning; 1 picks by the number of
 * terms).  All compute the same products with fp32 sums; they differ only in
 * the order of those sums.  The persistent launch relies on each cohort's
 * workgroups being resident at once; if they are not, its bounded waits
 * expire and approx_lstm_check reports APPROX_LSTM_ERR_DEVICE.  No effect on
 * fp32 models.  Errors: null model, persistent outside 0..3.
 */
approx_lstm_status approx_lstm_set_batched_path(approx_lstm_model* m, int32_t persistent);

/*
 * approx_lstm_set_timing -- enable (1) or disable (0) per-timestep device
 * timestamps in later runs (one device wall-clock read per phase by
 * workgroup 0; negligible cost).
 *
 * approx_lstm_get_timing -- synchronise hip_stream and copy the stamps of the
 * last run that recorded them, in microseconds from the start of its
 * recurrence, to host stamps_us[n], n >= 2 + 4T: [0] = 0, then for each
 * timestep t the starts of phase A (h-part dots), of the z wait, of the U
 * accumulation and of the h wait at [1+4t .. 4+4t], and the end at [1+4T].
 */
approx_lstm_status approx_lstm_set_timing(approx_lstm_model* m, int32_t enable);
approx_lstm_status approx_lstm_get_timing(approx_lstm_model* m, void* hip_stream, double* stamps_us, int32_t n);

/* approx_lstm_model_info -- sizes, live ranks and device footprint (host struct). */
approx_lstm_status approx_lstm_model_info(const approx_lstm_model* m, approx_lstm_info* out);

/*
 * approx_lstm_get_factors -- copy group g's refinement terms, in refinement
 * order, as the device store holds them (fp32; for a bf16 model the fp32
 * values are exactly the stored bf16 values), to host arrays:
 *   sigma [rank], u [rank][R_g], v_idx [rank][nz] (ascending column indices
 *   into [x; h], 0..C-1), v_val [rank][nz] (entries of prune(v) on v_idx).
 * Any output pointer may be NULL.  Reads the host copy kept by prepare.
 */
approx_lstm_status approx_lstm_get_factors(const approx_lstm_model* m, int32_t group, float* sigma,
                                           float* u, int32_t* v_idx, float* v_val);

/*
 * approx_lstm_get_factors_f64 -- the float64 sigma [rank], u [rank][R_g] and
 * unpruned v [rank][C] of group g before rounding (for certificates).  Needs
 * APPROX_LSTM_FLAG_KEEP_UNPRUNED at prepare time, else INVALID_ARG.
 */
approx_lstm_status approx_lstm_get_factors_f64(const approx_lstm_model* m, int32_t group,
                                               double* sigma, double* u, double* v_unpruned);

/*
 * Exact (dense) LSTM -- the baseline the progressive approximation is
 * measured against: gate pre-activations W_x x_t + W_h h_{t-1} + b with the
 * full weight matrices (Sec. II, Fig. 1; the faithful LSTM of the paper's
 * comparisons, Sec. VI-B), then the same cell update.  fp32.
 *
 * approx_lstm_exact_prepare -- copy the weights to the current device.
 *   w_ih host [4H][D], w_hh host [4H][H], bias host [4H] or NULL (zeros);
 *   gate rows i, f, g, o.  Synchronises hip_stream.
 * approx_lstm_exact_run -- the recurrence over x device [T][B][D] (T >= 0,
 *   B >= 1; T <= 65534) from h0, c0 device [B][H] or NULL (zeros); writes
 *   h_out device [T][B][H] and, if not NULL, c_out device [B][H].
 *   Asynchronous on hip_stream (allocates workspace on first use, blocking).
 *   Bounded device waits as for approx_lstm_run (see approx_lstm_exact_check).
 * approx_lstm_exact_run_rows -- the same recurrence stopped after `rows`
 *   rows of every gate (0 <= rows <= H): the anytime baseline of Sec. VI-B,
 *   whose dense products run in tiles of rows and whose output after each
 *   tile step is the baseline's intermediate result.  A row not reached holds
 *   the bias alone (rows = 0: every gate is its bias; rows = H: identical to
 *   approx_lstm_exact_run, bit for bit).  Same buffers and behaviour as
 *   approx_lstm_exact_run; rows outside [0, H] is APPROX_LSTM_ERR_INVALID_ARG.
 * approx_lstm_exact_check -- synchronise hip_stream and report an expired
 *   device wait (APPROX_LSTM_ERR_DEVICE); clears the flag.
 * approx_lstm_exact_set_launch -- workgroups of the recurrence kernel from
 *   the next run on (0 = automatic: one per 8 hidden units, at most the
 *   device's compute units); results do not depend on it.
 */
typedef struct approx_lstm_exact approx_lstm_exact;   /* opaque */

approx_lstm_status approx_lstm_exact_prepare(const float* w_ih, const float* w_hh, const float* bias,
                                             int32_t input_size, int32_t hidden_size, void* hip_stream,
                                             approx_lstm_exact** out);
approx_lstm_status approx_lstm_exact_run(approx_lstm_exact* m, const float* x, int32_t T, int32_t B,
                                         const float* h0, const float* c0, float* h_out, float* c_out,
                                         void* hip_stream);
approx_lstm_status approx_lstm_exact_run_rows(approx_lstm_exact* m, const float* x, int32_t T, int32_t B,
                                              const float* h0, const float* c0, int32_t rows, float* h_out,
                                              float* c_out, void* hip_stream);
approx_lstm_status approx_lstm_exact_check(approx_lstm_exact* m, void* hip_stream);
approx_lstm_status approx_lstm_exact_set_launch(approx_lstm_exact* m, int32_t blocks);
void approx_lstm_exact_destroy(approx_lstm_exact* m);

/* approx_lstm_destroy -- free the model and its device memory (NULL is a no-op). */
void approx_lstm_destroy(approx_lstm_model* m);

/* approx_lstm_last_error -- text of the last error on this thread ("" if none). */
const char* approx_lstm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* APPROX_LSTM_H */
