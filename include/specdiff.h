/*
 * specdiff.h — C ABI of the MI355X (gfx950) speculative-diffusion library.
 *
 * The library implements the parallel verification pass of speculative
 * diffusion sampling with block verification ("Accelerating Speculative
 * Diffusions via Block Verification"), driven by the paper's Free Drafter,
 * with a closed-form Gaussian-mixture target; and the paper's alternatives:
 * sample (token) verification, the reflection residual, the Frozen Drafter,
 * temperature, and the plain Euler-Maruyama chain they are measured against.
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless the comment says "host".
 *  - Arrays are row-major float32 unless stated.  A [B][rows][d] view is given
 *    by a base pointer and an sd_stride in ELEMENTS (chain stride, row stride);
 *    the d elements of a row are contiguous.
 *  - The caller owns all memory.  The library allocates device memory only in
 *    sd_target_create (freed by sd_target_destroy); everything else lives in
 *    caller buffers, including a caller workspace sized by the *_workspace query.
 *    sd_target_create also allocates 1 KB of mapped pinned host memory: the
 *    words through which a running sampler call learns, round by round,
 *    whether any chain is still active: 64 slots per target, one per running
 *    call and chain group (SD_EUNSUPPORTED beyond that).
 *    A sampler call that runs two chain groups (sd_sampler_options.groups)
 *    creates one HIP stream the first time it uses a given slot of those
 *    words; the target keeps it until sd_target_destroy.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *    null stream).  Only sd_run_sampler reads results back: a per-round "any
 *    chain active" flag that its kernels store into the mapped host memory,
 *    and the final statistics.
 *  - Arguments are validated before any HIP call: a bad argument returns
 *    SD_EINVAL, a HIP failure SD_EHIP; sd_last_error() then describes it (a
 *    thread-local string).  Outputs are undefined after an error.
 *  - Randomness: every draw comes from Philox4x32-10 keyed by `seed`, counter
 *    (c0, chain, round, tag<<24 | slot) with tags 1 INIT, 2 DRAFT (slot = draft
 *    step), 3 COIN, 4 USAMPLE, 5 RESID, 6 TARGET; uniform = ((w>>8)+0.5)*2^-24,
 *    normals by Box-Muller on word pairs; element e of a vector uses c0 = e>>2.
 *  - Notation: N steps, draft block K (<= SD_MAX_BLOCK), K_b = min(K, N - k)
 *    valid draft rows of a chain at step k.
 *  - Entry points are reentrant; an sd_target is immutable and may be shared
 *    by concurrent streams.
 */
#ifndef SPECDIFF_H
#define SPECDIFF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SD_ABI_VERSION 4
#define SD_MAX_BLOCK 64

typedef enum {
  SD_OK = 0,
  SD_EINVAL = -1,       /* invalid argument (checked before any HIP call)    */
  SD_EHIP = -2,         /* a HIP runtime call failed                          */
  SD_EUNSUPPORTED = -3, /* valid but not supported by the library            */
  SD_ENOMEM = -4,       /* device allocation failed (sd_target_create only)   */
  SD_ENUMERIC = -5      /* a non-finite value was met (sd_run_sampler)        */
} sd_status;

typedef enum { SD_BLOCK = 0, SD_TOKEN = 1 } sd_verify_mode;           /* Alg. 6 / Alg. 2 */
typedef enum { SD_FP32 = 0, SD_BF16 = 1 } sd_precision;               /* denoiser GEMMs  */
typedef enum { SD_USAMPLE_EXACT = 0, SD_USAMPLE_PAPER = 1 } sd_usample_mode; /* Alg. 7 */
/* The residual of a rejected draft: the Decomposition residual (Prop. 1,
 * Alg. 5) or the reflection residual (Alg. 4), which is valid with sample
 * (token) verification only (the impossibility proposition of Sec. 4). */
typedef enum { SD_RESIDUAL_DECOMPOSITION = 0, SD_RESIDUAL_REFLECTION = 1 } sd_residual_kind;
/* The drafter (Sec. 3.3, eq. frozen-draft-drift): FREE reuses the target score
 * the previous round already computed; FROZEN calls the target once per round
 * at the state Y_k and drafts with that score. */
typedef enum { SD_DRAFTER_FREE = 0, SD_DRAFTER_FROZEN = 1 } sd_drafter;

/* VP-SDE Euler-Maruyama chain (Sec. 2): beta(s) = beta_min + s (beta_max - beta_min),
 * t_n = n/N; m^q_n(y) = c1_n y + c2_n score(y), c1_n = 1 + beta_n/(2N),
 * c2_n = (1 + churn^2) beta_n/(2N), sigma_n = churn sqrt(beta_n/N), beta_n = beta(1 - n/N).
 * Requires n_steps >= 1, 0 < beta_min <= beta_max, churn > 0 (the paper requires eps > 0). */
typedef struct {
  int32_t n_steps;
  double beta_min, beta_max, churn;
} sd_schedule;

typedef struct {
  int64_t chain, row; /* element strides of a [B][rows][d] view */
} sd_stride;

typedef void* sd_stream;                /* hipStream_t */
typedef struct sd_target_s* sd_target;  /* opaque Gaussian-mixture target */

int32_t sd_abi_version(void);
const char* sd_last_error(void);

/* Host table of the schedule for n = 0..N (host out[4][N+1]): rows are the
 * signal level a_n = sqrt(abar(1 - t_n)), sigma_n, c1_n, c2_n (Sec. 2,
 * eq. target-distribution). */
sd_status sd_schedule_table(const sd_schedule* sched, double* host_out);

/* ---------------------------------------------------------------- target --
 * Closed-form Gaussian-mixture target q_data = sum_m w_m N(mu_m, var_m I):
 * q_s = sum_m w_m N(a mu_m, (a^2 var_m + 1 - a^2) I) and its score, and the EM
 * mean m^q_n(x) = c1_n x + c2_n score (eq. target-distribution).
 * mu [M][d], var [M], log_w [M] are HOST arrays copied at creation.
 * d >= 1, 1 <= n_comp <= 1024.  precision selects the GEMM operand type:
 * SD_FP32 multiplies float32 operands to float32 accuracy (on the aligned
 * path as six bf16 products of exact three-term bf16 splits of each operand,
 * whose dropped terms are below 2^-23 of |a b|, accumulated in float32;
 * elsewhere with float32 matrix instructions); SD_BF16 stores mu as bf16 (round to
 * nearest even) and rounds x and the softmax weights to bf16 before the two
 * products, accumulating in float32 (||x||^2, ||mu||^2 and the softmax stay
 * float64 from the float32 values, ||x||^2 on the widest logits tiles as a
 * float64 sum of float32 partials of four squares; the epilogue is float32).
 * Only the copies
 * of the chosen precision are allocated. */
sd_status sd_target_create(const sd_schedule* sched, int32_t d, int32_t n_comp,
                           const float* mu, const float* var, const float* log_w,
                           sd_precision precision, sd_target* out);
sd_status sd_target_destroy(sd_target target);
/* Workspace bytes sd_target_mean needs for `rows` rows. */
size_t sd_target_mean_workspace(sd_target target, int32_t rows);
/* For each row r: mq[r] = m^q_{step[r]}(x[r]) and, if score != NULL, score[r] =
 * s_{1 - t_step}(x[r]).  x, mq, score are [rows][d] with the given row strides
 * (>= d); step [rows] int32 in [0, N-1].  Rows are independent ("in parallel",
 * Alg. 1).  ws: device workspace of >= sd_target_mean_workspace bytes. */
sd_status sd_target_mean(sd_target target, int32_t rows, const float* x, int64_t x_row_stride,
                         const int32_t* step, float* mq, int64_t mq_row_stride,
                         float* score, int64_t score_row_stride, void* ws, size_t ws_bytes,
                         sd_stream stream);

/* sd_target_mean without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation and kernels, with the workspace in a
 * 128 MiB array of device memory that the library holds on every GPU it runs
 * on until the process ends (sd_target_mean_noalloc_max_bytes).  The call
 * allocates nothing (its first use on a GPU without a target created there
 * only looks up that GPU's copy).  Rows whose workspace
 * (sd_target_mean_workspace) exceeds it return SD_EINVAL: split them over
 * calls.  Every call on one GPU uses the same memory: calls that overlap on
 * one GPU (concurrent streams or threads) race and give undefined results.
 * Arguments, layouts and errors otherwise as sd_target_mean. */
sd_status sd_target_mean_noalloc(sd_target target, int32_t rows, const float* x,
                                 int64_t x_row_stride, const int32_t* step, float* mq,
                                 int64_t mq_row_stride, float* score, int64_t score_row_stride,
                                 sd_stream stream);
size_t sd_target_mean_noalloc_max_bytes(void);

/* ----------------------------------------------------------------- draft --
 * Y_0 ~ N(0, I) for B chains (Alg. 8, first line): y [B][d], INIT stream,
 * round 0. */
sd_status sd_init_chains(int32_t B, int32_t d, uint64_t seed, float* y, sd_stream stream);

/* Free Drafter block (Sec. 3.3, eq. frozen-draft-drift with the cached score):
 * for chain b at step k[b] (< N) with K_b = min(K, N - k), yhat_0 = y[b] and for
 * i = 1..K_b, n = k + i - 1:
 *   m^p_{i-1} = c1_n yhat_{i-1} + c2_n cache_score[b],  yhat_i = m^p_{i-1} + sigma_n xi_i
 * (xi_i: DRAFT stream, slot i, round round[b]).  Writes x rows 0..K (row 0 = y[b],
 * rows K_b+1..K repeat yhat_{K_b}) and mp rows 0..K-1 (rows >= K_b repeat the last
 * mean).  Chains with k[b] >= N are left untouched.  With cache_score = the
 * target score at (y, k) (sd_target_mean's score output) this is the Frozen
 * Drafter's block.
 * y, cache_score: [B][d] contiguous; x: [B][K+1][d] view; mp: [B][K][d] view. */
sd_status sd_draft_block(const sd_schedule* sched, int32_t B, int32_t K, int32_t d,
                         const float* y, const float* cache_score, const int32_t* k,
                         const uint32_t* round, uint64_t seed, float* x, sd_stride xs, float* mp,
                         sd_stride mps, sd_stream stream);

/* ---------------------------------------------------------------- verify --
 * Verification of B drafted blocks (Alg. 6 block / Alg. 2 token, with the
 * log-space ratios of App. A.2).  For chain b and j = 1..K_b (kb[b] in [0, K];
 * 0 = inactive chain):
 *   Delta_j = (mp_{j-1} - mq_{j-1}) / sigma_{j-1},  Z_j = (y_draft_{j-1} - mp_{j-1}) / sigma_{j-1},
 *   log_ratio[b][j-1] = -Z_j.Delta_j - ||Delta_j||^2/2,  delta_norm[b][j-1] = ||Delta_j||
 * (reductions over d accumulated in float64), then the acceptance scan:
 *   block: log alpha_j = min(0, log alpha_{j-1} + ell_j), h_j = v_j/(v_j + 1 - alpha_j)
 *          (h_{K_b} = alpha_{K_b}), coins eta_j < h_j, tau = 1 + max{j : c_j = 1},
 *          log_alpha_res = log alpha_{tau-1};
 *   token: coins eta_j < min(1, e^{ell_j}), tau = first rejected j (K_b + 1 if none),
 *          log_alpha_res = 0.
 * When tau <= K_b it also draws U ~ psi_{alpha_res} for ||Delta_tau|| by Alg. 7
 * (u_res[b]; NaN otherwise).  eta_j = uniform j-1 of (b, round[b], COIN); the
 * U-sample uniform is uniform 0 of (b, round[b], USAMPLE).
 * Inputs: y_draft [B][K][d] view (yhat_{k+1..}), mp [B][K][d] view (m^p_{k..}),
 * mq [B][>=K][d] view (m^q_{k..}), sigma [B][K+1] float64 (sigma_{k..k+K}),
 * kb [B] (values above K are clamped to K), round [B].  Outputs: tau [B] int32
 * (0 for inactive chains),
 * log_alpha_res [B], u_res [B], delta_norm [B][K], log_ratio [B][K] (float64),
 * coins [B] bitmask of c_1..c_K (nullable).  No workspace. */
sd_status sd_verify_block(int32_t B, int32_t K, int32_t d, sd_verify_mode mode,
                          const float* y_draft, sd_stride ys, const float* mp, sd_stride mps,
                          const float* mq, sd_stride mqs, const double* sigma, const int32_t* kb,
                          const uint32_t* round, uint64_t seed, sd_usample_mode usample_mode,
                          int32_t* tau, double* log_alpha_res, double* u_res, double* delta_norm,
                          double* log_ratio, uint64_t* coins, sd_stream stream);

/* sd_verify_block with temperature omega > 0 (App. "Temperature": the
 * tempered sample and block verification algorithms): p and q get the
 * covariance omega^2 sigma^2 I in the acceptance only, so every ell_j above
 * becomes ell_j / omega^2 (log alpha_j, the token threshold and the block
 * recursion), h_j keeps the untempered ||Delta_{j+1}||, log_alpha_res is the
 * tempered log alpha_{tau-1} (block) or 0 (token), and U is drawn for that
 * alpha_res and the untempered ||Delta_tau||.  log_ratio and delta_norm are
 * the untempered ell_j and ||Delta_j||.  omega = 1 is sd_verify_block; any
 * other value is lossy (the output no longer follows the target).  An omega
 * that is not positive and finite, or whose square over- or underflows in
 * float64, returns SD_EINVAL. */
sd_status sd_verify_block_tempered(int32_t B, int32_t K, int32_t d, sd_verify_mode mode,
                                   double omega, const float* y_draft, sd_stride ys,
                                   const float* mp, sd_stride mps, const float* mq,
                                   sd_stride mqs, const double* sigma, const int32_t* kb,
                                   const uint32_t* round, uint64_t seed,
                                   sd_usample_mode usample_mode, int32_t* tau,
                                   double* log_alpha_res, double* u_res, double* delta_norm,
                                   double* log_ratio, uint64_t* coins, sd_stream stream);

/* -------------------------------------------------------------- residual --
 * The new state Y_{k+tau} of each chain (Alg. 8, residual calculation):
 *  - tau <= K_b: Decomposition residual (Prop. 1, Alg. 5) with alpha = alpha_res:
 *      e = Delta_tau/||Delta_tau||, G ~ N(0, I) (RESID stream),
 *      y = mq_{tau-1} + sigma_{tau-1} (U e + G - e (e.G)),  U = u_res[b];
 *  - tau = K_b + 1 <= steps_left[b]: y = mq_{K_b} + sigma_{K_b} xi (TARGET stream);
 *  - tau = K_b + 1 >  steps_left[b]: y = y_draft_{K_b - 1} (the last draft is Y_N).
 * steps_left[b] = N - k[b] >= K_b; chains with tau[b] <= 0 are skipped.
 * delta_norm [B][K] as produced by sd_verify_block; mq is a [B][K+1][d] view
 * (row K_b feeds the full-accept draw).  kb is clamped to K and chains with
 * tau outside [1, K_b + 1] are skipped.  y_out [B][d] contiguous. */
sd_status sd_sample_residual(int32_t B, int32_t K, int32_t d, const float* y_draft, sd_stride ys,
                             const float* mp, sd_stride mps, const float* mq, sd_stride mqs,
                             const double* sigma, const int32_t* kb, const int32_t* steps_left,
                             const int32_t* tau, const double* u_res, const double* delta_norm,
                             const uint32_t* round, uint64_t seed, float* y_out,
                             sd_stream stream);

/* The reflection residual of sample verification (Alg. 4) for the chains
 * that rejected at tau <= K_b: with Z = (y_draft_{tau-1} - mp_{tau-1}) /
 * sigma_{tau-1} (the draft noise of the rejected step) and e = Delta_tau /
 * ||Delta_tau||,
 *     y = mq_{tau-1} + sigma_{tau-1} (I - 2 e e^T) Z,
 * computed as y_draft_{tau-1} - c (mp - mq), c = 1 + 2 (D.W)/(D.D), D = mp -
 * mq, W = y_draft - mp, with the two sums over d in float64.  The full-accept
 * cases (tau = K_b + 1) are those of sd_sample_residual; no U and no RESID
 * noise are used.  A tau that points at a step with mp = mq (no direction
 * e; a verification never rejects such a step) returns the draft, y =
 * y_draft_{tau-1}.  Same arguments and layouts as sd_sample_residual. */
sd_status sd_sample_residual_reflection(int32_t B, int32_t K, int32_t d, const float* y_draft,
                                        sd_stride ys, const float* mp, sd_stride mps,
                                        const float* mq, sd_stride mqs, const double* sigma,
                                        const int32_t* kb, const int32_t* steps_left,
                                        const int32_t* tau, const uint32_t* round, uint64_t seed,
                                        float* y_out, sd_stream stream);

/* --------------------------------------------------------------- sampler --
 * The full speculative sampler (Alg. 8) with the Free Drafter: Y_0 ~ N(0, I),
 * one explicit target call at Y_0 to seed the cached score, then rounds of
 * draft -> target means on all min(K_b+1, N-k) rows -> verify -> residual ->
 * commit until every chain has reached step N.  Chains run in lockstep rounds,
 * each with its own step k and round counter.  Returns Y_N in y_out [B][d]
 * (written only by a call that ends with every chain at step N).
 * tau_trace (nullable): [trace_rounds][B] int32, tau of each chain per round
 * (0 once a chain has finished).  stats (host, nullable): see sd_stats.
 * ws: >= sd_sampler_workspace bytes; it holds the whole sampler state between
 * rounds, so a run may be split over calls (sd_sampler_options).
 * Returns SD_ENUMERIC if a non-finite log-ratio was met, SD_EHIP also when no
 * round finishes within 120 s (the kernels are then left running and the call
 * returns without waiting for them).
 * Statistics are counted from the start of the run (Y_0), over every call. */
typedef struct {
  int64_t rounds;       /* rounds run so far: until all chains finished, or the
                           rounds a partial call has left in the workspace     */
  int64_t chain_rounds; /* sum over chains of rounds in which the chain was active */
  int64_t steps;        /* sum over chains of steps advanced (B * N when done) */
  int64_t ties;         /* coins with |eta_j - h_j| <= 1e-6 (alpha_j for token):
                           decisions another rounding may flip               */
  double mean_tau;      /* sum of tau over chain-rounds / chain_rounds        */
  int32_t finished;     /* 1 when every chain has reached step N              */
  int32_t groups;       /* chain groups this call ran (sd_sampler_options)    */
  int64_t tau_hist[SD_MAX_BLOCK + 2]; /* tau_hist[t] = number of chain-rounds with tau = t */
} sd_stats;

size_t sd_sampler_workspace(sd_target target, int32_t B, int32_t K);
sd_status sd_run_sampler(sd_target target, int32_t B, int32_t K, sd_verify_mode mode,
                         sd_usample_mode usample_mode, uint64_t seed, float* y_out,
                         int32_t* tau_trace, int32_t trace_rounds, sd_stats* stats, void* ws,
                         size_t ws_bytes, sd_stream stream);

/* The sampler's variants and how much of the run one call does (host struct,
 * read during the call only):
 *  mode, usample_mode   as in sd_run_sampler;
 *  residual             DECOMPOSITION (Alg. 5) or REFLECTION (Alg. 4; needs
 *                       mode == SD_TOKEN, else SD_EINVAL);
 *  drafter              FREE (the default sampler) or FROZEN: every round
 *                       first calls the target at (Y_k, k) and drafts with
 *                       that score, so Delta_1 = 0 and one extra target call
 *                       on B rows is made per round;
 *  omega                temperature > 0 of the verification (see
 *                       sd_verify_block_tempered); 1 is exact, other values
 *                       are lossy;
 *  start_round          0: a new run: the call first initialises the state
 *                       in ws (Y_0, the explicit target call at Y_0, the
 *                       first draft block).  r > 0: continue the run whose
 *                       first r rounds (stats.rounds of the call that left
 *                       them) are in ws, called with the same target, B, K,
 *                       options, seed and workspace (anything else is
 *                       undefined); a run split over calls gives the same
 *                       result as one call;
 *  max_rounds           the rounds this call may run: negative = until every
 *                       chain has reached step N; n >= 0 = at most n (0 with
 *                       start_round 0 only initialises).  The state stays in
 *                       ws (see sd_sampler_state); a call that ends before the
 *                       run is finished does not write y_out;
 *  groups               1: every round runs as one sequence of kernels on
 *                       `stream`; 2: the chains are split into two halves
 *                       (the first B/2 and the rest) whose rounds run on
 *                       `stream` and on a second stream of the library at
 *                       the same time, so that one half's latency-bound
 *                       kernels overlap the other's matrix work (joined back
 *                       into `stream` before the call returns); 0: the
 *                       library chooses (two when each half has at least
 *                       2048 target rows, B/2 (K+1)).  The results do not
 *                       depend on it:
 *                       every row is computed in the same order either way,
 *                       so y_out, tau_trace, the statistics and the state are
 *                       bit-identical.  A run split over calls may change it
 *                       between calls.  With B = 1 it is 1. */
typedef struct {
  sd_verify_mode mode;
  sd_usample_mode usample_mode;
  sd_residual_kind residual;
  sd_drafter drafter;
  double omega;
  int32_t start_round;
  int32_t max_rounds;
  int32_t groups;
} sd_sampler_options;

/* sd_run_sampler with options (sd_run_sampler is this call with DECOMPOSITION,
 * FREE, omega = 1, start_round = 0, max_rounds = -1 and groups = 0).  Same
 * workspace (sd_sampler_workspace, sized for either grouping), outputs and
 * errors; SD_EINVAL also for a negative start_round or groups outside 0..2. */
sd_status sd_run_sampler_ex(sd_target target, int32_t B, int32_t K,
                            const sd_sampler_options* options, uint64_t seed, float* y_out,
                            int32_t* tau_trace, int32_t trace_rounds, sd_stats* stats, void* ws,
                            size_t ws_bytes, sd_stream stream);

/* The sampler state that a workspace holds after `rounds` rounds (stats.rounds
 * of the last call), as device pointers into ws (test hook: for checking a
 * round against another implementation, or reading a partial run):
 *  x           [B][K+1][d]  the next round's block: row 0 = Y_k of every chain
 *                           with k < N; with the Free Drafter rows 1..K are its
 *                           drafts (rows past K_b repeat the last one);
 *  y           [B][d]       Y_N of the chains that have reached step N;
 *  cache       [B][d]       c2_c S_c, the Free Drafter's cached score S_c times
 *                           c2 at its step c = cache_step[b] (Sec. 3.3);
 *  cache_step, k, round [B] the cache's step, the chain's step k and its round
 *                           counter for the next round;
 *  mq          [B][K+1][d]  the last round's target means m^q (row j at step
 *                           k + j of that round; rows past min(K_b, N-k-1)
 *                           are not meaningful);
 *  lrp         [B (K+1)][n_tiles][3] float64: the last round's verification
 *                           partial sums per draft row j < K_b over column
 *                           tiles: ||m^p - m^q||^2, (yhat_{j+1} - m^p).(m^p - m^q),
 *                           G.(m^p - m^q) (G the residual's normals); sums over
 *                           the tiles divided by sigma^2 give ||Delta_{j+1}||^2
 *                           and -ell_{j+1} - ||Delta_{j+1}||^2/2;
 *  tau, coins, log_alpha_res, u [B]: the last round's decision record (tau 0
 *                           for a chain that was inactive; coins bit j-1 = c_j;
 *                           u = U of the residual draw, NaN when none);
 *  ties        [B]          running count of the chain's tied coins.
 * SD_EINVAL for a NULL or short workspace, or rounds < 0. */
typedef struct {
  float* x;
  float* y;
  float* cache;
  int32_t* cache_step;
  int32_t* k;
  uint32_t* round;
  float* mq;
  double* lrp;
  int32_t n_tiles;
  int32_t* tau;
  uint64_t* coins;
  double* log_alpha_res;
  double* u;
  int32_t* ties;
} sd_sampler_view;

sd_status sd_sampler_state(sd_target target, int32_t B, int32_t K, void* ws, size_t ws_bytes,
                           int64_t rounds, sd_sampler_view* out);

/* ------------------------------------------------------------- plain EM --
 * The plain Euler-Maruyama chain (Sec. 2), the non-speculative baseline whose
 * law the sampler reproduces: Y_0 ~ N(0, I) (INIT stream, as sd_run_sampler)
 * and for n = 0..N-1
 *     Y_{n+1} = m^q_n(Y_n) + sigma_n xi_n,   xi_n: TARGET stream, round n, slot 1,
 * one target call on B rows per step.  y_out [B][d] holds the state during
 * the call and Y_N at the end.  ws: >= sd_plain_em_workspace bytes, 256-byte
 * aligned. */
size_t sd_plain_em_workspace(sd_target target, int32_t B);
sd_status sd_run_plain_em(sd_target target, int32_t B, uint64_t seed, float* y_out, void* ws,
                          size_t ws_bytes, sd_stream stream);

/* ------------------------------------------------------------- profiling --
 * Per-kernel timing with HIP events recorded around every launch on the
 * launch's own stream.  sd_profile_enable(1) clears and starts collection,
 * (0) stops it.  sd_profile_read waits for the recorded events and returns up
 * to `capacity` entries (host out), *count = number of kernels seen; its
 * `launches` counts the timed launches. */
typedef struct {
  char name[48];
  int64_t launches;
  double total_ms;
} sd_kernel_stat;

sd_status sd_profile_enable(int32_t on);
/* Restrict collection to launches of the kernel named `name` (host string,
 * copied); NULL times every kernel again. */
sd_status sd_profile_only(const char* name);
/* Time only every n-th launch of each profiled kernel (n >= 1, default 1;
 * counted per kernel name from the last sd_profile_enable(1)): a systematic
 * sample that keeps the events' cost off most launches.  SD_EINVAL for n < 1. */
sd_status sd_profile_every(int32_t n);
/* Launches of the kernel `name` (host string) seen while collecting, timed or
 * not (host out *count; 0 for a kernel not profiled). */
sd_status sd_profile_seen(const char* name, int64_t* count);
sd_status sd_profile_read(sd_kernel_stat* out, int32_t capacity, int32_t* count);

/* ----------------------------------------------------------- test hooks --
 * Raw Philox4x32-10 outputs for n counters (device [n][4] uint32 in/out) with
 * key = seed, and the float32 normals of one (chain, round, tag, slot) stream
 * (device out [d]).  Used to check the generator against its definition. */
sd_status sd_philox_words(uint64_t seed, int32_t n, const uint32_t* counters, uint32_t* out,
                          sd_stream stream);
sd_status sd_philox_normals(uint64_t seed, uint32_t chain, uint32_t round, uint32_t tag,
                            uint32_t slot, int32_t d, float* out, sd_stream stream);

/* Calibration of the matrix cores (not part of the sampler): `blocks`
 * workgroups of four wavefronts, each issuing iters x 4
 * v_mfma_f32_32x32x16_bf16 (32768 flops each) on register operands with no
 * memory traffic, so blocks x 16 x iters x 32768 flops in all; one float per
 * wavefront is written to out (device, [blocks][4], caller-owned) so the loop
 * is kept.  Timing it gives the bf16 matrix rate this GPU sustains, the
 * practical ceiling beside the published dense peak.  SD_EINVAL unless
 * blocks >= 1, iters >= 1 and out is non-null. */
sd_status sd_mfma_loop(int32_t blocks, int32_t iters, float* out, sd_stream stream);

#ifdef __cplusplus
}
#endif
#endif /* SPECDIFF_H */
