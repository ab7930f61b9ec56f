// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "specdiff.h"

namespace sd {

// Thread-local error message behind sd_last_error().
void set_error(const char* fmt, ...);

// ------------------------------------------------------------- profiling --
bool prof_on(const char* name);
void prof_push(const char* name, hipEvent_t start, hipEvent_t stop);
void prof_events(hipEvent_t* start, hipEvent_t* stop);

// Enqueue one kernel launch through `launch`; when profiling is on, bracket it
// with events on the same stream.  Returns the launch error, if any.
template <class F>
hipError_t timed(const char* name, hipStream_t s, F&& launch) {
  if (!prof_on(name)) {
    launch();
    return hipGetLastError();
  }
  hipEvent_t a, b;
  prof_events(&a, &b);
  (void)hipEventRecord(a, s);
  launch();
  hipError_t e = hipGetLastError();
  (void)hipEventRecord(b, s);
  prof_push(name, a, b);
  return e;
}

#ifdef __HIPCC__
}  // namespace sd
#include <hip/hip_ext.h>
namespace sd {
// One launch of `kernel`; when profiling is on for `name` the launch carries
// the start and stop events in its own dispatch (hipExtLaunchKernelGGL), which
// times the kernel alone and costs the stream less than two event records.
template <class Kern, class... Args>
hipError_t launch_timed(const char* name, Kern kernel, dim3 grid, dim3 block, hipStream_t s,
                        Args... args) {
  if (!prof_on(name)) {
    kernel<<<grid, block, 0, s>>>(args...);
    return hipGetLastError();
  }
  hipEvent_t a, b;
  prof_events(&a, &b);
  hipExtLaunchKernelGGL(kernel, grid, block, 0, s, a, b, 0, args...);
  const hipError_t e = hipGetLastError();
  prof_push(name, a, b);
  return e;
}
#endif

// ------------------------------------------------------------- schedule --
struct Sched {
  int N;
  double bmin, bmax, eps;
};

__host__ __device__ inline double sched_beta(const Sched& s, int n) {
  const double fwd = 1.0 - (double)n / (double)s.N;
  return s.bmin + fwd * (s.bmax - s.bmin);
}
__host__ __device__ inline double sched_sigma(const Sched& s, int n) {
  return s.eps * sqrt(sched_beta(s, n) / (double)s.N);
}
__host__ __device__ inline double sched_c1(const Sched& s, int n) {
  return 1.0 + 0.5 * sched_beta(s, n) / (double)s.N;
}
__host__ __device__ inline double sched_c2(const Sched& s, int n) {
  return 0.5 * (1.0 + s.eps * s.eps) * sched_beta(s, n) / (double)s.N;
}
__host__ __device__ inline double sched_signal(const Sched& s, int n) {
  const double fwd = 1.0 - (double)n / (double)s.N;
  return sqrt(exp(-(s.bmin * fwd + 0.5 * (s.bmax - s.bmin) * fwd * fwd)));
}

inline Sched to_sched(const sd_schedule* p) {
  return Sched{p->n_steps, p->beta_min, p->beta_max, p->churn};
}

// ------------------------------------------------------- target internals --
struct Target {
  Sched sc;
  int d, M;
  sd_precision prec;
  float* mu;      // [M][d]
  float* muT;     // [d][M]
  uint16_t* mu16;   // [M][d] bf16 (round to nearest even), bf16 precision only
  uint16_t* muT16;  // [d][M] bf16, bf16 precision only
  // float32 precision: the exact three-term bf16 splits of mu and mu^T
  // (planes hi, mid, lo, each [M][d] resp. [d][M]) for the matrix-core
  // contractions of gemm_split.hpp
  uint16_t* mu_split;   // [3][M][d]
  uint16_t* muT_split;  // [3][d][M]
  double* logw;   // [M]
  double* musq;   // [M] ||mu_m||^2 (float64 from the float32 means)
  float4* coef;   // [N+1] per step: (c1_n, c2_n, sigma_n, 1/c2_n) rounded to float32
  double2* ls;    // [N][M] per step and component: (log s2, 1/s2), s2 = a_n^2 var_m + 1 - a_n^2
  int device;
  // Mapped pinned host words through which the sampler's kernels publish the
  // per-round "any chain active" flag: kFlagGroups groups of kFlagSlots words,
  // one group per running sampler call (bit g of flag_busy, taken and given
  // back atomically; a group whose call timed out is never given back).
  int32_t* host_flags;      // host address [kFlagGroups][kFlagSlots]
  int32_t* host_flags_dev;  // the same memory as the device sees it
  uint64_t flag_busy;
  // the second stream of a sampler call that runs two chain groups, one per
  // flag group (created at its first use, used only by the call that holds
  // that flag group)
  hipStream_t side[64];
};
constexpr int kFlagGroups = 64, kFlagSlots = 4;
static_assert(sizeof(Target::side) / sizeof(hipStream_t) == kFlagGroups, "one side stream per flag group");

// Workspace of a target call on `rows` rows whose logits GEMM is split over d
// as for plan_rows rows (0: rows).  The split fixes the order in which the
// partial logits are summed, so calls on parts of a batch that take the
// whole batch's row count here give every row the same result as one call.
size_t target_ws_bytes(const Target& t, int rows, int plan_rows = 0);
size_t target_ws_bytes_bf16(const Target& t, int rows, int plan_rows = 0);
// Rows' EM means (and scores if score != nullptr).  gate: nullable device flag;
// when it reads 0 every kernel exits at once (finished sampler rounds).
hipError_t target_mean_launch(const Target& t, int rows, const float* x, int64_t ldx,
                              const int32_t* step, float* mq, int64_t ldq, float* score,
                              int64_t lds, void* ws, hipStream_t s, const int* gate,
                              int plan_rows = 0);

// The sampler's target call on its [B][K+1][d] block (x rows contiguous,
// row stride d) that also leaves the verification's partial sums in
// lrp[row][lr_tiles(t, K1)][3] (see gmm_mean_lr_kernel); the draft means are
// recomputed from x, the cache rows sv [B][d] and the cache steps cstep [B];
// rnd = chains' rounds; chain0 = the generator's chain index of the first
// chain (a part of a batch); plan_rows as for target_ws_bytes.
hipError_t target_mean_lr_launch(const Target& t, int rows, int K1, const float* x,
                                 const int32_t* step, float* mq, const float* sv,
                                 const int32_t* cstep, double* lrp, const uint32_t* rnd,
                                 uint64_t seed, void* ws, hipStream_t s, const int* gate,
                                 int plan_rows = 0, int chain0 = 0);
int lr_tiles(const Target& t, int K1);
// bf16 versions of the three calls above (dispatched to by them).
hipError_t target_mean_bf16_launch(const Target& t, int rows, const float* x, int64_t ldx,
                                   const int32_t* step, float* mq, int64_t ldq, float* score,
                                   int64_t lds, void* ws, hipStream_t s, const int* gate,
                                   int plan_rows = 0);
hipError_t target_mean_lr_bf16_launch(const Target& t, int rows, int K1, const float* x,
                                      const int32_t* step, float* mq, const float* sv,
                                      const int32_t* cstep, double* lrp, const uint32_t* rnd,
                                      uint64_t seed, void* ws, hipStream_t s, const int* gate,
                                      int plan_rows = 0, int chain0 = 0);
int lr_tiles_bf16(const Target& t, int K1);
// Softmax over the split logits partials part[S][rows][M] (+ xsq[S][rows]):
// P[rows][M] = r a / s2 (float32, or bf16 when p_bf16) and rowc[rows][3] =
// (c1, c2, rho) of each row's step.
hipError_t gmm_softmax_launch(const Target& t, int rows, int S, const float* part,
                              const double* xsq, const int32_t* step, void* P, bool p_bf16,
                              float* rowc, hipStream_t s, const int* gate);
// Sampler verification on the fused partials (see scan_fused_kernel).
// w2 = omega^2 (temperature; 1 = exact); reflect: the reflection residual.
// coins, lar, ures [B]: the round's decision record; ties [B]: running count
// of coins within 1e-6 of their thresholds; chain0: the generator's chain
// index of chain 0.
hipError_t scan_fused_launch(int B, int K, int d, int N, int mode, int umode, const double* lrp,
                             int nct, const double* sigma, const int32_t* kcur,
                             const uint32_t* rcur, uint64_t seed, double w2, bool reflect,
                             int32_t* tau, int32_t* rmode, float* rcoef, float* rsig,
                             uint64_t* coins, double* lar, double* ures, int32_t* ties,
                             int* nanflag, int* act_next, int* host_prev, int pub_round,
                             hipStream_t s, const int* gate, int chain0 = 0);
// Residual, commit and the next round's Free-Drafter block, elementwise over
// (chain, four coordinates); per-chain state is read from the *cur arrays and
// written to the *next arrays (round parity), so no workgroup races another.
// frozen: the Frozen Drafter drafts after its own target call, so the round
// ends with the new state in x row 0 and the next cache at (row 0, step k).
// chain0: the generator's chain index of chain 0; trace rows are trace_ld
// chains apart (0: B).  stream_bytes: the draft block whose size decides
// whether its rows are streamed past the caches (0: this call's block).
hipError_t advance_launch(const Sched& sc, const float4* coef, int B, int K, int d,
                          uint64_t seed, const int32_t* kcur, const uint32_t* rcur,
                          const int32_t* crow_cur, const int32_t* cstep_cur, int32_t* knext,
                          uint32_t* rnext, int32_t* crow_next, int32_t* cstep_next,
                          const int32_t* tau, const int32_t* rmode, const float* rcoef,
                          const float* rsig, float* x, float* sv, const float* mq, float* y,
                          int32_t* step, double* sigma, int32_t* hist, int64_t* steps,
                          int* act_next, int32_t* trace, int r, int trace_rounds, bool frozen,
                          hipStream_t s, const int* gate, int chain0 = 0, int trace_ld = 0,
                          int64_t stream_bytes = 0);

// ---------------------------------------------------------------- kernels --
hipError_t init_chains_launch(int B, int d, uint64_t seed, float* y, float* x0, int64_t x0c,
                              hipStream_t s);
hipError_t draft_launch(const Sched& sc, int B, int K, int d, const float* y, const float* cs,
                        const int32_t* k, const uint32_t* rnd, uint64_t seed, float* x,
                        sd_stride xs, float* mp, sd_stride mps, hipStream_t s, const int* gate);
// Draft whose cached score is recovered from row crow[b] of the previous
// round's x / target means at step cstep[b] (the sampler's Free Drafter):
// writes the draft rows and the cache row sv[b] = c2_c S_c ([B][d]), no means.
hipError_t draft_cached_launch(const Sched& sc, const float4* coef, int B, int K, int d,
                               const float* y,
                               const int32_t* crow, const int32_t* cstep, const float* mqprev,
                               sd_stride mqs, const int32_t* k, const uint32_t* rnd,
                               uint64_t seed, float* x, sd_stride xs, float* sv,
                               hipStream_t s, const int* gate, int chain0 = 0,
                               int64_t stream_bytes = 0);
hipError_t verify_launch(int B, int K, int d, int mode, const float* yd, sd_stride ys,
                         const float* mp, sd_stride mps, const float* mq, sd_stride mqs,
                         const double* sigma, const int32_t* kb, const uint32_t* rnd,
                         uint64_t seed, int umode, double w2, int32_t* tau, double* lar,
                         double* ures, double* dn, double* lr, uint64_t* coins, int* nanflag,
                         hipStream_t s, const int* gate);
hipError_t residual_launch(int B, int K, int d, const float* yd, sd_stride ys, const float* mp,
                           sd_stride mps, const float* mq, sd_stride mqs, const double* sigma,
                           const int32_t* kb, const int32_t* left, const int32_t* tau,
                           const double* ures, const double* dn, const uint32_t* rnd,
                           uint64_t seed, float* y, hipStream_t s);
// The reflection residual (Alg. 4) for rejected chains, the same full-accept
// cases as residual_launch otherwise.
hipError_t reflection_launch(int B, int K, int d, const float* yd, sd_stride ys, const float* mp,
                             sd_stride mps, const float* mq, sd_stride mqs, const double* sigma,
                             const int32_t* kb, const int32_t* left, const int32_t* tau,
                             const uint32_t* rnd, uint64_t seed, float* y, hipStream_t s);
// One plain Euler-Maruyama step on B rows: y = mq + sigma_n xi (TARGET
// stream, round n, slot 1), and step[b] = n + 1 for the next target call.
hipError_t em_noise_launch(int B, int d, int n, float sigma_n, uint64_t seed, const float* mq,
                           float* y, int32_t* step, hipStream_t s);
// Sampler-only kernels.
hipError_t residual_commit_launch(int B, int K, int d, int N, const float* yd, sd_stride ys,
                                  const float* mp, sd_stride mps, const float* mq, sd_stride mqs,
                                  const double* sigma, const int32_t* kb, const int32_t* left,
                                  const int32_t* tau, const double* ures, const double* dn,
                                  uint32_t* rnd, uint64_t seed, float* y, int32_t* k,
                                  int32_t* crow, int32_t* cstep, int32_t* adv, int32_t* trace,
                                  int r, int trace_rounds, hipStream_t s, const int* gate);
hipError_t fill_i32_launch(int32_t* p, int64_t n, int32_t v, hipStream_t s);
// *f0 = 1 if a chain of [0, split) has k < N, else 0; *f1 the same for
// [split, B) (one workgroup).
hipError_t chains_active_launch(int B, int split, int N, const int32_t* k, int* f0, int* f1,
                                hipStream_t s);
hipError_t fill_i64_launch(int64_t* p, int64_t n, int64_t v, hipStream_t s);
hipError_t prepare_launch(const Sched& sc, int B, int K, const int32_t* k, int32_t* kb,
                          int32_t* left, int32_t* step, double* sigma, int32_t* tau,
                          int32_t* adv, int* cnt_cur, int* cnt_next, int64_t* hist,
                          int64_t* steps, hipStream_t s);
hipError_t philox_words_launch(uint64_t seed, int n, const uint32_t* ctr, uint32_t* out,
                               hipStream_t s);
hipError_t philox_normals_launch(uint64_t seed, uint32_t chain, uint32_t rnd, uint32_t tag,
                                 uint32_t slot, int d, float* out, hipStream_t s);
// blocks workgroups of four wavefronts, each issuing iters x 4 bf16 matrix
// instructions on registers; one float per wavefront to out ([blocks][4]).
hipError_t mfma_loop_launch(int blocks, int iters, float* out, hipStream_t s);

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Whether a kernel that writes a block of `bytes` of draft rows uses
// non-temporal stores for them.  The next target call reads the whole block
// back: while it is at most half of the 256 MB infinity cache most of it is
// still there for that read, so the rows are stored normally; a larger block
// mostly leaves the cache before it is read, and normal stores then only
// displace other lines (measured: streaming a 113 MB block slowed the next
// logits GEMM by 5 us; streaming 151 MB and 428 MB blocks made the advance
// kernel 10 and 25 us faster and the logits GEMM no slower).
constexpr int64_t kStreamRowsBytes = (int64_t)128 << 20;
inline bool stream_rows(int64_t bytes) { return bytes > kStreamRowsBytes; }

#ifdef __HIPCC__
// Workgroups are dispatched round-robin over the eight XCDs, each with its own
// L2.  Remap the linear workgroup id so that XCD x works on a contiguous
// range of the tile space (tiles that share operand rows stay on one L2); the
// innermost tile index is the fastest-varying one.  Workgroup L runs on XCD
// x = L % 8 as its (L / 8)-th; with total = 8 q + r, XCDs x < r receive q + 1
// workgroups and the others q, so XCD x takes the range starting at
// x q + min(x, r) (a bijection of [0, total)).
__device__ __forceinline__ int xcd_tile(int total) {
  const int L = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  const int x = L % 8, q = total / 8, r = total % 8;
  return x * q + min(x, r) + L / 8;
}
#endif

}  // namespace sd
