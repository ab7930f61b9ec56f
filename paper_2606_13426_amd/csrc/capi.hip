// C ABI: argument validation (always before any HIP call), the Gaussian-mixture
// target object, the sampler's round loop (Alg. 8) and the event profiler.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <map>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "common.hpp"
#include "gemm_split.hpp"

namespace sd {

static thread_local char g_err[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

// ------------------------------------------------------------- profiling --
namespace {
struct PendingEv {
  std::string name;
  hipEvent_t a, b;
};
struct Stat {
  int64_t launches = 0;
  double ms = 0.0;
};
std::mutex g_prof_mu;
std::atomic<bool> g_prof{false};  // read without the lock on every launch
std::vector<PendingEv> g_pending;
std::vector<hipEvent_t> g_pool;
std::map<std::string, Stat> g_stats;

void drain_locked() {
  for (auto& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      Stat& s = g_stats[p.name];
      s.launches += 1;
      s.ms += ms;
    }
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
  }
  g_pending.clear();
}
}  // namespace

std::string g_prof_only;
int64_t g_prof_every = 1;
std::map<std::string, int64_t> g_prof_seen;  // launches of each profiled kernel so far

bool prof_on(const char* name) {
  if (!g_prof.load(std::memory_order_relaxed)) return false;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof || !(g_prof_only.empty() || g_prof_only == name)) return false;
  return g_prof_seen[name]++ % g_prof_every == 0;
}

void prof_events(hipEvent_t* a, hipEvent_t* b) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (g_pending.size() > 4096) drain_locked();
  for (hipEvent_t* e : {a, b}) {
    if (!g_pool.empty()) {
      *e = g_pool.back();
      g_pool.pop_back();
    } else {
      // timing only: no system-scope fence (cache writeback and invalidation)
      // when the event is recorded, so the timed launch and the work after it
      // run as they would untimed
      (void)hipEventCreateWithFlags(e, hipEventDisableSystemFence);
    }
  }
}

void prof_push(const char* name, hipEvent_t a, hipEvent_t b) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_pending.push_back(PendingEv{name, a, b});
}

}  // namespace sd

using namespace sd;

// --------------------------------------------------- no-allocation scratch --
// Device memory for sd_target_mean_noalloc: the target call's workspace (the
// split logits partials, the softmax weights and per-row coefficients) for
// callers that cannot allocate.  Every GPU the library runs on holds one copy
// until the process ends.  Host code must not use the array's name as an
// address: the device address of each GPU's copy comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kScratchBytes = (size_t)128 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_addr;  // device -> address of its copy of scratch

// The current device's copy of scratch (resolved on the first use on a device).
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  const auto it = g_scratch_addr.find(dev);
  if (it != g_scratch_addr.end()) {
    *out = it->second;
    return hipSuccess;
  }
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch_addr[dev] = ptr;
  *out = ptr;
  return hipSuccess;
}
}  // namespace

#define SD_CHECK_ARG(cond, ...)     \
  do {                              \
    if (!(cond)) {                  \
      set_error(__VA_ARGS__);       \
      return SD_EINVAL;             \
    }                               \
  } while (0)

#define SD_HIP(call)                                                           \
  do {                                                                         \
    hipError_t e_ = (call);                                                    \
    if (e_ != hipSuccess) {                                                    \
      set_error("%s failed: %s", #call, hipGetErrorString(e_));                \
      return SD_EHIP;                                                          \
    }                                                                          \
  } while (0)

static bool sched_ok(const sd_schedule* s) {
  return s && s->n_steps >= 1 && s->beta_min > 0.0 && s->beta_max >= s->beta_min &&
         s->churn > 0.0 && isfinite(s->beta_max) && isfinite(s->churn);
}

static bool stride_ok(sd_stride st, int d, int rows) {
  return st.row >= d && st.chain >= (int64_t)rows * st.row;
}

extern "C" {

int32_t sd_abi_version(void) { return SD_ABI_VERSION; }

const char* sd_last_error(void) { return g_err; }

sd_status sd_schedule_table(const sd_schedule* sched, double* host_out) {
  SD_CHECK_ARG(sched_ok(sched), "sd_schedule_table: invalid schedule (need N >= 1, 0 < beta_min <= beta_max, churn > 0)");
  SD_CHECK_ARG(host_out, "sd_schedule_table: host_out is NULL");
  const Sched sc = to_sched(sched);
  const int n1 = sc.N + 1;
  for (int n = 0; n <= sc.N; ++n) {
    host_out[n] = sched_signal(sc, n);
    host_out[n1 + n] = sched_sigma(sc, n);
    host_out[2 * n1 + n] = sched_c1(sc, n);
    host_out[3 * n1 + n] = sched_c2(sc, n);
  }
  return SD_OK;
}

// ---------------------------------------------------------------- target --
// float32 -> bf16 bits, round to nearest even (finite inputs).
static uint16_t bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

sd_status sd_target_create(const sd_schedule* sched, int32_t d, int32_t n_comp, const float* mu,
                           const float* var, const float* log_w, sd_precision precision,
                           sd_target* out) {
  SD_CHECK_ARG(out, "sd_target_create: out is NULL");
  *out = nullptr;
  SD_CHECK_ARG(sched_ok(sched), "sd_target_create: invalid schedule (need N >= 1, 0 < beta_min <= beta_max, churn > 0)");
  SD_CHECK_ARG(d >= 1, "sd_target_create: d = %d < 1", d);
  SD_CHECK_ARG(n_comp >= 1 && n_comp <= 1024, "sd_target_create: n_comp = %d not in [1, 1024]", n_comp);
  SD_CHECK_ARG(mu && var && log_w, "sd_target_create: mu/var/log_w must be host arrays");
  SD_CHECK_ARG(precision == SD_FP32 || precision == SD_BF16, "sd_target_create: unknown precision");
  for (int m = 0; m < n_comp; ++m) {
    SD_CHECK_ARG(var[m] > 0.0f && var[m] < 1.0e30f, "sd_target_create: var[%d] must be positive and finite", m);
    SD_CHECK_ARG(isfinite(log_w[m]), "sd_target_create: log_w[%d] is not finite", m);
  }
  const size_t M = (size_t)n_comp, D = (size_t)d;
  std::vector<float> muT(D * M);
  std::vector<double> vv(M), lw(M), msq(M);
  for (size_t m = 0; m < M; ++m) {
    double s = 0.0;
    for (size_t i = 0; i < D; ++i) {
      const float x = mu[m * D + i];
      if (!isfinite(x)) {
        set_error("sd_target_create: mu[%zu][%zu] is not finite", m, i);
        return SD_EINVAL;
      }
      s += (double)x * (double)x;
      muT[i * M + m] = x;
    }
    msq[m] = s;
    vv[m] = var[m];
    lw[m] = log_w[m];
  }
  Target* t = new Target();  // value-initialised: every pointer starts NULL
  t->sc = to_sched(sched);
  t->d = d;
  t->M = n_comp;
  t->prec = precision;
  (void)hipGetDevice(&t->device);
  const bool bf = precision == SD_BF16;
  // the operand copies of the chosen precision only
  bool ok = (bf ? hipMalloc(&t->mu16, sizeof(uint16_t) * M * D) == hipSuccess &&
                      hipMalloc(&t->muT16, sizeof(uint16_t) * M * D) == hipSuccess
                : hipMalloc(&t->mu, sizeof(float) * M * D) == hipSuccess &&
                      hipMalloc(&t->muT, sizeof(float) * M * D) == hipSuccess &&
                      hipMalloc(&t->mu_split, sizeof(uint16_t) * 3 * M * D) == hipSuccess &&
                      hipMalloc(&t->muT_split, sizeof(uint16_t) * 3 * M * D) == hipSuccess) &&
            hipMalloc(&t->ls, sizeof(double2) * M * (size_t)sched->n_steps) == hipSuccess &&
            hipMalloc(&t->logw, sizeof(double) * M) == hipSuccess &&
            hipMalloc(&t->musq, sizeof(double) * M) == hipSuccess &&
            hipMalloc(&t->coef, sizeof(float4) * (size_t)(sched->n_steps + 1)) == hipSuccess;
  if (!ok) {
    set_error("sd_target_create: device allocation failed");
    sd_target_destroy(reinterpret_cast<sd_target>(t));
    return SD_ENOMEM;
  }
  // the sampler's per-round flags: mapped pinned host words, one group per
  // concurrent sampler call
  if (hipHostMalloc(reinterpret_cast<void**>(&t->host_flags),
                    sizeof(int32_t) * kFlagGroups * kFlagSlots, hipHostMallocDefault) != hipSuccess ||
      hipHostGetDevicePointer(reinterpret_cast<void**>(&t->host_flags_dev), t->host_flags, 0) !=
          hipSuccess) {
    set_error("sd_target_create: mapped host flags could not be allocated");
    sd_target_destroy(reinterpret_cast<sd_target>(t));
    return SD_ENOMEM;
  }
  t->flag_busy = 0;
  // set-up of the no-allocation scratch on this device
  void* scr = nullptr;
  if (scratch_address(&scr) != hipSuccess) {
    set_error("sd_target_create: the scratch array's device address is not available");
    sd_target_destroy(reinterpret_cast<sd_target>(t));
    return SD_EHIP;
  }
  if (bf) {
    std::vector<uint16_t> h(M * D), hT(M * D);
    for (size_t m = 0; m < M; ++m)
      for (size_t i = 0; i < D; ++i) {
        const uint16_t v = bf16_rne(mu[m * D + i]);
        h[m * D + i] = v;
        hT[i * M + m] = v;
      }
    ok = hipMemcpy(t->mu16, h.data(), sizeof(uint16_t) * M * D, hipMemcpyHostToDevice) ==
             hipSuccess &&
         hipMemcpy(t->muT16, hT.data(), sizeof(uint16_t) * M * D, hipMemcpyHostToDevice) ==
             hipSuccess;
  } else {
    const size_t n = M * D;
    std::vector<uint16_t> sp(3 * n), spT(3 * n);
    split::split_host(mu, n, sp.data(), sp.data() + n, sp.data() + 2 * n);
    split::split_host(muT.data(), n, spT.data(), spT.data() + n, spT.data() + 2 * n);
    ok = hipMemcpy(t->mu, mu, sizeof(float) * n, hipMemcpyHostToDevice) == hipSuccess &&
         hipMemcpy(t->muT, muT.data(), sizeof(float) * n, hipMemcpyHostToDevice) == hipSuccess &&
         hipMemcpy(t->mu_split, sp.data(), sizeof(uint16_t) * 3 * n, hipMemcpyHostToDevice) ==
             hipSuccess &&
         hipMemcpy(t->muT_split, spT.data(), sizeof(uint16_t) * 3 * n, hipMemcpyHostToDevice) ==
             hipSuccess;
  }
  ok = ok &&

       hipMemcpy(t->logw, lw.data(), sizeof(double) * M, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(t->musq, msq.data(), sizeof(double) * M, hipMemcpyHostToDevice) == hipSuccess;
  std::vector<double2> ls(M * (size_t)sched->n_steps);
  for (int n = 0; n < sched->n_steps; ++n) {
    const double a = sched_signal(t->sc, n), a2 = a * a;
    for (size_t m = 0; m < M; ++m) {
      const double s2 = a2 * vv[m] + 1.0 - a2;
      ls[(size_t)n * M + m] = make_double2(log(s2), 1.0 / s2);
    }
  }
  ok = ok && hipMemcpy(t->ls, ls.data(), sizeof(double2) * ls.size(), hipMemcpyHostToDevice) ==
                 hipSuccess;
  std::vector<float4> coef((size_t)sched->n_steps + 1);
  for (int n = 0; n <= sched->n_steps; ++n) {
    const double c2 = sched_c2(t->sc, n);
    coef[n] = make_float4((float)sched_c1(t->sc, n), (float)c2, (float)sched_sigma(t->sc, n),
                          (float)(1.0 / c2));
  }
  ok = ok && hipMemcpy(t->coef, coef.data(), sizeof(float4) * coef.size(), hipMemcpyHostToDevice) ==
                 hipSuccess;
  if (!ok) {
    set_error("sd_target_create: copy to device failed");
    sd_target_destroy(reinterpret_cast<sd_target>(t));
    return SD_EHIP;
  }
  *out = reinterpret_cast<sd_target>(t);
  return SD_OK;
}

sd_status sd_target_destroy(sd_target target) {
  if (!target) return SD_OK;
  Target* t = reinterpret_cast<Target*>(target);
  if (t->mu) (void)hipFree(t->mu);
  if (t->muT) (void)hipFree(t->muT);
  if (t->mu_split) (void)hipFree(t->mu_split);
  if (t->muT_split) (void)hipFree(t->muT_split);
  if (t->mu16) (void)hipFree(t->mu16);
  if (t->muT16) (void)hipFree(t->muT16);
  if (t->ls) (void)hipFree(t->ls);
  if (t->logw) (void)hipFree(t->logw);
  if (t->musq) (void)hipFree(t->musq);
  if (t->coef) (void)hipFree(t->coef);
  // a flag group still held by a call that timed out may be written by its
  // kernels later: that memory and those side streams are then left alone
  const bool idle = __atomic_load_n(&t->flag_busy, __ATOMIC_ACQUIRE) == 0;
  if (t->host_flags && idle) (void)hipHostFree(t->host_flags);
  for (int g = 0; g < kFlagGroups && idle; ++g)
    if (t->side[g]) (void)hipStreamDestroy(t->side[g]);
  delete t;
  return SD_OK;
}

size_t sd_target_mean_workspace(sd_target target, int32_t rows) {
  if (!target || rows < 1) return 0;
  return target_ws_bytes(*reinterpret_cast<Target*>(target), rows);
}

sd_status sd_target_mean(sd_target target, int32_t rows, const float* x, int64_t x_row_stride,
                         const int32_t* step, float* mq, int64_t mq_row_stride, float* score,
                         int64_t score_row_stride, void* ws, size_t ws_bytes, sd_stream stream) {
  SD_CHECK_ARG(target, "sd_target_mean: target is NULL");
  const Target& t = *reinterpret_cast<Target*>(target);
  SD_CHECK_ARG(rows >= 1, "sd_target_mean: rows = %d < 1", rows);
  SD_CHECK_ARG(x && step && mq && ws, "sd_target_mean: x, step, mq and ws must be non-NULL");
  SD_CHECK_ARG(x_row_stride >= t.d && mq_row_stride >= t.d, "sd_target_mean: row strides must be >= d = %d", t.d);
  SD_CHECK_ARG(!score || score_row_stride >= t.d, "sd_target_mean: score row stride must be >= d");
  SD_CHECK_ARG(ws_bytes >= target_ws_bytes(t, rows), "sd_target_mean: workspace %zu < %zu bytes", ws_bytes, target_ws_bytes(t, rows));
  SD_CHECK_ARG(((uintptr_t)ws & 255u) == 0, "sd_target_mean: workspace must be 256-byte aligned");
  SD_HIP(target_mean_launch(t, rows, x, x_row_stride, step, mq, mq_row_stride, score,
                            score_row_stride, ws, (hipStream_t)stream, nullptr));
  return SD_OK;
}

sd_status sd_target_mean_noalloc(sd_target target, int32_t rows, const float* x,
                                 int64_t x_row_stride, const int32_t* step, float* mq,
                                 int64_t mq_row_stride, float* score, int64_t score_row_stride,
                                 sd_stream stream) {
  SD_CHECK_ARG(target, "sd_target_mean_noalloc: target is NULL");
  const Target& t = *reinterpret_cast<Target*>(target);
  SD_CHECK_ARG(rows >= 1, "sd_target_mean_noalloc: rows = %d < 1", rows);
  SD_CHECK_ARG(x && step && mq, "sd_target_mean_noalloc: x, step and mq must be non-NULL");
  SD_CHECK_ARG(x_row_stride >= t.d && mq_row_stride >= t.d, "sd_target_mean_noalloc: row strides must be >= d = %d", t.d);
  SD_CHECK_ARG(!score || score_row_stride >= t.d, "sd_target_mean_noalloc: score row stride must be >= d");
  const size_t need = target_ws_bytes(t, rows);
  SD_CHECK_ARG(need <= kScratchBytes,
               "sd_target_mean_noalloc: %d rows need %zu bytes of scratch, more than the %zu it holds "
               "(split the rows over calls)", rows, need, kScratchBytes);
  void* ws = nullptr;
  SD_HIP(scratch_address(&ws));
  SD_HIP(target_mean_launch(t, rows, x, x_row_stride, step, mq, mq_row_stride, score,
                            score_row_stride, ws, (hipStream_t)stream, nullptr));
  return SD_OK;
}

size_t sd_target_mean_noalloc_max_bytes(void) { return kScratchBytes; }

// ----------------------------------------------------------------- draft --
sd_status sd_init_chains(int32_t B, int32_t d, uint64_t seed, float* y, sd_stream stream) {
  SD_CHECK_ARG(B >= 1 && d >= 1, "sd_init_chains: need B >= 1 and d >= 1");
  SD_CHECK_ARG(y, "sd_init_chains: y is NULL");
  SD_HIP(init_chains_launch(B, d, seed, y, nullptr, 0, (hipStream_t)stream));
  return SD_OK;
}

sd_status sd_draft_block(const sd_schedule* sched, int32_t B, int32_t K, int32_t d,
                         const float* y, const float* cache_score, const int32_t* k,
                         const uint32_t* round, uint64_t seed, float* x, sd_stride xs, float* mp,
                         sd_stride mps, sd_stream stream) {
  SD_CHECK_ARG(sched_ok(sched), "sd_draft_block: invalid schedule");
  SD_CHECK_ARG(B >= 1 && d >= 1, "sd_draft_block: need B >= 1 and d >= 1");
  SD_CHECK_ARG(K >= 1 && K <= SD_MAX_BLOCK, "sd_draft_block: K = %d not in [1, %d]", K, SD_MAX_BLOCK);
  SD_CHECK_ARG(y && cache_score && k && round && x && mp, "sd_draft_block: NULL pointer argument");
  SD_CHECK_ARG(stride_ok(xs, d, K + 1), "sd_draft_block: x stride too small for [B][K+1][d]");
  SD_CHECK_ARG(stride_ok(mps, d, K), "sd_draft_block: mp stride too small for [B][K][d]");
  SD_HIP(draft_launch(to_sched(sched), B, K, d, y, cache_score, k, round, seed, x, xs, mp, mps,
                      (hipStream_t)stream, nullptr));
  return SD_OK;
}

// ---------------------------------------------------------------- verify --
static sd_status verify_impl(const char* fn, int32_t B, int32_t K, int32_t d, sd_verify_mode mode,
                             double omega, const float* y_draft, sd_stride ys, const float* mp,
                             sd_stride mps, const float* mq, sd_stride mqs, const double* sigma,
                             const int32_t* kb, const uint32_t* round, uint64_t seed,
                             sd_usample_mode usample_mode, int32_t* tau, double* log_alpha_res,
                             double* u_res, double* delta_norm, double* log_ratio,
                             uint64_t* coins, sd_stream stream) {
  SD_CHECK_ARG(B >= 1 && d >= 1, "%s: need B >= 1 and d >= 1", fn);
  SD_CHECK_ARG(K >= 1 && K <= SD_MAX_BLOCK, "%s: K = %d not in [1, %d]", fn, K, SD_MAX_BLOCK);
  SD_CHECK_ARG(mode == SD_BLOCK || mode == SD_TOKEN, "%s: unknown mode", fn);
  SD_CHECK_ARG(usample_mode == SD_USAMPLE_EXACT || usample_mode == SD_USAMPLE_PAPER, "%s: unknown usample mode", fn);
  SD_CHECK_ARG(omega > 0.0 && isfinite(omega) && omega * omega > 0.0 && isfinite(omega * omega),
               "%s: omega must be positive and finite, with omega^2 too", fn);
  SD_CHECK_ARG(y_draft && mp && mq && sigma && kb && round && tau && log_alpha_res && u_res &&
                   delta_norm && log_ratio,
               "%s: NULL pointer argument", fn);
  SD_CHECK_ARG(stride_ok(ys, d, K) && stride_ok(mps, d, K) && stride_ok(mqs, d, K),
               "%s: stride too small for [B][K][d]", fn);
  SD_HIP(verify_launch(B, K, d, (int)mode, y_draft, ys, mp, mps, mq, mqs, sigma, kb, round, seed,
                       (int)usample_mode, omega * omega, tau, log_alpha_res, u_res, delta_norm,
                       log_ratio, coins, nullptr, (hipStream_t)stream, nullptr));
  return SD_OK;
}

sd_status sd_verify_block(int32_t B, int32_t K, int32_t d, sd_verify_mode mode,
                          const float* y_draft, sd_stride ys, const float* mp, sd_stride mps,
                          const float* mq, sd_stride mqs, const double* sigma, const int32_t* kb,
                          const uint32_t* round, uint64_t seed, sd_usample_mode usample_mode,
                          int32_t* tau, double* log_alpha_res, double* u_res, double* delta_norm,
                          double* log_ratio, uint64_t* coins, sd_stream stream) {
  return verify_impl("sd_verify_block", B, K, d, mode, 1.0, y_draft, ys, mp, mps, mq, mqs, sigma,
                     kb, round, seed, usample_mode, tau, log_alpha_res, u_res, delta_norm,
                     log_ratio, coins, stream);
}

sd_status sd_verify_block_tempered(int32_t B, int32_t K, int32_t d, sd_verify_mode mode,
                                   double omega, const float* y_draft, sd_stride ys,
                                   const float* mp, sd_stride mps, const float* mq,
                                   sd_stride mqs, const double* sigma, const int32_t* kb,
                                   const uint32_t* round, uint64_t seed,
                                   sd_usample_mode usample_mode, int32_t* tau,
                                   double* log_alpha_res, double* u_res, double* delta_norm,
                                   double* log_ratio, uint64_t* coins, sd_stream stream) {
  return verify_impl("sd_verify_block_tempered", B, K, d, mode, omega, y_draft, ys, mp, mps, mq,
                     mqs, sigma, kb, round, seed, usample_mode, tau, log_alpha_res, u_res,
                     delta_norm, log_ratio, coins, stream);
}

// -------------------------------------------------------------- residual --
sd_status sd_sample_residual(int32_t B, int32_t K, int32_t d, const float* y_draft, sd_stride ys,
                             const float* mp, sd_stride mps, const float* mq, sd_stride mqs,
                             const double* sigma, const int32_t* kb, const int32_t* steps_left,
                             const int32_t* tau, const double* u_res, const double* delta_norm,
                             const uint32_t* round, uint64_t seed, float* y_out,
                             sd_stream stream) {
  SD_CHECK_ARG(B >= 1 && d >= 1, "sd_sample_residual: need B >= 1 and d >= 1");
  SD_CHECK_ARG(K >= 1 && K <= SD_MAX_BLOCK, "sd_sample_residual: K = %d not in [1, %d]", K, SD_MAX_BLOCK);
  SD_CHECK_ARG(y_draft && mp && mq && sigma && kb && steps_left && tau && u_res && delta_norm &&
                   round && y_out,
               "sd_sample_residual: NULL pointer argument");
  SD_CHECK_ARG(stride_ok(ys, d, K) && stride_ok(mps, d, K), "sd_sample_residual: stride too small for [B][K][d]");
  SD_CHECK_ARG(mqs.row >= d && mqs.chain >= (int64_t)(K + 1) * mqs.row,
               "sd_sample_residual: mq stride too small for [B][K+1][d]");
  SD_HIP(residual_launch(B, K, d, y_draft, ys, mp, mps, mq, mqs, sigma, kb, steps_left, tau,
                         u_res, delta_norm, round, seed, y_out, (hipStream_t)stream));
  return SD_OK;
}

sd_status sd_sample_residual_reflection(int32_t B, int32_t K, int32_t d, const float* y_draft,
                                        sd_stride ys, const float* mp, sd_stride mps,
                                        const float* mq, sd_stride mqs, const double* sigma,
                                        const int32_t* kb, const int32_t* steps_left,
                                        const int32_t* tau, const uint32_t* round, uint64_t seed,
                                        float* y_out, sd_stream stream) {
  SD_CHECK_ARG(B >= 1 && d >= 1, "sd_sample_residual_reflection: need B >= 1 and d >= 1");
  SD_CHECK_ARG(K >= 1 && K <= SD_MAX_BLOCK, "sd_sample_residual_reflection: K = %d not in [1, %d]", K, SD_MAX_BLOCK);
  SD_CHECK_ARG(y_draft && mp && mq && sigma && kb && steps_left && tau && round && y_out,
               "sd_sample_residual_reflection: NULL pointer argument");
  SD_CHECK_ARG(stride_ok(ys, d, K) && stride_ok(mps, d, K), "sd_sample_residual_reflection: stride too small for [B][K][d]");
  SD_CHECK_ARG(mqs.row >= d && mqs.chain >= (int64_t)(K + 1) * mqs.row,
               "sd_sample_residual_reflection: mq stride too small for [B][K+1][d]");
  SD_HIP(reflection_launch(B, K, d, y_draft, ys, mp, mps, mq, mqs, sigma, kb, steps_left, tau,
                           round, seed, y_out, (hipStream_t)stream));
  return SD_OK;
}

}  // extern "C"

// --------------------------------------------------------------- sampler --
namespace {

struct SamplerLayout {
  size_t y, x, sv, mq, sigma, step, k2, rnd2, crow2, cstep2, tau, rmode, rcoef, rsig, hist, steps,
      act, nan, kb, left, dummy_i32, dummy_i64, coins, lar, ures, ties, lrp, tws, tws1, total;
  size_t tws_bytes, tws1_bytes;
  int nct;
};

// With two chain groups, group 0 holds chains [0, B / 2) and group 1 the rest.
inline int group_chain0(int B, int groups, int g) { return groups == 2 && g == 1 ? B / 2 : 0; }
inline int group_chains(int B, int groups, int g) {
  return groups == 2 ? (g == 0 ? B / 2 : B - B / 2) : B;
}

// The library's choice of chain groups (sd_sampler_options.groups = 0): two
// when each half still has 2048 target rows or more.  Measured (one group /
// two, ms per run): pixel3072 30.6 / 29.0, pixel12288 232 / 222, latent16384
// 249 / 255 -- its 2304 rows make a logits grid of 252 one-per-CU workgroups,
// and two halves need 280, a second wave.
inline int choose_groups(int B, int K, int requested) {
  if (B < 2) return 1;
  if (requested == 1 || requested == 2) return requested;
  return (int64_t)(B / 2) * (K + 1) >= 2048 ? 2 : 1;
}

inline size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

SamplerLayout sampler_layout(const Target& t, int B, int K) {
  SamplerLayout L{};
  const size_t d = t.d, Bs = B, K1 = K + 1;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = a256(off + bytes);
    return o;
  };
  L.nct = lr_tiles(t, (int)K1);
  L.y = take(4 * Bs * d);
  L.x = take(4 * Bs * K1 * d);
  L.sv = take(4 * Bs * d);
  L.mq = take(4 * Bs * K1 * d);
  L.sigma = take(8 * Bs * K1);
  L.step = take(4 * Bs * K1);
  L.k2 = take(4 * 2 * Bs);
  L.rnd2 = take(4 * 2 * Bs);
  L.crow2 = take(4 * 2 * Bs);
  L.cstep2 = take(4 * 2 * Bs);
  L.tau = take(4 * Bs);
  L.rmode = take(4 * Bs);
  L.rcoef = take(4 * Bs);
  L.rsig = take(4 * Bs);
  L.hist = take(4 * Bs * (SD_MAX_BLOCK + 2));
  L.steps = take(8 * Bs);
  L.act = take(4 * 2 * 2);  // [group][round parity]
  L.nan = take(4);
  L.kb = take(4 * Bs);
  L.left = take(4 * Bs);
  L.dummy_i32 = take(4 * (Bs + 2));
  L.dummy_i64 = take(8 * (SD_MAX_BLOCK + 3));
  L.coins = take(8 * Bs);
  L.lar = take(8 * Bs);
  L.ures = take(8 * Bs);
  L.ties = take(4 * Bs);
  L.lrp = take(8 * 3 * Bs * K1 * (size_t)L.nct);
  // the target calls on all B (K + 1) rows and, with the Frozen Drafter, on the
  // B states alone (fewer rows may take more splits of the logits GEMM); with
  // two chain groups each group's calls on its own rows, split as for all
  // rows (so that every row is summed in the same order)
  const int rows = (int)(Bs * K1);
  L.tws_bytes = std::max(target_ws_bytes(t, rows), target_ws_bytes(t, B));
  L.tws1_bytes = 0;
  if (B >= 2) {
    const int b0 = B / 2, b1 = B - B / 2;
    L.tws_bytes = std::max({L.tws_bytes, target_ws_bytes(t, b0 * (int)K1, rows), target_ws_bytes(t, b0, B)});
    L.tws1_bytes = std::max(target_ws_bytes(t, b1 * (int)K1, rows), target_ws_bytes(t, b1, B));
  }
  L.tws = take(L.tws_bytes);
  L.tws1 = take(L.tws1_bytes);
  L.total = off;
  return L;
}

}  // namespace

extern "C" {

size_t sd_sampler_workspace(sd_target target, int32_t B, int32_t K) {
  if (!target || B < 1 || K < 1 || K > SD_MAX_BLOCK) return 0;
  return sampler_layout(*reinterpret_cast<Target*>(target), B, K).total;
}

sd_status sd_run_sampler(sd_target target, int32_t B, int32_t K, sd_verify_mode mode,
                         sd_usample_mode usample_mode, uint64_t seed, float* y_out,
                         int32_t* tau_trace, int32_t trace_rounds, sd_stats* stats, void* ws,
                         size_t ws_bytes, sd_stream stream) {
  const sd_sampler_options o{mode, usample_mode, SD_RESIDUAL_DECOMPOSITION, SD_DRAFTER_FREE, 1.0, 0, -1, 0};
  return sd_run_sampler_ex(target, B, K, &o, seed, y_out, tau_trace, trace_rounds, stats, ws,
                           ws_bytes, stream);
}

}  // extern "C"

namespace {

using Clock = std::chrono::steady_clock;

// A sampler call gives up on a GPU that finishes no round for this long.
constexpr int kStallSeconds = 120;

// Wait for the stream without blocking in the runtime past the deadline:
// hipSuccess, the stream's error, or hipErrorNotReady with *timed_out set.
hipError_t wait_bounded(hipStream_t s, Clock::time_point deadline, bool* timed_out) {
  *timed_out = false;
  for (;;) {
    const hipError_t q = hipStreamQuery(s);
    if (q != hipErrorNotReady) return q;
    (void)hipGetLastError();  // not-ready is a status, not a failure
    if (Clock::now() >= deadline) {
      *timed_out = true;
      return q;
    }
    std::this_thread::sleep_for(std::chrono::microseconds(50));
  }
}

// One group of the target's mapped flag words for the duration of a call.
int acquire_flags(Target* t) {
  uint64_t cur = __atomic_load_n(&t->flag_busy, __ATOMIC_ACQUIRE);
  while (cur != ~0ull) {
    const int g = __builtin_ctzll(~cur);
    if (__atomic_compare_exchange_n(&t->flag_busy, &cur, cur | (1ull << g), false,
                                    __ATOMIC_ACQ_REL, __ATOMIC_ACQUIRE))
      return g;
  }
  return -1;
}

void release_flags(Target* t, int g) {
  __atomic_fetch_and(&t->flag_busy, ~(1ull << g), __ATOMIC_RELEASE);
}

}  // namespace

extern "C" {

sd_status sd_run_sampler_ex(sd_target target, int32_t B, int32_t K,
                            const sd_sampler_options* opts, uint64_t seed, float* y_out,
                            int32_t* tau_trace, int32_t trace_rounds, sd_stats* stats, void* ws,
                            size_t ws_bytes, sd_stream stream) {
  SD_CHECK_ARG(opts, "sd_run_sampler: options are NULL");
  const sd_verify_mode mode = opts->mode;
  const sd_usample_mode usample_mode = opts->usample_mode;
  SD_CHECK_ARG(mode == SD_BLOCK || mode == SD_TOKEN, "sd_run_sampler: unknown mode");
  SD_CHECK_ARG(usample_mode == SD_USAMPLE_EXACT || usample_mode == SD_USAMPLE_PAPER, "sd_run_sampler: unknown usample mode");
  SD_CHECK_ARG(opts->residual == SD_RESIDUAL_DECOMPOSITION || opts->residual == SD_RESIDUAL_REFLECTION,
               "sd_run_sampler: unknown residual");
  SD_CHECK_ARG(opts->residual == SD_RESIDUAL_DECOMPOSITION || mode == SD_TOKEN,
               "sd_run_sampler: the reflection residual needs sample (token) verification");
  SD_CHECK_ARG(opts->drafter == SD_DRAFTER_FREE || opts->drafter == SD_DRAFTER_FROZEN,
               "sd_run_sampler: unknown drafter");
  SD_CHECK_ARG(opts->omega > 0.0 && isfinite(opts->omega) && opts->omega * opts->omega > 0.0 &&
                   isfinite(opts->omega * opts->omega),
               "sd_run_sampler: omega must be positive and finite, with omega^2 too");
  SD_CHECK_ARG(opts->start_round >= 0, "sd_run_sampler: start_round must be >= 0");
  SD_CHECK_ARG(opts->groups >= 0 && opts->groups <= 2, "sd_run_sampler: groups = %d not in 0..2",
               opts->groups);
  SD_CHECK_ARG(target, "sd_run_sampler: target is NULL");
  Target* tp = reinterpret_cast<Target*>(target);
  const Target& t = *tp;
  SD_CHECK_ARG(B >= 1, "sd_run_sampler: B = %d < 1", B);
  SD_CHECK_ARG(K >= 1 && K <= SD_MAX_BLOCK, "sd_run_sampler: K = %d not in [1, %d]", K, SD_MAX_BLOCK);
  const bool frozen = opts->drafter == SD_DRAFTER_FROZEN;
  const bool reflect = opts->residual == SD_RESIDUAL_REFLECTION;
  const double w2 = opts->omega * opts->omega;
  SD_CHECK_ARG(y_out && ws, "sd_run_sampler: y_out and ws must be non-NULL");
  SD_CHECK_ARG(!tau_trace || trace_rounds >= 0, "sd_run_sampler: trace_rounds < 0");
  SD_CHECK_ARG(((uintptr_t)ws & 255u) == 0, "sd_run_sampler: workspace must be 256-byte aligned");
  const SamplerLayout L = sampler_layout(t, B, K);
  SD_CHECK_ARG(ws_bytes >= L.total, "sd_run_sampler: workspace %zu < %zu bytes", ws_bytes, L.total);
  SD_CHECK_ARG((int64_t)B * (K + 1) <= INT32_MAX, "sd_run_sampler: B*(K+1) rows exceed int32");
  const int N = t.sc.N;
  // a round advances every active chain by at least one step, so at most N
  // rounds have work
  constexpr int kLag = 3;
  static_assert(kLag + 1 <= kFlagSlots, "a flag group must hold kLag + 1 rounds");
  const int start = opts->start_round;
  const int64_t cap = (int64_t)N + 1 + kLag;
  SD_CHECK_ARG(start <= cap, "sd_run_sampler: start_round %d beyond the %lld rounds a run can have",
               start, (long long)cap);
  const int end = (int)std::min<int64_t>(cap, opts->max_rounds >= 0
                                                  ? (int64_t)start + opts->max_rounds
                                                  : cap);

  hipStream_t s = (hipStream_t)stream;
  char* base = static_cast<char*>(ws);
  auto F = [&](size_t o) { return reinterpret_cast<float*>(base + o); };
  auto I = [&](size_t o) { return reinterpret_cast<int32_t*>(base + o); };
  auto D = [&](size_t o) { return reinterpret_cast<double*>(base + o); };
  const int d = t.d, K1 = K + 1;
  float *y = F(L.y), *x = F(L.x), *sv = F(L.sv), *mq = F(L.mq), *rcoef = F(L.rcoef),
        *rsig = F(L.rsig);
  double *sigma = D(L.sigma), *lrp = D(L.lrp), *lar = D(L.lar), *ures = D(L.ures);
  int32_t *step = I(L.step), *k2 = I(L.k2), *crow2 = I(L.crow2), *cstep2 = I(L.cstep2),
          *tau = I(L.tau), *rmode = I(L.rmode), *hist = I(L.hist), *act = I(L.act),
          *nanflag = I(L.nan), *kb = I(L.kb), *left = I(L.left), *dummy = I(L.dummy_i32),
          *ties = I(L.ties);
  uint32_t* rnd2 = reinterpret_cast<uint32_t*>(base + L.rnd2);
  uint64_t* coins = reinterpret_cast<uint64_t*>(base + L.coins);
  int64_t* steps = reinterpret_cast<int64_t*>(base + L.steps);
  int64_t* dummy64 = reinterpret_cast<int64_t*>(base + L.dummy_i64);
  void* tws = base + L.tws;
  const sd_stride xs{(int64_t)K1 * d, d}, mqs{(int64_t)K1 * d, d};
  const int G = choose_groups(B, K, opts->groups);
  // the draft rows are streamed past the caches, or not, as for the whole block
  const int64_t block_bytes = (int64_t)B * K1 * d * 4;

  if (start == 0) {
    // Y_0 (also row 0 of x); the one explicit target call at Y_0, whose mean
    // (row 0 of mq) seeds the Free Drafter's cached score; the round-0 rows'
    // steps and sigmas; the first draft block.  The Frozen Drafter makes that
    // call and draft at the start of every round instead.
    SD_HIP(fill_i32_launch(k2, 2 * (int64_t)B, 0, s));
    SD_HIP(fill_i32_launch(reinterpret_cast<int32_t*>(rnd2), 2 * (int64_t)B, 0, s));
    SD_HIP(fill_i32_launch(crow2, 2 * (int64_t)B, 0, s));
    SD_HIP(fill_i32_launch(cstep2, 2 * (int64_t)B, 0, s));
    SD_HIP(fill_i32_launch(hist, (int64_t)B * (SD_MAX_BLOCK + 2), 0, s));
    SD_HIP(fill_i64_launch(steps, B, 0, s));
    SD_HIP(fill_i32_launch(ties, B, 0, s));
    SD_HIP(fill_i32_launch(act, 4, 0, s));
    SD_HIP(fill_i32_launch(nanflag, 1, 0, s));
    SD_HIP(fill_i32_launch(step, B, 0, s));
    SD_HIP(fill_i32_launch(tau, B, 0, s));
    SD_HIP(fill_i32_launch(dummy, B + 2, 0, s));
    SD_HIP(init_chains_launch(B, d, seed, y, x, (int64_t)K1 * d, s));
    if (!frozen)
      SD_HIP(target_mean_launch(t, B, x, (int64_t)K1 * d, step, mq, (int64_t)K1 * d, nullptr, 0,
                                tws, s, nullptr));
    SD_HIP(prepare_launch(t.sc, B, K, k2, kb, left, step, sigma, tau, dummy, dummy + B,
                          dummy + B + 1, dummy64, dummy64 + SD_MAX_BLOCK + 2, s));
    if (!frozen)
      SD_HIP(draft_cached_launch(t.sc, t.coef, B, K, d, y, crow2, cstep2, mq, mqs, k2, rnd2, seed,
                                 x, xs, sv, s, nullptr));
  }
  // each group's gate of round `start` (whether any of its chains is still
  // active), from the chains' steps: a resumed run may group its chains
  // differently from the call that left the state
  const int par0 = start & 1;
  SD_HIP(chains_active_launch(B, G == 2 ? B / 2 : B, N, k2 + par0 * B, act + par0, act + 2 + par0, s));

  // Round r's scan publishes round r - 1's active flag, tagged with r - 1, into
  // slot (r - 1) % kFlagSlots of its group's block of mapped host words.  After
  // enqueueing round r the host polls round r - kLag's slots until the tags are
  // there (the queue stays kLag rounds ahead) and stops enqueueing once every
  // group's flag is cleared.  No event or copy is queued per round: a marker
  // between rounds would hold the next round's first kernel back by several
  // microseconds.  The first flag this call reads is that of round start - 1
  // (published by round start's scan), so a finished run is seen at once.
  // With two chain groups the second group's rounds run on a second stream,
  // forked from `stream` after the first group's first target call (so that
  // the two run half a round apart: one group's latency-bound scan and
  // residual overlap the other's GEMMs) and joined back into it at the end.
  struct GroupRun {
    int c0, nb, grp;
    void* tws;
    hipStream_t st;
    int32_t* host_dev;
    volatile int32_t* pub;
  };
  GroupRun gr[2]{};
  auto release_all = [&]() {
    for (int g = 0; g < G; ++g)
      if (gr[g].grp >= 0) release_flags(tp, gr[g].grp);
  };
  for (int g = 0; g < G; ++g) gr[g].grp = -1;
  for (int g = 0; g < G; ++g) {
    GroupRun& q = gr[g];
    q.c0 = group_chain0(B, G, g);
    q.nb = group_chains(B, G, g);
    q.tws = g == 0 ? tws : base + L.tws1;
    q.grp = acquire_flags(tp);
    if (q.grp < 0) {
      release_all();
      set_error("sd_run_sampler: more than %d sampler calls (or chain groups) at once on one target",
                kFlagGroups);
      return SD_EUNSUPPORTED;
    }
    int32_t* const host_act = t.host_flags + q.grp * kFlagSlots;
    q.host_dev = t.host_flags_dev + q.grp * kFlagSlots;
    for (int i = 0; i < kFlagSlots; ++i) host_act[i] = -1;  // tag -1: nothing published
    q.pub = host_act;
    q.st = s;
    if (g == 1) {
      hipStream_t& side = tp->side[q.grp];
      if (!side && hipStreamCreateWithFlags(&side, hipStreamNonBlocking) != hipSuccess) {
        side = nullptr;
        release_all();
        set_error("sd_run_sampler: the second chain group's stream could not be created");
        return SD_EHIP;
      }
      q.st = side;
    }
  }
  std::atomic_thread_fence(std::memory_order_seq_cst);
  hipEvent_t fork = nullptr, join = nullptr;
  if (G == 2) {
    if (hipEventCreateWithFlags(&fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&join, hipEventDisableTiming) != hipSuccess) {
      release_all();
      set_error("sd_run_sampler: could not create the events of the second chain group");
      return SD_EHIP;
    }
  }
  bool forked = false;
  constexpr int kQuietMs = 20;
  const int first_flag = start > 0 ? start - 1 : 0;
  sd_status st = SD_OK;
  bool stalled = false;
  int64_t rounds = -1;
  Clock::time_point last_progress = Clock::now();
  int r = start;
  auto enqueue = [&](int g, int cur, int nxt) -> hipError_t {
    const GroupRun& q = gr[g];
    const int b0 = q.c0, nb = q.nb;
    const int64_t rows0 = (int64_t)b0 * K1;
    float *xg = x + rows0 * d, *mqg = mq + rows0 * d, *svg = sv + (int64_t)b0 * d,
          *yg = y + (int64_t)b0 * d;
    int32_t* stepg = step + rows0;
    double *sigmag = sigma + rows0, *lrpg = lrp + rows0 * L.nct * 3;
    const int32_t *kc = k2 + cur * B + b0, *crc = crow2 + cur * B + b0, *csc = cstep2 + cur * B + b0;
    const uint32_t* rc = rnd2 + cur * B + b0;
    const int* gate = act + 2 * g + cur;
    int* next = act + 2 * g + nxt;
    hipError_t e = hipSuccess;
    if (frozen) {
      // the Frozen Drafter's target call at (Y_k, k) into row 0 of m^q (the
      // cache steps hold min(k, N - 1)), then the block drafted with that score
      e = target_mean_launch(t, nb, xg, (int64_t)K1 * d, csc, mqg, (int64_t)K1 * d, nullptr, 0, q.tws,
                             q.st, gate, B);
      if (e == hipSuccess)
        e = draft_cached_launch(t.sc, t.coef, nb, K, d, yg, crc, csc, mqg, mqs, kc, rc, seed, xg, xs, svg,
                                q.st, gate, b0, block_bytes);
    }
    if (e == hipSuccess)
      e = target_mean_lr_launch(t, nb * K1, K1, xg, stepg, mqg, svg, csc, lrpg, rc, seed, q.tws, q.st,
                                gate, B * K1, b0);
    if (G == 2 && !forked && e == hipSuccess) {
      // (the first group's first round: everything before this is on `stream`)
      e = hipEventRecord(fork, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(gr[1].st, fork, 0);
      forked = e == hipSuccess;
    }
    int32_t* publish = r >= 1 ? q.host_dev + (r - 1) % kFlagSlots : nullptr;
    if (e == hipSuccess)
      e = scan_fused_launch(nb, K, d, N, (int)mode, (int)usample_mode, lrpg, L.nct, sigmag, kc, rc, seed,
                            w2, reflect, tau + b0, rmode + b0, rcoef + b0, rsig + b0, coins + b0,
                            lar + b0, ures + b0, ties + b0, nanflag, next, publish, r - 1, q.st, gate,
                            b0);
    if (e == hipSuccess)
      e = advance_launch(t.sc, t.coef, nb, K, d, seed, kc, rc, crc, csc, k2 + nxt * B + b0,
                         rnd2 + nxt * B + b0, crow2 + nxt * B + b0, cstep2 + nxt * B + b0, tau + b0,
                         rmode + b0, rcoef + b0, rsig + b0, xg, svg, mqg, yg, stepg, sigmag,
                         hist + (int64_t)b0 * (SD_MAX_BLOCK + 2), steps + b0, next,
                         tau_trace ? tau_trace + b0 : nullptr, r, tau_trace ? trace_rounds : 0,
                         frozen, q.st, gate, b0, B, block_bytes);
    return e;
  };
  for (; r < end && rounds < 0; ++r) {
    const int cur = r & 1, nxt = cur ^ 1;
    hipError_t e = hipSuccess;
    for (int g = 0; g < G && e == hipSuccess; ++g) e = enqueue(g, cur, nxt);
    if (e != hipSuccess) {
      set_error("sd_run_sampler: launch failed in round %d: %s", r, hipGetErrorString(e));
      st = SD_EHIP;
      break;
    }
    const int back = r - kLag;
    if (back >= first_flag) {
      // round back + 1's scans (enqueued) publish round back's flags; each
      // wait ends on the tag, or on an error or a drained stream reported by
      // the runtime.  The runtime is asked only after kQuietMs without the
      // tag: a stream query queues a marker whose system-scope release holds
      // the next kernel back by several microseconds.
      bool any = false;
      for (int g = 0; g < G && st == SD_OK; ++g) {
        volatile int32_t* slot = gr[g].pub + back % kFlagSlots;
        int32_t v;
        auto next_query = Clock::now() + std::chrono::milliseconds(kQuietMs);
        for (uint32_t spin = 1; ((v = *slot) >> 1) != back; ++spin) {
          if ((spin & 1023u) != 0) continue;
          const Clock::time_point now = Clock::now();
          if (now - last_progress > std::chrono::seconds(kStallSeconds)) {
            set_error("sd_run_sampler: no round finished within %d s (round %d); the GPU may be hung",
                      kStallSeconds, back);
            st = SD_EHIP;
            stalled = true;
            break;
          }
          if (now < next_query) continue;
          next_query = now + std::chrono::milliseconds(kQuietMs);
          const hipError_t q = hipStreamQuery(gr[g].st);
          // not-ready is a status, not a failure: keep it out of the launch checks
          if (q == hipErrorNotReady) {
            (void)hipGetLastError();
            continue;
          }
          v = *slot;
          if (q == hipSuccess && (v >> 1) == back) break;
          set_error("sd_run_sampler: round %d's flag was not published (%s)", back,
                    hipGetErrorString(q));
          st = SD_EHIP;
          break;
        }
        if (st == SD_OK && (v & 1) != 0) any = true;
      }
      if (st != SD_OK) break;
      last_progress = Clock::now();
      if (!any) rounds = back + 1;
    }
  }
  if (stalled) return st;  // the kernels may still write to the flag groups: keep them
  if (G == 2) {
    // the second group's work, done or failed, is ordered before what follows on `stream`
    hipError_t e = hipEventRecord(join, gr[1].st);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, join, 0);
    if (e != hipSuccess) {
      set_error("sd_run_sampler: could not join the second chain group's stream: %s",
                hipGetErrorString(e));
      return SD_EHIP;  // keep the flag groups: the second stream may still run
    }
  }
  const Clock::time_point deadline = Clock::now() + std::chrono::seconds(kStallSeconds);
  bool finished = rounds >= 0;
  if (st == SD_OK && !finished) {
    // every launched round finishes; the flags of rounds up to r - 2 are then
    // in their slots, and the last round's, which no later scan publishes, is
    // copied
    int32_t last_flag[2] = {1, 1};
    hipError_t e = hipSuccess;
    bool late = false;
    if (r > start) {
      for (int g = 0; g < G && e == hipSuccess; ++g)
        e = hipMemcpyAsync(&last_flag[g], act + 2 * g + (r & 1), sizeof(int32_t), hipMemcpyDeviceToHost, s);
      if (e == hipSuccess) e = wait_bounded(s, deadline, &late);
    }
    if (late) {
      set_error("sd_run_sampler: the last rounds did not finish within %d s", kStallSeconds);
      return SD_EHIP;  // keep the flag groups (see above)
    }
    if (e != hipSuccess) {
      set_error("sd_run_sampler: waiting for the last rounds failed: %s", hipGetErrorString(e));
      st = SD_EHIP;
    }
    for (int back = std::max(r - kLag, first_flag); st == SD_OK && back < r; ++back) {
      bool any = false;
      for (int g = 0; g < G; ++g) {
        const int32_t v = gr[g].pub[back % kFlagSlots];
        const int32_t flag = back == r - 1 ? last_flag[g] : ((v >> 1) == back ? (v & 1) : 1);
        if (flag != 0) any = true;
      }
      if (!any) {
        rounds = back + 1;
        finished = true;
        break;
      }
    }
    if (st == SD_OK && !finished) {
      if (r < cap) {
        rounds = r;  // a partial call: the state after round r - 1 is in ws
      } else {
        set_error("sd_run_sampler: chains still active after %d rounds", r);
        st = SD_EHIP;
      }
    }
  }
  if (st == SD_OK) {
    std::vector<int32_t> h_hist((size_t)B * (SD_MAX_BLOCK + 2)), h_ties(B);
    std::vector<int64_t> h_steps(B);
    int32_t h_nan = 0;
    hipError_t e = hipSuccess;
    if (finished)
      e = hipMemcpyAsync(y_out, y, sizeof(float) * (size_t)B * d, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(h_hist.data(), hist, sizeof(int32_t) * h_hist.size(), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(h_steps.data(), steps, sizeof(int64_t) * B, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(h_ties.data(), ties, sizeof(int32_t) * B, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&h_nan, nanflag, sizeof(int32_t), hipMemcpyDeviceToHost, s);
    bool late = false;
    if (e == hipSuccess) e = wait_bounded(s, deadline, &late);
    if (late) {
      set_error("sd_run_sampler: the final copies did not finish within %d s", kStallSeconds);
      return SD_EHIP;  // keep the flag groups (see above)
    }
    if (e != hipSuccess) {
      set_error("sd_run_sampler: final copy failed: %s", hipGetErrorString(e));
      st = SD_EHIP;
    } else {
      if (stats) {
        memset(stats, 0, sizeof(*stats));
        stats->rounds = rounds;
        stats->finished = finished ? 1 : 0;
        stats->groups = G;
        double tau_sum = 0.0;
        for (int b = 0; b < B; ++b) {
          stats->steps += h_steps[b];
          stats->ties += h_ties[b];
          for (int i = 0; i < SD_MAX_BLOCK + 2; ++i) stats->tau_hist[i] += h_hist[(size_t)b * (SD_MAX_BLOCK + 2) + i];
        }
        for (int i = 0; i < SD_MAX_BLOCK + 2; ++i) {
          stats->chain_rounds += stats->tau_hist[i];
          tau_sum += (double)i * (double)stats->tau_hist[i];
        }
        stats->mean_tau = stats->chain_rounds > 0 ? tau_sum / (double)stats->chain_rounds : 0.0;
      }
      if (h_nan) {
        set_error("sd_run_sampler: non-finite log-ratio met");
        st = SD_ENUMERIC;
      }
    }
  }
  bool late = false;
  (void)wait_bounded(s, deadline, &late);
  if (late) {
    if (st == SD_OK) {
      set_error("sd_run_sampler: the stream did not drain within %d s", kStallSeconds);
      st = SD_EHIP;
    }
    return st;  // keep the flag groups (see above)
  }
  release_all();
  if (fork) (void)hipEventDestroy(fork);
  if (join) (void)hipEventDestroy(join);
  return st;
}

sd_status sd_sampler_state(sd_target target, int32_t B, int32_t K, void* ws, size_t ws_bytes,
                           int64_t rounds, sd_sampler_view* out) {
  SD_CHECK_ARG(target && ws && out, "sd_sampler_state: NULL pointer argument");
  SD_CHECK_ARG(B >= 1 && K >= 1 && K <= SD_MAX_BLOCK, "sd_sampler_state: need B >= 1 and K in [1, %d]",
               SD_MAX_BLOCK);
  SD_CHECK_ARG(rounds >= 0, "sd_sampler_state: rounds < 0");
  const Target& t = *reinterpret_cast<Target*>(target);
  const SamplerLayout L = sampler_layout(t, B, K);
  SD_CHECK_ARG(ws_bytes >= L.total, "sd_sampler_state: workspace %zu < %zu bytes", ws_bytes, L.total);
  char* base = static_cast<char*>(ws);
  const int cur = (int)(rounds & 1);
  memset(out, 0, sizeof(*out));
  out->x = reinterpret_cast<float*>(base + L.x);
  out->y = reinterpret_cast<float*>(base + L.y);
  out->cache = reinterpret_cast<float*>(base + L.sv);
  out->cache_step = reinterpret_cast<int32_t*>(base + L.cstep2) + cur * B;
  out->k = reinterpret_cast<int32_t*>(base + L.k2) + cur * B;
  out->round = reinterpret_cast<uint32_t*>(base + L.rnd2) + cur * B;
  out->mq = reinterpret_cast<float*>(base + L.mq);
  out->lrp = reinterpret_cast<double*>(base + L.lrp);
  out->n_tiles = L.nct;
  out->tau = reinterpret_cast<int32_t*>(base + L.tau);
  out->coins = reinterpret_cast<uint64_t*>(base + L.coins);
  out->log_alpha_res = reinterpret_cast<double*>(base + L.lar);
  out->u = reinterpret_cast<double*>(base + L.ures);
  out->ties = reinterpret_cast<int32_t*>(base + L.ties);
  return SD_OK;
}

// ------------------------------------------------------------- plain EM --
static size_t em_ws_bytes(const Target& t, int B) {
  return a256(sizeof(float) * (size_t)B * t.d) + a256(sizeof(int32_t) * (size_t)B) +
         target_ws_bytes(t, B);
}

size_t sd_plain_em_workspace(sd_target target, int32_t B) {
  if (!target || B < 1) return 0;
  return em_ws_bytes(*reinterpret_cast<Target*>(target), B);
}

sd_status sd_run_plain_em(sd_target target, int32_t B, uint64_t seed, float* y_out, void* ws,
                          size_t ws_bytes, sd_stream stream) {
  SD_CHECK_ARG(target, "sd_run_plain_em: target is NULL");
  const Target& t = *reinterpret_cast<Target*>(target);
  SD_CHECK_ARG(B >= 1, "sd_run_plain_em: B = %d < 1", B);
  SD_CHECK_ARG(y_out && ws, "sd_run_plain_em: y_out and ws must be non-NULL");
  SD_CHECK_ARG(((uintptr_t)ws & 255u) == 0, "sd_run_plain_em: workspace must be 256-byte aligned");
  SD_CHECK_ARG(ws_bytes >= em_ws_bytes(t, B), "sd_run_plain_em: workspace %zu < %zu bytes", ws_bytes, em_ws_bytes(t, B));
  hipStream_t s = (hipStream_t)stream;
  char* base = static_cast<char*>(ws);
  float* mq = reinterpret_cast<float*>(base);
  int32_t* step = reinterpret_cast<int32_t*>(base + a256(sizeof(float) * (size_t)B * t.d));
  void* tws = base + a256(sizeof(float) * (size_t)B * t.d) + a256(sizeof(int32_t) * (size_t)B);
  const int d = t.d;
  SD_HIP(init_chains_launch(B, d, seed, y_out, nullptr, 0, s));
  SD_HIP(fill_i32_launch(step, B, 0, s));
  for (int n = 0; n < t.sc.N; ++n) {
    SD_HIP(target_mean_launch(t, B, y_out, d, step, mq, d, nullptr, 0, tws, s, nullptr));
    SD_HIP(em_noise_launch(B, d, n, (float)sched_sigma(t.sc, n), seed, mq, y_out, step, s));
  }
  return SD_OK;
}

// ------------------------------------------------------------- profiling --
sd_status sd_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (on) {
    drain_locked();
    g_stats.clear();
    g_prof_seen.clear();
  }
  g_prof = on != 0;
  return SD_OK;
}

sd_status sd_profile_only(const char* name) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_only = name ? name : "";
  return SD_OK;
}

sd_status sd_profile_every(int32_t n) {
  SD_CHECK_ARG(n >= 1, "sd_profile_every: n < 1");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_every = n;
  g_prof_seen.clear();
  return SD_OK;
}

sd_status sd_profile_seen(const char* name, int64_t* count) {
  SD_CHECK_ARG(name && count, "sd_profile_seen: NULL pointer argument");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  const auto it = g_prof_seen.find(name);
  *count = it == g_prof_seen.end() ? 0 : it->second;
  return SD_OK;
}

sd_status sd_profile_read(sd_kernel_stat* out, int32_t capacity, int32_t* count) {
  SD_CHECK_ARG(count, "sd_profile_read: count is NULL");
  SD_CHECK_ARG(capacity >= 0 && (capacity == 0 || out), "sd_profile_read: out is NULL");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  drain_locked();
  int i = 0;
  for (auto& kv : g_stats) {
    if (i < capacity) {
      memset(&out[i], 0, sizeof(out[i]));
      strncpy(out[i].name, kv.first.c_str(), sizeof(out[i].name) - 1);
      out[i].launches = kv.second.launches;
      out[i].total_ms = kv.second.ms;
    }
    ++i;
  }
  *count = i;
  return SD_OK;
}

// ----------------------------------------------------------- test hooks --
sd_status sd_philox_words(uint64_t seed, int32_t n, const uint32_t* counters, uint32_t* out,
                          sd_stream stream) {
  SD_CHECK_ARG(n >= 0, "sd_philox_words: n < 0");
  SD_CHECK_ARG(n == 0 || (counters && out), "sd_philox_words: NULL pointer argument");
  SD_HIP(philox_words_launch(seed, n, counters, out, (hipStream_t)stream));
  return SD_OK;
}

sd_status sd_philox_normals(uint64_t seed, uint32_t chain, uint32_t round, uint32_t tag,
                            uint32_t slot, int32_t d, float* out, sd_stream stream) {
  SD_CHECK_ARG(d >= 1 && out, "sd_philox_normals: need d >= 1 and out");
  SD_CHECK_ARG(tag < 256 && slot < (1u << 24), "sd_philox_normals: tag < 256 and slot < 2^24");
  SD_HIP(philox_normals_launch(seed, chain, round, tag, slot, d, out, (hipStream_t)stream));
  return SD_OK;
}

sd_status sd_mfma_loop(int32_t blocks, int32_t iters, float* out, sd_stream stream) {
  SD_CHECK_ARG(blocks >= 1 && iters >= 1, "sd_mfma_loop: need blocks >= 1 and iters >= 1");
  SD_CHECK_ARG(out, "sd_mfma_loop: NULL out");
  SD_HIP(mfma_loop_launch(blocks, iters, out, (hipStream_t)stream));
  return SD_OK;
}

}  // extern "C"
