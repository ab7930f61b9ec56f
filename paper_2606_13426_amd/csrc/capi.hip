// C ABI: argument validation (always before any HIP call), the Gaussian-mixture
// target object, the sampler's round loop (Alg. 8) and the event profiler.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

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
bool g_prof = false;
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

bool prof_on() { return g_prof; }

void prof_events(hipEvent_t* a, hipEvent_t* b) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (g_pending.size() > 4096) drain_locked();
  for (hipEvent_t* e : {a, b}) {
    if (!g_pool.empty()) {
      *e = g_pool.back();
      g_pool.pop_back();
    } else {
      (void)hipEventCreate(e);
    }
  }
}

void prof_push(const char* name, hipEvent_t a, hipEvent_t b) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_pending.push_back(PendingEv{name, a, b});
}

}  // namespace sd

using namespace sd;

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
sd_status sd_target_create(const sd_schedule* sched, int32_t d, int32_t n_comp, const float* mu,
                           const float* var, const float* log_w, sd_precision precision,
                           sd_target* out) {
  SD_CHECK_ARG(out, "sd_target_create: out is NULL");
  *out = nullptr;
  SD_CHECK_ARG(sched_ok(sched), "sd_target_create: invalid schedule (need N >= 1, 0 < beta_min <= beta_max, churn > 0)");
  SD_CHECK_ARG(d >= 1, "sd_target_create: d = %d < 1", d);
  SD_CHECK_ARG(n_comp >= 1 && n_comp <= 4096, "sd_target_create: n_comp = %d not in [1, 4096]", n_comp);
  SD_CHECK_ARG(mu && var && log_w, "sd_target_create: mu/var/log_w must be host arrays");
  SD_CHECK_ARG(precision == SD_FP32 || precision == SD_BF16, "sd_target_create: unknown precision");
  if (precision == SD_BF16) {
    set_error("sd_target_create: the bf16 GEMM path is not built in this version");
    return SD_EUNSUPPORTED;
  }
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
  Target* t = new Target();
  t->sc = to_sched(sched);
  t->d = d;
  t->M = n_comp;
  t->prec = precision;
  (void)hipGetDevice(&t->device);
  bool ok = hipMalloc(&t->mu, sizeof(float) * M * D) == hipSuccess &&
            hipMalloc(&t->muT, sizeof(float) * M * D) == hipSuccess &&
            hipMalloc(&t->var, sizeof(double) * M) == hipSuccess &&
            hipMalloc(&t->logw, sizeof(double) * M) == hipSuccess &&
            hipMalloc(&t->musq, sizeof(double) * M) == hipSuccess;
  if (!ok) {
    set_error("sd_target_create: device allocation failed");
    sd_target_destroy(reinterpret_cast<sd_target>(t));
    return SD_ENOMEM;
  }
  ok = hipMemcpy(t->mu, mu, sizeof(float) * M * D, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(t->muT, muT.data(), sizeof(float) * M * D, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(t->var, vv.data(), sizeof(double) * M, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(t->logw, lw.data(), sizeof(double) * M, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(t->musq, msq.data(), sizeof(double) * M, hipMemcpyHostToDevice) == hipSuccess;
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
  if (t->var) (void)hipFree(t->var);
  if (t->logw) (void)hipFree(t->logw);
  if (t->musq) (void)hipFree(t->musq);
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

// ----------------------------------------------------------------- draft --
sd_status sd_init_chains(int32_t B, int32_t d, uint64_t seed, float* y, sd_stream stream) {
  SD_CHECK_ARG(B >= 1 && d >= 1, "sd_init_chains: need B >= 1 and d >= 1");
  SD_CHECK_ARG(y, "sd_init_chains: y is NULL");
  SD_HIP(init_chains_launch(B, d, seed, y, (hipStream_t)stream));
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
sd_status sd_verify_block(int32_t B, int32_t K, int32_t d, sd_verify_mode mode,
                          const float* y_draft, sd_stride ys, const float* mp, sd_stride mps,
                          const float* mq, sd_stride mqs, const double* sigma, const int32_t* kb,
                          const uint32_t* round, uint64_t seed, sd_usample_mode usample_mode,
                          int32_t* tau, double* log_alpha_res, double* u_res, double* delta_norm,
                          double* log_ratio, uint64_t* coins, sd_stream stream) {
  SD_CHECK_ARG(B >= 1 && d >= 1, "sd_verify_block: need B >= 1 and d >= 1");
  SD_CHECK_ARG(K >= 1 && K <= SD_MAX_BLOCK, "sd_verify_block: K = %d not in [1, %d]", K, SD_MAX_BLOCK);
  SD_CHECK_ARG(mode == SD_BLOCK || mode == SD_TOKEN, "sd_verify_block: unknown mode");
  SD_CHECK_ARG(usample_mode == SD_USAMPLE_EXACT || usample_mode == SD_USAMPLE_PAPER, "sd_verify_block: unknown usample mode");
  SD_CHECK_ARG(y_draft && mp && mq && sigma && kb && round && tau && log_alpha_res && u_res &&
                   delta_norm && log_ratio,
               "sd_verify_block: NULL pointer argument");
  SD_CHECK_ARG(stride_ok(ys, d, K) && stride_ok(mps, d, K) && stride_ok(mqs, d, K),
               "sd_verify_block: stride too small for [B][K][d]");
  SD_HIP(verify_launch(B, K, d, (int)mode, y_draft, ys, mp, mps, mq, mqs, sigma, kb, round, seed,
                       (int)usample_mode, tau, log_alpha_res, u_res, delta_norm, log_ratio, coins,
                       nullptr, (hipStream_t)stream, nullptr));
  return SD_OK;
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
                         u_res, delta_norm, round, seed, y_out, (hipStream_t)stream, nullptr));
  return SD_OK;
}

}  // extern "C"

// --------------------------------------------------------------- sampler --
namespace {

struct SamplerLayout {
  size_t y, cache, x, mp, mq, score, sigma, lar, ures, dn, lr, k, step, kb, left, tau, rnd, cnt,
      hist, steps, nan, tws, total;
  size_t tws_bytes;
};

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
  L.y = take(4 * Bs * d);
  L.cache = take(4 * Bs * d);
  L.x = take(4 * Bs * K1 * d);
  L.mp = take(4 * Bs * K * d);
  L.mq = take(4 * Bs * K1 * d);
  L.score = take(4 * Bs * K1 * d);
  L.sigma = take(8 * Bs * K1);
  L.lar = take(8 * Bs);
  L.ures = take(8 * Bs);
  L.dn = take(8 * Bs * K);
  L.lr = take(8 * Bs * K);
  L.k = take(4 * Bs);
  L.step = take(4 * Bs * K1);
  L.kb = take(4 * Bs);
  L.left = take(4 * Bs);
  L.tau = take(4 * Bs);
  L.rnd = take(4 * Bs);
  L.cnt = take(4 * 2);
  L.hist = take(8 * (SD_MAX_BLOCK + 2));
  L.steps = take(8);
  L.nan = take(4);
  const size_t rows = Bs * K1;
  L.tws_bytes = target_ws_bytes(t, (int)rows);
  L.tws = take(L.tws_bytes);
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
  SD_CHECK_ARG(target, "sd_run_sampler: target is NULL");
  const Target& t = *reinterpret_cast<Target*>(target);
  SD_CHECK_ARG(B >= 1, "sd_run_sampler: B = %d < 1", B);
  SD_CHECK_ARG(K >= 1 && K <= SD_MAX_BLOCK, "sd_run_sampler: K = %d not in [1, %d]", K, SD_MAX_BLOCK);
  SD_CHECK_ARG(mode == SD_BLOCK || mode == SD_TOKEN, "sd_run_sampler: unknown mode");
  SD_CHECK_ARG(usample_mode == SD_USAMPLE_EXACT || usample_mode == SD_USAMPLE_PAPER, "sd_run_sampler: unknown usample mode");
  SD_CHECK_ARG(y_out && ws, "sd_run_sampler: y_out and ws must be non-NULL");
  SD_CHECK_ARG(!tau_trace || trace_rounds >= 0, "sd_run_sampler: trace_rounds < 0");
  SD_CHECK_ARG(((uintptr_t)ws & 255u) == 0, "sd_run_sampler: workspace must be 256-byte aligned");
  const SamplerLayout L = sampler_layout(t, B, K);
  SD_CHECK_ARG(ws_bytes >= L.total, "sd_run_sampler: workspace %zu < %zu bytes", ws_bytes, L.total);
  SD_CHECK_ARG((int64_t)B * (K + 1) <= INT32_MAX, "sd_run_sampler: B*(K+1) rows exceed int32");

  hipStream_t s = (hipStream_t)stream;
  char* base = static_cast<char*>(ws);
  auto F = [&](size_t o) { return reinterpret_cast<float*>(base + o); };
  auto D = [&](size_t o) { return reinterpret_cast<double*>(base + o); };
  auto I = [&](size_t o) { return reinterpret_cast<int32_t*>(base + o); };
  const int d = t.d, N = t.sc.N, K1 = K + 1;
  float *y = F(L.y), *cache = F(L.cache), *x = F(L.x), *mp = F(L.mp), *mq = F(L.mq),
        *score = F(L.score);
  double *sigma = D(L.sigma), *lar = D(L.lar), *ures = D(L.ures), *dn = D(L.dn), *lr = D(L.lr);
  int32_t *kk = I(L.k), *step = I(L.step), *kb = I(L.kb), *left = I(L.left), *tau = I(L.tau);
  uint32_t* rnd = reinterpret_cast<uint32_t*>(base + L.rnd);
  int* cnt = I(L.cnt);
  int64_t* hist = reinterpret_cast<int64_t*>(base + L.hist);
  int64_t* steps = reinterpret_cast<int64_t*>(base + L.steps);
  int* nanflag = I(L.nan);
  void* tws = base + L.tws;

  const sd_stride xs{(int64_t)K1 * d, d}, mps{(int64_t)K * d, d}, mqs{(int64_t)K1 * d, d};
  const sd_stride ys{(int64_t)K1 * d, d};  // drafts are rows 1..K of x
  const float* ydraft = x + d;

  // Y_0 and the one explicit target call that seeds the Free-Drafter cache
  SD_HIP(init_chains_launch(B, d, seed, y, s));
  SD_HIP(fill_i32_launch(kk, B, 0, s));
  SD_HIP(fill_i32_launch(reinterpret_cast<int32_t*>(rnd), B, 0, s));
  SD_HIP(fill_i32_launch(step, B, 0, s));
  SD_HIP(fill_i32_launch(cnt, 2, B, s));
  SD_HIP(fill_i32_launch(nanflag, 1, 0, s));
  SD_HIP(fill_i64_launch(hist, SD_MAX_BLOCK + 2, 0, s));
  SD_HIP(fill_i64_launch(steps, 1, 0, s));
  SD_HIP(target_mean_launch(t, B, y, d, step, mq, d, cache, d, tws, s, nullptr));

  int32_t* host_cnt = nullptr;
  constexpr int kLag = 3;
  hipEvent_t ev[kLag + 1];
  SD_HIP(hipHostMalloc(reinterpret_cast<void**>(&host_cnt), sizeof(int32_t) * (kLag + 1), hipHostMallocDefault));
  for (int i = 0; i <= kLag; ++i) {
    host_cnt[i] = -1;
    (void)hipEventCreateWithFlags(&ev[i], hipEventDisableTiming);
  }
  sd_status st = SD_OK;
  int64_t rounds = 0;
  const int max_rounds = N + kLag + 2;
  int r = 0;
  bool done = false;
  for (; r < max_rounds && !done; ++r) {
    int* cur = cnt + (r & 1);
    const int* gate = cnt + ((r + 1) & 1);
    hipError_t e = prepare_launch(t.sc, B, K, kk, kb, left, step, sigma, cur, s, gate);
    if (e == hipSuccess) e = draft_launch(t.sc, B, K, d, y, cache, kk, rnd, seed, x, xs, mp, mps, s, gate);
    if (e == hipSuccess) e = target_mean_launch(t, B * K1, x, d, step, mq, d, score, d, tws, s, gate);
    if (e == hipSuccess)
      e = verify_launch(B, K, d, (int)mode, ydraft, ys, mp, mps, mq, mqs, sigma, kb, rnd, seed,
                        (int)usample_mode, tau, lar, ures, dn, lr, nullptr, nanflag, s, gate);
    if (e == hipSuccess)
      e = residual_launch(B, K, d, ydraft, ys, mp, mps, mq, mqs, sigma, kb, left, tau, ures, dn,
                          rnd, seed, y, s, gate);
    if (e == hipSuccess)
      e = commit_launch(B, K, d, N, tau, kb, kk, rnd, score, mqs, cache, cur, hist, steps,
                        tau_trace, r, tau_trace ? trace_rounds : 0, s, gate);
    const int slot = r % (kLag + 1);
    if (e == hipSuccess) e = hipMemcpyAsync(&host_cnt[slot], cur, sizeof(int32_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipEventRecord(ev[slot], s);
    if (e != hipSuccess) {
      set_error("sd_run_sampler: launch failed in round %d: %s", r, hipGetErrorString(e));
      st = SD_EHIP;
      break;
    }
    // look at the counter of round r - kLag (the queue keeps kLag rounds ahead)
    const int back = r - kLag;
    if (back >= 0) {
      const int bs = back % (kLag + 1);
      if (hipEventSynchronize(ev[bs]) != hipSuccess) {
        set_error("sd_run_sampler: event wait failed");
        st = SD_EHIP;
        break;
      }
      if (host_cnt[bs] == 0) {
        done = true;
        rounds = back + 1;
      }
    }
  }
  if (st == SD_OK && !done) {
    // drain: find the first round whose counter read zero
    for (int back = r - kLag < 0 ? 0 : r - kLag; back < r; ++back) {
      const int bs = back % (kLag + 1);
      (void)hipEventSynchronize(ev[bs]);
      if (host_cnt[bs] == 0) {
        done = true;
        rounds = back + 1;
        break;
      }
    }
    if (!done) {
      set_error("sd_run_sampler: chains still active after %d rounds", r);
      st = SD_EHIP;
    }
  }
  if (st == SD_OK) {
    hipError_t e = hipMemcpyAsync(y_out, y, sizeof(float) * (size_t)B * d, hipMemcpyDeviceToDevice, s);
    int64_t h_hist[SD_MAX_BLOCK + 2];
    int64_t h_steps = 0;
    int32_t h_nan = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(h_hist, hist, sizeof(h_hist), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&h_steps, steps, sizeof(int64_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&h_nan, nanflag, sizeof(int32_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      set_error("sd_run_sampler: final copy failed: %s", hipGetErrorString(e));
      st = SD_EHIP;
    } else {
      if (stats) {
        memset(stats, 0, sizeof(*stats));
        stats->rounds = rounds;
        stats->steps = h_steps;
        for (int i = 0; i < SD_MAX_BLOCK + 2; ++i) {
          stats->tau_hist[i] = h_hist[i];
          stats->chain_rounds += h_hist[i];
        }
      }
      if (h_nan) {
        set_error("sd_run_sampler: non-finite log-ratio met");
        st = SD_ENUMERIC;
      }
    }
  }
  (void)hipStreamSynchronize(s);
  for (int i = 0; i <= kLag; ++i) (void)hipEventDestroy(ev[i]);
  (void)hipHostFree(host_cnt);
  return st;
}

// ------------------------------------------------------------- profiling --
sd_status sd_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (on) {
    drain_locked();
    g_stats.clear();
  }
  g_prof = on != 0;
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

}  // extern "C"
