"""ctypes binding of libspecdiff.so (include/specdiff.h), same names as the C ABI.

Argument marshalling only: torch tensors are passed as device pointers with
their element strides, the stream is torch's current stream, and every status
other than SD_OK raises SpecDiffError with sd_last_error().  There is no
fallback: if the library has not been built, loading raises.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspecdiff.so")

SD_OK, SD_EINVAL, SD_EHIP, SD_EUNSUPPORTED, SD_ENOMEM, SD_ENUMERIC = 0, -1, -2, -3, -4, -5
SD_BLOCK, SD_TOKEN = 0, 1
SD_FP32, SD_BF16 = 0, 1
SD_USAMPLE_EXACT, SD_USAMPLE_PAPER = 0, 1
SD_RESIDUAL_DECOMPOSITION, SD_RESIDUAL_REFLECTION = 0, 1
SD_DRAFTER_FREE, SD_DRAFTER_FROZEN = 0, 1
SD_MAX_BLOCK = 64
TAG_INIT, TAG_DRAFT, TAG_COIN, TAG_USAMPLE, TAG_RESID, TAG_TARGET = 1, 2, 3, 4, 5, 6

c_int32, c_int64, c_uint32, c_uint64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64
c_double, c_size_t, c_void_p, c_char_p = ctypes.c_double, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_char_p


class sd_schedule(ctypes.Structure):
    _fields_ = [("n_steps", c_int32), ("beta_min", c_double), ("beta_max", c_double),
                ("churn", c_double)]


class sd_stride(ctypes.Structure):
    _fields_ = [("chain", c_int64), ("row", c_int64)]


class sd_stats(ctypes.Structure):
    _fields_ = [("rounds", c_int64), ("chain_rounds", c_int64), ("steps", c_int64),
                ("ties", c_int64), ("mean_tau", c_double), ("finished", c_int32),
                ("groups", c_int32), ("tau_hist", c_int64 * (SD_MAX_BLOCK + 2))]


class sd_sampler_options(ctypes.Structure):
    _fields_ = [("mode", c_int32), ("usample_mode", c_int32), ("residual", c_int32),
                ("drafter", c_int32), ("omega", c_double), ("start_round", c_int32),
                ("max_rounds", c_int32), ("groups", c_int32)]


class sd_sampler_view(ctypes.Structure):
    _fields_ = [("x", c_void_p), ("y", c_void_p), ("cache", c_void_p), ("cache_step", c_void_p),
                ("k", c_void_p), ("round", c_void_p), ("mq", c_void_p), ("lrp", c_void_p),
                ("n_tiles", c_int32), ("tau", c_void_p), ("coins", c_void_p),
                ("log_alpha_res", c_void_p), ("u", c_void_p), ("ties", c_void_p)]


class sd_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", c_int64), ("total_ms", c_double)]


class SpecDiffError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"status {status}: {msg}")
        self.status = status


P = c_void_p
S = sd_stride
# (name, restype, argtypes) of every exported function, in header order
SIGNATURES = [
    ("sd_abi_version", c_int32, []),
    ("sd_last_error", c_char_p, []),
    ("sd_schedule_table", c_int32, [ctypes.POINTER(sd_schedule), P]),
    ("sd_target_create", c_int32, [ctypes.POINTER(sd_schedule), c_int32, c_int32, P, P, P, c_int32,
                                   ctypes.POINTER(c_void_p)]),
    ("sd_target_destroy", c_int32, [P]),
    ("sd_target_mean_workspace", c_size_t, [P, c_int32]),
    ("sd_target_mean", c_int32, [P, c_int32, P, c_int64, P, P, c_int64, P, c_int64, P, c_size_t, P]),
    ("sd_target_mean_noalloc", c_int32, [P, c_int32, P, c_int64, P, P, c_int64, P, c_int64, P]),
    ("sd_target_mean_noalloc_max_bytes", c_size_t, []),
    ("sd_init_chains", c_int32, [c_int32, c_int32, c_uint64, P, P]),
    ("sd_draft_block", c_int32, [ctypes.POINTER(sd_schedule), c_int32, c_int32, c_int32, P, P, P, P,
                                 c_uint64, P, S, P, S, P]),
    ("sd_verify_block", c_int32, [c_int32, c_int32, c_int32, c_int32, P, S, P, S, P, S, P, P, P,
                                  c_uint64, c_int32, P, P, P, P, P, P, P]),
    ("sd_verify_block_tempered", c_int32, [c_int32, c_int32, c_int32, c_int32, c_double, P, S, P, S, P,
                                           S, P, P, P, c_uint64, c_int32, P, P, P, P, P, P, P]),
    ("sd_sample_residual", c_int32, [c_int32, c_int32, c_int32, P, S, P, S, P, S, P, P, P, P, P, P, P,
                                     c_uint64, P, P]),
    ("sd_sample_residual_reflection", c_int32, [c_int32, c_int32, c_int32, P, S, P, S, P, S, P, P, P, P,
                                                P, c_uint64, P, P]),
    ("sd_sampler_workspace", c_size_t, [P, c_int32, c_int32]),
    ("sd_run_sampler", c_int32, [P, c_int32, c_int32, c_int32, c_int32, c_uint64, P, P, c_int32,
                                 ctypes.POINTER(sd_stats), P, c_size_t, P]),
    ("sd_run_sampler_ex", c_int32, [P, c_int32, c_int32, ctypes.POINTER(sd_sampler_options), c_uint64, P,
                                    P, c_int32, ctypes.POINTER(sd_stats), P, c_size_t, P]),
    ("sd_sampler_state", c_int32, [P, c_int32, c_int32, P, c_size_t, c_int64,
                                   ctypes.POINTER(sd_sampler_view)]),
    ("sd_plain_em_workspace", c_size_t, [P, c_int32]),
    ("sd_run_plain_em", c_int32, [P, c_int32, c_uint64, P, P, c_size_t, P]),
    ("sd_profile_enable", c_int32, [c_int32]),
    ("sd_profile_only", c_int32, [c_char_p]),
    ("sd_profile_every", c_int32, [c_int32]),
    ("sd_profile_seen", c_int32, [c_char_p, ctypes.POINTER(c_int64)]),
    ("sd_profile_read", c_int32, [ctypes.POINTER(sd_kernel_stat), c_int32, ctypes.POINTER(c_int32)]),
    ("sd_philox_words", c_int32, [c_uint64, c_int32, P, P, P]),
    ("sd_philox_normals", c_int32, [c_uint64, c_uint32, c_uint32, c_uint32, c_uint32, c_int32, P, P]),
    ("sd_mfma_loop", c_int32, [c_int32, c_int32, P, P]),
]

_lib = None


def load():
    """Load the library (once).  Raises if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        for name, res, args in SIGNATURES:
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def last_error():
    return load().sd_last_error().decode(errors="replace")


def _check(status, name):
    if status != SD_OK:
        raise SpecDiffError(status, f"{name}: {last_error()}")


def _p(t):
    return None if t is None else c_void_p(t.data_ptr())


def _stream():
    import torch
    return c_void_p(torch.cuda.current_stream().cuda_stream)


def stride3(t):
    """sd_stride of a [B][rows][d] view whose last dimension is contiguous."""
    assert t.dim() == 3 and t.stride(2) == 1, "need a [B][rows][d] view with contiguous rows"
    return sd_stride(t.stride(0), t.stride(1))


def schedule(n_steps, beta_min=0.1, beta_max=20.0, churn=1.0):
    return sd_schedule(int(n_steps), float(beta_min), float(beta_max), float(churn))


def sd_abi_version():
    return load().sd_abi_version()


def sd_schedule_table(sched):
    import numpy as np
    out = np.empty((4, sched.n_steps + 1), dtype=np.float64)
    _check(load().sd_schedule_table(ctypes.byref(sched), out.ctypes.data_as(c_void_p)), "sd_schedule_table")
    return out


class Target:
    """Owner of an sd_target handle (Gaussian-mixture target on the current device)."""

    def __init__(self, sched, mu, var, log_w, precision=SD_FP32):
        import numpy as np
        mu = np.ascontiguousarray(mu, dtype=np.float32)
        var = np.ascontiguousarray(var, dtype=np.float32)
        log_w = np.ascontiguousarray(log_w, dtype=np.float32)
        self.sched = sched
        self.M, self.d = mu.shape
        h = c_void_p()
        _check(load().sd_target_create(ctypes.byref(sched), self.d, self.M,
                                       mu.ctypes.data_as(c_void_p), var.ctypes.data_as(c_void_p),
                                       log_w.ctypes.data_as(c_void_p), precision, ctypes.byref(h)),
               "sd_target_create")
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            load().sd_target_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def sd_target_mean_workspace(target, rows):
    return load().sd_target_mean_workspace(target.handle, rows)


def sd_target_mean(target, x, step, mq, score=None, ws=None):
    """x, mq, score: [rows][d] float32 (row stride >= d); step: [rows] int32."""
    import torch
    rows = x.shape[0]
    if ws is None:
        ws = torch.empty(sd_target_mean_workspace(target, rows), dtype=torch.uint8, device=x.device)
    _check(load().sd_target_mean(target.handle, rows, _p(x), x.stride(0), _p(step), _p(mq), mq.stride(0),
                                 _p(score), score.stride(0) if score is not None else 0, _p(ws),
                                 ws.numel(), _stream()), "sd_target_mean")


def sd_target_mean_noalloc(target, x, step, mq, score=None):
    """sd_target_mean with the library's own scratch memory (no workspace)."""
    rows = x.shape[0]
    _check(load().sd_target_mean_noalloc(target.handle, rows, _p(x), x.stride(0), _p(step), _p(mq),
                                         mq.stride(0), _p(score),
                                         score.stride(0) if score is not None else 0, _stream()),
           "sd_target_mean_noalloc")


def sd_target_mean_noalloc_max_bytes():
    return load().sd_target_mean_noalloc_max_bytes()


def sd_init_chains(y, seed):
    B, d = y.shape
    _check(load().sd_init_chains(B, d, seed, _p(y), _stream()), "sd_init_chains")


def sd_draft_block(sched, y, cache_score, k, rnd, seed, x, mp):
    """y, cache_score [B][d]; k int32 [B]; rnd int32/uint32 [B]; x [B][K+1][d]; mp [B][K][d] views."""
    B, d = y.shape
    K = mp.shape[1]
    _check(load().sd_draft_block(ctypes.byref(sched), B, K, d, _p(y), _p(cache_score), _p(k), _p(rnd),
                                 seed, _p(x), stride3(x), _p(mp), stride3(mp), _stream()),
           "sd_draft_block")


def _verify_out(B, K, dev):
    import torch
    return dict(tau=torch.empty(B, dtype=torch.int32, device=dev),
                log_alpha_res=torch.empty(B, dtype=torch.float64, device=dev),
                u_res=torch.empty(B, dtype=torch.float64, device=dev),
                delta_norm=torch.empty(B, K, dtype=torch.float64, device=dev),
                log_ratio=torch.empty(B, K, dtype=torch.float64, device=dev),
                coins=torch.empty(B, dtype=torch.int64, device=dev))


def sd_verify_block(y_draft, mp, mq, sigma, kb, rnd, seed, mode=SD_BLOCK, usample_mode=SD_USAMPLE_EXACT,
                    out=None):
    """Views [B][K][d] (mq: [B][>=K][d]); sigma [B][K+1] float64; kb, rnd [B] int32.

    Returns dict of device tensors tau, log_alpha_res, u_res, delta_norm, log_ratio, coins.
    """
    B, K, d = y_draft.shape
    if out is None:
        out = _verify_out(B, K, y_draft.device)
    _check(load().sd_verify_block(B, K, d, mode, _p(y_draft), stride3(y_draft), _p(mp), stride3(mp),
                                  _p(mq), stride3(mq), _p(sigma), _p(kb), _p(rnd), seed, usample_mode,
                                  _p(out["tau"]), _p(out["log_alpha_res"]), _p(out["u_res"]),
                                  _p(out["delta_norm"]), _p(out["log_ratio"]), _p(out.get("coins")),
                                  _stream()), "sd_verify_block")
    return out


def sd_verify_block_tempered(y_draft, mp, mq, sigma, kb, rnd, seed, omega, mode=SD_BLOCK,
                             usample_mode=SD_USAMPLE_EXACT, out=None):
    """sd_verify_block with temperature omega (same arguments and outputs)."""
    B, K, d = y_draft.shape
    if out is None:
        out = _verify_out(B, K, y_draft.device)
    _check(load().sd_verify_block_tempered(B, K, d, mode, float(omega), _p(y_draft), stride3(y_draft),
                                           _p(mp), stride3(mp), _p(mq), stride3(mq), _p(sigma), _p(kb),
                                           _p(rnd), seed, usample_mode, _p(out["tau"]),
                                           _p(out["log_alpha_res"]), _p(out["u_res"]),
                                           _p(out["delta_norm"]), _p(out["log_ratio"]),
                                           _p(out.get("coins")), _stream()), "sd_verify_block_tempered")
    return out


def sd_sample_residual(y_draft, mp, mq, sigma, kb, steps_left, tau, u_res, delta_norm, rnd, seed, y_out):
    B, K, d = y_draft.shape
    _check(load().sd_sample_residual(B, K, d, _p(y_draft), stride3(y_draft), _p(mp), stride3(mp), _p(mq),
                                     stride3(mq), _p(sigma), _p(kb), _p(steps_left), _p(tau), _p(u_res),
                                     _p(delta_norm), _p(rnd), seed, _p(y_out), _stream()),
           "sd_sample_residual")


def sd_sample_residual_reflection(y_draft, mp, mq, sigma, kb, steps_left, tau, rnd, seed, y_out):
    B, K, d = y_draft.shape
    _check(load().sd_sample_residual_reflection(B, K, d, _p(y_draft), stride3(y_draft), _p(mp),
                                                stride3(mp), _p(mq), stride3(mq), _p(sigma), _p(kb),
                                                _p(steps_left), _p(tau), _p(rnd), seed, _p(y_out),
                                                _stream()), "sd_sample_residual_reflection")


def sd_sampler_workspace(target, B, K):
    return load().sd_sampler_workspace(target.handle, B, K)


def _stats_dict(st):
    return dict(rounds=st.rounds, chain_rounds=st.chain_rounds, steps=st.steps, ties=st.ties,
                mean_tau=st.mean_tau, finished=bool(st.finished), groups=st.groups,
                tau_hist=[st.tau_hist[i] for i in range(SD_MAX_BLOCK + 2)])


def sd_run_sampler(target, B, K, seed, mode=SD_BLOCK, usample_mode=SD_USAMPLE_EXACT, y_out=None,
                   trace_rounds=0, ws=None, device="cuda"):
    """Runs Alg. 8 for B chains; returns (y_out [B][d], stats dict, tau_trace or None)."""
    import torch
    if y_out is None:
        y_out = torch.empty(B, target.d, dtype=torch.float32, device=device)
    if ws is None:
        ws = torch.empty(sd_sampler_workspace(target, B, K), dtype=torch.uint8, device=device)
    trace = torch.zeros(trace_rounds, B, dtype=torch.int32, device=device) if trace_rounds > 0 else None
    st = sd_stats()
    _check(load().sd_run_sampler(target.handle, B, K, mode, usample_mode, seed, _p(y_out), _p(trace),
                                 trace_rounds, ctypes.byref(st), _p(ws), ws.numel(), _stream()),
           "sd_run_sampler")
    return y_out, _stats_dict(st), trace


def sd_run_sampler_ex(target, B, K, seed, mode=SD_BLOCK, usample_mode=SD_USAMPLE_EXACT,
                      residual=SD_RESIDUAL_DECOMPOSITION, drafter=SD_DRAFTER_FREE, omega=1.0,
                      y_out=None, trace_rounds=0, ws=None, device="cuda", start_round=0,
                      max_rounds=-1, trace=None, groups=0):
    """Alg. 8 with the sampler options (residual, drafter, temperature, the
    rounds of a run this call does: max_rounds < 0 until done, 0 initialise
    only, and the chain groups run concurrently: 0 the library's choice, 1, 2);
    returns as sd_run_sampler.  A partial run continues with the same ws (and
    trace) and start_round = stats["rounds"]."""
    import torch
    if y_out is None:
        y_out = torch.empty(B, target.d, dtype=torch.float32, device=device)
    if ws is None:
        ws = torch.empty(sd_sampler_workspace(target, B, K), dtype=torch.uint8, device=device)
    if trace is None and trace_rounds > 0:
        trace = torch.zeros(trace_rounds, B, dtype=torch.int32, device=device)
    if trace is not None:
        trace_rounds = trace.shape[0]
    st = sd_stats()
    opts = sd_sampler_options(mode, usample_mode, residual, drafter, float(omega), int(start_round),
                              int(max_rounds), int(groups))
    _check(load().sd_run_sampler_ex(target.handle, B, K, ctypes.byref(opts), seed, _p(y_out), _p(trace),
                                    trace_rounds, ctypes.byref(st), _p(ws), ws.numel(), _stream()),
           "sd_run_sampler_ex")
    return y_out, _stats_dict(st), trace


def sd_sampler_state(target, B, K, ws, rounds):
    """Views (torch tensors aliasing ws) of the sampler state after `rounds` rounds:
    x [B][K+1][d], y [B][d], cache [B][d], cache_step, k, round [B] int32,
    mq [B][K+1][d], lrp [B(K+1)][n_tiles][3] float64, tau [B], coins [B] int64,
    log_alpha_res, u [B] float64, ties [B] int32."""
    import torch
    v = sd_sampler_view()
    _check(load().sd_sampler_state(target.handle, B, K, _p(ws), ws.numel(), int(rounds), ctypes.byref(v)),
           "sd_sampler_state")
    base = ws.data_ptr()
    d, K1 = target.d, K + 1

    def view(ptr, shape, dtype):
        esz = torch.empty((), dtype=dtype).element_size()
        off = ptr - base
        assert off % esz == 0
        n = 1
        for e in shape:
            n *= e
        return ws[off: off + n * esz].view(dtype).view(*shape)

    f32, i32, f64, i64 = torch.float32, torch.int32, torch.float64, torch.int64
    return dict(x=view(v.x, (B, K1, d), f32), y=view(v.y, (B, d), f32), cache=view(v.cache, (B, d), f32),
                cache_step=view(v.cache_step, (B,), i32), k=view(v.k, (B,), i32),
                round=view(v.round, (B,), i32), mq=view(v.mq, (B, K1, d), f32),
                lrp=view(v.lrp, (B * K1, v.n_tiles, 3), f64), tau=view(v.tau, (B,), i32),
                coins=view(v.coins, (B,), i64), log_alpha_res=view(v.log_alpha_res, (B,), f64),
                u=view(v.u, (B,), f64), ties=view(v.ties, (B,), i32))


def sd_plain_em_workspace(target, B):
    return load().sd_plain_em_workspace(target.handle, B)


def sd_run_plain_em(target, B, seed, y_out=None, ws=None, device="cuda"):
    """The plain EM chain for B chains (N target calls); returns Y_N [B][d]."""
    import torch
    if y_out is None:
        y_out = torch.empty(B, target.d, dtype=torch.float32, device=device)
    if ws is None:
        ws = torch.empty(sd_plain_em_workspace(target, B), dtype=torch.uint8, device=device)
    _check(load().sd_run_plain_em(target.handle, B, seed, _p(y_out), _p(ws), ws.numel(), _stream()),
           "sd_run_plain_em")
    return y_out


def sd_profile_enable(on=True):
    _check(load().sd_profile_enable(1 if on else 0), "sd_profile_enable")


def sd_profile_only(name=None):
    _check(load().sd_profile_only(None if name is None else name.encode()), "sd_profile_only")


def sd_profile_every(n):
    _check(load().sd_profile_every(int(n)), "sd_profile_every")


def sd_profile_seen(name):
    n = c_int64()
    _check(load().sd_profile_seen(name.encode(), ctypes.byref(n)), "sd_profile_seen")
    return n.value


def sd_profile_read():
    cap = 64
    arr = (sd_kernel_stat * cap)()
    n = c_int32()
    _check(load().sd_profile_read(arr, cap, ctypes.byref(n)), "sd_profile_read")
    return {arr[i].name.decode(): (arr[i].launches, arr[i].total_ms) for i in range(min(n.value, cap))}


def sd_philox_words(seed, counters, out):
    _check(load().sd_philox_words(seed, counters.shape[0], _p(counters), _p(out), _stream()),
           "sd_philox_words")


def sd_philox_normals(seed, chain, rnd, tag, slot, out):
    _check(load().sd_philox_normals(seed, chain, rnd, tag, slot, out.numel(), _p(out), _stream()),
           "sd_philox_normals")


def sd_mfma_loop(blocks, iters, out):
    """Matrix-core calibration loop: blocks x 16 x iters x 32768 bf16 flops; out [blocks][4] float32."""
    _check(load().sd_mfma_loop(blocks, iters, _p(out), _stream()), "sd_mfma_loop")
