"""Shared helpers of the GPU parity tests (comparison rules, oracle glue)."""
import numpy as np

from oracle import sampler as osamp
from oracle.schedule import Schedule

FP32_RTOL = 1e-4   # float32 path: states, means and scores


def row_scale(ref):
    ref = np.asarray(ref, dtype=np.float64)
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    return np.maximum(np.abs(ref), rms)


def assert_rows_close(got, ref, rtol=FP32_RTOL, what=""):
    """|got - ref| <= rtol * max(|ref|, rms(row of ref)) elementwise."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    err = np.abs(got - ref) / np.maximum(row_scale(ref), 1e-30)
    worst = float(err.max()) if err.size else 0.0
    assert worst <= rtol, f"{what}: max scaled error {worst:.3e} > {rtol:.1e} at {np.unravel_index(err.argmax(), err.shape)}"
    return worst


def sigma_table(N, churn=1.0):
    return Schedule(N, churn=churn).sigma(np.arange(N + 1))


def oracle_verify_chains(inp, chains, seed, mode, umode, omega=1.0):
    """Oracle verification of the given chains of an input dict of numpy arrays."""
    out = {}
    for b in chains:
        kb = int(inp["kb"][b])
        if kb == 0:
            out[b] = None
            continue
        out[b] = osamp.verify_chain(inp["y_draft"][b], inp["mp"][b], inp["mq"][b], inp["sigma"][b], kb,
                                    seed, b, int(inp["round"][b]), mode, umode, omega)
    return out


def to_numpy(d):
    return {k: v.detach().cpu().numpy() for k, v in d.items()}


# ------------------------------------------------ bf16 operand precision model --
def bf16_round(a):
    """float32 values rounded to bf16 (round to nearest, ties to even), as float64."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def target_mean_bf16_operands(gmm, sched, x, n, rnd=bf16_round):
    """m^q and score with the bf16 path's operand rounding and float64 elsewhere.

    The two products see bf16 operands: x . mu_m with x and mu rounded, and
    P mu with P_m = r_m a / s2_m rounded to float32 and then to bf16 (the
    softmax stores float32 before the conversion).  ||x||^2, ||mu_m||^2, the
    softmax and the epilogue use the unrounded values.  With rnd = identity
    this is the plain definition of the Gaussian-mixture score.
    """
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    n = np.broadcast_to(np.asarray(n), (x.shape[0],))
    a = sched.signal(n)
    mu = gmm.mu
    s2 = a[:, None] ** 2 * gmm.var[None, :] + 1.0 - a[:, None] ** 2
    dot = rnd(x.astype(np.float32)) @ rnd(mu.astype(np.float32)).T
    logit = (gmm.log_w[None, :] - 0.5 * gmm.d * np.log(s2)
             - 0.5 * ((x * x).sum(1)[:, None] - 2.0 * a[:, None] * dot
                      + a[:, None] ** 2 * (mu * mu).sum(1)[None, :]) / s2)
    logit -= logit.max(axis=1, keepdims=True)
    r = np.exp(logit)
    r /= r.sum(axis=1, keepdims=True)
    P = rnd((r * a[:, None] / s2).astype(np.float32))
    score = P @ rnd(mu.astype(np.float32)) - (r / s2).sum(1)[:, None] * x
    mq = sched.c1(n)[:, None] * x + sched.c2(n)[:, None] * score
    return mq, score


def rel_l2_rows(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.linalg.norm(got - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-300)
