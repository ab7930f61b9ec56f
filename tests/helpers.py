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


def oracle_verify_chains(inp, chains, seed, mode, umode):
    """Oracle verification of the given chains of an input dict of numpy arrays."""
    out = {}
    for b in chains:
        kb = int(inp["kb"][b])
        if kb == 0:
            out[b] = None
            continue
        out[b] = osamp.verify_chain(inp["y_draft"][b], inp["mp"][b], inp["mq"][b], inp["sigma"][b], kb,
                                    seed, b, int(inp["round"][b]), mode, umode)
    return out


def to_numpy(d):
    return {k: v.detach().cpu().numpy() for k, v in d.items()}
