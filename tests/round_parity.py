"""One sampler round of the GPU checked against the oracle (Alg. 8).

The GPU runs a round at a time (sd_run_sampler_ex with start_round /
max_rounds); before and after each round the state of some chains is read
through sd_sampler_state.  Two checks per chain and round:

stage-wise  the oracle's verification (Alg. 6 / Alg. 2, U draw of Alg. 7) and
            residual (Alg. 5 / Alg. 4) fed the round's GPU drafts, the GPU's
            m^q and the draft means m^p the GPU forms (reproduced bit for bit
            in float32 below).  Both sides then hold the same float32 inputs,
            so tau and the coins must match exactly except where the oracle
            records a coin within 1e-6 of its threshold; ||Delta||, ell and
            log alpha_res to 1e-10, U to 1e-7, the new state to 1e-4.
independent the oracle's own round (its drafts, its float64 target, its
            verification and residual) from the GPU's state Y_k, k, round and
            cached score: drafts, m^q, the new state and the next cached score
            to 1e-4.  tau may differ only where the float32 rounding of the
            GPU's inputs moves a threshold across its coin: the coin then lies
            between the oracle's threshold and the stage-wise one, and the
            log-ratios of the two differ by no more than the float32
            tolerance 1e-4 (||Z|| ||Delta|| + ||Delta||^2/2).
"""
import numpy as np

from helpers import assert_rows_close
from oracle import sampler as osamp
from oracle.residual import USAMPLE_EXACT
from oracle.verify import log_ratio_terms

F32 = np.float32
F64 = np.float64


def fma_f32(a, b, c):
    """Correctly rounded float32 fused multiply-add of float32 arrays.

    a*b is exact in float64 (48 significant bits); the float64 sum s = a*b + c
    and its rounding error e (TwoSum) give the exact result s + e.  Rounding s
    to float32 is then correct unless s lies exactly half-way between two
    float32 numbers, where the sign of e decides."""
    a = np.asarray(a, F32).astype(F64)
    b = np.asarray(b, F32).astype(F64)
    c = np.asarray(c, F32).astype(F64)
    p = a * b
    s = p + c
    bb = s - p
    e = (p - (s - bb)) + (c - bb)
    r = s.astype(F32)
    r64 = r.astype(F64)
    up = np.nextafter(r, F32(np.inf))
    dn = np.nextafter(r, F32(-np.inf))
    half_up = (s - r64) == (up.astype(F64) - r64) / 2
    half_dn = (r64 - s) == (r64 - dn.astype(F64)) / 2
    r = np.where(half_up & (e > 0), up, r)
    r = np.where(half_dn & (e < 0), dn, r)
    return r


def coef_f32(sched, n):
    """The per-step float32 coefficients (c1_n, c2_n, sigma_n, 1/c2_n)."""
    n = np.asarray(n)
    c2 = sched.c2(n)
    return (sched.c1(n).astype(F32), c2.astype(F32), sched.sigma(n).astype(F32),
            (1.0 / c2).astype(F32))


def draft_means_f32(sched, drafts_in, sv, k, cstep, kb):
    """m^p_{j} = c1_{k+j} yhat_j + (c2_{k+j} / c2_c) sv for j < kb, as the GPU
    forms it: c2s = c2_n * (1/c2_c) and c2s * sv rounded to float32, then one
    fused multiply-add.  drafts_in: [kb, d] rows yhat_0 .. yhat_{kb-1}."""
    c1, c2, _, _ = coef_f32(sched, k + np.arange(kb))
    inv_c = coef_f32(sched, cstep)[3]
    c2s = (c2.astype(F64) * F64(inv_c)).astype(F32)
    prod = (c2s[:, None].astype(F64) * np.asarray(sv, F32)[None, :].astype(F64)).astype(F32)
    return fma_f32(np.broadcast_to(c1[:, None], prod.shape), drafts_in, prod)


def snapshot(view, chains):
    """numpy copies of the sampler state of the given chains (see sd_sampler_state)."""
    import torch
    idx = torch.as_tensor(np.asarray(chains), device=view["x"].device, dtype=torch.long)
    K1 = view["x"].shape[1]
    rows = (idx[:, None] * K1 + torch.arange(K1, device=idx.device)[None, :]).reshape(-1)
    out = {}
    for key in ("x", "y", "cache", "cache_step", "k", "round", "mq", "tau", "coins",
                "log_alpha_res", "u", "ties"):
        out[key] = view[key].index_select(0, idx).cpu().numpy()
    out["lrp"] = view["lrp"].index_select(0, rows).reshape(len(chains), K1, -1, 3).cpu().numpy()
    return out


class RoundStats:
    def __init__(self):
        self.compared = self.independent = self.ties = self.f32_flips = 0
        self.worst = {}

    def note(self, what, err):
        self.worst[what] = max(self.worst.get(what, 0.0), float(err))


def _close_scalar(got, want, rtol, what):
    assert abs(got - want) <= rtol * max(1.0, abs(want)), f"{what}: {got!r} vs {want!r}"


def check_round(gmm, sched, K, seed, i, b, before, after, stats, mode=osamp.BLOCK,
                residual=osamp.DECOMPOSITION, drafter=osamp.FREE, independent=False, omega=1.0,
                usample=USAMPLE_EXACT):
    """Compare chain b (index i of the snapshots) over the round between `before`
    and `after` (see the module docstring).  Returns False for an inactive chain."""
    N = sched.n_steps
    k = int(before["k"][i])
    if k >= N:
        assert int(after["tau"][i]) == 0
        return False
    rnd = int(before["round"][i])
    kb = min(K, N - k)
    frozen = drafter == osamp.FROZEN
    # the round's drafts, cache row and its step: the Frozen Drafter drafts at
    # the start of the round (they are in the state after it)
    src = after if frozen else before
    xin = src["x"][i]
    sv = src["cache"][i]
    cstep = k if frozen else int(before["cache_step"][i])
    drafts = np.array(xin[: kb + 1], dtype=F32)  # a copy: row 0 is replaced below
    drafts[0] = before["x"][i][0]
    mp = draft_means_f32(sched, drafts[:kb], sv, k, cstep, kb)
    mq = after["mq"][i]
    sig = sched.sigma(k + np.arange(kb + 1))
    # ---- stage-wise: the oracle fed the GPU's float32 inputs
    v = osamp.verify_chain(drafts[1:], mp, mq, sig, kb, seed, b, rnd, mode, usample, omega)
    lrp = after["lrp"][i][:kb]
    s2 = lrp[:, :, 0].sum(axis=1)
    sz = lrp[:, :, 1].sum(axis=1)
    nrm2 = s2 / sig[:kb] ** 2
    ell = -sz / sig[:kb] ** 2 - 0.5 * nrm2
    # the float64 sums differ only in their order: 1e-10 of the terms' size
    zd = np.abs(v["dot"]) + 0.5 * v["nrm2"] + 1.0
    assert np.all(np.abs(nrm2 - v["nrm2"]) <= 1e-10 * np.maximum(v["nrm2"], 1.0)), (b, k, nrm2, v["nrm2"])
    assert np.all(np.abs(ell - v["ell"]) <= 1e-10 * zd), (b, k, ell, v["ell"])
    tau = int(after["tau"][i])
    stats.compared += 1
    if v["ties"]:
        stats.ties += 1
    else:
        assert tau == v["tau"], (b, k, rnd, tau, v["tau"])
        coins = int(after["coins"][i]) & ((1 << kb) - 1)
        want = sum(1 << j for j in range(kb) if v["coins"][j])
        assert coins == want, (b, k, bin(coins), bin(want))
    if tau == v["tau"]:
        if mode == osamp.BLOCK and tau >= 2:
            _close_scalar(float(after["log_alpha_res"][i]), v["log_alpha_res"], 1e-10, f"log alpha_res {b}")
        if tau <= kb and residual == osamp.DECOMPOSITION:
            _close_scalar(float(after["u"][i]), v["U"], 1e-7, f"U chain {b} round {rnd}")
    knew = min(k + tau, N)
    y_gpu = after["x"][i][0] if knew < N else after["y"][i]
    u_gpu = float(after["u"][i])
    y_ref = osamp.residual_chain(drafts[1:], mp, mq, sig, kb, tau, u_gpu, N - k, seed, b, rnd, residual)
    stats.note("state (stage-wise)", assert_rows_close(y_gpu[None], y_ref[None], what=f"Y chain {b} round {rnd}"))
    if knew < N and not frozen:
        c = min(tau, kb)
        assert int(after["cache_step"][i]) == min(k + c, N - 1), (b, k, tau)
        c1c = F64(coef_f32(sched, k + c)[0])
        want_sv = mq[c].astype(F64) - c1c * drafts[c].astype(F64)
        err = np.linalg.norm(after["cache"][i] - want_sv) / max(np.linalg.norm(want_sv), 1e-30)
        assert err <= 1e-6, (b, k, err)
    if not independent:
        return True
    # ---- independent: the oracle's own round from the GPU's state
    stats.independent += 1
    y0 = before["x"][i][0].astype(F64)
    c2c = float(sched.c2(int(before["cache_step"][i])))
    score_c = before["cache"][i].astype(F64) / c2c
    y_new, score_new, k_new, info = osamp.run_round(gmm, sched, K, y0, score_c, k, rnd, seed, b, mode,
                                                    usample, residual, drafter, omega)
    stats.note("drafts", assert_rows_close(drafts[1:], info["yh"][1:], what=f"drafts chain {b} round {rnd}"))
    nrows = info["mq"].shape[0]
    stats.note("m^q", assert_rows_close(mq[:nrows], info["mq"], what=f"m^q chain {b} round {rnd}"))
    if info["tau"] != tau:
        # a float32 tie: the coin lies between the two thresholds, and the
        # log-ratios are within the float32 tolerance of each other
        h_ind = np.exp(info["log_h"])
        h_stg = np.exp(v["log_h"])
        between = [j for j in range(kb)
                   if min(h_ind[j], h_stg[j]) <= info["eta"][j] <= max(h_ind[j], h_stg[j])]
        assert between, (b, k, rnd, tau, info["tau"], info["eta"], h_ind, h_stg)
        _, _, ell_i = log_ratio_terms(info["yh"][1:], info["mp"], info["mq"][:kb], sig[:kb])
        dn = np.sqrt(np.maximum(info["nrm2"], 0.0))
        zn = np.linalg.norm((info["yh"][1:] - info["mp"]) / sig[:kb, None], axis=1)
        assert np.all(np.abs(ell_i - v["ell"]) <= 1e-4 * (zn * dn + 0.5 * info["nrm2"]) + 1e-12), (b, k)
        stats.f32_flips += 1
        return True
    stats.note("state (independent)", assert_rows_close(y_gpu[None], y_new[None], what=f"Y vs oracle round, chain {b}"))
    if k_new < N and not frozen:
        got = after["cache"][i].astype(F64) / float(sched.c2(int(after["cache_step"][i])))
        stats.note("cache", assert_rows_close(got[None], score_new[None], what=f"cached score chain {b}"))
    return True
