"""Sampler rounds on the GPU against the oracle, one round at a time.

The sampler runs a round per call (start_round / max_rounds) and its state is
read through sd_sampler_state before and after each round; tests/round_parity.py
holds the comparison rules.

* bf16 fused rounds at the pixel12288 and latent16384 shapes (K + 1 = 17 and 9:
  the 128-row mean tiles whose rows straddle chains, and the chain-aligned
  288 x 256 tiles, 32 chains of 9 rows), and at shapes that give the
  chain-aligned tile other chain counts (K + 1 = 2, 5, 17, 32: 56, 56, 16
  and 9 chains per tile, partial last tiles, M not a power of two): m^q per-row relative
  L2 <= 2e-2 against the float64 oracle, then, stage-wise, ||Delta||, ell, tau,
  coins, alpha_res, U, the new state and the next cache against the oracle fed
  the GPU's own drafts and m^q.  Reduced B (row tiles that straddle chains,
  a ragged last tile) and one round at the full B.
* a whole bf16 run on the chain-aligned tile (d = 1024, M = 512, K = 8) in
  lockstep for the three modes: 24 chains stage-wise every round.
* pixel3072 in float32 at the benchmark's size (B = 1024, N = 200) in
  lockstep for block/Free, token/reflection and block/Frozen: 32 chains every
  round stage-wise and, in turn, every fourth round of each against the
  oracle's own round from the GPU's state.
* Temperature: pixel3072 at full size at omega = 2 (block/Free) and a whole
  bf16 run on the chain-aligned tile at omega = 0.5 (token/reflection).
* The U draw with the paper's caps (Alg. 7 as run in its experiments) on a
  pixel3072-shaped run.
* A run split over calls equals one call; the device's tie counts equal the
  oracle's.
"""
import numpy as np
import pytest
import torch

from helpers import rel_l2_rows, target_mean_bf16_operands
from oracle import sampler as osamp
from oracle.gmm import GMM, target_mean
from oracle.schedule import Schedule
from paper_2606_13426_amd import _lib
from paper_2606_13426_amd.inputs import WORKLOADS, make_gmm, workload_gmm
from round_parity import RoundStats, check_round, snapshot

pytestmark = pytest.mark.gpu
DEV = "cuda"
MQ_REL_L2 = 2e-2
SCORE_VS_MODEL = 2e-3

_MODES = {
    (_lib.SD_BLOCK, _lib.SD_RESIDUAL_DECOMPOSITION, _lib.SD_DRAFTER_FREE):
        (osamp.BLOCK, osamp.DECOMPOSITION, osamp.FREE),
    (_lib.SD_TOKEN, _lib.SD_RESIDUAL_REFLECTION, _lib.SD_DRAFTER_FREE):
        (osamp.TOKEN, osamp.REFLECTION, osamp.FREE),
    (_lib.SD_BLOCK, _lib.SD_RESIDUAL_DECOMPOSITION, _lib.SD_DRAFTER_FROZEN):
        (osamp.BLOCK, osamp.DECOMPOSITION, osamp.FROZEN),
}


def _straddling(B, K1, tile=128):
    """Chains whose K + 1 rows cross a boundary of the mean GEMM's row tiles."""
    return [b for b in range(B) if (b * K1) // tile != (b * K1 + K1 - 1) // tile]


# (workload or (d, M, K, N), B, sampled chains): the two bf16 workloads' shapes
# at reduced and full B, a block of K + 1 = 5 rows with M = 64 (the 128-row
# kernel's general epilogue), and M >= 512 with d a multiple of 256 (the
# chain-aligned tile) at K + 1 = 5, 17, 2 and 32
BF16_ROUNDS = [("latent16384", 16, None), ("pixel12288", 16, None), ("latent16384", 256, 20),
               ("pixel12288", 512, 20), ((1024, 64, 4, 40), 48, None), ((512, 512, 4, 40), 70, None),
               ((512, 512, 16, 60), 40, None), ((768, 576, 1, 30), 130, None),
               ((512, 1024, 31, 80), 20, None)]


@pytest.mark.parametrize("name,B,nsel", BF16_ROUNDS)
def test_bf16_fused_round_stagewise(name, B, nsel):
    if isinstance(name, str):
        cfg = WORKLOADS[name]
        K, N = cfg["K"], cfg["N"]
        p = workload_gmm(name)
        assert K + 1 >= 8
    else:
        d, M, K, N = name
        p = make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=9)
    seed = 3
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"], precision=_lib.SD_BF16)
    ws = torch.empty(_lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device=DEV)
    r0 = 3
    _, st0, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, ws=ws, max_rounds=r0)
    assert st0["rounds"] == r0 and not st0["finished"]
    if nsel is None:
        sel = list(range(B))
    else:
        strad = _straddling(B, K + 1)
        sel = sorted(set(np.linspace(0, B - 1, nsel).astype(int).tolist()) | set(strad[:4]))
    before = snapshot(_lib.sd_sampler_state(tgt, B, K, ws, r0), sel)
    _, st1, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, ws=ws, start_round=r0, max_rounds=1)
    assert st1["rounds"] == r0 + 1
    after = snapshot(_lib.sd_sampler_state(tgt, B, K, ws, r0 + 1), sel)
    torch.cuda.synchronize()
    g = GMM(p["mu"], p["var"], p["log_w"])
    sch = Schedule(N)
    # m^q of every target row of the round against the float64 oracle, and the
    # score against the model of the bf16 operand rounding
    xs, steps, mqs = [], [], []
    for i in range(len(sel)):
        k = int(before["k"][i])
        nrows = min(min(K, N - k) + 1, N - k)
        xs.append(before["x"][i][:nrows])
        steps.append(k + np.arange(nrows))
        mqs.append(after["mq"][i][:nrows])
    x = np.concatenate(xs).astype(np.float64)
    n = np.concatenate(steps)
    mq = np.concatenate(mqs)
    ref_mq, _ = target_mean(g, sch, x, n)
    e = rel_l2_rows(mq, ref_mq)
    assert e.max() <= MQ_REL_L2, f"m^q per-row relative L2 {e.max():.3e}"
    model_mq, _ = target_mean_bf16_operands(g, sch, x, n)
    c2 = sch.c2(n)[:, None]
    e_sc = rel_l2_rows((mq - sch.c1(n)[:, None] * x) / c2, (model_mq - sch.c1(n)[:, None] * x) / c2)
    assert e_sc.max() <= SCORE_VS_MODEL, f"score vs the bf16 model {e_sc.max():.3e}"
    stats = RoundStats()
    for i, b in enumerate(sel):
        assert check_round(g, sch, K, seed, i, b, before, after, stats)
    assert stats.compared == len(sel) and stats.ties <= max(1, len(sel) // 50)


def _lockstep(mode, residual, drafter, name="pixel3072", B=None, N=None, K=None, M=None, d=None,
              nchains=32, seed=0, every=4, precision=None, omega=1.0, usample=_lib.SD_USAMPLE_EXACT):
    """Run the sampler a round per call and check `nchains` chains every round
    stage-wise; with every > 0 also, in turn, every `every`-th round of each
    against the oracle's own round (float32 targets only)."""
    cfg = WORKLOADS[name]
    B, N, K = B or cfg["B"], N or cfg["N"], K or cfg["K"]
    p = workload_gmm(name) if d is None else make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0,
                                                      seed=d)
    kw_t = {} if precision is None else dict(precision=precision)
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"], **kw_t)
    ws = torch.empty(_lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device=DEV)
    trace = torch.zeros(N, B, dtype=torch.int32, device=DEV)
    chains = np.unique(np.linspace(0, B - 1, nchains).astype(int))
    g = GMM(p["mu"], p["var"], p["log_w"])
    sch = Schedule(N)
    om = _MODES[(mode, residual, drafter)]
    kw = dict(mode=mode, residual=residual, drafter=drafter, ws=ws, trace=trace, omega=omega,
              usample_mode=usample)
    _, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, max_rounds=0, **kw)
    assert st["rounds"] == 0
    stats = RoundStats()
    r = 0
    before = snapshot(_lib.sd_sampler_state(tgt, B, K, ws, 0), chains)
    while True:
        y_out, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, start_round=r, max_rounds=1, **kw)
        if st["finished"] and st["rounds"] <= r:
            break
        assert st["rounds"] == r + 1
        after = snapshot(_lib.sd_sampler_state(tgt, B, K, ws, r + 1), chains)
        active = 0
        for i, b in enumerate(chains):
            active += check_round(g, sch, K, seed, i, int(b), before, after, stats, *om,
                                  independent=every > 0 and (r + i) % every == 0, omega=omega,
                                  usample=usample)
        before = after
        r += 1
        if st["finished"]:
            break
        if active == 0:
            # the sampled chains are done: the rest of the run in one call
            _, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, start_round=r, **kw)
            break
    torch.cuda.synchronize()
    assert st["finished"] and st["steps"] == B * N
    return stats, st


@pytest.mark.parametrize("mode,residual,drafter", list(_MODES))
def test_pixel3072_full_size_lockstep(mode, residual, drafter):
    stats, st = _lockstep(mode, residual, drafter)
    assert stats.compared >= 32 * (200 // 9)
    assert stats.independent >= stats.compared // 4 - 32
    # decisions a float32 input rounding moved across a coin, each explained
    assert stats.f32_flips <= max(2, stats.independent // 500), stats.f32_flips
    assert stats.ties <= max(3, stats.compared // 200), stats.ties
    print(f"lockstep: {stats.compared} chain-rounds, {stats.independent} independent, "
          f"ties {stats.ties}, float32 flips {stats.f32_flips}, worst {stats.worst}")


@pytest.mark.parametrize("mode,residual,drafter", list(_MODES))
def test_bf16_chain_aligned_tile_lockstep(mode, residual, drafter):
    # a whole bf16 run on the chain-aligned mean tile (M = 512, d a multiple of
    # 256, K + 1 = 9: 32 chains per tile; 72 chains leave a last tile of 8),
    # 24 chains checked stage-wise every round: the oracle's verification and
    # residual fed the GPU's drafts, m^q and draft means
    stats, st = _lockstep(mode, residual, drafter, B=72, N=60, K=8, M=512, d=1024, nchains=24, seed=3,
                          every=0, precision=_lib.SD_BF16)
    assert stats.compared >= 24 * (60 // 9) and stats.independent == 0
    assert stats.ties <= max(3, stats.compared // 200), stats.ties
    print(f"bf16 lockstep: {stats.compared} chain-rounds, ties {stats.ties}, worst {stats.worst}")


def test_tempered_lockstep():
    # temperature (App. "Temperature"): pixel3072 at full size, block/Free at
    # omega = 2, in lockstep as above; and a whole bf16 run on the
    # chain-aligned tile, token/reflection at omega = 0.5, stage-wise
    stats, _ = _lockstep(_lib.SD_BLOCK, _lib.SD_RESIDUAL_DECOMPOSITION, _lib.SD_DRAFTER_FREE, omega=2.0,
                         nchains=32, seed=2)
    assert stats.compared >= 32 * (200 // 9)
    assert stats.f32_flips <= max(2, stats.independent // 500), stats.f32_flips
    assert stats.ties <= max(3, stats.compared // 200), stats.ties
    b16, _ = _lockstep(_lib.SD_TOKEN, _lib.SD_RESIDUAL_REFLECTION, _lib.SD_DRAFTER_FREE, B=72, N=60, K=8,
                       M=512, d=1024, nchains=24, seed=3, every=0, precision=_lib.SD_BF16, omega=0.5)
    assert b16.compared >= 24 * (60 // 9) and b16.ties <= max(3, b16.compared // 200), b16.ties
    print(f"tempered lockstep: {stats.compared} / {b16.compared} chain-rounds, ties {stats.ties} / {b16.ties}, "
          f"worst {stats.worst}")


def test_paper_usample_lockstep():
    # the U draw with the paper's caps (Alg. 7: three doublings, four
    # bisections, tolerance 1e-6) inside the sampler: 24 chains of a
    # pixel3072-shaped run every round, every second one also against the
    # oracle's own round
    stats, _ = _lockstep(_lib.SD_BLOCK, _lib.SD_RESIDUAL_DECOMPOSITION, _lib.SD_DRAFTER_FREE, B=256, N=60,
                         nchains=24, seed=5, every=2, usample=_lib.SD_USAMPLE_PAPER)
    assert stats.compared >= 24 * (60 // 9) and stats.f32_flips <= 2
    assert stats.ties <= max(3, stats.compared // 200), stats.ties


def test_streamed_draft_rows_lockstep():
    # B (K + 1) d float32 = 1024 x 9 x 4096 x 4 = 151 MB of draft rows: above
    # the 128 MB at which the draft and advance kernels store them with
    # non-temporal stores
    B, K, N, d, M = 1024, 8, 16, 4096, 64
    assert B * (K + 1) * d * 4 > 128 << 20
    stats, _ = _lockstep(_lib.SD_BLOCK, _lib.SD_RESIDUAL_DECOMPOSITION, _lib.SD_DRAFTER_FREE,
                         B=B, N=N, K=K, M=M, d=d, nchains=16, seed=6, every=2)
    assert stats.compared >= 16 * 2 and stats.f32_flips <= 2


def test_small_lockstep_every_round_independent():
    # a few chains of pixel3072 on a short schedule: every round of every chain
    # against the oracle's own round (K > N - k ragged blocks at the end)
    stats, _ = _lockstep(_lib.SD_BLOCK, _lib.SD_RESIDUAL_DECOMPOSITION, _lib.SD_DRAFTER_FREE,
                         B=6, N=12, nchains=6, seed=4, every=1)
    assert stats.independent == stats.compared and stats.f32_flips == 0


@pytest.mark.parametrize("drafter", [_lib.SD_DRAFTER_FREE, _lib.SD_DRAFTER_FROZEN])
def test_split_run_equals_one_call(drafter):
    p = workload_gmm("tiny2d")
    B, K, N, seed = 64, 4, 40, 9
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"])
    y1, s1, t1 = _lib.sd_run_sampler_ex(tgt, B, K, seed, drafter=drafter, trace_rounds=N)
    ws = torch.empty(_lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device=DEV)
    trace = torch.zeros(N, B, dtype=torch.int32, device=DEV)
    y2 = torch.full_like(y1, float("nan"))
    r = 0
    for n in (0, 1, 3, 0, 2, 5):
        _, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, drafter=drafter, ws=ws, trace=trace, y_out=y2,
                                          start_round=r, max_rounds=n)
        assert st["rounds"] == r + n and not st["finished"]
        assert torch.isnan(y2).all()  # a partial call leaves y_out alone
        r = st["rounds"]
    _, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, drafter=drafter, ws=ws, trace=trace, y_out=y2,
                                      start_round=r)
    torch.cuda.synchronize()
    assert st["finished"] and st["rounds"] == s1["rounds"]
    assert torch.equal(y1, y2) and torch.equal(t1, trace)
    for key in ("chain_rounds", "steps", "ties", "tau_hist"):
        assert st[key] == s1[key], key
    assert st["mean_tau"] == pytest.approx(s1["mean_tau"])
    # a finished run continued is still finished and unchanged
    _, st2, _ = _lib.sd_run_sampler_ex(tgt, B, K, seed, drafter=drafter, ws=ws, y_out=y2,
                                       start_round=st["rounds"], max_rounds=3)
    assert st2["finished"] and st2["rounds"] == st["rounds"] and torch.equal(y1, y2)


@pytest.mark.parametrize("mode", [_lib.SD_BLOCK, _lib.SD_TOKEN])
def test_tie_counts_match_oracle(mode):
    # tiny2d end to end: the device counts the coins within 1e-6 of their
    # threshold per chain; on every chain whose rounds match the oracle's
    # the count equals the oracle's
    cfg = WORKLOADS["tiny2d"]
    B, K, N, seed = cfg["B"], cfg["K"], cfg["N"], 0
    p = workload_gmm("tiny2d")
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"])
    ws = torch.empty(_lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device=DEV)
    _, st, trace = _lib.sd_run_sampler_ex(tgt, B, K, seed, mode=mode, ws=ws, trace_rounds=N)
    ties = _lib.sd_sampler_state(tgt, B, K, ws, st["rounds"])["ties"].cpu().numpy()
    trace = trace.cpu().numpy()
    ref = osamp.run_sampler(GMM(p["mu"], p["var"], p["log_w"]), Schedule(N), B, K, seed, mode=mode)
    assert int(ties.sum()) == st["ties"]
    total = 0
    for i, b in enumerate(ref["chains"]):
        rec = ref["trace"][i]
        want = sum(len(info["ties"]) for info in rec)
        taus = [info["tau"] for info in rec]
        if list(trace[: len(taus), b]) == taus:
            assert int(ties[b]) == want, (b, int(ties[b]), want)
        else:
            assert want >= 1  # only a tie may send a chain another way
        total += want
    assert st["mean_tau"] == pytest.approx(
        sum(t * c for t, c in enumerate(st["tau_hist"])) / st["chain_rounds"])
    print(f"ties: device {st['ties']}, oracle {total}")
