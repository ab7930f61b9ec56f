"""Benchmark of the speculative-diffusion verification pass on one MI355X.

Step = one full run of the sampler (all hot-path steps: Free-Drafter drafts,
the Gaussian-mixture target on every draft state, log-ratio reductions, the
block-verification scan with U-sampling, the residual draw and the commit)
over one batch of B chains from Y_0 to Y_N, on the latent-sized workload
(d = 4*64*64, M = 1024 components, B = 256 chains, K = 8 drafts, N = 1000
steps, bf16 GEMM operands with float32 accumulation).  value = verified
chain-steps per second = B * N / seconds per run.

Per-kernel durations are measured live with HIP events on the launch's
stream; the dominant kernel's roofline uses its algorithmic work (see
algorithmic_work) over its measured time.  Runs use the library's choice of
chain groups (config.chain_groups); where it runs two concurrent groups, the
per-kernel times and the roofline come from extra one-group runs of the same
workload (roofline.chain_groups), since concurrent kernels share the GPU.  The pixel-sized float32 workload
(with token verification), the 64x64x3 pixel workload, the
verification-only workload (B = 4096, K = 32, d = 12288) and the paper's
variants are extra fields; the CPU oracle is timed on a bounded sample of
rounds of the headline workload.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_PEAK_TFLOPS = 157.3
BF16_PEAK_TFLOPS = 2500.0   # dense bf16 MFMA
GEMMS = ("gmm_logits", "gmm_mean", "gmm_mean_lr", "gmm_logits_bf16", "gmm_mean_bf16", "gmm_mean_lr_bf16")
METRIC = "verified chain-steps/sec + mean accepted steps per block; % MFMA / HBM peak"

# HBM bytes per launch of a workload's dominant kernel from two rocprofv3 passes
# (FETCH_SIZE x 2.000 and WRITE_SIZE x 1.000, the factors a 1 GiB device copy
# gives; profiles/sampler_latent16384_hbm_traffic.md), valid while the kernel's
# sources (its translation unit, every library header and the C header) have
# the digest (source_digest(unit)) recorded with them.
PROFILE_EVERY = 4  # the timed runs' event sample of the dominant kernel's launches

MEASURED_TRAFFIC = {
    ("verify12288", "logratio_reduce"): dict(bytes=(19344.1 + 8.5) * 1e6, unit="verify.hip",
                                             sources="7cb5cb276a21be1edb5612e45820ec882473a651"),
    ("pixel3072", "gmm_mean_lr"): dict(bytes=(136.1 + 122.0) * 1e6, unit="gmm.hip",
                                       sources="1d9832fb95c336178846c2f8d069c8aad7d8558d"),
    ("latent16384", "gmm_mean_lr_bf16"): dict(bytes=(277.7 + 154.0) * 1e6, unit="gmm_bf16.hip",
                                              sources="bc618f4030c65b9b569657e8f3ca128e666ddf1e"),
    ("pixel12288", "gmm_mean_lr_bf16"): dict(bytes=(511.7 + 445.9) * 1e6, unit="gmm_bf16.hip",
                                             sources="bc618f4030c65b9b569657e8f3ca128e666ddf1e"),
}


def measured_traffic(workload, kernel):
    """HBM bytes per launch from the committed counters, while the kernel's
    sources are those the counters were taken from; else None."""
    meas = MEASURED_TRAFFIC.get((workload, kernel))
    if meas and meas["sources"] == source_digest(meas["unit"]):
        return meas["bytes"]
    return None


def source_digest(unit):
    """sha1 over a kernel's translation unit csrc/<unit>, the library headers
    and the C header (names and contents with comments removed, so that a
    change to documentation alone keeps the counters valid)."""
    import glob
    import hashlib
    import re
    h = hashlib.sha1()
    files = sorted([os.path.join(ROOT, "paper_2606_13426_amd", "csrc", unit)] +
                   glob.glob(os.path.join(ROOT, "paper_2606_13426_amd", "csrc", "*.hpp")) +
                   [os.path.join(ROOT, "include", "specdiff.h")])
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f) as fh:
            code = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
        code = re.sub(r"//[^\n]*", "", code)
        h.update(code.encode())
    return h.hexdigest()


def _counts_from_trace(trace, N, K):
    """Per round: active chains, verified draft rows and drafted rows, from the tau trace."""
    R, B = trace.shape
    k = np.zeros(B, dtype=np.int64)
    act, rows_verified, rows_target = [], [], []
    for r in range(R):
        t = trace[r]
        a = t > 0
        if not a.any():
            break
        kb = np.minimum(K, N - k)
        act.append(int(a.sum()))
        rows_verified.append(int(kb[a].sum()))
        rows_target.append(int(np.minimum(kb + 1, N - k)[a].sum()))
        k = np.where(a, np.minimum(k + t, N), k)
    return np.array(act), np.array(rows_verified), np.array(rows_target)


def algorithmic_work(name, B, K, d, M, act, rows_verified, runs, nct=1):
    """(flops, bytes, dtype bytes) of a kernel's algorithmic work over `runs` sampler runs.

    Units per round: the GEMMs are launched on all B (K+1) rows (2 flops per
    multiply-add) and must move their operands and outputs once: the logits
    GEMM reads X and mu and produces the R x M logits, the mean GEMM reads X,
    each chain's cache row and mu and writes m^q (the draft means are
    recomputed, not stored); the explicit target call at Y_0 (one per run)
    covers B rows.  The streaming kernels count the float32 bytes their rows
    move once, for active chains only: advance reads the residual's state,
    mean and cache rows and the new cache's two rows, and writes the new
    state, K+1 draft rows and the new cache row.  Rounds launched after every
    chain has finished exit at once and count no work.  Returns None for
    kernels without a throughput roof (latency-bound scalar work).
    """
    rounds = len(act)
    R = B * (K + 1)
    bf = name.endswith("_bf16")
    eb = 2 if bf else 4
    if name in ("gmm_logits", "gmm_logits_bf16"):
        rows = R * rounds + B
        return 2.0 * rows * d * M * runs, (rows * d * 4 + rows * M * 4 + (rounds + 1) * M * d * eb) * runs, eb
    if name in ("gmm_mean_lr", "gmm_mean_lr_bf16"):
        rows = R * rounds
        return (2.0 * rows * M * d * runs,
                (rows * d * 8 + B * rounds * d * 4 + rounds * M * d * eb) * runs, eb)
    if name in ("gmm_mean", "gmm_mean_bf16"):
        return 2.0 * B * M * d * runs, (B * d * 8 + M * d * eb) * runs, eb
    if name == "gmm_softmax":
        rows = R * rounds + B
        return 0.0, rows * M * (4 + eb) * runs, eb
    if name == "logratio_reduce":
        return 0.0, 3.0 * 4 * d * rows_verified.sum() * runs, 4
    if name == "draft_block":   # one per run: reads y and the cached (x, m^q) row; K+1 drafts, the cache row
        return 0.0, 4.0 * d * (3 + (K + 1) + 1) * B * runs, 4
    if name == "advance":
        return 0.0, 4.0 * d * (5 + 1 + (K + 1) + 1) * act.sum() * runs, 4
    return None


def roof_entry(flops, nbytes, ms, eb):
    """Binding roof of a kernel: the one its algorithmic work needs more time on."""
    sec = ms * 1e-3
    mf_peak = (BF16_PEAK_TFLOPS if eb == 2 else FP32_PEAK_TFLOPS) * 1e12
    t_mfma, t_hbm = flops / mf_peak, nbytes / (HBM_PEAK_GBS * 1e9)
    if t_mfma >= t_hbm:
        return dict(bound="mfma", achieved=flops / sec / 1e12, unit="TFLOP/s", peak=mf_peak / 1e12,
                    frac=t_mfma / sec, algorithmic_flops=flops, algorithmic_bytes=nbytes)
    return dict(bound="hbm", achieved=nbytes / sec / 1e9, unit="GB/s", peak=HBM_PEAK_GBS,
                frac=t_hbm / sec, algorithmic_flops=flops, algorithmic_bytes=nbytes)


def run_sampler_bench(lib, name, mode, steps, warmup, profile, groups_req=0):
    """Whole sampler runs on the workload (Y_0 to Y_N) with the library's
    choice of chain groups: the seconds per run.  With profile, also the
    per-kernel breakdown of one profiled run and live HIP-event times of a
    systematic sample of the dominant kernel's launches over `steps` timed
    runs -- in the same timed runs when the sampler runs one chain group, else
    in `steps` extra runs with one group (the kernels of two concurrent groups
    share the GPU, so their event durations would not be the kernels' own)."""
    import torch
    from paper_2606_13426_amd.inputs import WORKLOADS, workload_gmm
    cfg = WORKLOADS[name]
    B, K, N, d, M = cfg["B"], cfg["K"], cfg["N"], cfg["d"], cfg["M"]
    p = workload_gmm(name)
    prec = lib.SD_BF16 if cfg["precision"] == "bf16" else lib.SD_FP32
    tgt = lib.Target(lib.schedule(N), p["mu"], p["var"], p["log_w"], precision=prec)
    ws = torch.empty(lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device="cuda")
    y = torch.empty(B, d, dtype=torch.float32, device="cuda")
    seed = 0

    def run(groups, trace_rounds=0):
        return lib.sd_run_sampler_ex(tgt, B, K, seed, mode=mode, y_out=y, ws=ws, groups=groups,
                                     trace_rounds=trace_rounds)

    for _ in range(max(warmup, 1)):
        _, st_w, _ = run(groups_req)
    torch.cuda.synchronize()
    groups = st_w["groups"]
    prof_groups = 1  # the grouping of the profiled runs

    def profile_begin():
        # one profiled run gives the per-kernel breakdown and names the
        # dominant kernel; the timed runs then bracket every PROFILE_EVERY-th
        # launch of it: a systematic sample whose events cost the stream a
        # quarter of what timing every launch does
        lib.sd_profile_only(None)
        lib.sd_profile_enable(True)
        run(prof_groups)
        bd = lib.sd_profile_read()
        lib.sd_profile_enable(False)
        dom = max(bd, key=lambda n: bd[n][1])
        torch.cuda.synchronize()
        lib.sd_profile_only(dom)
        lib.sd_profile_every(PROFILE_EVERY)
        lib.sd_profile_enable(True)
        return bd, dom

    def profile_end(dom):
        p, n = lib.sd_profile_read(), lib.sd_profile_seen(dom)
        lib.sd_profile_enable(False)
        lib.sd_profile_only(None)
        lib.sd_profile_every(1)
        return p, n

    breakdown, only, prof, seen = {}, None, {}, 0
    live = profile and groups == prof_groups
    if live:
        breakdown, only = profile_begin()
    stats = []
    t0 = time.perf_counter()
    for s in range(steps):
        _, st, trace = run(groups_req, trace_rounds=N if s == 0 else 0)
        stats.append(st)
        if s == 0:
            trace0 = trace.cpu().numpy()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if live:
        prof, seen = profile_end(only)
    elif profile:
        breakdown, only = profile_begin()
        for _ in range(steps):
            run(prof_groups)
        torch.cuda.synchronize()
        prof, seen = profile_end(only)
    sec = (t1 - t0) / steps
    st = stats[0]
    be = st["steps"] / st["chain_rounds"]
    act, rows_v, rows_t = _counts_from_trace(trace0, N, K)
    return dict(B=B, K=K, N=N, d=d, M=M, sec=sec, be=be, rounds=st["rounds"], prof=prof, seen=seen,
                mean_tau=st["mean_tau"], ties=st["ties"], groups=groups,
                profile_groups=prof_groups if profile else None,
                breakdown=breakdown,
                act=act, rows_verified=rows_v, rows_target=rows_t, tau_hist=st["tau_hist"][: K + 2],
                steps=steps)


def roofline_of(res, steps):
    """Roofline of the dominant kernel (timed live over the timed runs) and the
    per-kernel table of the profiled warm-up run (one sampler run)."""
    prof = res["prof"]
    if not prof:
        return None, {}
    name = max(prof, key=lambda n: prof[n][1])
    table = {}
    sources = dict(res["breakdown"])
    # the timed runs timed a systematic sample of the dominant kernel's
    # launches: its total time over all of them is the sample's mean duration
    # times the launches seen
    timed, ms_timed = prof[name]
    seen = max(res.get("seen", 0), timed)
    sources[name] = (seen, ms_timed * seen / max(timed, 1))
    for kname, (launches, ms) in sources.items():
        runs = steps if kname == name else 1
        entry = dict(launches=launches, avg_us=1e3 * ms / max(launches, 1), total_ms=ms)
        if kname == name:
            entry.update(timed_launches=timed)
        w = algorithmic_work(kname, res["B"], res["K"], res["d"], res["M"], res["act"],
                             res["rows_verified"], runs)
        if w is not None:
            entry.update(roof_entry(w[0], w[1], ms, w[2]))
        table[kname] = entry
    gem = [k for k in GEMMS if k in res["breakdown"]]
    if gem:
        # the denoiser's GEMMs together over the profiled run, against the matrix-core peak
        flops = sum(algorithmic_work(k, res["B"], res["K"], res["d"], res["M"], res["act"],
                                     res["rows_verified"], 1)[0] for k in gem)
        ms = sum(res["breakdown"][k][1] for k in gem)
        peak = BF16_PEAK_TFLOPS if gem[0].endswith("_bf16") else FP32_PEAK_TFLOPS
        table["denoiser_gemms"] = dict(bound="mfma", achieved=flops / (ms * 1e-3) / 1e12, unit="TFLOP/s",
                                       peak=peak, frac=flops / (ms * 1e-3) / 1e12 / peak, total_ms=ms)
    e = table[name]
    per = lambda v: v / max(e["launches"], 1) if v is not None else None
    roof = dict(kernel=name, bound=e.get("bound"), achieved=e.get("achieved"), peak=e.get("peak"),
                unit=e.get("unit"), frac=e.get("frac"), traffic=None,
                algorithmic_per_launch=per(e.get("algorithmic_bytes") if e.get("bound") == "hbm"
                                           else e.get("algorithmic_flops")),
                avg_launch_us=e["avg_us"], launches=e["launches"], timed_launches=timed)
    return roof, table


def _be_by_step(trace, N, nbins=10):
    """Steps advanced per chain-round for rounds starting in each tenth of the
    schedule (the acceptance-versus-step curve), from a tau trace [rounds][B]."""
    R, B = trace.shape
    k = np.zeros(B, dtype=np.int64)
    adv = np.zeros(nbins)
    cnt = np.zeros(nbins)
    for r in range(R):
        t = trace[r]
        a = t > 0
        if not a.any():
            break
        knew = np.minimum(k + t, N)
        bins = np.minimum(k * nbins // N, nbins - 1)
        np.add.at(adv, bins[a], (knew - k)[a])
        np.add.at(cnt, bins[a], 1)
        k = np.where(a, knew, k)
    return [float(a / c) if c else None for a, c in zip(adv, cnt)]


def variants_bench(lib, name, steps):
    """The paper's alternatives on the same workload and seed: the three
    residual/verification pairs of its comparison tables (reflection with
    sample verification R, decomposition with sample verification D, block B)
    at temperatures 0.5, 1, 2; the Frozen Drafter; and the plain
    Euler-Maruyama chain (one target call on B rows per step), with the terms
    of the paper's speedup decomposition (App. on Frozen and Free Drafters)
    from per-kernel event times of one profiled run each."""
    import torch
    from paper_2606_13426_amd.inputs import WORKLOADS, workload_gmm
    cfg = WORKLOADS[name]
    B, K, N, d = cfg["B"], cfg["K"], cfg["N"], cfg["d"]
    p = workload_gmm(name)
    prec = lib.SD_BF16 if cfg["precision"] == "bf16" else lib.SD_FP32
    tgt = lib.Target(lib.schedule(N), p["mu"], p["var"], p["log_w"], precision=prec)
    ws = torch.empty(lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device="cuda")
    y = torch.empty(B, d, dtype=torch.float32, device="cuda")
    seed = 0

    def timed_runs(fn, reps):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            out = fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / reps, out

    def profiled(fn):
        lib.sd_profile_only(None)
        lib.sd_profile_enable(True)
        fn()
        prof = lib.sd_profile_read()
        lib.sd_profile_enable(False)
        return prof

    def sampler(mode, residual, drafter, omega, trace_rounds=0, groups=0):
        return lambda: lib.sd_run_sampler_ex(tgt, B, K, seed, mode=mode, residual=residual, drafter=drafter,
                                             omega=omega, y_out=y, ws=ws, trace_rounds=trace_rounds,
                                             groups=groups)

    reps = max(2, steps // 3)
    kinds = {"R": (lib.SD_TOKEN, lib.SD_RESIDUAL_REFLECTION), "D": (lib.SD_TOKEN, lib.SD_RESIDUAL_DECOMPOSITION),
             "B": (lib.SD_BLOCK, lib.SD_RESIDUAL_DECOMPOSITION)}
    table = {}
    for omega in (0.5, 1.0, 2.0):
        for kind, (mode, resid) in kinds.items():
            sec, (_, st, _) = timed_runs(sampler(mode, resid, lib.SD_DRAFTER_FREE, omega), reps)
            table[f"{kind}_omega{omega:g}"] = dict(value=B * N / sec, ms_per_run=1e3 * sec,
                                                   mean_accepted_steps_per_block=st["steps"] / st["chain_rounds"],
                                                   rounds_per_run=st["rounds"])
    frozen = {}
    for label, mode in (("block", lib.SD_BLOCK), ("token", lib.SD_TOKEN)):
        sec, (_, st, _) = timed_runs(sampler(mode, lib.SD_RESIDUAL_DECOMPOSITION, lib.SD_DRAFTER_FROZEN, 1.0), reps)
        frozen[label] = dict(value=B * N / sec, ms_per_run=1e3 * sec,
                             mean_accepted_steps_per_block=st["steps"] / st["chain_rounds"],
                             rounds_per_run=st["rounds"])
    # the plain EM chain
    em_ws = torch.empty(lib.sd_plain_em_workspace(tgt, B), dtype=torch.uint8, device="cuda")
    em_sec, _ = timed_runs(lambda: lib.sd_run_plain_em(tgt, B, seed, y_out=y, ws=em_ws), reps)
    em_prof = profiled(lambda: lib.sd_run_plain_em(tgt, B, seed, y_out=y, ws=em_ws))
    # speedup terms, per round of the block sampler (Free and Frozen) and per EM step
    tq1 = 1e3 * sum(v[1] for k, v in em_prof.items() if k.startswith("gmm_")) / N   # us per target call on B rows
    # (one chain group: a round's kernels then run one after another, so
    # their event times add up to the round)
    free_prof = profiled(sampler(lib.SD_BLOCK, lib.SD_RESIDUAL_DECOMPOSITION, lib.SD_DRAFTER_FREE, 1.0, groups=1))
    frz_prof = profiled(sampler(lib.SD_BLOCK, lib.SD_RESIDUAL_DECOMPOSITION, lib.SD_DRAFTER_FROZEN, 1.0, groups=1))
    _, (_, _, trace) = timed_runs(sampler(lib.SD_BLOCK, lib.SD_RESIDUAL_DECOMPOSITION, lib.SD_DRAFTER_FREE,
                                          1.0, trace_rounds=N), 1)
    be_curve = _be_by_step(trace.cpu().numpy(), N)

    def terms(prof, be):
        # per round of the lockstep sampler, from the profiled run: the target
        # kernels (the Frozen Drafter's call on B rows included), the
        # verification + residual + commit (+ Free-Drafter draft, fused into
        # advance), the Frozen Drafter's separate draft kernel, and the whole
        # round; the one-time start (Y_0, the first draft) is spread over it
        rounds = prof["scan_fused"][0]
        per = lambda names: 1e3 * sum(prof[k][1] for k in names if k in prof) / rounds
        round_us = per(list(prof))
        return dict(target_us=per([k for k in prof if k.startswith("gmm_")]),
                    verify_residual_commit_us=per(["scan_fused", "advance"]),
                    draft_kernel_us=per(["draft_block"]),
                    round_us=round_us, target_over_time_q1=per([k for k in prof if k.startswith("gmm_")]) / tq1,
                    predicted_speedup=be * tq1 / round_us)

    # the latency-bound regime the paper's speedup assumes (a target call on a
    # few rows costs about what one row costs): the same target and schedule
    # with B = 8 chains
    Bs = 8
    ws_s = torch.empty(lib.sd_sampler_workspace(tgt, Bs, K), dtype=torch.uint8, device="cuda")
    em_ws_s = torch.empty(lib.sd_plain_em_workspace(tgt, Bs), dtype=torch.uint8, device="cuda")
    ys = torch.empty(Bs, d, dtype=torch.float32, device="cuda")
    em_s, _ = timed_runs(lambda: lib.sd_run_plain_em(tgt, Bs, seed, y_out=ys, ws=em_ws_s), reps)
    small = dict(B=Bs, plain_em=dict(value=Bs * N / em_s, ms_per_run=1e3 * em_s))
    for label, mode, resid, drafter in (("block_free", lib.SD_BLOCK, lib.SD_RESIDUAL_DECOMPOSITION, lib.SD_DRAFTER_FREE),
                                        ("block_frozen", lib.SD_BLOCK, lib.SD_RESIDUAL_DECOMPOSITION, lib.SD_DRAFTER_FROZEN),
                                        ("token_reflection_free", lib.SD_TOKEN, lib.SD_RESIDUAL_REFLECTION, lib.SD_DRAFTER_FREE)):
        sec, (_, st, _) = timed_runs(
            lambda: lib.sd_run_sampler_ex(tgt, Bs, K, seed, mode=mode, residual=resid, drafter=drafter,
                                          y_out=ys, ws=ws_s), reps)
        small[label] = dict(value=Bs * N / sec, ms_per_run=1e3 * sec, speedup_vs_plain_em=em_s / sec,
                            mean_accepted_steps_per_block=st["steps"] / st["chain_rounds"],
                            rounds_per_run=st["rounds"])

    be_free = table["B_omega1"]["mean_accepted_steps_per_block"]
    be_frz = frozen["block"]["mean_accepted_steps_per_block"]
    spec_ms = table["B_omega1"]["ms_per_run"]
    return dict(
        three_way=table, frozen_drafter=frozen,
        plain_em=dict(value=B * N / em_sec, ms_per_run=1e3 * em_sec, target_calls=N,
                      time_q1_us=tq1,
                      kernels={k: dict(launches=v[0], avg_us=1e3 * v[1] / max(v[0], 1)) for k, v in em_prof.items()}),
        speedup_vs_plain_em=dict(block_free=1e3 * em_sec / spec_ms,
                                 block_frozen=1e3 * em_sec / frozen["block"]["ms_per_run"],
                                 token_free=1e3 * em_sec / table["D_omega1"]["ms_per_run"]),
        speedup_terms=dict(free=terms(free_prof, be_free), frozen=terms(frz_prof, be_frz), time_q1_us=tq1),
        be_by_step_tenths=be_curve, small_batch=small)


def verify_bench(lib, steps, warmup):
    """Verification-only workload: one sd_verify_block + sd_sample_residual per step."""
    import torch
    from paper_2606_13426_amd.inputs import WORKLOADS, verify_inputs
    cfg = WORKLOADS["verify12288"]
    B, K, d, N = cfg["B"], cfg["K"], cfg["d"], cfg["N"]
    sig = lib.sd_schedule_table(lib.schedule(N))[1]
    inp = verify_inputs(B, K, d, N, sig, seed=1, device="cuda", perturb=cfg["perturb"])
    y = torch.empty(B, d, device="cuda")
    out = None
    seed = 11

    def step():
        nonlocal out
        out = lib.sd_verify_block(inp["y_draft"], inp["mp"], inp["mq"], inp["sigma"], inp["kb"],
                                  inp["round"], seed, out=out)
        lib.sd_sample_residual(inp["y_draft"], inp["mp"], inp["mq"], inp["sigma"], inp["kb"],
                               inp["steps_left"], out["tau"], out["u_res"], out["delta_norm"],
                               inp["round"], seed, y)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    lib.sd_profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = lib.sd_profile_read()
    lib.sd_profile_enable(False)
    sec = (t1 - t0) / steps
    tau = out["tau"].cpu().numpy()
    lr_launches, lr_ms = prof["logratio_reduce"]
    algo = 3.0 * 4 * d * B * K
    res_bytes = 4.0 * d * 3 * B
    del inp
    return dict(workload="verify12288", B=B, K=K, d=d,
                value=B * K / sec, unit="verified chain-steps/s", ms_per_step=1e3 * sec,
                mean_tau=float(tau.mean()),
                logratio=dict(bound="hbm", achieved=algo / (lr_ms / lr_launches * 1e-3) / 1e9,
                              peak=HBM_PEAK_GBS, unit="GB/s",
                              frac=algo / (lr_ms / lr_launches * 1e-3) / 1e9 / HBM_PEAK_GBS,
                              traffic=measured_traffic("verify12288", "logratio_reduce"),
                              algorithmic_per_launch=algo, avg_launch_us=1e3 * lr_ms / lr_launches),
                pass_GBps=(algo + res_bytes) / sec / 1e9,
                kernels={k: dict(launches=v[0], avg_us=1e3 * v[1] / max(v[0], 1)) for k, v in prof.items()})


def cpu_baseline(name, budget_s):
    """The oracle (NumPy float64) on a bounded sample of the workload: whole
    chains one after another, round by round (Alg. 8), until the budget is
    spent; value = steps advanced / seconds.  Its matrix products run on the
    BLAS thread pool (cores = that pool's threads), the rest on one thread."""
    from threadpoolctl import threadpool_info

    from oracle import sampler as osamp
    from oracle.gmm import GMM
    from oracle.schedule import Schedule
    from paper_2606_13426_amd.inputs import WORKLOADS, workload_gmm
    cfg = WORKLOADS[name]
    p = workload_gmm(name)
    g = GMM(p["mu"], p["var"], p["log_w"])
    sch = Schedule(cfg["N"])
    N, K = cfg["N"], cfg["K"]
    t0 = time.perf_counter()
    chains = rounds = steps = 0
    done = False
    while chains < cfg["B"] and not done:
        y, sc = osamp.init_state(g, sch, 0, chains)
        k = r = 0
        while k < N:
            y, sc, k, info = osamp.run_round(g, sch, K, y, sc, k, r, 0, chains)
            r += 1
            rounds += 1
            steps += info["steps"]
            if time.perf_counter() - t0 > budget_s:
                done = True
                break
        chains += 1
    el = time.perf_counter() - t0
    blas = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
    cores = max(blas) if blas else 1
    return dict(value=steps / el, unit="chain-steps/s", cores=cores, kind="oracle",
                sample=f"{name}: chains 0..{chains - 1} of {cfg['B']} from Y_0, {rounds} rounds, "
                       f"{steps} chain-steps in {el:.1f} s (NumPy float64, {cores} BLAS threads)")


def _dtype(name):
    from paper_2606_13426_amd.inputs import WORKLOADS
    return "bf16" if WORKLOADS[name].get("precision") == "bf16" else "f32"


def _precision(name):
    from paper_2606_13426_amd.inputs import WORKLOADS
    if WORKLOADS[name].get("precision") == "bf16":
        return ("bf16 operands of the two denoiser GEMMs with f32 accumulation; f32 states and "
                "epilogue, f64 softmax, log-ratio sums and scans")
    return "f32 (GEMMs as exact split-bf16 products, f32 accumulation); f64 softmax, log-ratio sums and scans"


# the denoiser GEMM shapes of the workloads (m x k @ k x n) and two square
# references, run through the vendor library (torch.mm -> hipBLASLt / rocBLAS)
LIBRARY_GEMMS = {
    "bf16_square_8192": (8192, 8192, 8192, "bf16", None),
    "bf16_latent16384_logits": (2304, 16384, 1024, "bf16", ("latent16384", "gmm_logits_bf16")),
    "bf16_latent16384_mean": (2304, 1024, 16384, "bf16", ("latent16384", "gmm_mean_lr_bf16")),
    "bf16_pixel12288_logits": (8704, 12288, 256, "bf16", ("pixel12288", "gmm_logits_bf16")),
    "fp32_square_4096": (4096, 4096, 4096, "f32", None),
    "fp32_pixel3072_logits": (9216, 3072, 64, "f32", ("pixel3072", "gmm_logits")),
    "fp32_pixel3072_mean": (9216, 64, 3072, "f32", ("pixel3072", "gmm_mean_lr")),
}


def mfma_calibration(lib, blocks=1024, iters=512, reps=5):
    """The bf16 matrix-core rate this GPU sustains: the library's register-only
    loop of v_mfma_f32_32x32x16_bf16 (sd_mfma_loop; four wavefronts per SIMD,
    four independent accumulators each), timed with events after a warm-up,
    against the published dense peak."""
    import torch
    out = torch.empty(blocks * 4, dtype=torch.float32, device="cuda")
    for _ in range(2):
        lib.sd_mfma_loop(blocks, iters, out)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        lib.sd_mfma_loop(blocks, iters, out)
    ev[1].record()
    torch.cuda.synchronize()
    s = ev[0].elapsed_time(ev[1]) / reps / 1e3
    tflops = blocks * 16 * iters * 32768 / s / 1e12
    return dict(kernel="mfma_loop", instruction="v_mfma_f32_32x32x16_bf16", blocks=blocks, iters=iters,
                us=s * 1e6, tflops=tflops, peak=2500.0, frac=tflops / 2500.0)


def library_gemms(reps=20):
    """The same products as plain library GEMMs (row-major, contiguous
    operands, output written), timed with events: what the vendor library
    reaches on these shapes.  The path's own kernels do more per launch (the
    logits kernels also round x to bf16 or accumulate ||x||^2, the mean
    kernels stream x and m^q and the verification sums)."""
    import torch
    out = {}
    for name, (m, k, n, dt, ours) in LIBRARY_GEMMS.items():
        dtype = torch.bfloat16 if dt == "bf16" else torch.float32
        g = torch.Generator(device="cuda").manual_seed(0)
        a = torch.randn(m, k, device="cuda", dtype=dtype, generator=g)
        b = torch.randn(k, n, device="cuda", dtype=dtype, generator=g)
        c = torch.empty(m, n, device="cuda", dtype=dtype)
        for _ in range(3):
            torch.mm(a, b, out=c)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(reps):
            torch.mm(a, b, out=c)
        ev[1].record()
        torch.cuda.synchronize()
        sec = ev[0].elapsed_time(ev[1]) / reps / 1e3
        peak = (BF16_PEAK_TFLOPS if dt == "bf16" else FP32_PEAK_TFLOPS) * 1e12
        out[name] = dict(m=m, k=k, n=n, dtype=dt, us=sec * 1e6, tflops=2 * m * k * n / sec / 1e12,
                         frac=2 * m * k * n / sec / peak,
                         path_kernel=None if ours is None else dict(workload=ours[0], kernel=ours[1]))
        del a, b, c
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="latent16384")
    ap.add_argument("--variants-workload", default="pixel3072",
                    help="workload of the variants field (the paper's R/D/B table, Frozen Drafter, plain EM)")
    ap.add_argument("--no-extra", action="store_true", help="skip the token and verification-only runs")
    ap.add_argument("--groups", dest="groups_req", type=int, default=0, choices=(0, 1, 2),
                    help="chain groups of the workload's sampler runs (0: the library's choice)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--calibrate-mfma", action="store_true",
                    help="only time the library's register-only bf16 matrix-instruction loop (the sustained "
                         "matrix-core rate beside the published peak) and exit")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of 1 GiB five times (the reference "
                         "kernel of known size for scaling the HBM byte counters) and exit")
    ap.add_argument("--library-gemms", action="store_true",
                    help="only time the workloads' denoiser GEMM shapes through the vendor library "
                         "(torch.mm) and exit")
    ap.add_argument("--verify-only", action="store_true",
                    help="only run the verification-only workload (verify12288: sd_verify_block + "
                         "sd_sample_residual) and exit")
    ap.add_argument("--variants", action="store_true",
                    help="only run the variants (reflection / decomposition / block at three "
                         "temperatures, the Frozen Drafter, the plain EM chain) on --workload and exit")
    args = ap.parse_args()
    if args.library_gemms:
        print(json.dumps(dict(library_gemms=library_gemms())))
        return
    if args.verify_only:
        import torch
        from paper_2606_13426_amd import _lib as lib
        lib.load()
        assert torch.cuda.is_available(), "bench.py needs a GPU"
        print(json.dumps(dict(verify_only=verify_bench(lib, args.steps, args.warmup))))
        return
    if args.variants:
        import torch
        from paper_2606_13426_amd import _lib as lib
        lib.load()
        # torch initialises the device before the library's first HIP call
        assert torch.cuda.is_available(), "bench.py needs a GPU"
        print(json.dumps(dict(workload=args.variants_workload,
                              variants=variants_bench(lib, args.variants_workload, args.steps))))
        return
    if args.calibrate_mfma:
        import torch
        from paper_2606_13426_amd import _lib as lib
        lib.load()
        assert torch.cuda.is_available(), "bench.py needs a GPU"
        print(json.dumps(dict(mfma_calibration=mfma_calibration(lib))))
        return
    if args.calibrate_copy:
        # also the achievable streaming rates of this machine: a read-plus-write
        # copy and a write-only fill of 1 GiB, timed with events (after a warm-up)
        import torch
        n = (1 << 30) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(6):
            dst.copy_(src)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record()
        for _ in range(10):
            dst.copy_(src)
        ev[1].record()
        for _ in range(10):
            dst.fill_(2.0)
        ev[2].record()
        torch.cuda.synchronize()
        copy_s = ev[0].elapsed_time(ev[1]) / 10 / 1e3
        fill_s = ev[1].elapsed_time(ev[2]) / 10 / 1e3
        print(json.dumps(dict(calibrate_copy_bytes_read=4 * n, calibrate_copy_bytes_written=4 * n,
                              copies=6, copy_us=copy_s * 1e6, copy_read_plus_write_GBs=8 * n / copy_s / 1e9,
                              fill_us=fill_s * 1e6, fill_write_GBs=4 * n / fill_s / 1e9)))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): chains are independent and "
              "would shard across GPUs without communication, but multi-GPU runs are not implemented",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_13426_amd import _lib as lib
    lib.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    res = run_sampler_bench(lib, args.workload, lib.SD_BLOCK, args.steps, args.warmup, profile=True,
                            groups_req=args.groups_req)
    roof, table = roofline_of(res, args.steps)
    if roof:
        roof["traffic"] = measured_traffic(args.workload, roof["kernel"])
        roof["chain_groups"] = res["profile_groups"]
    line = dict(metric=METRIC, value=res["B"] * res["N"] / res["sec"], unit="chain-steps/s", n_gpus=1,
                steps=args.steps, warmup=args.warmup, ms_per_step=1e3 * res["sec"], higher_is_better=True,
                scaling="weak", vs_baseline=None, dtype=_dtype(args.workload), data="synthetic",
                config=dict(workload=args.workload, d=res["d"], M=res["M"], B=res["B"], K=res["K"],
                            N=res["N"], verification="block", drafter="free", usample="exact",
                            chain_groups=res["groups"], parallelism="single-gpu"),
                precision=_precision(args.workload),
                mean_accepted_steps_per_block=res["be"], mean_tau=res["mean_tau"], ties=res["ties"],
                rounds_per_run=res["rounds"], roofline=roof, kernels=table)
    if not args.no_extra:
        # the other sampler workloads, each run end to end (not the headline
        # value); the pixel-sized one with block and token verification
        others = {}
        for wl in ("pixel3072", "pixel12288", "latent16384"):
            if wl == args.workload:
                continue
            r2 = run_sampler_bench(lib, wl, lib.SD_BLOCK, max(3, args.steps // 2), 1, profile=True)
            roof2, table2 = roofline_of(r2, max(3, args.steps // 2))
            if roof2:
                roof2["traffic"] = measured_traffic(wl, roof2["kernel"])
                roof2["chain_groups"] = r2["profile_groups"]
            others[wl] = dict(value=r2["B"] * r2["N"] / r2["sec"], unit="chain-steps/s",
                              ms_per_step=1e3 * r2["sec"], dtype=_dtype(wl),
                              mean_accepted_steps_per_block=r2["be"], rounds_per_run=r2["rounds"],
                              ties=r2["ties"],
                              config=dict(d=r2["d"], M=r2["M"], B=r2["B"], K=r2["K"], N=r2["N"],
                                          chain_groups=r2["groups"]),
                              roofline=roof2, denoiser_gemms=table2.get("denoiser_gemms"),
                              kernels={k: dict(avg_us=v["avg_us"], bound=v.get("bound"), frac=v.get("frac"))
                                       for k, v in table2.items() if "avg_us" in v})
            if wl == "pixel3072":
                tok = run_sampler_bench(lib, wl, lib.SD_TOKEN, max(2, args.steps // 2), 1, profile=False)
                others[wl]["token"] = dict(value=tok["B"] * tok["N"] / tok["sec"], ms_per_step=1e3 * tok["sec"],
                                           mean_accepted_steps_per_block=tok["be"],
                                           rounds_per_run=tok["rounds"])
        line["other_workloads"] = others
        line["verify_only"] = verify_bench(lib, args.steps, args.warmup)
        line["mfma_calibration"] = mfma_calibration(lib)
        line["library_gemms"] = library_gemms()
        line["variants"] = dict(workload=args.variants_workload,
                                **variants_bench(lib, args.variants_workload, args.steps))
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_budget)
    print(json.dumps(line))


if __name__ == "__main__":
    main()
