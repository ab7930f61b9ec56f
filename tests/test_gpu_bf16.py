"""bf16 denoiser path (SD_BF16): the target call against the float64 oracle
(the sampler's fused bf16 round is checked stage-wise in
test_gpu_round_parity.py).

Tolerances.  The stated bar for the bf16 GEMM path is a per-row relative L2
error of m^q of at most 2e-2 against the float64 oracle.  m^q = c1 x + c2 s is
dominated by c1 x, so the score s is also compared, per row, with a model of
the specified arithmetic (bf16-rounded operands of both products, float64
elsewhere; tests/helpers.py, pinned on the CPU): what remains is float32
accumulation and the occasional bf16 rounding of a weight P_m that lands on
the other side of a rounding boundary, held to 2e-3 relative L2.  Decisions in
bf16 are checked stage-wise: the oracle is fed the GPU's own m^q, never
compared against a float64 end-to-end run.
"""
import numpy as np
import pytest
import torch

from helpers import rel_l2_rows, target_mean_bf16_operands
from oracle.gmm import GMM, target_mean
from oracle.schedule import Schedule
from paper_2606_13426_amd import _lib
from paper_2606_13426_amd.inputs import make_gmm, workload_gmm

pytestmark = pytest.mark.gpu
DEV = "cuda"
MQ_REL_L2 = 2e-2
SCORE_VS_MODEL = 2e-3


def _check_bf16_rows(p, x, step, N, mq, sc):
    g = GMM(p["mu"], p["var"], p["log_w"])
    sch = Schedule(N)
    x64 = np.asarray(x, np.float64)
    ref_mq, _ = target_mean(g, sch, x64, step)
    e_mq = rel_l2_rows(mq, ref_mq)
    assert e_mq.max() <= MQ_REL_L2, f"m^q per-row relative L2 {e_mq.max():.3e} (row {e_mq.argmax()})"
    _, model_sc = target_mean_bf16_operands(g, sch, x64, step)
    e_sc = rel_l2_rows(sc, model_sc)
    assert e_sc.max() <= SCORE_VS_MODEL, f"score vs bf16 model {e_sc.max():.3e} (row {e_sc.argmax()})"
    return float(e_mq.max()), float(e_sc.max())


def _rows_near_data(p, rows, N, seed):
    rng = np.random.default_rng(seed)
    M, d = p["mu"].shape
    step = rng.integers(0, N, rows).astype(np.int32)
    a = Schedule(N).signal(step)
    comp = rng.integers(0, M, rows)
    x = (a[:, None] * p["mu"][comp]
         + np.sqrt(1 - a[:, None] ** 2 + a[:, None] ** 2 * p["var"][comp][:, None])
         * rng.standard_normal((rows, d)))
    x[::7] = rng.standard_normal((len(x[::7]), d))
    return x.astype(np.float32), step


@pytest.mark.parametrize("d,M,rows,N", [(33, 5, 70, 60), (300, 70, 257, 100), (3072, 64, 200, 200),
                                        (1024, 256, 130, 500), (256, 320, 90, 80), (512, 512, 131, 100)])
def test_bf16_target_mean_matches_oracle(d, M, rows, N):
    p = make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=d + M)
    x, step = _rows_near_data(p, rows, N, seed=rows)
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"], precision=_lib.SD_BF16)
    xt = torch.tensor(x, device=DEV)
    mq = torch.empty_like(xt)
    sc = torch.empty_like(xt)
    _lib.sd_target_mean(tgt, xt, torch.tensor(step, device=DEV), mq, sc)
    _check_bf16_rows(p, x, step, N, mq.cpu().numpy(), sc.cpu().numpy())


def test_bf16_target_mean_strided_rows():
    # row strides above d (views into wider buffers) on the unvectorised path
    d, M, rows, N = 130, 24, 90, 80
    p = make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=3)
    x, step = _rows_near_data(p, rows, N, seed=4)
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"], precision=_lib.SD_BF16)
    xw = torch.zeros(rows, d + 3, device=DEV)
    xw[:, :d] = torch.tensor(x, device=DEV)
    mqw = torch.full((rows, d + 5), 7.0, device=DEV)
    scw = torch.full((rows, d + 1), 7.0, device=DEV)
    _lib.sd_target_mean(tgt, xw[:, :d], torch.tensor(step, device=DEV), mqw[:, :d], scw[:, :d])
    assert torch.all(mqw[:, d:] == 7.0) and torch.all(scw[:, d:] == 7.0)
    _check_bf16_rows(p, x, step, N, mqw[:, :d].cpu().numpy(), scw[:, :d].cpu().numpy())


@pytest.mark.parametrize("name", ["pixel12288", "latent16384"])
def test_bf16_full_round_rows_sampled(name):
    # one full round's rows, B (K+1), at the workload's size; sampled rows checked
    p = workload_gmm(name)
    w = _lib_workload(name)
    N, R, d = w["N"], w["B"] * (w["K"] + 1), w["d"]
    x, step = _rows_near_data(p, R, N, seed=11)
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"], precision=_lib.SD_BF16)
    xt = torch.tensor(x, device=DEV)
    mq = torch.empty_like(xt)
    sc = torch.empty_like(xt)
    _lib.sd_target_mean(tgt, xt, torch.tensor(step, device=DEV), mq, sc)
    rows = np.sort(np.random.default_rng(1).choice(R, 24, replace=False))
    _check_bf16_rows(p, x[rows], step[rows], N, mq[rows].cpu().numpy(), sc[rows].cpu().numpy())


def _lib_workload(name):
    from paper_2606_13426_amd.inputs import WORKLOADS
    return WORKLOADS[name]


def test_bf16_sampler_deterministic_and_close_to_fp32_efficiency():
    d, M, N, B, K, seed = 512, 32, 60, 64, 6, 5
    p = make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=2)
    sched = _lib.schedule(N)
    t16 = _lib.Target(sched, p["mu"], p["var"], p["log_w"], precision=_lib.SD_BF16)
    t32 = _lib.Target(sched, p["mu"], p["var"], p["log_w"])
    y1, s1, _ = _lib.sd_run_sampler(t16, B, K, seed)
    y2, s2, _ = _lib.sd_run_sampler(t16, B, K, seed)
    assert torch.equal(y1, y2) and s1["rounds"] == s2["rounds"]
    assert torch.isfinite(y1).all()
    _, s32, _ = _lib.sd_run_sampler(t32, B, K, seed)
    be16 = s1["steps"] / s1["chain_rounds"]
    be32 = s32["steps"] / s32["chain_rounds"]
    assert abs(be16 - be32) <= 0.1 * be32, (be16, be32)


def test_bf16_sampler_variants_deterministic_and_close_to_fp32():
    """The variants on a bf16 target: deterministic, every chain reaches N, the
    Frozen Drafter accepts its first draft every round, and the block
    efficiency stays within 10 % of the float32 target's."""
    d, M, N, B, K, seed = 512, 32, 60, 64, 6, 8
    p = make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=4)
    sched = _lib.schedule(N)
    t16 = _lib.Target(sched, p["mu"], p["var"], p["log_w"], precision=_lib.SD_BF16)
    t32 = _lib.Target(sched, p["mu"], p["var"], p["log_w"])
    for kw in (dict(drafter=_lib.SD_DRAFTER_FROZEN),
               dict(mode=_lib.SD_TOKEN, residual=_lib.SD_RESIDUAL_REFLECTION),
               dict(omega=2.0)):
        y1, s1, tr = _lib.sd_run_sampler_ex(t16, B, K, seed, trace_rounds=N, **kw)
        y2, s2, _ = _lib.sd_run_sampler_ex(t16, B, K, seed, **kw)
        assert torch.equal(y1, y2) and s1["rounds"] == s2["rounds"], kw
        assert torch.isfinite(y1).all() and s1["steps"] == B * N, kw
        if kw.get("drafter") == _lib.SD_DRAFTER_FROZEN:
            t = tr.cpu().numpy()
            assert np.all(t[t > 0] >= 2)
        _, s32, _ = _lib.sd_run_sampler_ex(t32, B, K, seed, **kw)
        be16 = s1["steps"] / s1["chain_rounds"]
        be32 = s32["steps"] / s32["chain_rounds"]
        assert abs(be16 - be32) <= 0.1 * be32, (kw, be16, be32)
