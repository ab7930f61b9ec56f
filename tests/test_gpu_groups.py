"""Chain groups (sd_sampler_options.groups): the sampler with its chains split
into two halves whose rounds run on two streams at once gives the same run as
one sequence of kernels, bit for bit -- Y_N, every round's tau and the
statistics -- because every row is computed in the same order either way (the
target call of each half splits its logits GEMM as for all rows, and the
generator is keyed by the chain's index in the whole batch).

Cases: float32 and bf16 targets, the three sampler modes, K > N, an odd number
of chains, the chain-aligned bf16 mean tile (M >= 512) and the 128-row one,
both bf16 workloads at full size, a run split over calls that changes the
grouping between calls, and concurrent calls from several host threads on one
target.
"""
import threading

import pytest
import torch

from paper_2606_13426_amd import _lib
from paper_2606_13426_amd.inputs import WORKLOADS, make_gmm, workload_gmm

pytestmark = pytest.mark.gpu

FROZEN = dict(drafter=_lib.SD_DRAFTER_FROZEN)
TOKEN_R = dict(mode=_lib.SD_TOKEN, residual=_lib.SD_RESIDUAL_REFLECTION)

# (name or (d, M), B, K, N, precision, sampler options)
CASES = [
    ((5, 3), 7, 64, 40, None, {}),
    ((128, 64), 20, 4, 30, None, FROZEN),
    ((64, 320), 9, 3, 20, None, TOKEN_R),
    ((1024, 512), 72, 8, 60, _lib.SD_BF16, {}),
    ((1024, 512), 72, 8, 60, _lib.SD_BF16, FROZEN),
    ((512, 64), 33, 16, 50, _lib.SD_BF16, TOKEN_R),
    ("latent16384", None, None, None, _lib.SD_BF16, {}),
    ("pixel12288", None, None, None, _lib.SD_BF16, {}),
]


def _target(case):
    shape, B, K, N, prec, kw = case
    if isinstance(shape, str):
        cfg = WORKLOADS[shape]
        p = workload_gmm(shape)
        B, K, N = cfg["B"], cfg["K"], cfg["N"]
    else:
        d, M = shape
        p = make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=d + M)
    extra = {} if prec is None else dict(precision=prec)
    return _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"], **extra), B, K, N, kw


def _same(a, b):
    ya, sa, ta = a
    yb, sb, tb = b
    assert torch.equal(ya, yb), "Y_N differs"
    assert torch.equal(ta, tb), "tau trace differs"
    for key in ("rounds", "chain_rounds", "steps", "ties", "tau_hist", "finished", "mean_tau"):
        assert sa[key] == sb[key], key


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-{c[1]}-{c[2]}-{sorted(c[5].items())}")
def test_two_groups_equal_one(case):
    tgt, B, K, N, kw = _target(case)
    one = _lib.sd_run_sampler_ex(tgt, B, K, 11, trace_rounds=N, groups=1, **kw)
    two = _lib.sd_run_sampler_ex(tgt, B, K, 11, trace_rounds=N, groups=2, **kw)
    torch.cuda.synchronize()
    assert one[1]["finished"] and one[1]["steps"] == B * N
    assert one[1]["groups"] == 1 and two[1]["groups"] == 2
    _same(one, two)


def test_split_run_changing_groups_equals_one_call():
    tgt, B, K, N, kw = _target(((1024, 512), 72, 8, 60, _lib.SD_BF16, {}))
    one = _lib.sd_run_sampler_ex(tgt, B, K, 5, trace_rounds=N, groups=1)
    ws = torch.empty(_lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device="cuda")
    trace = torch.zeros(N, B, dtype=torch.int32, device="cuda")
    y = torch.full((B, tgt.d), float("nan"), device="cuda")
    r = 0
    for n, g in ((2, 2), (3, 1), (4, 2), (1, 0)):
        _, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, 5, ws=ws, trace=trace, y_out=y, start_round=r,
                                          max_rounds=n, groups=g)
        assert st["rounds"] == r + n and not st["finished"]
        r = st["rounds"]
    y, st, trace = _lib.sd_run_sampler_ex(tgt, B, K, 5, ws=ws, trace=trace, y_out=y, start_round=r,
                                          groups=2)
    torch.cuda.synchronize()
    _same(one, (y, st, trace))


def test_init_only_then_resume_with_two_groups():
    # max_rounds = 0 initialises the state only; the run resumed from it with
    # two groups equals one call with one group
    tgt, B, K, N, kw = _target(((128, 64), 20, 4, 30, None, {}))
    one = _lib.sd_run_sampler_ex(tgt, B, K, 7, trace_rounds=N, groups=1)
    ws = torch.empty(_lib.sd_sampler_workspace(tgt, B, K), dtype=torch.uint8, device="cuda")
    trace = torch.zeros(N, B, dtype=torch.int32, device="cuda")
    _, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, 7, ws=ws, trace=trace, max_rounds=0, groups=2)
    assert st["rounds"] == 0 and not st["finished"]
    two = _lib.sd_run_sampler_ex(tgt, B, K, 7, ws=ws, trace=trace, start_round=st["rounds"], groups=2)
    torch.cuda.synchronize()
    _same(one, two)


def test_library_choice_of_groups():
    # two groups from 2048 target rows per half (B/2 (K + 1)), else one
    p = make_gmm(64, 8, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=1)
    tgt = _lib.Target(_lib.schedule(6), p["mu"], p["var"], p["log_w"])
    for B, K, want in ((455, 8, 1), (456, 8, 2), (1, 8, 1)):
        _, st, _ = _lib.sd_run_sampler_ex(tgt, B, K, 0)
        assert st["groups"] == want, (B, K, st["groups"])


def test_concurrent_calls_on_one_target():
    # three host threads, each on its own stream, share one target (its flag
    # slots and second-group streams): each run equals the same run alone
    tgt, B, K, N, _ = _target(((512, 64), 40, 4, 40, None, {}))
    jobs = ((1, 2), (2, 1), (3, 2))
    ref = [_lib.sd_run_sampler_ex(tgt, B, K, seed, trace_rounds=N, groups=g) for seed, g in jobs]
    torch.cuda.synchronize()
    out, errors = [None] * len(jobs), []

    def work(i, seed, g):
        try:
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                out[i] = _lib.sd_run_sampler_ex(tgt, B, K, seed, trace_rounds=N, groups=g)
            stream.synchronize()
        except Exception as e:  # re-raised in the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i, seed, g)) for i, (seed, g) in enumerate(jobs)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not any(th.is_alive() for th in threads)
    if errors:
        raise errors[0]
    for a, b in zip(ref, out):
        _same(a, b)


def test_groups_out_of_range_rejected():
    tgt, B, K, N, _ = _target(((5, 3), 7, 4, 10, None, {}))
    with pytest.raises(_lib.SpecDiffError) as e:
        _lib.sd_run_sampler_ex(tgt, B, K, 0, groups=3)
    assert e.value.status == _lib.SD_EINVAL
