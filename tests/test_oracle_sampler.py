"""Pins of the oracle's full sampler (Alg. 8 with the Free Drafter) (no GPU).

* the final state of speculative sampling (block and token verification)
  follows the law of the plain Euler-Maruyama chain (two-sample KS, d = 1, 2);
* block verification advances at least as many steps per round as token;
* in the first round the Free Drafter's first draft mean equals the target
  mean, so Delta_1 = 0 and the first draft is always accepted;
* every chain ends exactly at step N; same seed, same result.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import sampler as S
from oracle.gmm import GMM
from oracle.schedule import Schedule


def _gmm(d, seed):
    rng = np.random.default_rng(seed)
    M = 3
    return GMM(rng.standard_normal((M, d)) * 2.0, rng.uniform(0.05, 0.5, M),
               np.log(rng.dirichlet(np.ones(M))))


@pytest.mark.parametrize("mode,d,K,N", [(S.BLOCK, 1, 3, 12), (S.TOKEN, 1, 3, 12), (S.BLOCK, 2, 4, 10)])
def test_final_law_matches_plain_em(mode, d, K, N):
    g = _gmm(d, 1)
    sch = Schedule(N)
    B = 900
    spec = S.run_sampler(g, sch, B, K, seed=11, mode=mode)["y"]
    em = S.run_plain_em(g, sch, B, seed=12)
    for i in range(d):
        assert stats.ks_2samp(spec[:, i], em[:, i]).pvalue > 1e-3


def test_block_efficiency_block_vs_token():
    g = _gmm(1, 2)
    sch = Schedule(20)
    rb = S.run_sampler(g, sch, 200, 4, seed=3, mode=S.BLOCK)
    rt = S.run_sampler(g, sch, 200, 4, seed=3, mode=S.TOKEN)
    be_b, be_t = S.block_efficiency(rb["trace"]), S.block_efficiency(rt["trace"])
    assert 1.0 <= be_t <= 5.0 and 1.0 <= be_b <= 5.0
    assert be_b >= be_t - 0.05


@pytest.mark.parametrize("mode", [S.BLOCK, S.TOKEN])
def test_first_round_accepts_first_draft_and_accounting(mode):
    g = _gmm(2, 4)
    sch = Schedule(15)
    res = S.run_sampler(g, sch, 40, 4, seed=5, mode=mode, keep_trace=True)
    for rec in res["trace"]:
        first = rec[0]
        assert first["nrm2"][0] == 0.0          # m^p_0 = m^q_0 exactly
        assert first["tau"] >= 2
        assert sum(info["steps"] for info in rec) == sch.n_steps
        ks = [info["k"] for info in rec]
        assert ks == sorted(ks) and ks[0] == 0
        for info in rec:
            assert 1 <= info["tau"] <= info["kb"] + 1


def test_deterministic():
    g = _gmm(2, 6)
    sch = Schedule(10)
    a = S.run_sampler(g, sch, 8, 3, seed=9)
    b = S.run_sampler(g, sch, 8, 3, seed=9)
    assert np.array_equal(a["y"], b["y"])
    c = S.run_sampler(g, sch, 8, 3, seed=10)
    assert not np.array_equal(a["y"], c["y"])
