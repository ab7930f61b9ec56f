"""Pins of the oracle's full sampler (Alg. 8 with the Free Drafter) (no GPU).

* the final state of speculative sampling (block and token verification)
  follows the law of the plain Euler-Maruyama chain (two-sample KS, d = 1, 2);
* block verification advances at least as many steps per round as token;
* in the first round the Free Drafter's first draft mean equals the target
  mean, so Delta_1 = 0 and the first draft is always accepted;
* every chain ends exactly at step N; same seed, same result;
* the Free Drafter's cached score is the target score at the rejected draft
  (or at the last draft after a full accept), at that draft's time.
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


def _fd_score(g, x, a, h=1e-5):
    """Central differences of log q_s at one point: the score without the oracle's score code."""
    d = x.shape[0]
    out = np.empty(d)
    for i in range(d):
        e = np.zeros(d)
        e[i] = h
        out[i] = (g.log_density((x + e)[None], a)[0] - g.log_density((x - e)[None], a)[0]) / (2 * h)
    return out


def test_free_drafter_cache_is_score_at_rejected_or_last_draft():
    """Sec. 3.3: the next round drafts with the target score the round already
    computed at the rejected draft yhat_{k+tau}, time t_{k+tau} (tau <= K_b), or
    after a full accept at the last draft yhat_{k+K_b}, time t_{k+K_b}.

    The score the next round actually used is read back from its first draft
    mean, S_c = (m^p_0 - c1_k' Y_k') / c2_k', and compared with finite
    differences of log q at the expected row and time; the neighbouring rows
    and the neighbouring time do not match it."""
    g = _gmm(2, 7)
    sch = Schedule(40)
    K = 4
    res = S.run_sampler(g, sch, 60, K, seed=13, keep_trace=True)
    rej = full = distinct = compared = 0
    for rec in res["trace"]:
        for cur, nxt in zip(rec[:-1], rec[1:]):
            k1 = nxt["k"]
            used = (nxt["mp"][0] - sch.c1(k1) * nxt["yh"][0]) / sch.c2(k1)
            c = min(cur["tau"], cur["kb"])
            n = cur["k"] + c
            assert k1 == min(cur["k"] + cur["tau"], sch.n_steps)
            want = _fd_score(g, cur["yh"][c], sch.signal(n))
            assert np.allclose(used, want, rtol=1e-6, atol=1e-6), (cur["k"], cur["tau"], used, want)
            alts = [_fd_score(g, cur["yh"][c], sch.signal(n - 1))]
            alts += [_fd_score(g, cur["yh"][j], sch.signal(cur["k"] + j))
                     for j in (c - 1, c + 1) if 0 <= j <= cur["kb"]]
            compared += 1
            distinct += all(np.max(np.abs(alt - used)) > 1e-4 for alt in alts)
            if cur["tau"] <= cur["kb"]:
                rej += 1
            else:
                full += 1
    assert rej >= 20 and full >= 20, (rej, full)
    assert distinct >= 0.95 * compared, (distinct, compared)
