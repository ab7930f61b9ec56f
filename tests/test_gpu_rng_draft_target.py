"""GPU parity of the Philox stream, the Free-Drafter block and the mixture target.

Philox words must be bit-exact; float32 normals, drafts, draft means, target
means and scores must match the float64 oracle within 1e-4 of max(|ref|,
rms(row)).  Sizes are chosen to span several tiles and ragged tails.
"""
import numpy as np
import pytest
import torch

from helpers import assert_rows_close, row_scale
from oracle import philox
from oracle import sampler as osamp
from oracle.gmm import GMM, target_mean
from oracle.schedule import Schedule
from paper_2606_13426_amd import _lib
from paper_2606_13426_amd.inputs import make_gmm, workload_gmm

pytestmark = pytest.mark.gpu
DEV = "cuda"


def test_philox_words_bit_exact():
    rng = np.random.default_rng(0)
    n = 5000
    ctr = rng.integers(0, 2 ** 32, size=(n, 4), dtype=np.uint64)
    ctr[:3] = [[0, 0, 0, 0], [0xFFFFFFFF] * 4, [0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344]]
    for seed in (0, 0xFFFFFFFFFFFFFFFF, 0x299F31D0A4093822, 12345):
        c = torch.tensor(ctr.astype(np.uint32).view(np.int32), device=DEV)
        out = torch.empty_like(c)
        _lib.sd_philox_words(seed, c, out)
        got = out.cpu().numpy().view(np.uint32).astype(np.uint64)
        ref = philox.philox4x32_10(ctr, philox.seed_key(seed))
        assert np.array_equal(got, ref)


@pytest.mark.parametrize("d", [1, 7, 4096])
def test_philox_normals(d):
    out = torch.empty(d, dtype=torch.float32, device=DEV)
    _lib.sd_philox_normals(99, 5, 17, philox.TAG_DRAFT, 3, out)
    ref = philox.normal_vector(99, 5, 17, philox.TAG_DRAFT, 3, d)
    err = np.abs(out.cpu().numpy() - ref) / np.maximum(1.0, np.abs(ref))
    assert err.max() < 2e-6


def test_init_chains_matches_oracle():
    B, d = 5, 37
    y = torch.empty(B, d, dtype=torch.float32, device=DEV)
    _lib.sd_init_chains(y, 42)
    ref = np.stack([philox.normal_vector(42, b, 0, philox.TAG_INIT, 0, d) for b in range(B)])
    assert np.abs(y.cpu().numpy() - ref).max() < 1e-5


@pytest.mark.parametrize("d", [70, 256])
def test_draft_block_matches_oracle(d):
    N, K, seed = 50, 6, 3
    ks = [0, 10, 44, 46, 49, 50, 13, 0]
    B = len(ks)
    sch = Schedule(N)
    rng = np.random.default_rng(d)
    y = rng.standard_normal((B, d)).astype(np.float32)
    cs = (3.0 * rng.standard_normal((B, d))).astype(np.float32)
    rnd = rng.integers(0, 1000, B).astype(np.int32)
    x = torch.full((B, K + 1, d), 7.0, device=DEV)
    mp = torch.full((B, K, d), 7.0, device=DEV)
    _lib.sd_draft_block(_lib.schedule(N), torch.tensor(y, device=DEV), torch.tensor(cs, device=DEV),
                        torch.tensor(ks, dtype=torch.int32, device=DEV), torch.tensor(rnd, device=DEV),
                        seed, x, mp)
    xg, mg = x.cpu().numpy(), mp.cpu().numpy()
    for b, k in enumerate(ks):
        if k >= N:
            assert np.all(xg[b] == 7.0) and np.all(mg[b] == 7.0)
            continue
        kb = min(K, N - k)
        yh, mpr = osamp.draft_chain(y[b].astype(np.float64), cs[b].astype(np.float64), k, kb, sch, seed, b,
                                    int(rnd[b]))
        assert_rows_close(xg[b, : kb + 1], yh, what=f"draft rows chain {b}")
        assert_rows_close(mg[b, :kb], mpr, what=f"draft means chain {b}")
        for i in range(kb + 1, K + 1):
            assert np.array_equal(xg[b, i], xg[b, kb])


def _target_case(d, M, rows, seed, mu_std=1.0, var=(0.01, 0.2)):
    p = make_gmm(d, M, mu_std=mu_std, var=var, dirichlet=1.0, seed=seed)
    return p


# the last two: 256 < M <= 512, two rows per softmax workgroup, each over two
# wavefronts (M = 320 leaves lanes past M)
@pytest.mark.parametrize("d,M,rows,N", [(2, 4, 300, 100), (33, 5, 70, 60), (130, 70, 129, 200),
                                        (3072, 64, 200, 200), (300, 320, 150, 100), (512, 512, 130, 100)])
def test_target_mean_matches_oracle(d, M, rows, N):
    p = _target_case(d, M, rows, seed=d + M)
    rng = np.random.default_rng(rows)
    step = rng.integers(0, N, rows).astype(np.int32)
    sch = Schedule(N)
    a = sch.signal(step)
    comp = rng.integers(0, M, rows)
    # rows near the data law at their own noise level, plus pure-noise rows
    x = (a[:, None] * p["mu"][comp] + np.sqrt(1 - a[:, None] ** 2 + a[:, None] ** 2 * p["var"][comp][:, None])
         * rng.standard_normal((rows, d)))
    x[::7] = rng.standard_normal((len(x[::7]), d))
    x = x.astype(np.float32)
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"])
    xt = torch.tensor(x, device=DEV)
    mq = torch.empty_like(xt)
    sc = torch.empty_like(xt)
    _lib.sd_target_mean(tgt, xt, torch.tensor(step, device=DEV), mq, sc)
    g = GMM(p["mu"], p["var"], p["log_w"])
    ref_mq, ref_sc = target_mean(g, sch, x.astype(np.float64), step)
    assert_rows_close(mq.cpu().numpy(), ref_mq, what="m^q")
    # the score sum_m r_m (a mu_m - x)/s2_m is formed as O - rho x from two
    # float32 products whose terms can be much larger than their difference
    # (x near a component with small s2): its float32 error is bounded by a
    # few rounding units of the terms' size, T = sum_m r_m a |mu_m| / s2_m +
    # |x| sum_m r_m / s2_m, on top of the 1e-4 relative bar
    a64 = a[:, None]
    s2 = a64 ** 2 * g.var[None, :] + 1 - a64 ** 2
    w = g.responsibilities(x.astype(np.float64), a) / s2
    T = (w * a64) @ np.abs(g.mu) + np.abs(x) * w.sum(1)[:, None]
    err = np.abs(sc.cpu().numpy() - ref_sc)
    bound = 1e-4 * row_scale(ref_sc) + 16 * M * 2.0 ** -24 * T
    assert np.all(err <= bound), f"score: worst error / bound {float((err / bound).max()):.3f}"


def test_target_mean_full_round_rows_sampled():
    # the row count of one pixel3072 round, B (K+1) = 9216 rows, as the sampler launches it
    p = workload_gmm("pixel3072")
    N, R, d = 200, 1024 * 9, 3072
    gen = torch.Generator(device=DEV)
    gen.manual_seed(5)
    x = torch.randn(R, d, generator=gen, device=DEV)
    step = torch.randint(0, N, (R,), generator=gen, device=DEV).to(torch.int32)
    tgt = _lib.Target(_lib.schedule(N), p["mu"], p["var"], p["log_w"])
    mq = torch.empty_like(x)
    _lib.sd_target_mean(tgt, x, step, mq)
    rows = np.random.default_rng(0).choice(R, 48, replace=False)
    g = GMM(p["mu"], p["var"], p["log_w"])
    xs = x[rows].cpu().numpy().astype(np.float64)
    ref, _ = target_mean(g, Schedule(N), xs, step[rows].cpu().numpy())
    assert_rows_close(mq[rows].cpu().numpy(), ref, what="m^q sampled rows")
