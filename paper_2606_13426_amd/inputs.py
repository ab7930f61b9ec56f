"""Seeded synthetic workloads for the speculative-diffusion verification pass.

This module only draws random arrays (NumPy's PCG64 for the mixture targets,
torch generators for the large verification-only tensors).  It holds none of
the method's arithmetic; quantities that the method defines (the per-step
sigma of the Euler-Maruyama kernel) are passed in by the caller.  It is the one
piece of code that both the HIP path and the CPU oracle consume, so that both
see bit-identical inputs.

Workloads (the paper's image datasets and trained U-Nets are not available;
a closed-form Gaussian-mixture data law stands in for them, with the
dimensions of its pixel- and latent-space experiments):
  tiny2d       d = 2,      M = 4,    mu ~ N(0, 4I), var ~ U[.05, .5], w ~ Dir(1);
               N = 100 steps, B = 256 chains, K = 4 drafts
  pixel3072    d = 3*32*32, M = 64,   mu ~ N(0, I), var ~ U[.01, .2], w ~ Dir(1);
               N = 200, B = 1024, K = 8          (CIFAR10-sized)
  pixel12288   d = 3*64*64, M = 256,  as above;  N = 500, B = 512, K = 16
  verify12288  verification only: B = 4096, K = 32, d = 12288, N = 1000,
               m^q = m^p + 0.05 N(0, I), drafts drawn from the draft kernels
  latent16384  d = 4*64*64, M = 1024, mu ~ N(0, I), var ~ U[.01, .1], w ~ Dir(.5);
               N = 1000, B = 256, K = 8
"""
import numpy as np

WORKLOADS = {
    "tiny2d": dict(d=2, M=4, mu_std=2.0, var=(0.05, 0.5), dirichlet=1.0,
                   N=100, B=256, K=4, precision="fp32"),
    "pixel3072": dict(d=3072, M=64, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0,
                      N=200, B=1024, K=8, precision="fp32"),
    "pixel12288": dict(d=12288, M=256, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0,
                       N=500, B=512, K=16, precision="bf16"),
    "verify12288": dict(d=12288, B=4096, K=32, N=1000, perturb=0.05),
    "latent16384": dict(d=16384, M=1024, mu_std=1.0, var=(0.01, 0.1), dirichlet=0.5,
                        N=1000, B=256, K=8, precision="bf16"),
}


def make_gmm(d, M, mu_std=1.0, var=(0.01, 0.2), dirichlet=1.0, seed=0):
    """Mixture parameters as float32 arrays: mu [M, d], var [M], log_w [M]."""
    rng = np.random.default_rng(seed)
    mu = (rng.standard_normal((M, d)) * mu_std).astype(np.float32)
    v = rng.uniform(var[0], var[1], size=M).astype(np.float32)
    w = rng.dirichlet(np.full(M, float(dirichlet)))
    log_w = np.log(np.maximum(w, 1e-300)).astype(np.float32)
    return dict(mu=mu, var=v, log_w=log_w)


def workload_gmm(name, seed=None):
    cfg = WORKLOADS[name]
    if seed is None:
        seed = sorted(WORKLOADS).index(name) + 1
    return make_gmm(cfg["d"], cfg["M"], cfg["mu_std"], cfg["var"], cfg["dirichlet"], seed)


def verify_inputs(B, K, d, N, sigma_table, seed, device="cpu", perturb=0.05,
                  scaled=False):
    """Inputs of one verification pass, laid out [B][rows][d] float32.

    sigma_table: float64 array of sigma_n for n = 0..N (supplied by the caller).
    Each chain starts at a step k_b ~ U{0..N-K}; m^p rows ~ N(0, I);
    m^q = m^p + perturb * N(0, I) (K+1 rows, the last one for a full accept);
    drafts yhat_j = m^p_{j-1} + sigma_{k_b+j-1} xi.  With scaled=True the
    perturbation is sigma/sqrt(d) per row, so ||Delta|| is of order one and
    every acceptance path is exercised.
    Returns dict of torch tensors: y_draft [B,K,d], mp [B,K,d], mq [B,K+1,d],
    sigma [B,K+1] float64, k0 [B] int32, kb [B] int32, steps_left [B] int32,
    round [B] int32.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    k0 = torch.randint(0, N - K + 1, (B,), generator=g, device=device)
    sig_t = torch.as_tensor(np.asarray(sigma_table, dtype=np.float64), device=device)
    idx = k0[:, None] + torch.arange(K + 1, device=device)[None, :]
    sigma = sig_t[idx]
    mp = torch.randn(B, K, d, generator=g, device=device)
    extra = torch.randn(B, 1, d, generator=g, device=device)
    mq = torch.cat([mp, extra], dim=1)
    if scaled:
        scale = (sigma / np.sqrt(d)).to(torch.float32)[:, :, None]
        mq = mq + scale * torch.randn(B, K + 1, d, generator=g, device=device)
    else:
        mq = mq + perturb * torch.randn(B, K + 1, d, generator=g, device=device)
    xi = torch.randn(B, K, d, generator=g, device=device)
    y_draft = mp + sigma[:, :K, None].to(torch.float32) * xi
    del xi
    rnd = torch.randint(0, 1 << 20, (B,), generator=g, device=device).to(torch.int32)
    kb = torch.full((B,), K, dtype=torch.int32, device=device)
    steps_left = (N - k0).to(torch.int32)
    return dict(y_draft=y_draft.contiguous(), mp=mp.contiguous(), mq=mq.contiguous(),
                sigma=sigma.contiguous(), k0=k0.to(torch.int32), kb=kb,
                steps_left=steps_left, round=rnd)
