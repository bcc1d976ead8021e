"""Generator mixture of each neighbourhood and the (1+1)-ES on its weights
(Section 3, step 4; mixture mutation scale from the experiment settings table).

The paper scores a mixture with FID, which needs a pretrained feature network
that is not available.  Reading used here: the same Frechet form on a fixed
random feature map with diagonal covariances,
    score(w) = ||mu_w - mu_r||^2 + ||sigma_w - sigma_r||^2,
features f = x P with P [x_dim, F] ~ N(0, 1/x_dim) (Philox tag PROJ),
mu_r, sigma_r the per-feature mean and standard deviation over the whole
dataset, and for the mixture of generators G_k with weights w_k evaluated on
a shared latent set zeta (S samples, tag MIXZ):
    mu_w = sum_k w_k mean(f_k),  sigma_w^2 = sum_k w_k mean(f_k^2) - mu_w^2.
This is the 2-Wasserstein distance between diagonal Gaussians with the first
two moments of the mixture and of the data.

ES step per cell: w' = max(w + sigma n, 0) / sum, n ~ N(0, I_5) (tag MIXN);
rejected if the sum is 0; accepted iff score(w') < score(w).
"""
import numpy as np

from . import rng


def projection(S):
    F = S.wl["mix_feat_dim"]
    return rng.normals(S.seed, S.xd * F, 0, 0, 0, "PROJ").reshape(S.xd, F) / np.sqrt(S.xd)


def real_stats(S, data):
    """Per-feature mean and (biased) standard deviation of the projected dataset."""
    P = projection(S)
    f = np.asarray(data, dtype=np.float64) @ P
    mu = f.mean(axis=0)
    sd = np.sqrt(((f - mu) ** 2).mean(axis=0))
    return dict(P=P, mu_r=mu, sd_r=sd)


def generator_moments(S, st, P, gen):
    """mean(f) and mean(f^2) per cell's generator on the shared latents of this generation."""
    Sm = S.wl["mix_samples"]
    zeta = rng.normals(S.seed, Sm * S.zd, 0, gen, 0, "MIXZ").reshape(Sm, S.zd)
    mu = np.zeros((S.C, P.shape[1]))
    s2 = np.zeros((S.C, P.shape[1]))
    for k in range(S.C):
        out = S.Gnet.forward(st.Gp[k], zeta)[1]
        f = out @ P
        mu[k] = f.mean(axis=0)
        s2[k] = (f * f).mean(axis=0)
    return mu, s2


def score(w, mus, s2s, mu_r, sd_r):
    mu_w = w @ mus
    var_w = np.maximum(w @ s2s - mu_w * mu_w, 0.0)
    return float(((mu_w - mu_r) ** 2).sum() + ((np.sqrt(var_w) - sd_r) ** 2).sum())


def propose(S, w, cell, gen):
    """w' = max(w + sigma n, 0) / sum, or None when every weight is clipped to 0."""
    n = rng.normals(S.seed, 5, cell, gen, 0, "MIXN")
    wp = np.maximum(w + S.wl["mix_sigma"] * n, 0.0)
    tot = wp.sum()
    if not tot > 0.0:
        return None
    return wp / tot


def update(S, st, stats, gen):
    """One ES step for every cell; returns (w[C,5], score[C] of the kept w, accepted[C])."""
    mu, s2 = generator_moments(S, st, stats["P"], gen)
    w_new = np.array(st.w, copy=True)
    sc = np.zeros(S.C)
    acc = np.zeros(S.C, dtype=np.int64)
    for c in range(S.C):
        ks = S.nbr[c]
        cur = score(st.w[c], mu[ks], s2[ks], stats["mu_r"], stats["sd_r"])
        wp = propose(S, st.w[c], c, gen)
        if wp is not None:
            new = score(wp, mu[ks], s2[ks], stats["mu_r"], stats["sd_r"])
            if new < cur:
                w_new[c], cur, acc[c] = wp, new, 1
        sc[c] = cur
    return w_new, sc, acc
