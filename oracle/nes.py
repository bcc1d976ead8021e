"""Gradient-free training of a cell's pair by Natural Evolution Strategies, in
fp64.  Test infrastructure: only the tests, the smoke check and the bench's
CPU baseline use it.

The paper lists, beside the gradient-based trainers, gradient-free trainers
for evolution strategies and Natural Evolution Strategies (Section 3,
"Implementation and Distribution"), and says the trainers differ in how they
update the weights and evaluate fitness.  It gives no more, so the reading
(workload trainer "nes") is the antithetic NES gradient estimate used with an
ordinary optimiser:

  for one role with parameters theta (P values), a training step s draws
    eps_k ~ N(0, I_P), k = 0 .. n-1: normal k P + e of stream
      (cell, gen, s + 1, NES_G / NES_D),
    F_k+ = loss(theta + sigma eps_k),  F_k- = loss(theta - sigma eps_k)
      on the step's minibatch,
    g = sum_k (F_k+ - F_k-) eps_k / (2 n sigma),
  and takes one Adam step of theta on g with the individual's own Adam state
  (then the critic clip of the Wasserstein loss).

As in the gradient trainer, a step is the discriminator first (its loss with
the generator's current samples), then the generator against the updated
discriminator, on the same latents; loss is the role's training loss
(coevo.pair_losses).  losses[c] = (L_D, L_G) at the unperturbed parameters,
before each update.
"""
import numpy as np

from . import coevo, rng


def nes_gradient(f, theta, eps, sigma):
    """Antithetic NES estimate of grad f at theta from the directions eps [n, P]."""
    n = eps.shape[0]
    fp = np.array([f(theta + sigma * eps[k]) for k in range(n)])
    fm = np.array([f(theta - sigma * eps[k]) for k in range(n)])
    return ((fp - fm)[:, None] * eps).sum(axis=0) / (2.0 * n * sigma)


def directions(S, role, cell, gen, step):
    n, P = S.wl["nes_pairs"], (S.PG if role == "G" else S.PD)
    return rng.normals(S.seed, n * P, cell, gen, step + 1, "NES_" + role).reshape(n, P)


def train_step(S, st, data, gen, step):
    """One NES step of every training unit's pair, in place; returns losses [U, 2]."""
    sigma = S.wl["nes_sigma"]
    losses = np.zeros((S.U, 2))
    for c in range(S.U):
        _, x, z = coevo.sample(S, data, c, gen, step + 1)
        xf = coevo.g_forward(S, st.Gp[c], z)[1]

        def loss_d(dp):
            return coevo.pair_losses(S, coevo.d_logits(S, dp, x)[1], coevo.d_logits(S, dp, xf)[1])[0]

        losses[c, 0] = loss_d(st.Dp[c])
        g = nes_gradient(loss_d, st.Dp[c], directions(S, "D", c, gen, step), sigma)
        st.Dt[c] = coevo.adam(S, st.Dp[c], st.Dm[c], st.Dv[c], st.Dt[c], st.Dlr[c], g)
        if S.loss == "wasserstein":
            np.clip(st.Dp[c], -S.clip, S.clip, out=st.Dp[c])

        def loss_g(gp):
            a = coevo.d_logits(S, st.Dp[c], coevo.g_forward(S, gp, z)[1])[1]
            return coevo.pair_losses(S, a, a)[1]

        losses[c, 1] = loss_g(st.Gp[c])
        g = nes_gradient(loss_g, st.Gp[c], directions(S, "G", c, gen, step), sigma)
        st.Gt[c] = coevo.adam(S, st.Gp[c], st.Gm[c], st.Gv[c], st.Gt[c], st.Glr[c], g)
    return losses
