"""Gradient-free training of a cell's pair by a (1+lambda) evolution strategy,
in fp64.  Test infrastructure: only the tests, the smoke check and the
bench's CPU baseline use it.

The paper lists gradient-free trainers for evolution strategies beside those
for Natural Evolution Strategies and the gradient-based ones (Section 3,
"Implementation and Distribution"), and evolves the mixture weights with a
(1+1)-ES (Section 3, step 4).  It gives no more, so the reading (workload
trainer "es") is plus-selection on the network parameters with lambda = 2n
antithetic Gaussian mutants:

  for one role with parameters theta, training step s draws the n directions
  eps_k of the NES trainer (the same streams, nes.directions), scores on the
  step's minibatch the mutants
      q = 0 .. n-1:   theta + sigma eps_q
      q = n .. 2n-1:  theta - sigma eps_(q-n)
  and the parent (q = 2n, theta itself), and keeps the candidate of lowest
  loss.  The parent stays unless a mutant's loss is strictly lower; among
  mutants of equal loss the lower q wins.  Adam's moments are not used and
  stay as they are; the step count advances as in the other trainers; the
  Wasserstein critic is clipped to [-c, c] after the replacement.

The order is that of the other trainers: the discriminator first (its loss
with the generator's current samples), then the generator against the updated
discriminator, on the same latents.  losses[c] = (L_D, L_G) at the parents,
before each replacement.
"""
import numpy as np

from . import coevo, nes


def choose(f):
    """Index of the kept candidate among losses f[0 .. 2n] (f[2n] = parent) and
    its margin: the distance to the nearest other candidate's loss.

    A NaN loss ranks as +infinity (a non-finite candidate loses, as in the
    tournament); two infinite candidates are a tie (margin 0)."""
    f = np.asarray(f, dtype=np.float64)
    key = np.where(np.isnan(f), np.inf, f)
    parent = len(f) - 1
    q = int(np.argmin(key[:parent]))  # first of equal minima
    w = q if key[q] < key[parent] else parent
    others = np.delete(key, w)
    if not len(others):
        return w, np.inf
    with np.errstate(invalid="ignore"):
        d = np.abs(others - key[w])
    d[np.isnan(d)] = 0.0  # inf - inf: a tie between two losing candidates
    return w, float(np.min(d))


def candidates(theta, eps, sigma):
    """The 2n + 1 candidates in the order above, [2n + 1, P]."""
    return np.concatenate([theta + sigma * eps, theta - sigma * eps, theta[None]], axis=0)


def train_step(S, st, data, gen, step, forced=None, info=None):
    """One ES step of every training unit's pair, in place; returns losses [U, 2].

    forced[u] = (q_D, q_G) overrides the choice (a caller replaying another
    implementation's decisions on near-ties); info, a dict, receives the
    choices "q" [U, 2] and their margins "margin" [U, 2]."""
    sigma = S.wl["nes_sigma"]
    losses = np.zeros((S.U, 2))
    qs = np.zeros((S.U, 2), dtype=np.int64)
    margins = np.zeros((S.U, 2))
    for c in range(S.U):
        _, x, z = coevo.sample(S, data, c, gen, step + 1)
        xf = coevo.g_forward(S, st.Gp[c], z)[1]

        def loss_d(dp):
            return coevo.pair_losses(S, coevo.d_logits(S, dp, x)[1], coevo.d_logits(S, dp, xf)[1])[0]

        cand = candidates(st.Dp[c], nes.directions(S, "D", c, gen, step), sigma)
        f = np.array([loss_d(p) for p in cand])
        losses[c, 0] = f[-1]
        qs[c, 0], margins[c, 0] = choose(f)
        if forced is not None:
            qs[c, 0] = forced[c][0]
        st.Dp[c] = cand[qs[c, 0]]
        if S.loss == "wasserstein":
            np.clip(st.Dp[c], -S.clip, S.clip, out=st.Dp[c])
        st.Dt[c] += 1

        def loss_g(gp):
            a = coevo.d_logits(S, st.Dp[c], coevo.g_forward(S, gp, z)[1])[1]
            return coevo.pair_losses(S, a, a)[1]

        cand = candidates(st.Gp[c], nes.directions(S, "G", c, gen, step), sigma)
        f = np.array([loss_g(p) for p in cand])
        losses[c, 1] = f[-1]
        qs[c, 1], margins[c, 1] = choose(f)
        if forced is not None:
            qs[c, 1] = forced[c][1]
        st.Gp[c] = cand[qs[c, 1]]
        st.Gt[c] += 1
    if info is not None:
        info["q"], info["margin"] = qs, margins
    return losses
