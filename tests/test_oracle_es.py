"""Pins of the oracle's (1+lambda)-ES trainer: the plus-selection rule on
hand-made losses, a 1x1 grid against the same loop written with torch
networks (every candidate scored by torch), a vanishing mutation keeping the
parent bit for bit, and the elitist invariant with the Wasserstein clip."""
import numpy as np
import pytest
import torch

import synth
from oracle import coevo, es, mlp, rng


def _setup(**kw):
    wl = synth.small_workload("mnist_mlp_3x3", data=dict(n=512), trainer="es", **kw)
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    return S, coevo.create(S), data


@pytest.mark.parametrize("f, w, margin", [
    ([3.0, 1.0, 2.0, 5.0, 4.0], 1, 1.0),     # the best mutant
    ([2.0, 2.0, 2.0], 2, 0.0),               # all equal: the parent stays
    ([1.0, 3.0, 1.0], 2, 0.0),               # a mutant only as good as the parent: the parent stays
    ([4.0, 1.0, 1.0, 3.0, 2.0], 1, 0.0),     # equal mutants: the lower index
    ([3.0, 4.0, 2.5, 5.0, 2.0], 4, 0.5),     # the parent is best
    ([np.nan, 1.0, 2.0], 1, 1.0),            # a NaN mutant loses; a later, better one is kept
    ([np.nan, np.nan, 2.0], 2, np.inf),      # only NaN mutants: the parent stays
    ([1.0, np.nan, np.nan], 0, np.inf),      # a NaN parent loses to a finite mutant
    ([np.nan, np.nan, np.nan], 2, 0.0),      # everything NaN: the parent stays, a tie
])
def test_choice_rule(f, w, margin):
    got_w, got_m = es.choose(f)
    assert got_w == w and got_m == margin


def test_one_by_one_grid_matches_torch_loop():
    """A 1x1 generation of the ES trainer against the same loop written with
    torch fp64 networks: every candidate scored by torch, the plus-selection
    written out, the critic first, then the generator against the updated
    critic."""
    S, st, data = _setup(rows=1, cols=1, g_hidden=[8], d_hidden=[8], z_dim=4, batch=5, steps=4,
                         lr_mutation=0, nes_pairs=3, nes_sigma=0.05)
    new, rec = coevo.generation(S, st, data, 1)

    def net(pt, sizes, acts, x):
        h = x
        for (off, fi, fo), a in zip(mlp.layout(sizes)[0], acts):
            h = torch.nn.functional.linear(h, pt[off:off + fi * fo].view(fi, fo).t(), pt[off + fi * fo:off + (fi + 1) * fo])
            if a == "relu":
                h = torch.relu(h)
            elif a == "lrelu":
                h = torch.nn.functional.leaky_relu(h, S.slope)
            elif a == "tanh":
                h = torch.tanh(h)
        return h

    def plus_select(theta, eps, loss):
        parent = loss(theta)
        best, best_f = theta, parent
        for sgn in (1.0, -1.0):
            for k in range(eps.shape[0]):
                cand = theta + sgn * 0.05 * eps[k]
                fk = loss(cand)
                if fk < best_f:
                    best, best_f = cand, fk
        return best, parent, best_f

    bce = torch.nn.functional.binary_cross_entropy_with_logits
    G = torch.tensor(st.Gp[0])
    D = torch.tensor(st.Dp[0])
    kept = 0
    for s in range(4):
        idx = rng.indices(S.seed, S.B, S.N, 0, 1, s + 1)
        z = torch.tensor(rng.normals(S.seed, S.B * S.zd, 0, 1, s + 1, "Z").reshape(S.B, S.zd))
        x = torch.tensor(data[idx], dtype=torch.float64)
        xf = net(G, S.g_sizes, S.g_acts, z)

        def ld(d):
            ar, af = net(d, S.d_sizes, S.d_acts, x), net(d, S.d_sizes, S.d_acts, xf)
            return float(bce(ar, torch.ones_like(ar)) + bce(af, torch.zeros_like(af)))

        eps = torch.tensor(rng.normals(S.seed, 3 * S.PD, 0, 1, s + 1, "NES_D").reshape(3, S.PD))
        D, fd0, fd1 = plus_select(D, eps, ld)

        def lg(g):
            af = net(D, S.d_sizes, S.d_acts, net(g, S.g_sizes, S.g_acts, z))
            return float(bce(af, torch.ones_like(af)))

        eps = torch.tensor(rng.normals(S.seed, 3 * S.PG, 0, 1, s + 1, "NES_G").reshape(3, S.PG))
        G, fg0, fg1 = plus_select(G, eps, lg)
        kept += (fd1 == fd0) + (fg1 == fg0)
        assert abs(rec["losses"][s, 0, 0] - fd0) < 1e-12 and abs(rec["losses"][s, 0, 1] - fg0) < 1e-12
    assert kept < 8  # some steps did move
    assert np.allclose(new.Dp[0], D.numpy(), rtol=1e-12, atol=1e-15)
    assert np.allclose(new.Gp[0], G.numpy(), rtol=1e-12, atol=1e-15)
    # Adam's state untouched, step counts advanced
    for f in ("Gm", "Gv", "Dm", "Dv"):
        assert np.array_equal(getattr(new, f), getattr(st, f))
    assert np.all(new.Gt == st.Gt + 4) and np.all(new.Dt == st.Dt + 4)


def test_vanishing_mutation_keeps_the_parent():
    """With sigma far below the parameters' spacing every mutant equals its
    parent, all losses tie, and the parent is kept bit for bit."""
    S, st, data = _setup(rows=2, cols=2, g_hidden=[6], d_hidden=[5], z_dim=3, batch=4, nes_pairs=2,
                         nes_sigma=1e-300)
    ref = st.copy()
    info = {}
    es.train_step(S, st, data, 0, 0, info=info)
    assert np.all(info["q"] == 2 * 2) and np.all(info["margin"] == 0.0)
    assert np.array_equal(st.Dp, ref.Dp) and np.array_equal(st.Gp, ref.Gp)
    assert np.all(st.Dt == ref.Dt + 1) and np.all(st.Gt == ref.Gt + 1)


@pytest.mark.parametrize("loss", ["bce", "wasserstein"])
def test_step_never_raises_the_minibatch_loss(loss):
    """Elitism: on the step's own minibatch the kept critic's loss is at most
    the parent's, and so is the kept generator's against the updated critic;
    the Wasserstein critic ends inside [-c, c]."""
    S, st, data = _setup(rows=1, cols=2, g_hidden=[6], d_hidden=[5], z_dim=3, batch=6, nes_pairs=4,
                         nes_sigma=0.2, loss=loss, wgan_clip=0.3)
    ref = st.copy()
    gen, step = 1, 2
    info = {}
    losses = es.train_step(S, st, data, gen, step, info=info)
    for c in range(S.C):
        _, x, z = coevo.sample(S, data, c, gen, step + 1)
        xf = coevo.g_forward(S, ref.Gp[c], z)[1]
        ld = lambda dp: coevo.pair_losses(S, coevo.d_logits(S, dp, x)[1], coevo.d_logits(S, dp, xf)[1])[0]  # noqa
        assert abs(losses[c, 0] - ld(ref.Dp[c])) < 1e-14
        if loss == "bce":
            assert ld(st.Dp[c]) <= losses[c, 0]
        else:  # the clip may move the kept critic; it stays inside the bound
            assert np.all(np.abs(st.Dp[c]) <= 0.3)
        a0 = coevo.d_logits(S, st.Dp[c], coevo.g_forward(S, ref.Gp[c], z)[1])[1]
        a1 = coevo.d_logits(S, st.Dp[c], coevo.g_forward(S, st.Gp[c], z)[1])[1]
        assert abs(losses[c, 1] - coevo.pair_losses(S, a0, a0)[1]) < 1e-14
        assert coevo.pair_losses(S, a1, a1)[1] <= losses[c, 1]
    assert np.any(info["q"] != 2 * 4)  # a mutant was kept somewhere
