"""Pins of the oracle's NES trainer: the antithetic estimate is exact on
quadratics, converges to the backpropagated gradient of the GAN losses, and
a step is one Adam step on it; a 1x1 grid matches the same loop written with
torch networks and torch.optim.Adam."""
import numpy as np
import pytest
import torch

import synth
from oracle import coevo, mlp, nes, rng


def _setup(**kw):
    wl = synth.small_workload("mnist_mlp_3x3", data=dict(n=512), trainer="nes", **kw)
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    return S, coevo.create(S), data


def test_estimate_is_exact_for_quadratics():
    """For f = theta' A theta / 2 + b' theta the quadratic terms cancel in each
    antithetic pair: the estimate equals (1/n) sum_k eps_k eps_k' (A theta + b)."""
    r = np.random.default_rng(3)
    P, n = 7, 5
    M = r.standard_normal((P, P))
    A = M @ M.T
    b = r.standard_normal(P)
    theta = r.standard_normal(P)
    eps = r.standard_normal((n, P))
    f = lambda t: 0.5 * t @ A @ t + b @ t + 3.0  # noqa: E731
    g = nes.nes_gradient(f, theta, eps, 0.3)
    ref = (eps.T @ (eps @ (A @ theta + b))) / n
    assert np.allclose(g, ref, rtol=1e-11, atol=1e-11)
    # a linear function: the same formula, independent of sigma
    g2 = nes.nes_gradient(lambda t: b @ t, theta, eps, 1e-3)
    assert np.allclose(g2, (eps.T @ (eps @ b)) / n, rtol=1e-9, atol=1e-9)


@pytest.mark.parametrize("loss", ["bce", "wasserstein"])
def test_estimate_converges_to_the_backpropagated_gradient(loss):
    """With many directions the NES estimate of the critic's and the generator's
    loss gradient approaches the gradient the backpropagating trainer feeds to Adam."""
    # 41 parameters per network: the estimate's error shrinks like sqrt(P / n)
    S, st, data = _setup(rows=1, cols=1, g_hidden=[3], d_hidden=[4], z_dim=2, x_dim=8, batch=3, loss=loss,
                         wgan_clip=100.0)
    assert S.PD == 41 and S.PG == 41
    _, x, z = coevo.sample(S, data, 0, 0, 1)
    xf = coevo.g_forward(S, st.Gp[0], z)[1]
    loss_d = lambda dp: coevo.pair_losses(S, coevo.d_logits(S, dp, x)[1], coevo.d_logits(S, dp, xf)[1])[0]  # noqa
    loss_g = lambda gp: -0.0 + coevo.pair_losses(  # noqa: E731
        S, *(2 * [coevo.d_logits(S, st.Dp[0], coevo.g_forward(S, gp, z)[1])[1]]))[1]
    # the backpropagated gradients: one step with lr 0 from zero Adam state leaves m = (1 - beta1) g
    st2 = st.copy()
    st2.Dlr[:] = 0.0
    st2.Glr[:] = 0.0
    coevo.train_step(S, st2, data, 0, 0)
    gD = st2.Dm[0] / (1 - S.wl["beta1"])
    gG = st2.Gm[0] / (1 - S.wl["beta1"])
    n = 20000
    for f, theta, ref, tag in ((loss_d, st.Dp[0], gD, "NES_D"), (loss_g, st.Gp[0], gG, "NES_G")):
        eps = rng.normals(S.seed, n * len(theta), 0, 0, 1, tag).reshape(n, len(theta))
        g = nes.nes_gradient(f, theta, eps, 1e-3)
        cos = g @ ref / (np.linalg.norm(g) * np.linalg.norm(ref))
        assert cos > 0.99, cos
        assert np.linalg.norm(g - ref) < 0.15 * np.linalg.norm(ref)


def test_step_is_one_adam_step_on_the_estimate():
    """train_step draws the step's directions from streams NES_D / NES_G, scores the
    discriminator with the generator's current samples and the generator against the
    updated discriminator, and applies one Adam step to each."""
    S, st, data = _setup(rows=1, cols=2, g_hidden=[6], d_hidden=[5], z_dim=3, batch=4, nes_pairs=3,
                         nes_sigma=0.05)
    ref = st.copy()
    gen, step = 2, 7
    losses = nes.train_step(S, st, data, gen, step)
    for c in range(S.C):
        _, x, z = coevo.sample(S, data, c, gen, step + 1)
        xf = coevo.g_forward(S, ref.Gp[c], z)[1]
        fd = lambda dp: coevo.pair_losses(S, coevo.d_logits(S, dp, x)[1], coevo.d_logits(S, dp, xf)[1])[0]  # noqa
        eps = rng.normals(S.seed, 3 * S.PD, c, gen, step + 1, "NES_D").reshape(3, S.PD)
        g = np.zeros(S.PD)
        for k in range(3):
            g += (fd(ref.Dp[c] + 0.05 * eps[k]) - fd(ref.Dp[c] - 0.05 * eps[k])) * eps[k]
        g /= 2 * 3 * 0.05
        # first Adam step from zero state: p - lr g / (|g| + eps) (bias corrections cancel)
        d_new = ref.Dp[c] - ref.Dlr[c] * g / (np.abs(g) + S.wl["eps"])
        assert np.allclose(st.Dp[c], d_new, rtol=1e-12, atol=1e-15)
        assert abs(losses[c, 0] - fd(ref.Dp[c])) < 1e-14
        a = coevo.d_logits(S, d_new, xf)[1]
        assert abs(losses[c, 1] - coevo.softplus(-a).mean()) < 1e-12
    assert np.all(st.Gt == 1) and np.all(st.Dt == 1)
    assert not np.allclose(st.Gp, ref.Gp)


def test_one_by_one_grid_matches_torch_loop():
    """A 1x1 generation of the NES trainer against the same loop written with
    torch fp64 networks and torch.optim.Adam, fed the same directions."""
    S, st, data = _setup(rows=1, cols=1, g_hidden=[8], d_hidden=[8], z_dim=4, batch=5, steps=3,
                         lr_mutation=0, nes_pairs=4, nes_sigma=0.02)
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

    bce = torch.nn.functional.binary_cross_entropy_with_logits
    Gp = torch.tensor(st.Gp[0])
    Dp = torch.tensor(st.Dp[0])
    b = (S.wl["beta1"], S.wl["beta2"])
    Gv, Dv = Gp.clone().requires_grad_(True), Dp.clone().requires_grad_(True)
    og = torch.optim.Adam([Gv], lr=float(st.Glr[0]), betas=b, eps=S.wl["eps"])
    od = torch.optim.Adam([Dv], lr=float(st.Dlr[0]), betas=b, eps=S.wl["eps"])
    n, sig = 4, 0.02
    for s in range(3):
        idx = rng.indices(S.seed, S.B, S.N, 0, 1, s + 1)
        z = torch.tensor(rng.normals(S.seed, S.B * S.zd, 0, 1, s + 1, "Z").reshape(S.B, S.zd))
        x = torch.tensor(data[idx], dtype=torch.float64)
        with torch.no_grad():
            xf = net(Gv, S.g_sizes, S.g_acts, z)

            def ld(d):
                ar, af = net(d, S.d_sizes, S.d_acts, x), net(d, S.d_sizes, S.d_acts, xf)
                return float(bce(ar, torch.ones_like(ar)) + bce(af, torch.zeros_like(af)))

            eps = torch.tensor(rng.normals(S.seed, n * S.PD, 0, 1, s + 1, "NES_D").reshape(n, S.PD))
            gd = sum((ld(Dv + sig * eps[k]) - ld(Dv - sig * eps[k])) * eps[k] for k in range(n)) / (2 * n * sig)
        od.zero_grad()
        Dv.grad = gd.clone()
        od.step()
        with torch.no_grad():
            def lg(g):
                af = net(Dv, S.d_sizes, S.d_acts, net(g, S.g_sizes, S.g_acts, z))
                return float(bce(af, torch.ones_like(af)))

            eps = torch.tensor(rng.normals(S.seed, n * S.PG, 0, 1, s + 1, "NES_G").reshape(n, S.PG))
            gg = sum((lg(Gv + sig * eps[k]) - lg(Gv - sig * eps[k])) * eps[k] for k in range(n)) / (2 * n * sig)
        og.zero_grad()
        Gv.grad = gg.clone()
        og.step()
    assert np.allclose(new.Dp[0], Dv.detach().numpy(), rtol=1e-9, atol=1e-12)
    assert np.allclose(new.Gp[0], Gv.detach().numpy(), rtol=1e-9, atol=1e-12)
    assert rec["losses"].shape == (3, 1, 2)
