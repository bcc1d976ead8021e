"""Pins of the oracle's evaluation, fitness, selection, mutation, Adam and
training step against closed forms, brute force and torch CPU fp64."""
import itertools
import math

import numpy as np
import pytest
import torch

import synth
from oracle import coevo, grid, mlp, rng


def _setup(name="mnist_mlp_3x3", n=512, **kw):
    wl = synth.small_workload(name, data=dict(n=n), **kw)
    data = synth.make_dataset(wl["data"])
    S = coevo.Setup(wl, len(data))
    return S, coevo.create(S), data


def _zero_d_output(S, st):
    off, fi, fo = mlp.layout(S.d_sizes)[0][-1]
    st.Dp[:, off:off + (fi + 1) * fo] = 0.0


def test_bce_closed_form_at_half():
    """A discriminator whose output layer is zero outputs sigmoid(0) = 1/2
    everywhere: every BCE term is ln 2, L = 2 ln 2, the generator loss ln 2."""
    S, st, data = _setup(rows=2, cols=3, g_hidden=[16], d_hidden=[16, 8],
                         z_dim=8, x_dim=784, batch=10)
    _zero_d_output(S, st)
    L, Lg, fg, fd = coevo.evaluate(S, st, data, 0)
    assert np.allclose(L, 2 * math.log(2), rtol=0, atol=1e-15)
    assert np.allclose(Lg, math.log(2), rtol=0, atol=1e-15)
    assert np.allclose(fd, 2 * math.log(2)) and np.allclose(fg, -2 * math.log(2))


def test_generator_untouched_when_discriminator_is_constant():
    """With the output layer zero and a frozen discriminator (lr 0), the generator
    gradient vanishes, so Adam leaves the generator unchanged."""
    S, st, data = _setup(rows=1, cols=2, g_hidden=[16], d_hidden=[16], z_dim=8, batch=6,
                         lr0_d=0.0)
    _zero_d_output(S, st)
    g0 = st.Gp.copy()
    losses = coevo.train_step(S, st, data, 0, 0)
    assert np.array_equal(st.Gp, g0)
    assert np.allclose(losses, [2 * math.log(2), math.log(2)])
    assert np.all(st.Gt == 1)


def test_pair_losses_match_torch_bce():
    S, st, data = _setup(rows=2, cols=2, g_hidden=[32, 32], d_hidden=[32, 32], batch=9)
    L, Lg, fg, fd = coevo.evaluate(S, st, data, 3)
    bce = torch.nn.functional.binary_cross_entropy_with_logits
    for c in range(S.C):
        idx = rng.indices(S.seed, S.B, S.N, c, 3, 0)
        z = rng.normals(S.seed, S.B * S.zd, c, 3, 0, "Z").reshape(S.B, S.zd)
        x = torch.tensor(data[idx], dtype=torch.float64)
        for i, j in itertools.product(range(5), range(5)):
            gi, dj = S.nbr[c, i], S.nbr[c, j]
            xf = _torch_mlp(st.Gp[gi], S.g_sizes, S.g_acts, torch.tensor(z), S.slope)
            ar = _torch_mlp(st.Dp[dj], S.d_sizes, S.d_acts, x, S.slope)[:, 0]
            af = _torch_mlp(st.Dp[dj], S.d_sizes, S.d_acts, xf, S.slope)[:, 0]
            ref = bce(ar, torch.ones_like(ar)) + bce(af, torch.zeros_like(af))
            assert abs(L[c, i, j] - float(ref)) < 1e-12
            assert abs(Lg[c, i, j] - float(bce(af, torch.ones_like(af)))) < 1e-12
    # fitness: discriminators averaged, generators negative-averaged
    assert np.allclose(fd, L.mean(axis=1)) and np.allclose(fg, -L.mean(axis=2))
    # 2x2 duplicates (N == S, W == E) give identical rows / columns
    assert np.array_equal(L[:, 1], L[:, 2]) and np.array_equal(L[:, :, 3], L[:, :, 4])


def _torch_mlp(p, sizes, acts, x, slope):
    pt = torch.as_tensor(p, dtype=torch.float64)
    h = x
    for (off, fi, fo), a in zip(mlp.layout(sizes)[0], acts):
        h = h @ pt[off:off + fi * fo].view(fi, fo) + pt[off + fi * fo: off + (fi + 1) * fo]
        if a == "relu":
            h = torch.relu(h)
        elif a == "lrelu":
            h = torch.nn.functional.leaky_relu(h, slope)
        elif a == "tanh":
            h = torch.tanh(h)
    return h


def test_tournament_rank_distribution_by_brute_force():
    """Size-2 tournaments over 5 slots with distinct fitness: every ordered pair
    of distinct slots is equally likely, so the winner of rank r (0 = best) has
    probability (4 - r) / 10 = (0.4, 0.3, 0.2, 0.1, 0)."""
    S, _, _ = _setup(rows=1, cols=1, g_hidden=[4], d_hidden=[4], z_dim=2, batch=2)
    fit = np.array([0.3, -1.0, 2.0, 0.1, 0.7])
    rank = np.argsort(np.argsort(fit))
    # the draw map sends word pairs to ordered pairs: enumerate interval midpoints
    counts = np.zeros(5)
    seen = set()
    for k1 in range(5):
        for p in range(4):
            w0 = int((k1 + 0.5) * 2 ** 32 / 5)
            w1 = int((p + 0.5) * 2 ** 32 / 4)
            a = (w0 * 5) >> 32
            rem = [s for s in range(5) if s != a]
            b = rem[(w1 * 4) >> 32]
            seen.add((a, b))
            counts[rank[coevo.tournament_winner(fit, [a, b])]] += 1
    assert len(seen) == 20
    assert np.allclose(counts / 20, [0.4, 0.3, 0.2, 0.1, 0.0])
    # the Philox-driven draws cover the 20 ordered pairs evenly
    freq = {}
    for c in range(4000):
        d = tuple(coevo.tournament_draw(S, c, 0, "TOURN_G"))
        assert len(set(d)) == 2
        freq[d] = freq.get(d, 0) + 1
    assert len(freq) == 20
    assert max(freq.values()) < 1.35 * 200 and min(freq.values()) > 0.65 * 200


def test_tournament_ties_and_nan():
    assert coevo.tournament_winner(np.array([1.0, 1.0, 0, 0, 0]), [1, 0]) == 1
    assert coevo.tournament_winner(np.array([1.0, 1.0, 0, 0, 0]), [0, 1]) == 0
    assert coevo.tournament_winner(np.array([np.nan, 5.0, 0, 0, 0]), [0, 1]) == 1
    assert coevo.tournament_winner(np.array([np.nan, 5.0, 0, 0, 0]), [1, 0]) == 1
    assert coevo.tournament_winner(np.array([np.inf, np.nan, 0, 0, 0]), [0, 1]) == 0


def test_tournament_larger_sizes_draw_distinct_slots():
    for size in (1, 3, 4, 5):
        S, _, _ = _setup(rows=1, cols=1, g_hidden=[4], d_hidden=[4], z_dim=2, batch=2,
                         tournament_size=size)
        for c in range(50):
            d = coevo.tournament_draw(S, c, 1, "TOURN_D")
            assert len(d) == size and len(set(d)) == size


def test_select_replace_copies_winner_bitwise_and_mutates_lr():
    S, st, data = _setup(rows=3, cols=3, g_hidden=[8], d_hidden=[8], batch=4)
    g = np.random.default_rng(0)
    for f in ("Gm", "Gv", "Dm", "Dv"):
        getattr(st, f)[...] = g.normal(size=getattr(st, f).shape)
    st.Gt[:] = np.arange(S.C) + 10
    st.Dt[:] = np.arange(S.C) + 20
    fg = g.normal(size=(S.C, 5))
    fd = g.normal(size=(S.C, 5))
    new, sel = coevo.select_replace(S, st, fg, fd, 4)
    n_mut = 0
    for c in range(S.C):
        for r, (fit, tag, pre) in enumerate(((fg, "TOURN_G", "G"), (fd, "TOURN_D", "D"))):
            d = coevo.tournament_draw(S, c, 4, tag)
            best = min(d, key=lambda k: fit[c, k])
            assert sel[c, r] == S.nbr[c, best]
            for f in ("p", "m", "v", "t"):
                assert np.array_equal(getattr(new, pre + f)[c], getattr(st, pre + f)[sel[c, r]])
            lr_old = getattr(st, pre + "lr")[sel[c, r]]
            lr_new = getattr(new, pre + "lr")[c]
            n_mut += lr_new != lr_old
            assert abs(lr_new - lr_old) < 6e-4
    assert 0 < n_mut < 2 * S.C
    forced = np.tile(np.array([[4, 7]]), (S.C, 1))
    new2, sel2 = coevo.select_replace(S, st, fg, fd, 4, forced=forced)
    assert np.array_equal(sel2, forced)
    assert np.array_equal(new2.Gp, np.repeat(st.Gp[4:5], S.C, 0))
    assert np.array_equal(new2.Dp, np.repeat(st.Dp[7:8], S.C, 0))


def test_lr_mutation_statistics():
    """Gaussian hyper-parameter mutation: probability 0.5, N(0, (1e-4)^2), clamp at 0."""
    S, _, _ = _setup(rows=1, cols=1, g_hidden=[4], d_hidden=[4], z_dim=2, batch=2)
    d = np.array([coevo.mutate_lr(S, 1.0, c, 0, "LRMUT_G") - 1.0 for c in range(20000)])
    mutated = d != 0.0
    assert abs(mutated.mean() - 0.5) < 0.015
    assert abs(d[mutated].std() / 1e-4 - 1.0) < 0.03
    assert abs(d[mutated].mean()) < 5e-6
    assert coevo.mutate_lr(S, 0.0, 3, 0, "LRMUT_G") >= 0.0
    S2, _, _ = _setup(rows=1, cols=1, g_hidden=[4], d_hidden=[4], z_dim=2, batch=2, lr_mutation=0)
    assert coevo.mutate_lr(S2, 0.3, 3, 0, "LRMUT_G") == 0.3


def test_adam_closed_forms_and_torch():
    S, _, _ = _setup(rows=1, cols=1, g_hidden=[4], d_hidden=[4], z_dim=2, batch=2)
    lr, eps = 2e-4, S.wl["eps"]
    # constant gradient: m_hat = g and v_hat = g^2 exactly, so each step is -lr g / (|g| + eps)
    g = np.array([3.0, -0.5, 1e-3])
    p, m, v, t = np.zeros(3), np.zeros(3), np.zeros(3), 0
    for k in range(1, 6):
        t = coevo.adam(S, p, m, v, t, lr, g)
        assert np.allclose(p, -k * lr * g / (np.abs(g) + eps), rtol=1e-12, atol=0)
    # two hand-computed steps with g1 = 1, g2 = -2:
    # m1 = .1, v1 = .001 -> step lr * 1/(1+eps); m2 = .09 - .2 = -.11, v2 = .000999 + .004 = .004999
    p, m, v = np.zeros(1), np.zeros(1), np.zeros(1)
    t = coevo.adam(S, p, m, v, 0, lr, np.array([1.0]))
    t = coevo.adam(S, p, m, v, t, lr, np.array([-2.0]))
    mhat, vhat = -0.11 / (1 - 0.81), 0.004999 / (1 - 0.998001)
    expect = -lr / (1 + eps) - lr * mhat / (math.sqrt(vhat) + eps)
    assert abs(p[0] - expect) < 1e-15
    # random gradients against torch.optim.Adam
    gr = np.random.default_rng(0).normal(size=(30, 50))
    p0 = np.random.default_rng(1).normal(size=50)
    p, m, v, t = p0.copy(), np.zeros(50), np.zeros(50), 0
    pt = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.Adam([pt], lr=1e-2, betas=(0.9, 0.999), eps=1e-8)
    for k in range(30):
        t = coevo.adam(S, p, m, v, t, 1e-2, gr[k])
        opt.zero_grad()
        pt.grad = torch.tensor(gr[k])
        opt.step()
    assert np.allclose(p, pt.detach().numpy(), rtol=1e-12, atol=1e-14)


def _textbook_gan_generation(S, st, data, gen):
    """Plain alternating GAN training with torch fp64 autograd and torch.optim.Adam."""
    def net(pt, sizes, acts, x):
        h = x
        for (off, fi, fo), a in zip(mlp.layout(sizes)[0], acts):
            h = torch.nn.functional.linear(h, pt[off:off + fi * fo].view(fi, fo).t(),
                                           pt[off + fi * fo: off + (fi + 1) * fo])
            if a == "relu":
                h = torch.relu(h)
            elif a == "lrelu":
                h = torch.nn.functional.leaky_relu(h, S.slope)
            elif a == "tanh":
                h = torch.tanh(h)
        return h
    Gp = torch.tensor(st.Gp[0], requires_grad=True)
    Dp = torch.tensor(st.Dp[0], requires_grad=True)
    b = (S.wl["beta1"], S.wl["beta2"])
    og = torch.optim.Adam([Gp], lr=float(st.Glr[0]), betas=b, eps=S.wl["eps"])
    od = torch.optim.Adam([Dp], lr=float(st.Dlr[0]), betas=b, eps=S.wl["eps"])
    bce = torch.nn.functional.binary_cross_entropy_with_logits
    wgan = S.wl.get("loss", "bce") == "wasserstein"
    for s in range(S.wl["steps"]):
        idx = rng.indices(S.seed, S.B, S.N, 0, gen, s + 1)
        z = torch.tensor(rng.normals(S.seed, S.B * S.zd, 0, gen, s + 1, "Z").reshape(S.B, S.zd))
        x = torch.tensor(data[idx], dtype=torch.float64)
        xf = net(Gp, S.g_sizes, S.g_acts, z)
        ar = net(Dp, S.d_sizes, S.d_acts, x)
        af = net(Dp, S.d_sizes, S.d_acts, xf.detach())
        if wgan:  # critic loss, then weight clipping
            ld = af.mean() - ar.mean()
        else:
            ld = bce(ar, torch.ones_like(ar)) + bce(af, torch.zeros_like(af))
        od.zero_grad()
        ld.backward()
        od.step()
        if wgan:
            with torch.no_grad():
                Dp.clamp_(-S.wl["wgan_clip"], S.wl["wgan_clip"])
        af2 = net(Dp, S.d_sizes, S.d_acts, xf)
        lg = -af2.mean() if wgan else bce(af2, torch.ones_like(af2))
        og.zero_grad()
        lg.backward()
        og.step()
    return Gp.detach().numpy(), Dp.detach().numpy()


@pytest.mark.parametrize("name,loss", [("ring8_mlp_2x2", "bce"), ("mnist_mlp_3x3", "bce"),
                                       ("mnist_mlp_3x3", "wasserstein")])
def test_one_by_one_grid_is_plain_gan_training(name, loss):
    """On a 1x1 torus all five slots are the cell itself: selection is the
    identity and a generation reduces to textbook alternating GAN training
    (for the Wasserstein trainer: critic loss mean D(fake) - mean D(real),
    clamp of the critic's weights after its step, generator loss -mean D(fake))."""
    over = dict(rows=1, cols=1, steps=4, lr_mutation=0, loss=loss, wgan_clip=0.05)
    if name == "mnist_mlp_3x3":
        over.update(g_hidden=[32, 32], d_hidden=[32, 32], batch=16)
    S, st, data = _setup(name, n=1000, **over)
    new, rec = coevo.generation(S, st, data, 2)
    assert np.all(rec["sel"] == 0)
    assert np.allclose(rec["L"], rec["L"][0, 0, 0])
    gref, dref = _textbook_gan_generation(S, st, data, 2)
    assert np.allclose(new.Gp[0], gref, rtol=1e-10, atol=1e-13)
    assert np.allclose(new.Dp[0], dref, rtol=1e-10, atol=1e-13)
    assert new.Gt[0] == 4 and new.Dt[0] == 4


def test_train_step_gradients_match_finite_differences():
    """The discriminator and generator gradients the step feeds to Adam equal
    central differences of the two losses (tiny nets, fp64)."""
    S, st, data = _setup(rows=1, cols=1, g_hidden=[3], d_hidden=[4], z_dim=2, x_dim=784, batch=3)
    _, x, z = coevo.sample(S, data, 0, 0, 1)

    def loss_d(dp):
        ar = coevo.d_logits(S, dp, x)[1]
        af = coevo.d_logits(S, dp, coevo.g_forward(S, st.Gp[0], z)[1])[1]
        return coevo.softplus(-ar).mean() + coevo.softplus(af).mean()

    def loss_g(gp, dp):
        af = coevo.d_logits(S, dp, coevo.g_forward(S, gp, z)[1])[1]
        return coevo.softplus(-af).mean()

    # recover the gradients from one Adam step: with lr tiny the first step is
    # -lr * g / (|g| + eps); use t = 0, so m_hat = g and v_hat = g^2
    st2 = st.copy()
    st2.Dlr[:] = 0.0
    st2.Glr[:] = 0.0
    coevo.train_step(S, st2, data, 0, 0)
    gD = st2.Dm[0] / (1 - S.wl["beta1"])
    gG = st2.Gm[0] / (1 - S.wl["beta1"])
    h = 1e-6
    for k in range(len(gD)):
        e = np.zeros_like(gD)
        e[k] = h
        fd = (loss_d(st.Dp[0] + e) - loss_d(st.Dp[0] - e)) / (2 * h)
        assert abs(fd - gD[k]) < 1e-7 + 1e-6 * abs(fd)
    for k in range(len(gG)):
        e = np.zeros_like(gG)
        e[k] = h
        fd = (loss_g(st.Gp[0] + e, st.Dp[0]) - loss_g(st.Gp[0] - e, st.Dp[0])) / (2 * h)
        assert abs(fd - gG[k]) < 1e-7 + 1e-6 * abs(fd)


def test_wasserstein_closed_form_constant_critic():
    """A critic whose output layer is zero but for its bias b outputs b on every
    row: each pair's critic loss mean a_fake - mean a_real is 0 and the
    generator's own loss is -b."""
    S, st, data = _setup(rows=2, cols=3, g_hidden=[16], d_hidden=[16, 8], z_dim=8, batch=10,
                         loss="wasserstein")
    off, fi, fo = mlp.layout(S.d_sizes)[0][-1]
    st.Dp[:, off:off + fi * fo] = 0.0
    st.Dp[:, off + fi * fo] = 0.3
    L, Lg, fg, fd = coevo.evaluate(S, st, data, 0)
    assert np.all(np.abs(L) < 1e-15) and np.allclose(Lg, -0.3, rtol=0, atol=1e-15)
    assert np.all(np.abs(fd) < 1e-15) and np.all(np.abs(fg) < 1e-15)


def test_wasserstein_gradients_match_finite_differences():
    """The critic and generator gradients of the Wasserstein step equal central
    differences of mean D(fake) - mean D(real) and of -mean D(G(z)); the clip
    bound is set out of reach so that the step itself is a plain Adam step."""
    S, st, data = _setup(rows=1, cols=1, g_hidden=[3], d_hidden=[4], z_dim=2, x_dim=784, batch=3,
                         loss="wasserstein", wgan_clip=100.0)
    _, x, z = coevo.sample(S, data, 0, 0, 1)

    def loss_d(dp):
        ar = coevo.d_logits(S, dp, x)[1]
        af = coevo.d_logits(S, dp, coevo.g_forward(S, st.Gp[0], z)[1])[1]
        return af.mean() - ar.mean()

    def loss_g(gp, dp):
        return -coevo.d_logits(S, dp, coevo.g_forward(S, gp, z)[1])[1].mean()

    st2 = st.copy()
    st2.Dlr[:] = 0.0
    st2.Glr[:] = 0.0
    losses = coevo.train_step(S, st2, data, 0, 0)
    assert abs(losses[0, 0] - loss_d(st.Dp[0])) < 1e-14 and abs(losses[0, 1] - loss_g(st.Gp[0], st.Dp[0])) < 1e-14
    gD = st2.Dm[0] / (1 - S.wl["beta1"])
    gG = st2.Gm[0] / (1 - S.wl["beta1"])
    h = 1e-6
    for k in range(len(gD)):
        e = np.zeros_like(gD)
        e[k] = h
        fd = (loss_d(st.Dp[0] + e) - loss_d(st.Dp[0] - e)) / (2 * h)
        assert abs(fd - gD[k]) < 1e-7 + 1e-6 * abs(fd)
    for k in range(len(gG)):
        e = np.zeros_like(gG)
        e[k] = h
        fd = (loss_g(st.Gp[0] + e, st.Dp[0]) - loss_g(st.Gp[0] - e, st.Dp[0])) / (2 * h)
        assert abs(fd - gG[k]) < 1e-7 + 1e-6 * abs(fd)


def test_wasserstein_critic_weights_are_clipped():
    """After a Wasserstein step every critic parameter lies in [-c, c]; the
    ones the Adam step left inside are exactly the Adam results, the others
    sit on the bound with the sign of the Adam result."""
    c = 0.02
    S, st, data = _setup(rows=1, cols=2, g_hidden=[16], d_hidden=[16], z_dim=8, batch=6,
                         loss="wasserstein", wgan_clip=c, lr0_d=0.05)
    free = coevo.Setup(dict(S.wl, wgan_clip=1e9), S.N)
    st_free = st.copy()
    coevo.train_step(S, st, data, 0, 0)
    coevo.train_step(free, st_free, data, 0, 0)
    assert np.all(np.abs(st.Dp) <= c)
    inside = np.abs(st_free.Dp) <= c
    assert np.array_equal(st.Dp[inside], st_free.Dp[inside])
    assert np.array_equal(st.Dp[~inside], np.sign(st_free.Dp[~inside]) * c)
    assert inside.mean() < 1.0  # the bound was hit somewhere
    assert np.array_equal(st.Dm, st_free.Dm) and np.array_equal(st.Dv, st_free.Dv)
