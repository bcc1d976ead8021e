"""Pins of the oracle's mixture score and (1+1)-ES."""
import numpy as np
import scipy.linalg
from scipy import stats

import synth
from oracle import coevo, mixture, rng


def _setup(**kw):
    wl = synth.small_workload("mnist_mlp_4x4_mix", data=dict(n=600), g_hidden=[16, 16],
                              d_hidden=[16, 16], mix_samples=256, mix_feat_dim=8, **kw)
    data = synth.make_dataset(wl["data"])
    S = coevo.Setup(wl, len(data))
    return S, coevo.create(S), data


def test_one_dimensional_score_is_w2_between_gaussians():
    """With one feature and a one-hot w the score is (mu1-mu2)^2 + (s1-s2)^2,
    the squared 2-Wasserstein distance between N(mu1, s1^2) and N(mu2, s2^2):
    check it against the quantile-function integral int_0^1 (F1^-1 - F2^-1)^2."""
    mu1, s1, mu2, s2 = 0.3, 1.7, -0.4, 0.6
    q = (np.arange(200000) + 0.5) / 200000
    w2 = np.mean((stats.norm.ppf(q, mu1, s1) - stats.norm.ppf(q, mu2, s2)) ** 2)
    sc = mixture.score(np.array([1.0]), np.array([[mu1]]), np.array([[s1 ** 2 + mu1 ** 2]]),
                       np.array([mu2]), np.array([s2]))
    assert abs(sc - w2) < 2e-4


def test_score_is_frechet_distance_with_diagonal_covariances():
    g = np.random.default_rng(0)
    F = 6
    mu, var = g.normal(size=F), g.uniform(0.2, 2.0, size=F)
    mu_r, sd_r = g.normal(size=F), g.uniform(0.2, 2.0, size=F)
    s1, s2 = np.diag(var), np.diag(sd_r ** 2)
    fid = np.sum((mu - mu_r) ** 2) + np.trace(s1 + s2 - 2 * scipy.linalg.sqrtm(s1 @ s2)).real
    sc = mixture.score(np.array([1.0]), mu[None], (var + mu ** 2)[None], mu_r, sd_r)
    assert abs(sc - fid) < 1e-10


def test_mixture_moments_equal_pooled_samples():
    """Integer weights: the mixture moments equal the moments of the pooled
    sample in which generator k contributes n_k copies of its features."""
    g = np.random.default_rng(1)
    feats = [g.normal(k, 1 + 0.3 * k, size=(50, 4)) for k in range(5)]
    counts = np.array([3, 0, 1, 2, 4])
    w = counts / counts.sum()
    mus = np.stack([f.mean(0) for f in feats])
    s2s = np.stack([(f * f).mean(0) for f in feats])
    pooled = np.concatenate([np.repeat(f, n, axis=0) for f, n in zip(feats, counts) if n])
    mu_r, sd_r = np.zeros(4), np.ones(4)
    expect = np.sum((pooled.mean(0) - mu_r) ** 2) + np.sum((pooled.std(0) - sd_r) ** 2)
    assert abs(mixture.score(w, mus, s2s, mu_r, sd_r) - expect) < 1e-10


def test_es_keeps_simplex_and_never_worsens():
    S, st, data = _setup()
    stats_ = mixture.real_stats(S, data)
    for gen in range(3):
        w_before = st.w.copy()
        mu, s2 = mixture.generator_moments(S, st, stats_["P"], gen)
        w, sc, acc = mixture.update(S, st, stats_, gen)
        assert np.all(w >= 0) and np.allclose(w.sum(1), 1.0)
        for c in range(S.C):
            ks = S.nbr[c]
            old = mixture.score(w_before[c], mu[ks], s2[ks], stats_["mu_r"], stats_["sd_r"])
            assert sc[c] <= old
            assert (acc[c] == 1) == (not np.array_equal(w[c], w_before[c]))
            assert abs(sc[c] - mixture.score(w[c], mu[ks], s2[ks], stats_["mu_r"], stats_["sd_r"])) < 1e-12
        st.w[...] = w
    assert 0 < (w != 1 / 5).any(axis=1).sum()


def test_identical_generators_make_score_independent_of_w():
    """If every generator is the same network, the mixture has the moments of
    that one network for any w: score(w) is constant up to rounding, so the ES
    can only accept on rounding noise."""
    S, st, data = _setup()
    st.Gp[:] = st.Gp[0]
    stats_ = mixture.real_stats(S, data)
    mu, s2 = mixture.generator_moments(S, st, stats_["P"], 0)
    g = np.random.default_rng(3)
    ref = mixture.score(np.full(5, 0.2), mu[:5], s2[:5], stats_["mu_r"], stats_["sd_r"])
    for _ in range(20):
        w = g.dirichlet(np.ones(5))
        assert abs(mixture.score(w, mu[:5], s2[:5], stats_["mu_r"], stats_["sd_r"]) - ref) < 1e-12 * ref
    w, sc, acc = mixture.update(S, st, stats_, 0)
    assert np.allclose(sc, ref, rtol=1e-12)


def test_projection_and_real_stats():
    S, _, data = _setup()
    st_ = mixture.real_stats(S, data)
    P = st_["P"]
    assert P.shape == (784, 8)
    assert abs(P.std() * np.sqrt(784) - 1) < 0.05
    f = data.astype(np.float64) @ P
    assert np.allclose(st_["mu_r"], f.mean(0)) and np.allclose(st_["sd_r"], f.std(0))


def _torch_generator(p, sizes, acts, slope):
    """The generator written with torch fp64 layers: layer l's block of the
    parameter row is W_l [fan_in][fan_out] row-major, then b_l [fan_out]."""
    import torch

    pt = torch.from_numpy(np.asarray(p, dtype=np.float64))
    layers, off = [], 0
    for fi, fo in zip(sizes[:-1], sizes[1:]):
        lin = torch.nn.Linear(fi, fo, dtype=torch.float64)
        with torch.no_grad():
            lin.weight.copy_(pt[off:off + fi * fo].view(fi, fo).t())
            lin.bias.copy_(pt[off + fi * fo:off + (fi + 1) * fo])
        off += (fi + 1) * fo
        layers.append(lin)

    def run(z):
        h = torch.from_numpy(z)
        for lin, a in zip(layers, acts):
            h = lin(h)
            h = {"relu": torch.relu, "tanh": torch.tanh, "linear": lambda x: x,
                 "lrelu": lambda x: torch.nn.functional.leaky_relu(x, slope)}[a](h)
        return h

    return run


def test_generator_moments_equal_torch_on_the_shared_latents():
    """mu_k = mean over the S shared latents of the projected samples and
    s2_k = the mean of their squares (not the variance), recomputed for every
    cell with torch fp64 layers on the generation's MIXZ latents (one set for
    all cells) and the PROJ projection."""
    import torch

    S, st, data = _setup()
    P = mixture.projection(S)
    gen = 3
    mu, s2 = mixture.generator_moments(S, st, P, gen)
    Sm = S.wl["mix_samples"]
    zeta = rng.normals(S.seed, Sm * S.zd, 0, gen, 0, "MIXZ").reshape(Sm, S.zd)
    Pt = torch.from_numpy(P)
    for k in range(S.C):
        with torch.no_grad():
            f = _torch_generator(st.Gp[k], S.g_sizes, S.g_acts, S.slope)(zeta) @ Pt
        assert np.allclose(mu[k], f.mean(0).numpy(), rtol=1e-12, atol=1e-14)
        assert np.allclose(s2[k], (f * f).mean(0).numpy(), rtol=1e-12, atol=1e-14)
        assert np.all(s2[k] >= mu[k] ** 2 * (1 - 1e-12))  # E[f^2] >= E[f]^2


def test_generator_moments_of_a_constant_generator():
    """Closed form: a generator whose weights are all zero except the output
    bias b emits tanh(b) for every latent, so its features are the constant
    f = tanh(b) P: mu = f, s2 = f^2, and the mixture of such generators has
    variance 0 (sum_k w_k f_k^2 - (sum_k w_k f_k)^2 with equal f_k)."""
    S, st, data = _setup()
    P = mixture.projection(S)
    lay_off = sum((fi + 1) * fo for fi, fo in zip(S.g_sizes[:-2], S.g_sizes[1:-1]))
    fi = S.g_sizes[-2]
    g = np.random.default_rng(5)
    for k in range(S.C):
        st.Gp[k][:] = 0.0
        b = g.normal(size=S.xd)
        st.Gp[k][lay_off + fi * S.xd:lay_off + (fi + 1) * S.xd] = b
    mu, s2 = mixture.generator_moments(S, st, P, 0)
    for k in range(S.C):
        b = st.Gp[k][lay_off + fi * S.xd:lay_off + (fi + 1) * S.xd]
        f = np.tanh(b) @ P
        assert np.allclose(mu[k], f, rtol=1e-12, atol=1e-15)
        assert np.allclose(s2[k], f * f, rtol=1e-12, atol=1e-15)
    # same constant in every slot: any weights give zero variance, score = |f - mu_r|^2 + |sd_r|^2
    st.Gp[:] = st.Gp[0]
    mu, s2 = mixture.generator_moments(S, st, P, 0)
    stats_ = mixture.real_stats(S, data)
    w = g.dirichlet(np.ones(5))
    expect = np.sum((mu[0] - stats_["mu_r"]) ** 2) + np.sum(stats_["sd_r"] ** 2)
    # var_w = 0 up to the rounding of s2 - mu^2 (~1e-16 |f|^2), whose square
    # root (~1e-8 |f|) enters the score linearly: 1e-6 relative
    assert abs(mixture.score(w, mu[:5], s2[:5], stats_["mu_r"], stats_["sd_r"]) - expect) < 1e-6 * expect


def test_generator_moments_share_one_latent_set_per_generation():
    """All cells' generators see the same latents: two cells with the same
    generator get identical moments; the next generation's latents differ."""
    S, st, data = _setup()
    P = mixture.projection(S)
    st.Gp[3] = st.Gp[0]
    mu, s2 = mixture.generator_moments(S, st, P, 1)
    assert np.array_equal(mu[0], mu[3]) and np.array_equal(s2[0], s2[3])
    assert not np.array_equal(mu[0], mu[1])
    mu2, _ = mixture.generator_moments(S, st, P, 2)
    assert not np.allclose(mu[0], mu2[0], rtol=1e-6)
