"""Pins of the oracle's mixture score and (1+1)-ES."""
import numpy as np
import scipy.linalg
from scipy import stats

import synth
from oracle import coevo, mixture


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
