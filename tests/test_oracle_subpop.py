"""Pins of the oracle's sub-populations (pop_size s > 1 per cell) and of its
post-training re-evaluation and elitist replacement: uniform tournaments over
the 5 s neighbourhood individuals, individuals and training units indexed like
the cells of a wider grid, every pair of the neighbourhood population scored
(against torch networks), the elitist truncation on hand-made fitness values
and the re-evaluated fitness against torch."""
import numpy as np
import pytest
import torch

import synth
from oracle import coevo, es, mlp, nes

SMALL = dict(g_hidden=[6], d_hidden=[5], z_dim=3, x_dim=7, batch=4)


def _setup(**kw):
    wl = synth.small_workload("mnist_mlp_3x3", data=dict(n=512), **kw)
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    return S, coevo.create(S), data


def _torch_net(S, p, role, x):
    sizes, acts = (S.g_sizes, S.g_acts) if role == "G" else (S.d_sizes, S.d_acts)
    h = torch.tensor(x)
    pt = torch.tensor(p)
    for (off, fi, fo), a in zip(mlp.layout(sizes)[0], acts):
        h = torch.nn.functional.linear(h, pt[off:off + fi * fo].view(fi, fo).t(), pt[off + fi * fo:off + (fi + 1) * fo])
        if a == "relu":
            h = torch.relu(h)
        elif a == "lrelu":
            h = torch.nn.functional.leaky_relu(h, S.slope)
        elif a == "tanh":
            h = torch.tanh(h)
    return h


def _torch_bce(S, dp, x, xf):
    ar, af = _torch_net(S, dp, "D", x), _torch_net(S, dp, "D", xf)
    bce = torch.nn.functional.binary_cross_entropy_with_logits
    return float(bce(ar, torch.ones_like(ar)) + bce(af, torch.zeros_like(af))), float(bce(af, torch.ones_like(af)))


@pytest.mark.parametrize("s, size", [(2, 2), (3, 3), (4, 3), (1, 5)])
def test_tournament_draws_are_uniform_over_ordered_tuples(monkeypatch, s, size):
    """Words at the centres of the draw intervals reach every ordered tuple of
    distinct neighbourhood indices exactly once, for every member's words."""
    S, _, _ = _setup(rows=2, cols=2, pop_size=s, tournament_size=size, **SMALL)
    n = S.n
    member = s - 1
    tuples = []

    def grid_words(ks):
        w = np.zeros(8 * (member + 1), dtype=np.uint64)
        for j, k in enumerate(ks):
            w[8 * member + j] = int((k + 0.5) * 2.0 ** 32 / (n - j))
        return w
    import itertools
    depth = min(size, n - 1)
    for ks in itertools.product(*[range(n - j) for j in range(depth)]):
        monkeypatch.setattr(coevo.rng, "raw_words", lambda *a, _w=grid_words(ks), **k: _w)
        tuples.append(tuple(coevo.tournament_draw(S, 0, 0, "TOURN_G", member)))
    assert len(set(tuples)) == len(tuples) and all(len(set(t)) == size for t in tuples)
    # with distinct fitness 0 < 1 < ... the winner of size 2 has rank r with probability 2 (n-1-r) / (n (n-1))
    if size == 2:
        wins = np.bincount([coevo.tournament_winner(np.arange(n, dtype=float), list(t)) for t in tuples], minlength=n)
        assert np.array_equal(wins, 2 * (n - 1 - np.arange(n)))  # of n (n - 1) ordered pairs


@pytest.mark.parametrize("trainer", ["gradient", "nes", "es"])
def test_members_train_like_the_cells_of_a_wider_grid(trainer):
    """Individual u of a 1x1 grid with s = 2 is created and trained from stream
    u, as cell u of a 1x2 grid with one individual per cell."""
    kw = dict(SMALL, trainer=trainer, nes_pairs=2, nes_sigma=0.05)
    S2, st2, data = _setup(rows=1, cols=1, pop_size=2, **kw)
    S1, st1, _ = _setup(rows=1, cols=2, pop_size=1, **kw)
    for f in coevo.State.FIELDS[:-1]:
        assert np.array_equal(getattr(st2, f), getattr(st1, f)), f
    step = {"gradient": coevo.train_step, "nes": nes.train_step, "es": es.train_step}[trainer]
    for s in range(2):
        assert np.array_equal(step(S2, st2, data, 3, s), step(S1, st1, data, 3, s))
    for f in coevo.State.FIELDS[:-1]:
        assert np.array_equal(getattr(st2, f), getattr(st1, f)), f


def test_evaluation_scores_every_pair_of_the_neighbourhood_population():
    """2x2 grid, s = 2: L[c][k s + i][k' s + j] is the loss of member i of slot
    k's generator against member j of slot k''s discriminator (torch)."""
    S, st, data = _setup(rows=2, cols=2, pop_size=2, **SMALL)
    for f in ("Gp", "Dp"):  # distinct individuals
        getattr(st, f)[...] += 0.01 * np.random.default_rng(1).standard_normal(getattr(st, f).shape)
    L, Lg, fg, fd = coevo.evaluate(S, st, data, 4)
    assert L.shape == (4, 10, 10) and fg.shape == (4, 10)
    for c in range(S.C):
        _, x, z = coevo.sample(S, data, c, 4, 0)
        for gi in range(10):
            g_ind = S.nbr[c, gi // 2] * 2 + gi % 2
            xf = _torch_net(S, st.Gp[g_ind], "G", z).numpy()
            for dj in range(10):
                d_ind = S.nbr[c, dj // 2] * 2 + dj % 2
                l, lg = _torch_bce(S, st.Dp[d_ind], x, xf)
                assert abs(L[c, gi, dj] - l) < 1e-12 and abs(Lg[c, gi, dj] - lg) < 1e-12
    assert np.allclose(fd, L.mean(axis=1)) and np.allclose(fg, -L.mean(axis=2))


def test_each_member_has_its_own_tournament_and_mutation(monkeypatch):
    """s = 3 (15 neighbourhood individuals), tournaments of 2: words placed at
    chosen draw positions for each member (words 8 i ..) give hand-checked
    winners; a mutation word below the probability for member 1 only (words
    4 i ..) mutates member 1's learning rate only."""
    S, st, data = _setup(rows=2, cols=3, pop_size=3, tournament_size=2, lr_mut_prob=0.5, **SMALL)
    n = S.n
    pos = {0: (3, 0), 1: (14, 13), 2: (7, 7)}          # drawn: [3, 0], [14, 13], [7, 8]
    fit = np.arange(n, dtype=float)[::-1].copy()        # index 14 best, 0 worst
    fit[8] = -1.0                                       # index 8 best of all
    winners = {0: 3, 1: 14, 2: 8}

    def words(seed, count, cell, gen, step_field, tag):
        w = np.full(count, 0xFFFFFFFF, dtype=np.uint64)
        if tag.startswith("TOURN"):
            for i, (a, b) in pos.items():
                if 8 * i + 1 < count:
                    w[8 * i] = int((a + 0.5) * 2.0 ** 32 / n)
                    w[8 * i + 1] = int((b + 0.5) * 2.0 ** 32 / (n - 1))
        elif count > 4:
            w[4] = 0                                    # member 1: u0 < 0.5
            w[5:8] = 0x80000000
        return w
    monkeypatch.setattr(coevo.rng, "raw_words", words)
    st.Glr[:] = np.arange(S.U) * 1e-3 + 1e-3
    new, sel = coevo.select_replace(S, st, np.tile(fit, (S.C, 1)), np.tile(fit, (S.C, 1)), 1)
    for c in range(S.C):
        for i in range(3):
            u = c * 3 + i
            src = S.pool[c, winners[i]]
            assert sel[u, 0] == src and sel[u, 1] == src
            assert np.array_equal(new.Gp[u], st.Gp[src])
            assert (new.Glr[u] != st.Glr[src]) == (i == 1)


@pytest.mark.parametrize("f_old, f_new, src", [
    ([1.0, 5.0], [2.0, 3.0], [-1, 0]),          # the old best takes the dropped trained slot
    ([3.0, 4.0], [1.0, 2.0], [-1, -1]),         # both trained members better
    ([1.0, 2.0], [3.0, 4.0], [0, 1]),           # both previous members better, best first
    ([2.0], [2.0], [-1]),                       # a tie keeps the trained member
    ([0.5, 3.0], [np.nan, 1.0], [0, -1]),       # NaN loses
    ([5.0, 1.0, 3.0], [9.0, 2.0, 8.0], [1, -1, 2]),
])
def test_elitist_truncation(f_old, f_new, src):
    assert np.array_equal(coevo.merge_elite(np.array(f_old), np.array(f_new)), src)


@pytest.mark.parametrize("mode", [0, 1])
def test_reevaluation_and_replacement(mode):
    """1x2 grid, s = 2: the trained members' fitness against the previous
    neighbourhood (torch), the kept set is the s best of the 2 s, and a slot
    given back to a previous member carries its Adam state and lr."""
    S, st, data = _setup(rows=1, cols=2, pop_size=2, elitism=1, fitness_mode=mode, lr0_g=0.05, lr0_d=0.05,
                         **SMALL)
    gen = 3
    L, Lg, fg, fd = coevo.evaluate(S, st, data, gen)
    st2, _ = coevo.select_replace(S, st, fg, fd, gen)
    for s in range(3):
        coevo.train_step(S, st2, data, gen, s)
    out, info = coevo.elitist_replace(S, st, st2, data, gen, fg, fd)
    for c in range(S.C):
        _, x, z = coevo.sample(S, data, c, gen, 0)
        for i in range(2):
            xf = _torch_net(S, st2.Gp[c * 2 + i], "G", z).numpy()
            ls = [_torch_bce(S, st.Dp[S.pool[c, j]], x, xf) for j in range(S.n)]
            ref = -np.mean([a for a, _ in ls]) if mode == 0 else np.mean([b for _, b in ls])
            assert abs(info["fit_g2"][c, i] - ref) < 1e-12
            dref = np.mean([_torch_bce(S, st2.Dp[c * 2 + i], x,
                                       _torch_net(S, st.Gp[S.pool[c, k]], "G", z).numpy())[0] for k in range(S.n)])
            assert abs(info["fit_d2"][c, i] - dref) < 1e-12
        for r, (f_old, f_new, pre) in enumerate(((fg[c, :2], info["fit_g2"][c], "G"),
                                                 (fd[c, :2], info["fit_d2"][c], "D"))):
            kept = []
            for i in range(2):
                j = info["src"][c * 2 + i, r]
                if j < 0:
                    kept.append(f_new[i])
                    assert np.array_equal(getattr(out, pre + "p")[c * 2 + i], getattr(st2, pre + "p")[c * 2 + i])
                else:
                    kept.append(f_old[j])
                    for f in ("p", "m", "v", "t", "lr"):
                        assert np.array_equal(getattr(out, pre + f)[c * 2 + i], getattr(st, pre + f)[c * 2 + j])
            assert np.allclose(sorted(kept), np.sort(np.concatenate([f_old, f_new]))[:2])
