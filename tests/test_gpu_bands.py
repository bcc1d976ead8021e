"""The row-band executor (lipz_run_generations with bands >= 2, the paper's
asynchronous cells scheduled by neighbour readiness) against the oracle and
against the one-batch schedule: the same generations give the same state bit
for bit.

Against the oracle: one banded generation from a state loaded on both sides.
Its selections are read back from a banded run without training steps (each
cell's individuals are then bit-exact copies of their sources); the
tournaments must agree with the oracle's where decisive, and the oracle
replays them.  After evaluation, selection, the training steps and the
mixture step: parameters 1e-3 per tensor, step counts bit-exact, learning
rates 1e-6, mixture weights where the oracle's ES margin is decisive.  The
one-batch schedule is also checked against the entry points called one by
one.
"""
import numpy as np
import pytest

import synth
from oracle import coevo, mixture

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_1811_12843_amd as L  # noqa: E402
from harness import GpuGrid, check_selection, fp32_state, per_tensor_rel  # noqa: E402

RAGGED = dict(z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
              data=dict(kind="mnist_like", n=3000))

CASES = {
    # 8 rows in 4 bands: bands 0 and 2 (and 1 and 3) share no neighbour row and may drift apart
    "ragged_8x3_b4": dict(RAGGED, rows=8, cols=3, bands=4),
    # one row per band, uneven split of 7 rows into 3 bands, sub-populations with elitism
    "ragged_7x2_b3_s2": dict(RAGGED, rows=7, cols=2, bands=3, pop_size=2, elitism=1),
    "ragged_5x3_b5": dict(RAGGED, rows=5, cols=3, bands=5),
    # MNIST-shaped networks, 8x8 grid in 8 bands
    "mnist_8x8_b8": dict(rows=8, cols=8, bands=8, batch=32, data=dict(n=4000)),
    # the 4x4 grid with the mixture step, in 2 and 4 bands (its ES waits for the neighbour bands' moments)
    "mnist_4x4_mix_b2": dict(rows=4, cols=4, bands=2, batch=32, mix_enable=1, mix_samples=300, data=dict(n=4000)),
    "ragged_6x2_mix_b3": dict(RAGGED, rows=6, cols=2, bands=3, mix_enable=1, mix_samples=130, mix_feat_dim=24),
    # the gradient-free trainers
    "ragged_8x3_b4_nes": dict(RAGGED, rows=8, cols=3, bands=4, trainer="nes", nes_pairs=3),
    "ragged_6x2_b3_es_s2": dict(RAGGED, rows=6, cols=2, bands=3, trainer="es", nes_pairs=2, pop_size=2, elitism=1),
}


def _setup(key):
    wl = synth.small_workload("mnist_mlp_3x3", **CASES[key])
    data = synth.make_dataset(wl["data"])
    if data.shape[1] != wl["x_dim"]:
        data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    return wl, data


@pytest.mark.parametrize("key", list(CASES))
def test_bands_match_one_batch(key):
    wl, data = _setup(key)
    gens, steps = 3, 4
    print(f"[case] bands key={key}", flush=True)
    with GpuGrid(dict(wl, bands=0), data) as one:
        L.lipz_run_generations(one.g, 2, gens, steps)
        assert one.sync() == L.LIPZ_OK
        ref = one.save_blob()
    with GpuGrid(wl, data) as banded:
        L.lipz_run_generations(banded.g, 2, gens, steps)
        assert banded.sync() == L.LIPZ_OK
        got = banded.save_blob()
    assert np.array_equal(got, ref)


def test_one_batch_matches_the_entry_points():
    wl, data = _setup("ragged_7x2_b3_s2")
    wl = dict(wl, bands=0)
    print("[case] run_generations vs entry points", flush=True)
    with GpuGrid(wl, data) as a:
        L.lipz_run_generations(a.g, 0, 2, 3)
        assert a.sync() == L.LIPZ_OK
        ref = a.save_blob()
    with GpuGrid(wl, data) as b:
        for gen in range(2):
            b.eval(gen)
            b.select(gen)
            b.train(gen, 0, 3)
            b.elite(gen)
        got = b.save_blob()
    assert np.array_equal(got, ref)


def _sources(before, after, S):
    """Source individual of every unit and role: the row of `before` that the
    unit's parameters in `after` copy bit for bit."""
    sel = np.zeros((S.U, 2), dtype=np.int64)
    for r, f in enumerate(("Gp", "Dp")):
        a, b = getattr(after, f), getattr(before, f)
        for u in range(S.U):
            hits = [k for k in range(S.U) if np.array_equal(a[u], b[k])]
            assert len(hits) == 1, (u, f, hits)
            sel[u, r] = hits[0]
    return sel


@pytest.mark.parametrize("key", ["mnist_4x4_mix_b2", "ragged_8x3_b4"])
def test_banded_generation_matches_oracle(key):
    wl, data = _setup(key)
    steps, gen = 3, 1
    wl = dict(wl, steps=steps)
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    for s in range(2):  # a trained state
        coevo.train_step(S, st, data, 0, 60 + s)
    st = fp32_state(st)
    if wl["mix_enable"]:
        st.w = np.random.default_rng(2).dirichlet(np.ones(5), size=S.C).astype(np.float32).astype(np.float64)
    print(f"[case] banded generation vs oracle key={key}", flush=True)
    # the banded schedule's selections: a generation without training steps
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        L.lipz_run_generations(gg.g, gen, 1, 0)
        assert gg.sync() == L.LIPZ_OK
        gsel = _sources(st, gg.get_state(), S)
    _, _, ofg, ofd = coevo.evaluate(S, st, data, gen)
    n_dec = check_selection(S, gsel, ofg, ofd, gen)
    assert n_dec > 0
    # the whole banded generation
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        L.lipz_run_generations(gg.g, gen, 1, steps)
        assert gg.sync() == L.LIPZ_OK
        got = gg.get_state()
    ref, _ = coevo.select_replace(S, st, ofg, ofd, gen, forced=gsel)
    for s in range(steps):
        coevo.train_step(S, ref, data, gen, s)
    assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
    assert np.all(np.abs(got.Glr - ref.Glr) <= 1e-6 * np.abs(ref.Glr))
    assert np.all(np.abs(got.Dlr - ref.Dlr) <= 1e-6 * np.abs(ref.Dlr))
    for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
        e = per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes)
        print(f"  {p}: params rel {e:.2e}")
        assert e <= 1e-3
    if wl["mix_enable"]:
        stats = mixture.real_stats(S, data)
        # the ES step scores the generators the banded run trained (shared state)
        mu, s2 = mixture.generator_moments(S, got, stats["P"], gen)
        n_dec = 0
        for c in range(S.C):
            ks = S.nbr[c]
            cur = mixture.score(st.w[c], mu[ks], s2[ks], stats["mu_r"], stats["sd_r"])
            wp = mixture.propose(S, st.w[c], c, gen)
            new = None if wp is None else mixture.score(wp, mu[ks], s2[ks], stats["mu_r"], stats["sd_r"])
            kept_old = np.array_equal(got.w[c], st.w[c])
            if new is None or abs(new - cur) > 1e-4 * max(new, cur):
                n_dec += 1
                assert kept_old == (new is None or not new < cur), c
            if not kept_old:
                assert np.all(np.abs(got.w[c] - wp) <= 1e-6), c
        assert 4 * n_dec >= S.C
