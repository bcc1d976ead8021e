"""GPU parity of sub-populations (pop_size s > 1 individuals per role and
cell) and of the post-training re-evaluation with elitist replacement, against
the oracle, from identical states.

Tolerances as in the single-individual tests: losses and fitness 1e-4
relative; tournament decisions identical wherever the drawn individuals'
fitness margins are decisive (1e-4), else the GPU's choice is replayed;
parameters after training per tensor 1e-3.  The elitist truncation compares
2 s fitness values per cell and role: its decisions must equal the oracle's
unless two of those values lie within 1e-4 of each other, where the GPU's
choice is replayed.  The re-evaluation is checked on the GPU's own trained
individuals (the oracle re-scores them), so its fitness carries the
evaluation's tolerance, and the final state, copies of individuals on both
sides, is compared bit for bit.
"""
import numpy as np
import pytest

import synth
from oracle import coevo

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_1811_12843_amd as L  # noqa: E402
from harness import GpuGrid, check_selection, fp32_state, per_tensor_rel  # noqa: E402

RAGGED = dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
              data=dict(kind="mnist_like", n=3000))

CASES = {
    # two members per cell, every dimension ragged against the tiles
    "ragged_2x3_s2": dict(name="mnist_mlp_3x3", over=dict(RAGGED, pop_size=2, elitism=1, lr0_g=2e-3, lr0_d=2e-3)),
    # MNIST-shaped networks, three members, duplicate neighbours, generators ranked by their own loss
    "mnist_2x2_s3": dict(name="mnist_mlp_3x3", over=dict(rows=2, cols=2, batch=40, pop_size=3, elitism=1,
                                                          fitness_mode=1, data=dict(n=4000))),
    # one cell holding four members: 20 neighbourhood individuals, tournaments of 5
    "ring_1x1_s4": dict(name="ring8_mlp_2x2", over=dict(rows=1, cols=1, pop_size=4, elitism=1,
                                                         tournament_size=5, lr0_g=5e-3, lr0_d=5e-3)),
    # learning rates so large that training mostly spoils the members: the
    # previous ones come back (s = 2, and s = 1, where the better of the two stays)
    "ragged_2x3_s2_hot": dict(name="mnist_mlp_3x3", over=dict(RAGGED, pop_size=2, elitism=1, lr0_g=0.3, lr0_d=0.3)),
    "ragged_2x3_s1_hot": dict(name="mnist_mlp_3x3", over=dict(RAGGED, pop_size=1, elitism=1, lr0_g=0.3, lr0_d=0.3)),
}
BASE_CASES = ["ragged_2x3_s2", "mnist_2x2_s3", "ring_1x1_s4"]


def _setup(key):
    c = CASES[key]
    wl = synth.small_workload(c["name"], **dict(c["over"]))
    data = synth.make_dataset(wl["data"])
    if data.shape[1] != wl["x_dim"]:
        data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    for s in range(2):  # trained members, so they differ from their initialisation
        coevo.train_step(S, st, data, 0, 40 + s)
    return wl, data, S, fp32_state(st)


def _close(a, b, rtol=1e-4):
    return np.all(np.abs(a - b) <= rtol * np.abs(b))


@pytest.mark.parametrize("key", BASE_CASES)
def test_subpop_eval_matches_oracle(key):
    wl, data, S, st = _setup(key)
    print(f"[case] subpop-eval key={key}", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        for gen in (0, 3):
            got = gg.eval(gen)
            ref = coevo.evaluate(S, st, data, gen)
            for a, b in zip(got, ref):
                assert a.shape == b.shape and _close(a, b), np.max(np.abs(a - b) / np.abs(b))
        if S.C == 1:  # every slot is the cell itself: the 5 copies of a member score alike, bit for bit
            Lm = got[0][0].reshape(5, S.s, 5, S.s)
            assert all(np.array_equal(Lm[k], Lm[0]) and np.array_equal(Lm[:, :, k], Lm[:, :, 0]) for k in range(5))


@pytest.mark.parametrize("key", BASE_CASES)
def test_subpop_select_matches_oracle(key):
    wl, data, S, st = _setup(key)
    gen = 5
    print(f"[case] subpop-select key={key}", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        gg.eval(gen)
        gsel, glr = gg.select(gen)
        _, _, ofg, ofd = coevo.evaluate(S, st, data, gen)
        assert check_selection(S, gsel, ofg, ofd, gen) > 0
        new, _ = coevo.select_replace(S, st, ofg, ofd, gen, forced=gsel)
        got = gg.get_state()
        for f in ("Gp", "Gm", "Gv", "Dp", "Dm", "Dv", "Gt", "Dt"):
            assert np.array_equal(getattr(got, f), getattr(new, f)), f
        for f, col in (("Glr", 0), ("Dlr", 1)):
            assert np.all(np.abs(getattr(got, f) - getattr(new, f)) <= 1e-6 * np.abs(getattr(new, f)) + 1e-12)
            assert np.array_equal(glr[:, col], getattr(got, f))
        # forced sources: individual ids in [0, U)
        forced = np.stack([np.arange(S.U)[::-1], np.zeros(S.U, dtype=np.int64)], axis=1)
        sel2, _ = gg.select(gen + 1, forced=forced)
        assert np.array_equal(sel2, forced)
        assert gg.sync() == L.LIPZ_OK


@pytest.mark.parametrize("key", ["ragged_2x3_s2", "mnist_2x2_s3"])
def test_subpop_train_matches_oracle(key):
    wl, data, S, st = _setup(key)
    gen, step0, steps = 1, 4, 2
    print(f"[case] subpop-train key={key}", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        gl = gg.train(gen, step0, steps)
        got = gg.get_state()
    ref = st.copy()
    ol = np.array([coevo.train_step(S, ref, data, gen, step0 + k) for k in range(steps)])
    assert gl.shape == (steps, S.U, 2)
    assert _close(gl[0], ol[0]) and np.all(np.abs(gl - ol) <= 1e-3 * np.abs(ol))
    assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
    for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
        assert per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes) <= 1e-3


def _near_tie(f, tol=1e-4):
    f = np.sort(np.asarray(f, dtype=np.float64))
    return np.any(np.diff(f) <= tol * np.maximum(np.abs(f[1:]), np.abs(f[:-1])))


@pytest.mark.parametrize("key", list(CASES))
def test_elitist_replace_matches_oracle(key):
    """Evaluation, selection, three training steps and the elitist replacement
    on the GPU; the oracle re-scores the GPU's trained individuals against the
    previous neighbourhood and truncates."""
    wl, data, S, st = _setup(key)
    gen = 2
    print(f"[case] elitist key={key}", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        _, _, gfg, gfd = gg.eval(gen)
        gg.select(gen)
        gg.train(gen, 0, 3)
        trained = gg.get_state()
        gsrc, gf2g, gf2d = gg.elite(gen)
        got = gg.get_state()
        # a second replacement without a new evaluation and selection is out of order
        with pytest.raises(L.LipzError):
            gg.elite(gen)
    _, _, ofg, ofd = coevo.evaluate(S, st, data, gen)
    _, info = coevo.elitist_replace(S, st, trained, data, gen, ofg, ofd)
    assert _close(gf2g, info["fit_g2"]) and _close(gf2d, info["fit_d2"])
    s = S.s
    replayed = 0
    for c in range(S.C):
        for r, (fo, fn) in enumerate(((ofg[c, :s], info["fit_g2"][c]), (ofd[c, :s], info["fit_d2"][c]))):
            a, b = gsrc[c * s:(c + 1) * s, r], info["src"][c * s:(c + 1) * s, r]
            if not np.array_equal(a, b):
                assert _near_tie(np.concatenate([fo, fn])), (c, r, a, b, fo, fn)
                replayed += 1
    ref, _ = coevo.elitist_replace(S, st, trained, data, gen, ofg, ofd, forced=gsrc)
    for f in ("Gp", "Gm", "Gv", "Dp", "Dm", "Dv", "Gt", "Dt"):
        assert np.array_equal(getattr(got, f), getattr(ref, f).astype(getattr(got, f).dtype)), f
    for f in ("Glr", "Dlr"):
        assert np.array_equal(getattr(got, f), getattr(ref, f)), f
    restored = int(np.sum(gsrc >= 0))
    print(f"  previous members restored {restored} of {2 * S.U}, replayed {replayed}")
    if key.endswith("_hot"):
        assert restored > 0


def test_elitism_call_order():
    wl, data, S, st = _setup("ragged_2x3_s2")
    print("[case] elitism call order", flush=True)
    with GpuGrid(wl, data) as gg:
        with pytest.raises(L.LipzError):  # no evaluation yet
            gg.elite(0)
        gg.eval(0)
        with pytest.raises(L.LipzError):  # no selection after it
            gg.elite(0)
        gg.select(0)
        with pytest.raises(L.LipzError):  # another generation's minibatch
            gg.elite(1)
        gg.elite(0)
    wl0 = dict(wl, elitism=0)
    with GpuGrid(wl0, data) as gg:
        gg.eval(0)
        gg.select(0)
        with pytest.raises(L.LipzError):  # created without elitism
            gg.elite(0)
