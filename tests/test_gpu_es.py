"""GPU parity of the (1+lambda)-ES trainer against the oracle, from an
identical state.

The trainer's decisions are argmins over fp32 losses on the GPU and fp64
losses in the oracle.  Each decision is read back from the GPU's parameters:
the kept set is the oracle's candidate (parent or theta +- sigma eps_k)
nearest to them, at most a few fp32 roundings away, while every other
candidate is sigma |eps| away.  The decisions must agree wherever the
oracle's margin (the gap to the nearest other candidate's loss) exceeds 1e-4
relative; nearer ties may go either way, and the oracle then replays the
GPU's choice.  Compared after that: losses at the parents 1e-4 relative (the
generator's against the kept critic), parameters per tensor 1e-5 (a kept set
is one fp32 add away from the oracle's), Adam moments untouched and step
counts bit-exact, the Wasserstein critic inside its clip.
"""
import numpy as np
import pytest

import synth
from oracle import coevo, es, nes

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_1811_12843_amd as L  # noqa: E402
from harness import GpuGrid, fp32_state, per_tensor_rel  # noqa: E402

RAGGED = dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
              data=dict(kind="mnist_like", n=3000))

CASES = {
    "mnist_3x3_es": dict(name="mnist_mlp_3x3_es", over=dict(nes_pairs=4)),
    "ragged_2x3_es": dict(name="mnist_mlp_3x3_es", over=dict(RAGGED, nes_pairs=9, nes_sigma=0.02)),
    "ragged_2x3_es_wgan": dict(name="mnist_mlp_3x3_es", over=dict(RAGGED, nes_pairs=3, loss="wasserstein",
                                                                   wgan_clip=0.05)),
}


def _setup(key):
    c = CASES[key]
    wl = synth.small_workload(c["name"], **dict(c["over"]))
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    for s in range(2):  # a trained state, so the losses are not those of the initial networks
        coevo.train_step(S, st, data, 0, 50 + s)
    return wl, data, S, fp32_state(st)


def _kept(S, before, after, gen, step):
    """The GPU's choice per cell and role (0: D, 1: G), read from its parameters."""
    sigma = S.wl["nes_sigma"]
    q = np.zeros((S.C, 2), dtype=np.int64)
    for c in range(S.C):
        for r, (role, P) in enumerate((("D", "Dp"), ("G", "Gp"))):
            cand = es.candidates(getattr(before, P)[c], nes.directions(S, role, c, gen, step), sigma)
            if role == "D" and S.loss == "wasserstein":
                cand = np.clip(cand, -S.clip, S.clip)
            d = np.max(np.abs(cand - getattr(after, P)[c][None]), axis=1)
            q[c, r] = int(np.argmin(d))
            assert d[q[c, r]] < 1e-5 and np.sort(d)[1] > 1e-4, (c, role, np.sort(d)[:3])
    return q


def _step_and_compare(S, data, st, got, gl, gen, step, wl):
    """Check one GPU step (state st -> got, losses gl [C, 2]) against the oracle;
    returns the number of decisions replayed from the GPU."""
    info = {}
    es.train_step(S, st.copy(), data, gen, step, info=info)
    q = _kept(S, st, got, gen, step)
    f = np.abs(gl) + 1e-30
    loose = info["margin"] <= 1e-4 * f
    assert np.all((q == info["q"]) | loose), (q, info["q"], info["margin"])
    ref = st.copy()
    ol = es.train_step(S, ref, data, gen, step, forced=q)
    atol = 1e-6 if wl.get("loss") == "wasserstein" else 0.0
    assert np.all(np.abs(gl - ol) <= 1e-4 * np.abs(ol) + atol), np.max(np.abs(gl - ol))
    for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
        e = per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes)
        assert e <= 1e-5, (p, e)
        for f_ in (p + "m", p + "v"):
            assert np.array_equal(getattr(got, f_), getattr(st, f_)), f_
    assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
    if wl.get("loss") == "wasserstein":
        assert np.all(np.abs(got.Dp) <= np.float32(wl["wgan_clip"]))
    return int(np.sum(q != info["q"])), q


@pytest.mark.parametrize("key", list(CASES))
def test_es_step_matches_oracle(key):
    wl, data, S, st = _setup(key)
    gen, step = 1, 3
    print(f"[case] es-step key={key}", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        gl = gg.train(gen, step, 1)[0]
        got = gg.get_state()
    replayed, q = _step_and_compare(S, data, st, got, gl, gen, step, wl)
    moved = int(np.sum(q != 2 * wl["nes_pairs"]))
    print(f"  mutants kept {moved} of {2 * S.C}, near ties replayed {replayed}")
    assert moved > 0  # the step exercised the replacement, not only the parent's copy


def test_es_generation_matches_oracle():
    """Evaluation, selection and four ES steps in one call, against the same
    steps one call each (bitwise), each checked against the oracle."""
    wl, data, S, st = _setup("ragged_2x3_es")
    gen = 2
    print("[case] es-generation", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        gg.eval(gen)
        gg.select(gen)
        after_sel = gg.get_state()
        gl4 = gg.train(gen, 0, 4)
        got4 = gg.get_state()
        gg.set_state(after_sel)
        cur = after_sel
        for s in range(4):
            gl = gg.train(gen, s, 1)[0]
            nxt = gg.get_state()
            assert np.array_equal(gl, gl4[s])
            _step_and_compare(S, data, cur, nxt, gl, gen, s, wl)
            cur = nxt
    for f in ("Gp", "Dp", "Gt", "Dt"):
        assert np.array_equal(getattr(cur, f), getattr(got4, f)), f


@pytest.mark.parametrize("losses", [
    [np.nan, 1.0, 2.0, 3.0, 2.5],            # a NaN first mutant loses; the better later one is kept
    [np.nan, np.nan, np.nan, np.nan, 2.0],   # only NaN mutants: the parent stays
    [1.5, np.nan, 0.5, 0.5, np.nan],         # a NaN parent loses to the best finite mutant
    [np.nan] * 5,                            # all NaN: the parent stays
    [2.0, 1.0, 1.0, 3.0, 1.0],               # equal losses: the parent stays
])
def test_plus_selection_ranks_nan_last(losses):
    """The selection kernel on hand-made losses with NaN entries against the
    oracle's rule (NaN ranks as +infinity): the kept candidate's values land
    in the parameter row, bit for bit."""
    n, P, stride = 2, 37, 40
    f = np.array(losses, dtype=np.float32)
    g = np.random.default_rng(7)
    sets = g.normal(size=(1, 2 * n, stride)).astype(np.float32)
    parent = g.normal(size=(1, stride)).astype(np.float32)
    d_f = torch.from_numpy(f).cuda()
    d_s = torch.from_numpy(sets).cuda()
    d_p = torch.from_numpy(parent.copy()).cuda()
    L.lipz_test_es_select(torch.cuda.current_stream().cuda_stream, d_f.data_ptr(), d_s.data_ptr(), d_p.data_ptr(),
                          1, n, P, stride)
    torch.cuda.synchronize()
    w, _ = es.choose(f.astype(np.float64))
    expect = parent[0].copy()
    if w < 2 * n:
        expect[:P] = sets[0, w, :P]
    assert np.array_equal(d_p.cpu().numpy()[0], expect)
