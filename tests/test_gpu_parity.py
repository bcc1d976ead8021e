"""GPU parity: every C-ABI call against the oracle from an identical state
("teacher forcing": the oracle state is rounded to fp32, loaded into the
library, and both sides run one call from there).

Tolerances (from the arithmetic: fp32 accumulation over K <= 800 terms
against fp64, and Adam's first steps being ~ lr * sign(g)):
  losses and fitness        |gpu - oracle| <= 1e-4 |oracle| elementwise
  parameters after steps    per-tensor ||gpu - oracle|| / ||oracle|| <= 1e-3
  parameter updates         per-tensor relative error of (p_after - p_before) <= 5e-2
  decisions                 identical wherever the fitness margin > 1e-4 relative;
                            otherwise the GPU's choice is forced into the oracle
  copies, indices, counts   bit-exact
"""
import numpy as np
import pytest

import synth
from oracle import coevo, grid, mixture, mlp

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_1811_12843_amd as L  # noqa: E402
from harness import GpuGrid, check_mixture, check_selection, fp32_state, per_tensor_rel, rel_err  # noqa: E402

RTOL = 1e-4

# Small workload with every dimension ragged against the 64x64 tiles and 16-deep K slices.
RAGGED = dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
              data=dict(kind="mnist_like", n=3000))


def _data_for(wl):
    d = synth.make_dataset(wl["data"])
    if wl["x_dim"] != d.shape[1]:
        d = np.ascontiguousarray(d[:, :wl["x_dim"]])
    return d


def _workload(name, **kw):
    return synth.small_workload(name, **kw)


WORKLOADS = {
    "ring8_2x2": lambda: _workload("ring8_mlp_2x2"),
    "ragged_2x3": lambda: _workload("mnist_mlp_3x3", **RAGGED),
    "ragged_lin_relu": lambda: _workload("mnist_mlp_3x3", **dict(RAGGED, g_out_act="linear",
                                                                 d_hidden_act="relu", g_hidden_act="lrelu",
                                                                 rows=1, cols=3, batch=70)),
    "mnist_3x3": lambda: _workload("mnist_mlp_3x3"),
    "mnist_4x4_mix": lambda: _workload("mnist_mlp_4x4_mix"),
    "mnist_8x8": lambda: _workload("mnist_mlp_8x8"),
    # generators ranked by their own non-saturating loss (fitness_mode 1)
    "mnist_3x3_fm1": lambda: _workload("mnist_mlp_3x3", fitness_mode=1),
    # the Wasserstein trainer: linear critic, clipped critic weights
    "mnist_3x3_wgan": lambda: _workload("mnist_mlp_3x3", loss="wasserstein", wgan_clip=0.01),
    "ragged_2x3_wgan": lambda: _workload("mnist_mlp_3x3", **dict(RAGGED, loss="wasserstein", wgan_clip=0.05)),
}


def _close(a, b, wl, rtol=RTOL):
    """|a - b| <= rtol |b|; the Wasserstein losses are differences of two
    means that can nearly cancel, so they also get an absolute term of
    rtol * 1e-2 (critic outputs are O(1e-2 .. 1) here)."""
    atol = rtol * 1e-2 if wl.get("loss") == "wasserstein" else 0.0
    return np.all(np.abs(a - b) <= rtol * np.abs(b) + atol)

_DATA_CACHE = {}


def _setup(key):
    wl = WORKLOADS[key]()
    dk = (wl["data"]["kind"], wl["data"]["n"], wl["x_dim"])
    if dk not in _DATA_CACHE:
        _DATA_CACHE[dk] = _data_for(wl)
    data = _DATA_CACHE[dk]
    S = coevo.Setup(wl, len(data))
    return wl, data, S


def _warm_state(S, data, steps=2, gen=0):
    """An oracle state with non-zero Adam moments and step counts."""
    st = coevo.create(S)
    for s in range(steps):
        coevo.train_step(S, st, data, gen, 50 + s)
    return fp32_state(st)


def _print_case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


# ---------------------------------------------------------------------------
def test_gemm_kernel_against_matmul():
    """The grouped MFMA GEMM on one problem, every operand layout and epilogue,
    against an fp64 matrix product (the plain definition)."""
    g = np.random.default_rng(0)
    dev = "cuda"
    desc = torch.zeros(256, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream().cuda_stream
    # (37, 52, 600) and (200, 256, 784) reach the wave-split kernel (K >= 512) with
    # ragged M, N and K tails; (37, 53, 19) is unaligned and takes the generic kernel.
    # The depths give the register-staged kernel 1 to 32 slices of 32 (its K loop
    # drains 1, 2 or 3 slices, with and without a steady-state pass before) and
    # the wave-split kernel (variants 2, 6) waves with 0 to 16 k blocks of 16,
    # a partial last block among them
    shapes = [(1, 1, 1), (64, 64, 16), (37, 53, 19), (129, 65, 33), (100, 256, 64), (200, 256, 784),
              (257, 784, 100), (37, 52, 600), (100, 96, 200), (40, 8, 1000), (44, 72, 96), (36, 132, 148)]
    for (M, N, K), tile_rows in [(s, tr) for s in shapes for tr in (32, 64)]:
        for a_trans in (0, 1):
            for b_trans in (0, 1):
                lda, ldb = (M if a_trans else K), (K if b_trans else N)
                aligned = lda % 4 == 0 and ldb % 4 == 0 and not (a_trans and b_trans)
                # variant 0: the library's choice; 1, 2: each aligned kernel (register-staged,
                # wave-split) on the same problem; + 4: the same with write-back stores
                variants = (0, 1, 2, 4, 5, 6) if aligned else (0, 4)
                for variant, (epi, act) in [(v, e) for v in variants
                                            for e in ((0, 0), (1, 1), (1, 2), (1, 3), (2, 2), (2, 3))]:
                    _print_case("gemm", M=M, N=N, K=K, at=a_trans, bt=b_trans, epi=epi, act=act,
                                tile_rows=tile_rows, variant=variant)
                    A = g.normal(size=(M, K)).astype(np.float32)
                    Bm = g.normal(size=(K, N)).astype(np.float32)
                    bias = g.normal(size=N).astype(np.float32)
                    aux = np.tanh(g.normal(size=(M, N))).astype(np.float32)
                    dA = torch.from_numpy(np.ascontiguousarray(A.T if a_trans else A)).to(dev)
                    dB = torch.from_numpy(np.ascontiguousarray(Bm.T if b_trans else Bm)).to(dev)
                    dC = torch.full((M, N), 7.0, device=dev)
                    db = torch.from_numpy(bias).to(dev)
                    daux = torch.from_numpy(aux).to(dev)
                    L.lipz_test_gemm(stream, desc.data_ptr(), M, N, K, dA.data_ptr(),
                                     M if a_trans else K, a_trans, -1, dB.data_ptr(),
                                     K if b_trans else N, b_trans, dC.data_ptr(), N, epi, act, 0.2,
                                     d_bias=db.data_ptr(), d_aux=daux.data_ptr(), tile_rows=tile_rows,
                                     variant=variant)
                    torch.cuda.synchronize()
                    acc = A.astype(np.float64) @ Bm.astype(np.float64)
                    scale = np.abs(A).astype(np.float64) @ np.abs(Bm).astype(np.float64)
                    if epi == 0:
                        ref = acc
                    elif epi == 1:
                        x = acc + bias
                        ref = mlp.act(["linear", "relu", "lrelu", "tanh"][act], x, 0.2)
                        scale = scale + np.abs(bias)
                    else:
                        y = aux.astype(np.float64)
                        d = {2: np.where(y > 0, 1.0, 0.2), 3: 1 - y * y}[act]
                        ref = acc * d
                        scale = scale * np.abs(d)
                    out = dC.cpu().numpy()
                    assert np.all(np.abs(out - ref) <= 3e-5 * scale + 1e-6), (M, N, K, a_trans, b_trans, epi,
                                                                              variant)


def test_gemm_weight_gradient_with_bias_row_and_adam():
    """[X | 1]^T dY accumulated over the batch and applied by the fused Adam epilogue."""
    g = np.random.default_rng(1)
    dev = "cuda"
    desc = torch.zeros(256, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream().cuda_stream
    cases = [(s, tr, v) for s in [(200, 784, 256), (100, 256, 784), (19, 37, 45), (64, 2, 64), (100, 64, 256),
                                  (520, 72, 36), (100, 256, 256)]
             for tr in (32, 64) for v in ((0, 1, 2, 4, 5, 6) if s[1] % 4 == 0 and s[2] % 4 == 0 else (0, 4))]
    for (rows, fi, fo), tile_rows, variant in cases:
        _print_case("wgrad_adam", rows=rows, fi=fi, fo=fo, tile_rows=tile_rows, variant=variant)
        X = g.normal(size=(rows, fi)).astype(np.float32)
        dY = (g.normal(size=(rows, fo)) * 1e-2).astype(np.float32)
        P0 = g.normal(size=(fi + 1, fo)).astype(np.float32)
        m0 = (g.normal(size=(fi + 1, fo)) * 1e-3).astype(np.float32)
        v0 = (np.abs(g.normal(size=(fi + 1, fo))) * 1e-5).astype(np.float32)
        t0, step_local, lr = 7, 2, 3e-4
        dP = torch.from_numpy(P0.copy()).to(dev)
        dm = torch.from_numpy(m0.copy()).to(dev)
        dv = torch.from_numpy(v0.copy()).to(dev)
        dX = torch.from_numpy(X).to(dev)
        ddY = torch.from_numpy(dY).to(dev)
        dlr = torch.tensor([lr], dtype=torch.float32, device=dev)
        dt = torch.tensor([t0], dtype=torch.int32, device=dev)
        L.lipz_test_gemm(stream, desc.data_ptr(), fi + 1, fo, rows, dX.data_ptr(), fi, 1, fi,
                         ddY.data_ptr(), fo, 0, dP.data_ptr(), fo, 3, 0, 0.2, d_m=dm.data_ptr(),
                         d_v=dv.data_ptr(), d_lr=dlr.data_ptr(), d_t=dt.data_ptr(), step_local=step_local,
                         tile_rows=tile_rows, variant=variant)
        torch.cuda.synchronize()
        Xe = np.concatenate([X, np.ones((rows, 1), np.float32)], axis=1).astype(np.float64)
        grad = Xe.T @ dY.astype(np.float64)
        S = coevo.Setup(synth.workload("mnist_mlp_3x3"), 10)
        p, m, v = P0.astype(np.float64), m0.astype(np.float64), v0.astype(np.float64)
        coevo.adam(S, p, m, v, t0 + step_local, lr, grad)
        assert rel_err(dm.cpu().numpy(), m) < 1e-5
        assert rel_err(dv.cpu().numpy(), v) < 1e-4
        assert rel_err(dP.cpu().numpy() - P0, p - P0) < 1e-3
        assert rel_err(dP.cpu().numpy(), p) < 1e-6


# ---------------------------------------------------------------------------
@pytest.mark.parametrize("key", ["ring8_2x2", "ragged_2x3", "mnist_4x4_mix"])
def test_create_matches_oracle_init(key):
    wl, data, S = _setup(key)
    _print_case("create", key=key)
    with GpuGrid(wl, data) as gg:
        assert gg.sync() == L.LIPZ_OK
        assert np.array_equal(np.array(L.lipz_get_neighbors(gg.g, S.C)), grid.neighbours(wl["rows"], wl["cols"]))
        for role, sizes in ((L.LIPZ_ROLE_G, S.g_sizes), (L.LIPZ_ROLE_D, S.d_sizes)):
            assert L.lipz_param_layout(gg.g, role) == [tuple(x) for x in mlp.layout(sizes)[0]]
        got = gg.get_state()
        ref = fp32_state(coevo.create(S))
        for f in ("Gp", "Dp"):
            a, b = getattr(got, f), getattr(ref, f)
            ulp = np.spacing(np.abs(b).astype(np.float32)).astype(np.float64)
            assert np.all(np.abs(a - b) <= ulp), f
        for f in ("Gm", "Gv", "Dm", "Dv", "Gt", "Dt", "Glr", "Dlr", "w"):
            assert np.array_equal(getattr(got, f), getattr(ref, f)), f


@pytest.mark.parametrize("key", ["ring8_2x2", "ragged_2x3", "ragged_lin_relu", "mnist_3x3", "mnist_4x4_mix",
                                 "mnist_3x3_fm1", "mnist_3x3_wgan", "ragged_2x3_wgan"])
def test_eval_matches_oracle(key):
    wl, data, S = _setup(key)
    st = _warm_state(S, data, steps=1)
    _print_case("eval", key=key)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        for gen in (0, 3):
            Lm, Lg, fg, fd = gg.eval(gen)
            oL, oLg, ofg, ofd = coevo.evaluate(S, st, data, gen)
            for a, b in ((Lm, oL), (Lg, oLg), (fg, ofg), (fd, ofd)):
                assert _close(a, b, wl), np.max(np.abs(a - b) / np.abs(b))
            if wl["rows"] == 2 and wl["cols"] == 2:
                # duplicate neighbours (N == S, W == E) are bit-identical on the GPU too
                assert np.array_equal(Lm[:, 1], Lm[:, 2]) and np.array_equal(Lm[:, :, 3], Lm[:, :, 4])


@pytest.mark.parametrize("key", ["ring8_2x2", "ragged_2x3", "mnist_4x4_mix", "mnist_3x3_fm1", "mnist_3x3_wgan"])
def test_select_replace_matches_oracle(key):
    wl, data, S = _setup(key)
    st = _warm_state(S, data, steps=2)
    gen = 5
    _print_case("select", key=key)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        gg.eval(gen)
        gsel, glr = gg.select(gen)
        _, _, ofg, ofd = coevo.evaluate(S, st, data, gen)
        assert check_selection(S, gsel, ofg, ofd, gen) > 0
        new, osel = coevo.select_replace(S, st, ofg, ofd, gen, forced=gsel)
        got = gg.get_state()
        for f in ("Gp", "Gm", "Gv", "Dp", "Dm", "Dv", "Gt", "Dt", "w"):
            assert np.array_equal(getattr(got, f), getattr(new, f)), f
        for f, col in (("Glr", 0), ("Dlr", 1)):
            assert np.all(np.abs(getattr(got, f) - getattr(new, f)) <= 1e-6 * np.abs(getattr(new, f)) + 1e-12)
            assert np.array_equal(glr[:, col], getattr(got, f))
        # forced selection bypasses the tournament
        forced = np.stack([np.arange(S.C)[::-1], np.zeros(S.C, dtype=np.int64)], axis=1)
        sel2, _ = gg.select(gen + 1, forced=forced)
        assert np.array_equal(sel2, forced)


@pytest.mark.parametrize("key,steps", [("ring8_2x2", 3), ("ragged_2x3", 3), ("ragged_lin_relu", 2),
                                       ("mnist_3x3", 2), ("mnist_4x4_mix", 1)])
def test_train_step_matches_oracle(key, steps):
    wl, data, S = _setup(key)
    st = _warm_state(S, data, steps=2)
    gen, step0 = 1, 4
    _print_case("train", key=key, steps=steps)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        glosses = gg.train(gen, step0, steps)
        ref = st.copy()
        olosses = np.array([coevo.train_step(S, ref, data, gen, step0 + k) for k in range(steps)])
        got = gg.get_state()
        assert np.all(np.abs(glosses[0] - olosses[0]) <= RTOL * np.abs(olosses[0]))
        assert np.all(np.abs(glosses - olosses) <= 1e-3 * np.abs(olosses))
        assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
        for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
            e = per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes)
            du = per_tensor_rel(getattr(got, p + "p") - getattr(st, p + "p"),
                                getattr(ref, p + "p") - getattr(st, p + "p"), sizes)
            print(f"  {p}: params rel {e:.2e}, updates rel {du:.2e}")
            assert e <= 1e-3 and du <= 5e-2


@pytest.mark.parametrize("key", ["mnist_3x3_wgan", "ragged_2x3_wgan"])
def test_wasserstein_train_step_matches_oracle(key):
    """One Wasserstein step from an identical state.  The critic loss comes
    before any update and must agree to 1e-4.  The generator loss is taken
    after the critic's Adam step and clip: Adam's first steps move a weight
    by about lr whatever the size of its gradient, so a weight whose gradient
    is near zero can step the other way in fp32 than in fp64, and one output
    weight of the critic moves -mean D(fake) (~1e-2 here) by ~1e-5.  The
    generator loss is therefore checked with the GPU's own updated critic
    (teacher forcing), and the parameters per tensor as in the other tests."""
    wl, data, S = _setup(key)
    st = _warm_state(S, data, steps=2)
    gen, step0 = 1, 4
    _print_case("train-wgan", key=key)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        glosses = gg.train(gen, step0, 1)[0]
        got = gg.get_state()
        ref = st.copy()
        olosses = coevo.train_step(S, ref, data, gen, step0)
        assert _close(glosses[:, 0], olosses[:, 0], wl)
        lg = np.zeros(S.C)
        for c in range(S.C):
            _, _, z = coevo.sample(S, data, c, gen, step0 + 1)
            xf = coevo.g_forward(S, st.Gp[c], z)[1]
            lg[c] = -coevo.d_logits(S, got.Dp[c], xf)[1].mean()
        assert _close(glosses[:, 1], lg, wl)
        assert np.all(np.abs(got.Dp) <= np.float32(wl["wgan_clip"]))
        assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
        for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
            e = per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes)
            print(f"  {p}: params rel {e:.2e}")
            assert e <= 1e-3
        # the same from the state after one step, three more steps in one call
        gg.set_state(fp32_state(ref))
        gg.train(gen, step0 + 1, 3)
        got = gg.get_state()
        for k in range(3):
            coevo.train_step(S, ref, data, gen, step0 + 1 + k)
        for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
            assert per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes) <= 1e-3


def _generation_parity(key, **over):
    wl, data, S = _setup(key)
    wl.update(over)
    S = coevo.Setup(wl, len(data))
    st = _warm_state(S, data, steps=1)
    gen = 2
    stats = mixture.real_stats(S, data) if wl["mix_enable"] else None
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        Lm, _, fg, fd = gg.eval(gen)
        oL, _, ofg, ofd = coevo.evaluate(S, st, data, gen)
        assert _close(Lm, oL, wl)
        gsel, _ = gg.select(gen)
        check_selection(S, gsel, ofg, ofd, gen)
        ref, _ = coevo.select_replace(S, st, ofg, ofd, gen, forced=gsel)
        glosses = gg.train(gen, 0, wl["steps"])
        olosses = np.array([coevo.train_step(S, ref, data, gen, s) for s in range(wl["steps"])])
        if wl.get("loss") == "wasserstein":
            # losses after critic updates are checked with teacher forcing in
            # test_wasserstein_train_step_matches_oracle; here the first critic loss
            assert _close(glosses[0, :, 0], olosses[0, :, 0], wl)
        else:
            assert np.all(np.abs(glosses - olosses) <= 1e-3 * np.abs(olosses) + 1e-5)
        got = gg.get_state()
        for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
            assert per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes) <= 1e-3
        if wl["mix_enable"]:
            w, sc, acc = gg.mixture(gen)
            check_mixture(S, fp32_state(got), stats, gen, w, sc, acc)


def test_generation_ring8_2x2_full():
    _print_case("generation", key="ring8_2x2")
    _generation_parity("ring8_2x2")


def test_generation_mnist_4x4_mix_short():
    _print_case("generation", key="mnist_4x4_mix")
    _generation_parity("mnist_4x4_mix", steps=3)


def test_generation_wasserstein_3x3_short():
    _print_case("generation", key="mnist_3x3_wgan")
    _generation_parity("mnist_3x3_wgan", steps=5)


@pytest.mark.parametrize("key,n_steps", [("mnist_3x3", None), ("mnist_4x4_mix", None), ("mnist_8x8", None)])
def test_generation_full_length_each_step(key, n_steps):
    """A whole generation at the workload's own length (100 training steps):
    evaluation and selection, then every training step on the GPU from the
    state the GPU reached, the oracle taking the same step from that state;
    per step losses 1e-4, parameters 1e-3 and their updates 5e-2; then the
    mixture update from the GPU's final state.

    Left to run free for 100 steps the two sides part by more than 1e-3 (the
    4x4 grid: 5e-3 in D's parameters), because the GAN dynamics amplify every
    rounding: the oracle parts nearly as far from a copy of itself whose state
    is rounded to fp32 after each step (the 4x4 grid: 1.7e-3 in G's
    parameters).  So the steps are compared from a shared state.  The 8x8
    grid (64 cells) too runs its whole generation."""
    wl, data, S = _setup(key)
    st = _warm_state(S, data, steps=1)
    gen = 2
    steps = n_steps or wl["steps"]
    _print_case("generation-each-step", key=key, steps=steps)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        gg.eval(gen)
        _, _, ofg, ofd = coevo.evaluate(S, st, data, gen)
        gsel, _ = gg.select(gen)
        check_selection(S, gsel, ofg, ofd, gen)
        ref, _ = coevo.select_replace(S, st, ofg, ofd, gen, forced=gsel)
        cur = gg.get_state()
        for f in ("Gp", "Gm", "Gv", "Dp", "Dm", "Dv", "Gt", "Dt"):
            assert np.array_equal(getattr(cur, f), getattr(ref, f)), f
        worst = dict(loss=0.0, G=0.0, D=0.0, dG=0.0, dD=0.0)
        for s in range(steps):
            gl = gg.train(gen, s, 1)[0]
            nxt = gg.get_state()
            ref = cur.copy()
            ol = coevo.train_step(S, ref, data, gen, s)
            e = float(np.max(np.abs(gl - ol) / np.abs(ol)))
            assert e <= RTOL, (s, e)
            worst["loss"] = max(worst["loss"], e)
            assert np.array_equal(nxt.Gt, ref.Gt) and np.array_equal(nxt.Dt, ref.Dt)
            for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
                e = per_tensor_rel(getattr(nxt, p + "p"), getattr(ref, p + "p"), sizes)
                du = per_tensor_rel(getattr(nxt, p + "p") - getattr(cur, p + "p"),
                                    getattr(ref, p + "p") - getattr(cur, p + "p"), sizes)
                assert e <= 1e-3 and du <= 5e-2, (s, p, e, du)
                worst[p], worst["d" + p] = max(worst[p], e), max(worst["d" + p], du)
            cur = nxt
        print("  worst over the steps: " + ", ".join(f"{k} {v:.2e}" for k, v in worst.items()))
        if wl["mix_enable"]:
            stats = mixture.real_stats(S, data)
            w, sc, acc = gg.mixture(gen)
            assert check_mixture(S, cur, stats, gen, w, sc, acc) > 0


@pytest.mark.parametrize("key", ["ragged_2x3", "mnist_4x4_mix"])
def test_mixture_matches_oracle(key):
    """Two mixture steps from random simplex weights: decisions, kept scores
    (1e-4 relative) and weights wherever the oracle's score margin exceeds
    1e-4; at least a quarter of the cells must be decisive."""
    wl, data, S = _setup(key)
    wl = dict(wl, mix_enable=1, mix_samples=1024 if key == "mnist_4x4_mix" else 77, mix_feat_dim=64 if key == "mnist_4x4_mix" else 9)
    S = coevo.Setup(wl, len(data))
    st = _warm_state(S, data, steps=1)
    g0 = np.random.default_rng(0)
    st.w = fp32_state(coevo.State(**{**{f: getattr(st, f) for f in coevo.State.FIELDS},
                                     "w": g0.dirichlet(np.ones(5), size=S.C)})).w
    stats = mixture.real_stats(S, data)
    _print_case("mixture", key=key)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        for gen in (0, 1):
            w, sc, acc = gg.mixture(gen)
            n_dec = check_mixture(S, st, stats, gen, w, sc, acc)
            print(f"  gen {gen}: {n_dec} of {S.C} cells decisive, {int(acc.sum())} accepted")
            assert 4 * n_dec >= S.C
            st.w = w.astype(np.float64)


def test_mixture_large_grid_many_features():
    """C x F = 1024 x 4096 > 2^21 feature moments (a 32x32 grid with 4096
    features, tiny networks): every cell's moments are formed and its ES step
    matches the oracle."""
    wl = synth.small_workload("mnist_mlp_4x4_mix", rows=32, cols=32, z_dim=4, x_dim=16, g_hidden=[8],
                              d_hidden=[8], batch=4, mix_samples=8, mix_feat_dim=4096,
                              data=dict(kind="mnist_like", n=256))
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    st = fp32_state(coevo.create(S))
    g0 = np.random.default_rng(1)
    st.w = g0.dirichlet(np.ones(5), size=S.C).astype(np.float32).astype(np.float64)
    stats = mixture.real_stats(S, data)
    _print_case("mixture-32x32-F4096")
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        w, sc, acc = gg.mixture(0)
        n_dec = check_mixture(S, st, stats, 0, w, sc, acc)
        print(f"  {n_dec} of {S.C} cells decisive, {int(acc.sum())} accepted")
        assert 4 * n_dec >= S.C


def test_full_size_8x8_eval_and_one_step():
    """The largest MLP grid (64 cells, 1600 pairings) at full size."""
    wl = synth.workload("mnist_mlp_8x8")
    dk = ("mnist_like", 60000, 784)
    if dk not in _DATA_CACHE:
        _DATA_CACHE[dk] = synth.make_dataset(wl["data"])
    data = _DATA_CACHE[dk]
    S = coevo.Setup(wl, len(data))
    st = fp32_state(coevo.create(S))
    _print_case("full_8x8")
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        Lm, _, _, _ = gg.eval(0)
        oL, _, _, _ = coevo.evaluate(S, st, data, 0)
        assert np.all(np.abs(Lm - oL) <= RTOL * np.abs(oL))
        gl = gg.train(0, 0, 1)
        ref = st.copy()
        ol = coevo.train_step(S, ref, data, 0, 0)
        assert np.all(np.abs(gl[0] - ol) <= RTOL * np.abs(ol))
        got = gg.get_state()
        for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
            assert per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes) <= 1e-3


# ---------------------------------------------------------------------------
def test_determinism_bitwise():
    wl, data, S = _setup("ragged_2x3")
    st = _warm_state(S, data, steps=1)
    outs = []
    _print_case("determinism")
    with GpuGrid(wl, data) as gg:
        for _ in range(2):
            gg.set_state(st)
            e = gg.eval(1)
            s = gg.select(1)
            l = gg.train(1, 0, 3)
            outs.append((e, s, l, gg.save_blob()))
    for a, b in zip(outs[0][0], outs[1][0]):
        assert np.array_equal(a, b)
    assert np.array_equal(outs[0][1][0], outs[1][1][0])
    assert np.array_equal(outs[0][2], outs[1][2])
    assert np.array_equal(outs[0][3], outs[1][3])


@pytest.mark.filterwarnings("ignore:invalid value encountered in logaddexp:RuntimeWarning")
def test_nonfinite_individual_loses_and_is_flagged():
    """A collapsed (NaN) discriminator sorts as +inf and is replaced by a
    neighbour's winner; the sticky non-finite flag is reported by lipz_sync."""
    wl, data, S = _setup("ragged_2x3")
    st = _warm_state(S, data, steps=1)
    st.Dp[2, :10] = np.nan
    _print_case("nonfinite")
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        Lm, Lg, fg, fd = gg.eval(0)
        assert gg.sync() == L.LIPZ_E_NONFINITE
        oL, _, ofg, ofd = coevo.evaluate(S, st, data, 0)
        assert np.array_equal(np.isnan(Lm), np.isnan(oL))
        assert np.array_equal(np.isnan(fd), np.isnan(ofd))
        gsel, _ = gg.select(0)
        check_selection(S, gsel, ofg, ofd, 0)
        for c in range(S.C):
            drawn = coevo.tournament_draw(S, c, 0, "TOURN_D")
            if any(not np.isnan(ofd[c, k]) for k in drawn):
                assert gsel[c, 1] != 2


def test_call_order_and_argument_errors():
    wl, data, S = _setup("ragged_2x3")
    _print_case("errors")
    with GpuGrid(wl, data) as gg:
        with pytest.raises(L.LipzError) as e:
            L.lipz_select_replace(gg.g, 0)
        assert e.value.status == L.LIPZ_E_ORDER
        with pytest.raises(L.LipzError) as e:
            L.lipz_mixture_update(gg.g, 0)
        assert e.value.status == L.LIPZ_E_ORDER
        with pytest.raises(L.LipzError) as e:
            L.lipz_eval_neighborhoods(gg.g, 70000)
        assert e.value.status == L.LIPZ_E_INVAL
        with pytest.raises(L.LipzError) as e:
            L.lipz_train_step(gg.g, 0, 65535, 1)
        assert e.value.status == L.LIPZ_E_INVAL
        gg.eval(0)
        gg.select(0)
        with pytest.raises(L.LipzError) as e:  # the fitness is stale after a replacement
            L.lipz_select_replace(gg.g, 0)
        assert e.value.status == L.LIPZ_E_ORDER
        assert gg.sync() == L.LIPZ_OK


@pytest.mark.parametrize("key", ["ring8_2x2", "ragged_2x3", "mnist_4x4_mix"])
def test_train_calls_split_anywhere_give_the_same_state(key):
    """Steps 3..9 of a generation in one call, in calls of 1, 2, 3 and 1 steps,
    in calls of 2 and 5 steps without the loss output: the state after them
    is bit for bit the same.  A step's minibatch is drawn by the call's first
    launch (the call's first step) or, one step ahead, inside a launch of the
    step before, into the minibatch buffer of the step's parity; a call may
    start at an odd or an even step."""
    wl, data, S = _setup(key)
    st = _warm_state(S, data, steps=1)
    gen = 2
    _print_case("train-split", key=key)
    with GpuGrid(wl, data) as gg:
        blobs = []
        for plan, with_losses in (([(3, 7)], True), ([(3, 1), (4, 2), (6, 3), (9, 1)], True),
                                  ([(3, 2), (5, 5)], False)):
            gg.set_state(st)
            for step0, n in plan:
                if with_losses:
                    gg.train(gen, step0, n)
                else:
                    L.lipz_train_step(gg.g, gen, step0, n, None)
                    gg.sync()
            blobs.append(gg.save_blob())
        assert not np.array_equal(blobs[0], _blob_of(gg, st))
        for b in blobs[1:]:
            assert np.array_equal(b, blobs[0])


def _blob_of(gg, st):
    gg.set_state(st)
    return gg.save_blob()
