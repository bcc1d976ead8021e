"""Edge cases of the MLP path on the GPU against the oracle: one-wide
networks and a batch of one on a 1x1 grid, the deepest networks the
configuration allows with tournaments of one, the largest batch, a zero
learning rate, and calls that do no work."""
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

CASES = {
    # every width 1, one sample per batch, the cell its own neighbourhood
    "unit_1x1_b1": dict(rows=1, cols=1, z_dim=1, x_dim=1, g_hidden=[1], d_hidden=[1], batch=1,
                        data=dict(kind="mnist_like", n=64)),
    # four hidden layers (the most the configuration takes), odd widths, tournaments of one
    "deep_2x2_t1": dict(rows=2, cols=2, z_dim=5, x_dim=29, g_hidden=[17, 9, 33, 70], d_hidden=[45, 3, 19, 66],
                        batch=13, tournament_size=1, g_hidden_act="lrelu", d_hidden_act="tanh",
                        data=dict(kind="mnist_like", n=500)),
    # the largest batch
    "batch2048_1x2": dict(rows=1, cols=2, z_dim=6, x_dim=40, g_hidden=[24], d_hidden=[20], batch=2048,
                          data=dict(kind="mnist_like", n=5000)),
    # a zero learning rate: Adam's moments move, the parameters do not
    "lr0_2x3": dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
                    lr0_g=0.0, lr0_d=0.0, lr_mutation=0, data=dict(kind="mnist_like", n=3000)),
}


def _setup(key):
    wl = synth.small_workload("mnist_mlp_3x3", **CASES[key])
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    if wl["lr0_g"] > 0:
        for s in range(2):
            coevo.train_step(S, st, data, 0, 30 + s)
    return wl, data, S, fp32_state(st)


def _close(a, b, rtol=1e-4):
    return np.all(np.abs(a - b) <= rtol * np.abs(b) + 1e-7)


@pytest.mark.parametrize("key", list(CASES))
def test_edge_generation_matches_oracle(key):
    wl, data, S, st = _setup(key)
    gen = 1
    print(f"[case] edges key={key}", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        got_eval = gg.eval(gen)
        ref_eval = coevo.evaluate(S, st, data, gen)
        for a, b in zip(got_eval, ref_eval):
            assert _close(a, b), np.max(np.abs(a - b))
        gsel, _ = gg.select(gen)
        _, _, ofg, ofd = ref_eval
        check_selection(S, gsel, ofg, ofd, gen)
        ref, _ = coevo.select_replace(S, st, ofg, ofd, gen, forced=gsel)
        gl = gg.train(gen, 0, 2)
        got = gg.get_state()
    ol = np.array([coevo.train_step(S, ref, data, gen, k) for k in range(2)])
    assert _close(gl[0], ol[0])
    assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
    for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
        assert per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes) <= 1e-3
        if wl["lr0_g"] == 0.0:
            assert np.array_equal(getattr(got, p + "p"), getattr(ref, p + "p"))
            assert per_tensor_rel(getattr(got, p + "m"), getattr(ref, p + "m"), sizes) <= 1e-3


def test_calls_without_work_leave_the_state():
    wl, data, S, st = _setup("deep_2x2_t1")
    print("[case] no-op calls", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        before = gg.save_blob()
        L.lipz_train_step(gg.g, 0, 5, 0)
        L.lipz_run_generations(gg.g, 3, 0, 4)
        assert gg.sync() == L.LIPZ_OK
        assert np.array_equal(gg.save_blob(), before)
