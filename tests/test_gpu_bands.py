"""The row-band executor (lipz_run_generations with bands >= 2, the paper's
asynchronous cells scheduled by neighbour readiness) against the one-batch
schedule: the same generations give the same state bit for bit.

The one-batch schedule is itself checked against the oracle call by call
(tests/test_gpu_parity.py, tests/test_gpu_subpop.py); here it is also checked
against the entry points called one by one.
"""
import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_1811_12843_amd as L  # noqa: E402
from harness import GpuGrid  # noqa: E402

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
