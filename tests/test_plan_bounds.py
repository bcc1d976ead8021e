"""Host-only check of every launch plan (no GPU): each GEMM, convolution,
batch-norm, reduction and dot descriptor the library builds for a workload
stays inside the workspace and the dataset, with the kernels' own index
formulas (lipz_test_plan_bounds)."""
import pytest

import paper_1811_12843_amd as L
import synth

SMALL_DCGAN = [
    dict(rows=2, cols=2, img=(16, 16, 3), x_dim=768, z_dim=8, g_hidden=[32, 16], d_hidden=[16, 32], batch=5,
         data=dict(n=512, h=16, w=16)),
    dict(rows=3, cols=3, img=(32, 32, 3), x_dim=3072, z_dim=12, g_hidden=[64, 32, 16], d_hidden=[16, 32, 64],
         batch=6, data=dict(n=512, h=32, w=32)),
    dict(rows=1, cols=3, img=(8, 8, 1), x_dim=64, z_dim=5, g_hidden=[8], d_hidden=[12], batch=3,
         data=dict(n=100, h=8, w=8, c=1)),
]


@pytest.fixture(scope="module", autouse=True)
def _lib():
    try:
        L.load_library()
    except RuntimeError as e:  # pragma: no cover
        pytest.skip(str(e))


@pytest.mark.parametrize("name", sorted(synth.WORKLOADS))
def test_workload_plans_stay_in_bounds(name):
    wl = synth.workload(name)
    n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(wl), wl["data"]["n"])
    assert n_bad == 0, msg


@pytest.mark.parametrize("i", range(len(SMALL_DCGAN)))
def test_small_dcgan_plans_stay_in_bounds(i):
    wl = synth.small_workload("celeba_dcgan_4x4", **SMALL_DCGAN[i])
    n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(wl), wl["data"]["n"])
    assert n_bad == 0, msg


SMALL_NES = [
    dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19, nes_pairs=3,
         data=dict(kind="mnist_like", n=300)),
    dict(rows=1, cols=1, z_dim=3, x_dim=5, g_hidden=[6], d_hidden=[7], batch=2, nes_pairs=1,
         data=dict(kind="mnist_like", n=50)),
    dict(rows=2, cols=2, z_dim=9, x_dim=11, g_hidden=[13], d_hidden=[17, 3], batch=4, nes_pairs=64,
         loss="wasserstein", data=dict(kind="mnist_like", n=50)),
]


@pytest.mark.parametrize("i", range(len(SMALL_NES)))
def test_small_nes_plans_stay_in_bounds(i):
    """Parameter counts that are not multiples of 4, so a thread's four
    directions straddle two directions and the end of the stream."""
    for trainer in ("nes", "es"):
        wl = synth.small_workload("mnist_mlp_3x3_nes", trainer=trainer, **SMALL_NES[i])
        n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(wl), wl["data"]["n"])
        assert n_bad == 0, msg


SMALL_SUBPOP = [
    dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19, pop_size=2,
         elitism=1, data=dict(kind="mnist_like", n=300)),
    dict(rows=1, cols=1, z_dim=3, x_dim=5, g_hidden=[6], d_hidden=[7], batch=2, pop_size=4, elitism=1,
         tournament_size=5, data=dict(kind="mnist_like", n=50)),
    dict(rows=3, cols=2, z_dim=9, x_dim=70, g_hidden=[13, 8], d_hidden=[130], batch=5, pop_size=3,
         elitism=0, data=dict(kind="mnist_like", n=50)),
]


@pytest.mark.parametrize("i", range(len(SMALL_SUBPOP)))
@pytest.mark.parametrize("trainer", ["gradient", "nes", "es"])
def test_subpopulation_plans_stay_in_bounds(i, trainer):
    """Sub-populations (training per individual, evaluation over 5 s
    neighbourhood individuals, the re-evaluation of elitism)."""
    wl = synth.small_workload("mnist_mlp_3x3", trainer=trainer, nes_pairs=2, **SMALL_SUBPOP[i])
    n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(wl), wl["data"]["n"])
    assert n_bad == 0, msg


@pytest.mark.parametrize("over", [dict(rows=8, cols=3, bands=4), dict(rows=7, cols=2, bands=3, pop_size=2, elitism=1),
                                  dict(rows=5, cols=3, bands=5), dict(rows=8, cols=8, bands=8),
                                  dict(rows=4, cols=4, bands=2, mix_enable=1, mix_samples=200)])
def test_band_plans_stay_in_bounds(over):
    wl = synth.small_workload("mnist_mlp_3x3", z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
                              **over)
    n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(wl), wl["data"]["n"])
    assert n_bad == 0, msg
    for trainer in ("nes", "es"):
        n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(dict(wl, trainer=trainer, nes_pairs=3)),
                                             wl["data"]["n"])
        assert n_bad == 0, msg
    for bad in (dict(wl, bands=wl["rows"] + 1), dict(wl, bands=9)):
        assert L.lipz_workspace_bytes(L.config_from_dict(bad), wl["data"]["n"]) == 0


@pytest.mark.parametrize("over", [
    dict(rows=1, cols=1, z_dim=1, x_dim=1, g_hidden=[1], d_hidden=[1], batch=1, data=dict(n=64)),
    dict(rows=2, cols=2, z_dim=5, x_dim=29, g_hidden=[17, 9, 33, 70], d_hidden=[45, 3, 19, 66], batch=13),
    dict(rows=1, cols=2, z_dim=6, x_dim=40, g_hidden=[24], d_hidden=[20], batch=2048, data=dict(n=5000)),
])
def test_edge_plans_stay_in_bounds(over):
    """One-wide networks and a batch of one, four hidden layers, the largest batch."""
    wl = synth.small_workload("mnist_mlp_3x3", **over)
    n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(wl), wl["data"]["n"])
    assert n_bad == 0, msg


def test_invalid_dcgan_shapes_are_rejected():
    wl = synth.small_workload("celeba_dcgan_4x4", img=(48, 48, 3), x_dim=48 * 48 * 3)
    assert L.lipz_workspace_bytes(L.config_from_dict(wl), 100) == 0
    wl = synth.small_workload("celeba_dcgan_4x4", g_hidden=[512, 256, 128, 66])
    assert L.lipz_workspace_bytes(L.config_from_dict(wl), 100) == 0
    wl = synth.small_workload("celeba_dcgan_4x4", mix_enable=1)
    assert L.lipz_workspace_bytes(L.config_from_dict(wl), 100) == 0


def test_outputs_reaching_2_29_elements_are_rejected():
    """The GEMM epilogue addresses its output through buffer resources with
    32-bit byte offsets below 2^31: a batch of 512 rows of 2^20 generated
    values (2^29 elements, 2 GiB, in one problem's output) is not planned;
    one row fewer is."""
    base = dict(rows=1, cols=1, z_dim=4, x_dim=1 << 20, g_hidden=[8], d_hidden=[8], data=dict(n=64))
    for batch in (512, 2048):
        over = synth.small_workload("mnist_mlp_3x3", batch=batch, **base)
        assert L.lipz_workspace_bytes(L.config_from_dict(over), 64) == 0
        with pytest.raises(RuntimeError):
            L.lipz_test_plan_bounds(L.config_from_dict(over), 64)
    under = synth.small_workload("mnist_mlp_3x3", batch=511, **base)
    assert L.lipz_workspace_bytes(L.config_from_dict(under), 64) > 0
    n_bad, msg = L.lipz_test_plan_bounds(L.config_from_dict(under), 64)
    assert n_bad == 0, msg


@pytest.mark.parametrize("groups,nb", [
    ([0], 1), ([0], 7), ([0], 8), ([0], 256), ([0], 2176),
    ([0, 144], 400),            # short tiles then long ones
    ([0, 256], 2128), ([0, 1600], 2176), ([0, 3, 10], 13), ([0, 1, 2, 3], 4),
    ([0, 5, 11, 30], 47), ([0, 100, 101, 350], 357),
])
def test_tile_map_covers_every_tile_once_and_spreads_groups(groups, nb):
    """Block b runs on XCD b % 8.  The map is a permutation of the tiles; each
    group's tiles on one XCD are a contiguous run, and the XCDs' shares of a
    group differ by at most one tile."""
    t = L.lipz_test_tile_map(groups, nb)
    assert sorted(t) == list(range(nb))
    bounds = groups + [nb]
    for gi in range(len(groups)):
        lo, hi = bounds[gi], bounds[gi + 1]
        per = [[tt for b, tt in enumerate(t) if b % 8 == x and lo <= tt < hi] for x in range(8)]
        sizes = [len(p) for p in per]
        assert max(sizes) - min(sizes) <= 1, sizes
        for p in per:  # contiguous, in block order
            assert p == list(range(p[0], p[0] + len(p))) if p else True
        assert sum(sizes) == hi - lo


def test_tile_map_rejects_bad_groups():
    for groups, nb in [([1], 4), ([0, 0], 4), ([0, 5], 5), ([0, 1, 2, 3, 4], 9), ([], 3)]:
        with pytest.raises(RuntimeError):
            L.lipz_test_tile_map(groups, nb)
