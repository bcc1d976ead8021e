"""lipz_grid_create_static (the create that takes its workspace from the
library's static per-device array instead of the caller) against
lipz_grid_create on a caller workspace: the same configuration, state and
calls give bit-identical outputs and states, for two static grids in a row,
the second smaller than the first (the array keeps the first grid's
contents).  Also the refusals: a second live static grid on the device, a
configuration larger than the array, row bands."""
import numpy as np
import pytest

import synth
from oracle import coevo

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_1811_12843_amd as L  # noqa: E402
from harness import GpuGrid, fp32_state  # noqa: E402

FIRST = dict(name="mnist_mlp_4x4_mix",
             over=dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
                       mix_samples=77, mix_feat_dim=9, data=dict(kind="mnist_like", n=3000)))
SECOND = dict(name="ring8_mlp_2x2", over=dict(rows=1, cols=2, batch=16, data=dict(n=2048)))


def _case(c):
    wl = synth.small_workload(c["name"], **c["over"])
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    return wl, data


def _run(gg, wl, st0):
    """Evaluation, selection, three training steps and (if enabled) the mixture
    step of generation 1 from state st0; every output and the final state."""
    gg.set_state(st0)
    out = {}
    out["L"], out["Lg"], out["fg"], out["fd"] = gg.eval(1)
    out["sel"], out["lr"] = gg.select(1)
    out["losses"] = gg.train(1, 0, 3)
    if wl["mix_enable"]:
        out["w"], out["score"], out["acc"] = gg.mixture(1)
    out["blob"] = gg.save_blob()
    return out


def _compare(wl, data):
    S = coevo.Setup(wl, len(data))
    st0 = coevo.create(S)
    for s in range(2):  # a trained state
        coevo.train_step(S, st0, data, 0, 40 + s)
    st0 = fp32_state(st0)
    with GpuGrid(wl, data) as ref:
        want = _run(ref, wl, st0)
    with GpuGrid(wl, data, static_ws=True) as gg:
        got = _run(gg, wl, st0)
        # while this grid holds the array a second static create is refused
        with pytest.raises(L.LipzError) as e:
            L.lipz_grid_create_static(L.config_from_dict(wl), gg.data.data_ptr(), len(data), gg.stream)
        assert e.value.status == L.LIPZ_E_ORDER
    for k in want:
        assert np.array_equal(np.asarray(got[k]), np.asarray(want[k])), k
    # the step really changed the state, the outputs are finite
    assert np.all(np.isfinite(want["L"])) and np.all(np.isfinite(want["losses"]))


def test_static_workspace_matches_caller_workspace_twice():
    wl, data = _case(FIRST)
    nb1 = L.lipz_workspace_bytes(L.config_from_dict(wl), len(data))
    print(f"first: {wl['rows']}x{wl['cols']} grid, workspace {nb1} bytes", flush=True)
    _compare(wl, data)
    wl2, data2 = _case(SECOND)
    nb2 = L.lipz_workspace_bytes(L.config_from_dict(wl2), len(data2))
    print(f"second: {wl2['rows']}x{wl2['cols']} grid, workspace {nb2} bytes", flush=True)
    assert nb2 < nb1
    _compare(wl2, data2)


def test_static_workspace_refusals():
    wl = synth.workload("mnist_mlp_3x3")  # 214 MiB of workspace
    cfg = L.config_from_dict(wl)
    n = wl["data"]["n"]
    assert L.lipz_workspace_bytes(cfg, n) > L.LIPZ_STATIC_WORKSPACE_BYTES
    d = torch.zeros(16, wl["x_dim"], device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    with pytest.raises(L.LipzError) as e:
        L.lipz_grid_create_static(cfg, d.data_ptr(), 16, stream)
    assert e.value.status == L.LIPZ_E_WORKSPACE
    wl = synth.small_workload("mnist_mlp_3x3", rows=4, cols=2, z_dim=7, x_dim=37, g_hidden=[33], d_hidden=[45],
                              batch=19, bands=2, data=dict(kind="mnist_like", n=300))
    with pytest.raises(L.LipzError) as e:
        L.lipz_grid_create_static(L.config_from_dict(wl), d.data_ptr(), 16, stream)
    assert e.value.status == L.LIPZ_E_UNSUPPORTED
