"""GPU parity of the NES trainer (gradient-free, antithetic estimate + Adam)
against the oracle, from an identical state.

What is compared, and why (tolerances from fp32 against fp64):
  * the critic loss at the unperturbed parameters, before any update: 1e-4;
  * the generator loss follows the critic's update, so it is recomputed by
    the oracle on the GPU's own updated critic (teacher forcing), 1e-4;
  * Adam's first moment after the step, per tensor 1e-3: it carries the NES
    estimate itself, a weighted sum of directions with weights F_k+ - F_k-
    (differences of fp32 losses, ~1e-2 apart for sigma = 1e-2);
  * parameters per tensor 1e-3, step counts bit-exact, Wasserstein critic
    parameters inside the clip bound.
"""
import numpy as np
import pytest

import synth
from oracle import coevo, nes

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("no GPU", allow_module_level=True)

from harness import GpuGrid, fp32_state, per_tensor_rel  # noqa: E402

RAGGED = dict(rows=2, cols=3, z_dim=7, x_dim=37, g_hidden=[33, 70], d_hidden=[45, 19], batch=19,
              data=dict(kind="mnist_like", n=3000))

CASES = {
    "mnist_3x3_nes": dict(name="mnist_mlp_3x3_nes", over=dict(nes_pairs=4)),
    "ragged_2x3_nes": dict(name="mnist_mlp_3x3_nes", over=dict(RAGGED, nes_pairs=9, nes_sigma=0.02)),
    "ragged_2x3_nes_wgan": dict(name="mnist_mlp_3x3_nes", over=dict(RAGGED, nes_pairs=3, loss="wasserstein",
                                                                     wgan_clip=0.05)),
}


def _setup(key):
    c = CASES[key]
    wl = synth.small_workload(c["name"], **dict(c["over"]))
    data = synth.make_dataset(wl["data"])
    data = np.ascontiguousarray(data[:, :wl["x_dim"]])
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    for s in range(2):  # warm Adam state and step counts
        coevo.train_step(S, st, data, 0, 50 + s)
    return wl, data, S, fp32_state(st)


def _close(a, b, wl, rtol=1e-4):
    atol = rtol * 1e-2 if wl.get("loss") == "wasserstein" else 0.0
    return np.all(np.abs(a - b) <= rtol * np.abs(b) + atol)


@pytest.mark.parametrize("key", list(CASES))
def test_nes_step_matches_oracle(key):
    wl, data, S, st = _setup(key)
    gen, step = 1, 3
    print(f"[case] nes-step key={key}", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        gl = gg.train(gen, step, 1)[0]
        got = gg.get_state()
    ref = st.copy()
    ol = nes.train_step(S, ref, data, gen, step)
    assert _close(gl[:, 0], ol[:, 0], wl), np.max(np.abs(gl[:, 0] - ol[:, 0]))
    lg = np.zeros(S.C)
    for c in range(S.C):
        _, _, z = coevo.sample(S, data, c, gen, step + 1)
        a = coevo.d_logits(S, got.Dp[c], coevo.g_forward(S, st.Gp[c], z)[1])[1]
        lg[c] = coevo.pair_losses(S, a, a)[1]
    assert _close(gl[:, 1], lg, wl), np.max(np.abs(gl[:, 1] - lg))
    assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
    if wl.get("loss") == "wasserstein":
        assert np.all(np.abs(got.Dp) <= np.float32(wl["wgan_clip"]))
    for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
        em = per_tensor_rel(getattr(got, p + "m"), getattr(ref, p + "m"), sizes)
        ep = per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes)
        print(f"  {p}: first moment rel {em:.2e}, params rel {ep:.2e}")
        assert em <= 1e-3 and ep <= 1e-3


def test_nes_generation_matches_oracle():
    """Evaluation, selection and three NES steps in one generation; the
    parameters after it per tensor."""
    wl, data, S, st = _setup("ragged_2x3_nes")
    gen = 2
    print("[case] nes-generation", flush=True)
    with GpuGrid(wl, data) as gg:
        gg.set_state(st)
        _, _, fg, fd = gg.eval(gen)
        gsel, _ = gg.select(gen)
        gg.train(gen, 0, 3)
        got = gg.get_state()
    _, _, ofg, ofd = coevo.evaluate(S, st, data, gen)
    ref, _ = coevo.select_replace(S, st, ofg, ofd, gen, forced=gsel)
    for s in range(3):
        nes.train_step(S, ref, data, gen, s)
    for p, sizes in (("G", S.g_sizes), ("D", S.d_sizes)):
        e = per_tensor_rel(getattr(got, p + "p"), getattr(ref, p + "p"), sizes)
        print(f"  {p}: params rel {e:.2e}")
        assert e <= 1e-3
    assert np.array_equal(got.Gt, ref.Gt) and np.array_equal(got.Dt, ref.Dt)
