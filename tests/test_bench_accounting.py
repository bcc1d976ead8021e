"""The benchmark's algorithmic FLOP count (the numerator of every matrix-core
fraction it reports) against the per-sample multiply-add counts and the
per-generation totals worked out by hand from the layer shapes of each
workload (2 FLOP per multiply-add, bias terms excluded)."""
import pytest

import bench
import synth


def test_mlp_multiply_adds_per_sample():
    wl = synth.workload("mnist_mlp_4x4_mix")
    g, g_first, d, d_first = bench.macs_per_sample(wl)
    # G 64-256-256-784, D 784-256-256-1
    assert (g, g_first) == (64 * 256 + 256 * 256 + 256 * 784, 64 * 256) == (282_624, 16_384)
    assert (d, d_first) == (784 * 256 + 256 * 256 + 256, 784 * 256) == (266_496, 200_704)


def test_training_step_multiply_adds():
    """Per sample: the D step is G's forward, D's forward and weight gradients
    on the 2B rows and D's input gradients below its first layer (1,480,192);
    the G step is D's forward and input gradients down to the image on the B
    fakes, G's weight gradients and G's input gradients above z (1,081,856)."""
    wl = dict(synth.workload("mnist_mlp_4x4_mix"), rows=1, cols=1, batch=1, steps=1, mix_enable=0)
    _, train, rest = bench.gemm_flops_per_generation(wl)
    assert train == 2.0 * (1_480_192 + 1_081_856)
    assert rest == 0.0


@pytest.mark.parametrize("name,ev,train,rest", [
    ("ring8_mlp_2x2", None, None, 0.0),
    ("mnist_mlp_3x3", 16.93e9, 461.2e9, 0.0),
    ("mnist_mlp_4x4_mix", 30.10e9, 819.9e9, 10.90e9),
    ("mnist_mlp_8x8", 120.4e9, 3279.4e9, 0.0),
])
def test_mlp_generation_totals(name, ev, train, rest):
    wl = synth.workload(name)
    e, t, r = bench.gemm_flops_per_generation(wl)
    if ev is not None:
        assert e == pytest.approx(ev, rel=2e-3)
        assert t == pytest.approx(train, rel=2e-3)
    assert r == pytest.approx(rest, rel=2e-3, abs=1.0)
    if name == "ring8_mlp_2x2":
        # 2x2 grid, B 64, 20 steps: 0.5669 GFLOP per generation in all
        assert e + t + r == pytest.approx(0.5669e9, rel=1e-3)


def test_dcgan_generation_total():
    """64x64 DCGAN grid: 123.9 TFLOP per generation, 7.45 of them in the
    evaluation (104.6 M multiply-adds per sample through G, 103.8 M through D)."""
    wl = synth.workload("celeba_dcgan_4x4")
    g, _, d, _ = bench.macs_per_sample(wl)
    assert g == pytest.approx(104.6e6, rel=1e-3) and d == pytest.approx(103.8e6, rel=1e-3)
    e, t, r = bench.gemm_flops_per_generation(wl)
    assert e == pytest.approx(7.45e12, rel=2e-3)
    assert e + t + r == pytest.approx(123.9e12, rel=1e-3)
