"""CPU checks of the C ABI: the library loads, exports every declared symbol,
the ctypes struct matches the C compiler's layout, and host-side validation
works (no GPU needed: nothing here launches a kernel)."""
import ctypes
import glob
import os
import re
import subprocess

import pytest

import paper_1811_12843_amd as L
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        txt = open(h).read()
        txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
        for m in re.finditer(r"\b(lipz_[a-z0-9_]+)\s*\(", txt):
            names.add(m.group(1))
    return names


def test_library_exports_every_declared_function():
    lib = L.load_library()
    names = _declared_functions()
    assert len(names) >= 19
    for n in sorted(names):
        assert hasattr(lib, n), n
    assert names == set(L.lipz._SIGS)


def test_config_struct_layout_matches_c(tmp_path):
    fields = [f for f, _ in L.lipz_config._fields_]
    src = ['#include <stdio.h>', '#include <stddef.h>', '#include "lipz.h"', "int main(void) {",
           'printf("%zu\\n", sizeof(lipz_config));']
    src += [f'printf("%zu\\n", offsetof(lipz_config, {f}));' for f in fields]
    src += ["return 0; }"]
    (tmp_path / "t.c").write_text("\n".join(src))
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(tmp_path / "t.c"), "-o",
                    str(tmp_path / "t")], check=True)
    out = [int(x) for x in subprocess.run([str(tmp_path / "t")], capture_output=True, text=True,
                                          check=True).stdout.split()]
    assert out[0] == ctypes.sizeof(L.lipz_config)
    for f, off in zip(fields, out[1:]):
        assert getattr(L.lipz_config, f).offset == off, f


def test_workspace_sizing_and_validation():
    for name in ("ring8_mlp_2x2", "mnist_mlp_3x3", "mnist_mlp_4x4_mix", "mnist_mlp_8x8"):
        w = synth.workload(name)
        c = L.config_from_dict(w)
        nb = L.lipz_workspace_bytes(c, w["data"]["n"])
        assert nb > 0 and nb % 256 == 0
    w = synth.workload("mnist_mlp_3x3")
    base = L.lipz_workspace_bytes(L.config_from_dict(w), 60000)
    # the mixture buffers only exist with mix_enable
    w2 = dict(w, mix_enable=1)
    assert L.lipz_workspace_bytes(L.config_from_dict(w2), 60000) > base
    bad = [dict(w, batch=0), dict(w, tournament_size=6), dict(w, rows=0), dict(w, g_hidden=[]),
           dict(w, lrelu_slope=0.0), dict(w, beta1=1.0), dict(w, fitness_mode=2),
           dict(w, loss="wasserstein", wgan_clip=0.0), dict(w, loss="wasserstein", wgan_clip=float("inf"))]
    for b in bad:
        assert L.lipz_workspace_bytes(L.config_from_dict(b), 60000) == 0
    c = L.config_from_dict(w)
    c.loss_kind = 2
    assert L.lipz_workspace_bytes(c, 60000) == 0
    # the Wasserstein trainer: same buffers as the BCE one, for both network kinds
    assert L.lipz_workspace_bytes(L.config_from_dict(dict(w, loss="wasserstein")), 60000) == base
    assert L.lipz_workspace_bytes(L.config_from_dict(synth.workload("mnist_mlp_4x4_wgan")), 60000) > 0
    d = synth.workload("celeba_dcgan_4x4")
    assert L.lipz_workspace_bytes(L.config_from_dict(dict(d, loss="wasserstein")), 1000) == \
        L.lipz_workspace_bytes(L.config_from_dict(d), 1000) > 0
    # the NES trainer: its Q = 2 nes_pairs + 1 parameter sets per role and cell add to the workspace
    nes = synth.workload("mnist_mlp_3x3_nes")
    assert L.lipz_workspace_bytes(L.config_from_dict(nes), 60000) > base
    for b in (dict(nes, nes_pairs=0), dict(nes, nes_pairs=65), dict(nes, nes_sigma=0.0),
              dict(nes, g_hidden=[65536, 8192])):  # nes_pairs x parameters >= 2^31
        assert L.lipz_workspace_bytes(L.config_from_dict(b), 60000) == 0
    c = L.config_from_dict(nes)
    c.trainer = 3
    assert L.lipz_workspace_bytes(c, 60000) == 0
    for t in ("nes", "es"):
        d = dict(synth.workload("celeba_dcgan_4x4"), trainer=t)
        assert L.lipz_workspace_bytes(L.config_from_dict(d), 1000) == 0
    # sub-populations: per-individual state and training buffers grow with s; elitism adds the re-evaluation
    w1 = synth.workload("mnist_mlp_3x3")
    b1 = L.lipz_workspace_bytes(L.config_from_dict(w1), 60000)
    b2 = L.lipz_workspace_bytes(L.config_from_dict(dict(w1, pop_size=2)), 60000)
    b2e = L.lipz_workspace_bytes(L.config_from_dict(dict(w1, pop_size=2, elitism=1)), 60000)
    assert 0 < b1 < b2 < b2e
    for b in (dict(w1, pop_size=0), dict(w1, pop_size=5), dict(w1, elitism=2),
              dict(w2, pop_size=2),  # the mixture step needs one generator per cell
              dict(synth.workload("celeba_dcgan_4x4"), pop_size=2),
              dict(synth.workload("celeba_dcgan_4x4"), elitism=1)):
        assert L.lipz_workspace_bytes(L.config_from_dict(b), 60000) == 0
    # the ES trainer: the same sets, no direction buffer
    es = synth.workload("mnist_mlp_3x3_es")
    assert base < L.lipz_workspace_bytes(L.config_from_dict(es), 60000) < L.lipz_workspace_bytes(
        L.config_from_dict(nes), 60000)
    for b in (dict(es, nes_pairs=0), dict(es, nes_sigma=-1.0), dict(es, g_hidden=[65536, 8192])):
        assert L.lipz_workspace_bytes(L.config_from_dict(b), 60000) == 0
    c = L.config_from_dict(w)
    c.abi_version = 99
    assert L.lipz_workspace_bytes(c, 60000) == 0
    assert L.lipz_workspace_bytes(L.config_from_dict(w), 0) == 0
    # the 64x64 DCGAN grid: ~24 GiB (evaluation activations of 80 (cell, slot) pairs dominate)
    nb = L.lipz_workspace_bytes(L.config_from_dict(synth.workload("celeba_dcgan_4x4")), 1000)
    assert 20 * 2**30 < nb < 28 * 2**30 and nb % 256 == 0


def test_create_rejects_bad_arguments_without_touching_the_gpu():
    w = synth.workload("ring8_mlp_2x2")
    c = L.config_from_dict(w)
    with pytest.raises(L.LipzError) as e:
        L.lipz_grid_create(c, 0, 0, 0, 100, None)
    assert e.value.status == L.LIPZ_E_INVAL
    with pytest.raises(L.LipzError) as e:
        L.lipz_grid_create(c, 256, 1, 512, 100, None)  # workspace too small, checked first on host
    assert e.value.status == L.LIPZ_E_WORKSPACE
    with pytest.raises(L.LipzError) as e:
        L.lipz_grid_create(c, 257, 1 << 40, 512, 100, None)  # misaligned
    assert e.value.status == L.LIPZ_E_WORKSPACE
    # the mixture step is defined for the MLP networks only: rejected on the host
    d = L.config_from_dict(dict(synth.workload("celeba_dcgan_4x4"), mix_enable=1))
    with pytest.raises(L.LipzError) as e:
        L.lipz_grid_create(d, 256, 1 << 40, 512, 100, None)
    assert e.value.status == L.LIPZ_E_INVAL


def test_error_strings():
    for s in range(0, -7, -1):
        assert L.lipz_error_string(s) not in ("", "unknown status")
    assert L.lipz_error_string(-100) == "unknown status"
    assert L.lipz_last_error(None) == ""
