"""Throughput of one grid generation on one MI355X.

A step is one generation of the 4x4 MNIST-shaped MLP grid with mixture
weights: lipz_eval_neighborhoods (400 generator x discriminator pairings),
lipz_select_replace, 100 x lipz_train_step, lipz_mixture_update.  Inputs
(dataset, state) are resident in HBM before the timed region starts.

Prints one JSON line:
  value            grid generations per second (whole job, one GPU)
  pair_evals_per_s pairings evaluated per second by lipz_eval_neighborhoods
  mfma_frac        algorithmic GEMM FLOPs of a generation / time / fp32 MFMA peak
  roofline         the grouped-GEMM kernel: algorithmic FLOPs per launch over its
                   average launch time (HIP events stamped by each GEMM dispatch);
                   traffic = HBM bytes per launch from the FETCH_SIZE / WRITE_SIZE
                   passes stored in profiles/ (null once the GEMM source changed)
  cpu_baseline     the oracle (fp64 NumPy) on this host's cores, on a bounded sample
  per_config       the other workloads of the benchmark (the 2x2 ring grid, the 3x3
                   and 8x8 MNIST-shaped grids, the 64x64 DCGAN grid), one warm-up
                   and one timed generation each: generations/s, ms/generation,
                   mfma_frac, and the matrix-core kernels' own rate and fraction

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Other workloads (--workload): ring8_mlp_2x2, mnist_mlp_3x3, mnist_mlp_8x8,
mnist_mlp_4x4_wgan (the Wasserstein trainer), mnist_mlp_3x3_nes and
mnist_mlp_3x3_es (the gradient-free NES and (1+lambda)-ES trainers),
mnist_mlp_4x4_pop2 (two individuals per role and cell, elitist replacement) and
celeba_dcgan_4x4 (the 64x64 DCGAN grid; its
roofline kernel is the implicit-GEMM convolution together with the grouped
GEMM).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "G×D pair-evals/sec + grid generations/sec (4x4 MLP grid); % fp32 MFMA peak"
FP32_MFMA_PEAK = 157.3e12  # MI355X dense fp32 matrix peak, FLOP/s


def macs_per_sample(wl):
    """Multiply-adds per sample of one forward pass: (G, G's first layer, D,
    D's first layer).  Convolutions count their real taps only (a stride-2
    transposed convolution: 16 taps per input pixel)."""
    if wl["net"] == "mlp":
        g = [wl["z_dim"]] + list(wl["g_hidden"]) + [wl["x_dim"]]
        d = [wl["x_dim"]] + list(wl["d_hidden"]) + [1]
        gl = [g[i] * g[i + 1] for i in range(len(g) - 1)]
        dl = [d[i] * d[i + 1] for i in range(len(d) - 1)]
    else:
        h, _, c = wl["img"]
        gc, dc = list(wl["g_hidden"]), list(wl["d_hidden"])
        n = len(gc)
        gl = [wl["z_dim"] * 16 * gc[0]]
        gl += [16 * (4 << (k - 1)) ** 2 * gc[k - 1] * gc[k] for k in range(1, n)]
        gl += [16 * (h // 2) ** 2 * gc[n - 1] * c]
        cin = [c] + dc[:-1]
        dl = [16 * (h >> (k + 1)) ** 2 * cin[k] * dc[k] for k in range(n)] + [16 * dc[-1]]
    return sum(gl), gl[0], sum(dl), dl[0]


def gemm_flops_per_generation(wl):
    """Algorithmic matrix-core FLOPs (2 per multiply-add, bias terms excluded)
    of one generation: evaluation, S training steps, and the rest (the
    mixture step, the re-evaluation of elitist replacement)."""
    C, B = wl["rows"] * wl["cols"], wl["batch"]
    s = wl.get("pop_size", 1)
    n = 5 * s  # neighbourhood population
    macs_g, g_first, macs_d, d_first = macs_per_sample(wl)
    # evaluation: n G forwards per cell, D forwards on B real + n B fake rows per D
    ev = C * (n * B * macs_g + n * (1 + n) * B * macs_d)
    rest = 0
    if wl.get("elitism", 0):
        # re-evaluation: s trained G forwards, n previous D on their s B rows,
        # s trained D on the (1 + n) B evaluation rows
        rest += C * (s * B * macs_g + n * s * B * macs_d + s * (1 + n) * B * macs_d)
    if wl["mix_enable"]:
        rest += C * wl["mix_samples"] * (macs_g + wl["x_dim"] * wl["mix_feat_dim"])
    C = C * s  # training units
    if wl.get("trainer", "gradient") in ("nes", "es"):
        # NES / ES: G fwd; Q = 2 pairs + 1 critic parameter sets, each D fwd over 2B rows;
        # Q generator sets, each G fwd, and the updated D over their Q B rows
        Q = 2 * wl["nes_pairs"] + 1
        train = C * wl["steps"] * (B * macs_g + Q * 2 * B * macs_d + Q * B * macs_g + Q * B * macs_d)
        return 2.0 * ev, 2.0 * train, 2.0 * rest
    # D step: G fwd, D fwd (2B), D weight grads (2B), D input grads below layer 1 (2B)
    d_step = B * macs_g + 2 * B * macs_d + 2 * B * macs_d + 2 * B * (macs_d - d_first)
    # G step: D fwd (B), D input grads down to x (B), G weight grads, G input grads above z
    g_step = B * macs_d + B * macs_d + B * macs_g + B * (macs_g - g_first)
    train = C * wl["steps"] * (d_step + g_step)
    return 2.0 * ev, 2.0 * train, 2.0 * rest


def gemm_source_digest():
    """SHA-256 of the GEMM kernels' code: gemm.hip and the part of
    lipz_internal.h up to the declaration of launch_gemm_grouped (the device
    helpers and the GEMM's descriptor types; the rest of the header declares
    other kernels), with comments and whitespace removed, so that a change
    of wording alone keeps counters taken from the same code valid."""
    import hashlib
    import re
    csrc = os.path.join(ROOT, "paper_1811_12843_amd", "csrc")
    with open(os.path.join(csrc, "gemm.hip"), "rb") as f:
        gemm = f.read()
    with open(os.path.join(csrc, "lipz_internal.h"), "rb") as f:
        head = f.read()
    cut = head.index(b";", head.index(b"hipError_t launch_gemm_grouped(")) + 1
    code = gemm + b"\n" + head[:cut]
    code = re.sub(rb"/\*.*?\*/", b" ", code, flags=re.S)   # block comments
    code = re.sub(rb"//[^\n]*", b"", code)                  # line comments
    code = re.sub(rb"\s+", b"", code)
    return hashlib.sha256(code).hexdigest()


def stored_gemm_traffic(workload):
    """HBM bytes per grouped-GEMM launch from the FETCH_SIZE / WRITE_SIZE passes
    recorded in profiles/, or None when the GEMM source changed since."""
    path = os.path.join(ROOT, "profiles", f"gemm_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("gemm_source_sha256") != gemm_source_digest():
        return None
    return rec.get("traffic_bytes_per_launch")


def _oracle_cores():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return int(os.environ.get("OMP_NUM_THREADS", "1"))


def cpu_baseline(wl, data, budget_s=20.0):
    """Time the oracle on a bounded sample of the same workload and scale it to
    generations/s.  MLP: one whole evaluation, k training steps (k chosen to
    fit the budget), one mixture step; a generation = eval + S * mean step +
    mixture.  DCGAN: one cell's evaluation (5 generator and 30 discriminator
    forwards) and one cell's training step (a 1x1 grid draws cell 0's samples),
    each scaled by the number of cells."""
    import numpy as np
    from oracle import coevo, es, mixture, nes
    cores = _oracle_cores()
    step_fn = {"nes": nes.train_step, "es": es.train_step}.get(wl.get("trainer", "gradient"), coevo.train_step)
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    if wl["net"] != "mlp":
        t0 = time.perf_counter()
        _, x, z = coevo.sample(S, data, 0, 0, 0)
        fakes = [coevo.g_forward(S, st.Gp[S.nbr[0, i]], z)[1] for i in range(5)]
        for j in range(5):
            dp = st.Dp[S.nbr[0, j]]
            coevo.d_logits(S, dp, x)
            for i in range(5):
                coevo.d_logits(S, dp, fakes[i])
        t_cell_eval = time.perf_counter() - t0
        S1 = coevo.Setup(dict(wl, rows=1, cols=1), len(data))
        st1 = coevo.State(**{f: np.array(getattr(st, f)[:1]) for f in coevo.State.FIELDS})
        t0 = time.perf_counter()
        coevo.train_step(S1, st1, data, 0, 0)
        t_cell_step = time.perf_counter() - t0
        t_eval = S.C * t_cell_eval
        t_gen = t_eval + wl["steps"] * S.C * t_cell_step
        return {"value": 1.0 / t_gen, "unit": "generations/s", "cores": int(cores), "kind": "oracle",
                "sample": (f"cell 0's evaluation ({t_cell_eval:.2f} s) and one training step of cell 0 "
                           f"({t_cell_step:.2f} s) of the {wl['rows']}x{wl['cols']} grid; generation = "
                           f"{S.C} x eval + {wl['steps']} x {S.C} x step (extrapolated from one cell)"),
                "pair_evals_per_s": S.C * 25 / t_eval}
    t0 = time.perf_counter()
    coevo.evaluate(S, st, data, 0)
    t_eval = time.perf_counter() - t0
    t0 = time.perf_counter()
    k = 0
    while True:
        step_fn(S, st, data, 0, k)
        k += 1
        el = time.perf_counter() - t0
        if el > budget_s * 0.5 or k >= wl["steps"]:
            break
    t_step = el / k
    t_mix = 0.0
    if wl["mix_enable"]:
        stats = mixture.real_stats(S, data)
        t0 = time.perf_counter()
        mixture.update(S, st, stats, 0)
        t_mix = time.perf_counter() - t0
    t_elite = 0.0
    if wl.get("elitism", 0):
        _, _, fg, fd = coevo.evaluate(S, st, data, 0)
        t0 = time.perf_counter()
        coevo.elitist_replace(S, st, st, data, 0, fg, fd)
        t_elite = time.perf_counter() - t0
    t_gen = t_eval + wl["steps"] * t_step + t_mix + t_elite
    return {"value": 1.0 / t_gen, "unit": "generations/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"1 evaluation ({t_eval:.2f} s), {k} training steps ({t_step:.3f} s each)"
                       + (f", 1 mixture step ({t_mix:.2f} s)" if wl["mix_enable"] else "")
                       + (f", 1 elitist replacement ({t_elite:.2f} s)" if wl.get("elitism", 0) else "")
                       + f" of {wl['rows']}x{wl['cols']} grid; generation = eval + "
                       f"{wl['steps']} x step + mixture"),
            "pair_evals_per_s": S.C * S.n * S.n / t_eval}


def mfma_ceiling(torch, L, n=8192, reps=6):
    """The fp32 matrix-core rate that one large square product reaches on this
    GPU: torch.matmul (the vendor BLAS, fp32 without reduced-precision inputs)
    and this library's grouped GEMM on the same n x n x n problem (through its
    single-problem test entry point).  Both in TFLOP/s, HIP events."""
    torch.backends.cuda.matmul.allow_tf32 = False
    g = torch.Generator(device="cuda").manual_seed(0)
    a = torch.randn(n, n, device="cuda", generator=g)
    b = torch.randn(n, n, device="cuda", generator=g)
    c = torch.empty(n, n, device="cuda")
    flop = 2.0 * n * n * n

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        return flop * reps / (e0.elapsed_time(e1) * 1e-3) / 1e12

    vendor = timed(lambda: torch.matmul(a, b, out=c))
    # the vendor product's precision: a 256 x 256 corner against fp64 (fp32
    # inputs give ~1e-6 here; reduced-precision inputs would give ~1e-3)
    ref = a[:256].double() @ b[:, :256].double()
    vendor_err = float((c[:256, :256].double() - ref).norm() / ref.norm())
    desc = torch.zeros(256, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def own():
        L.lipz_test_gemm(stream, desc.data_ptr(), n, n, n, a.data_ptr(), n, 0, -1, b.data_ptr(), n, 0,
                         c.data_ptr(), n, 0, 0)

    ours = timed(own)
    del a, b, c
    return {"shape": [n, n, n], "vendor_tflops": vendor, "vendor_rel_err": vendor_err, "own_gemm_tflops": ours}


# The configurations reported beside the headline one (dataset rows; 0 = the
# workload's own): the 2x2 ring grid, the 3x3 and 8x8 MNIST-shaped grids and
# the 64x64 DCGAN grid on a small synthetic image set (minibatch rows are drawn
# uniformly, so the work per step does not depend on the dataset size).
PER_CONFIG = {"mnist_mlp_3x3": 0, "mnist_mlp_4x4_mix": 0, "mnist_mlp_8x8": 0, "ring8_mlp_2x2": 0,
              "celeba_dcgan_4x4": 512}
# workloads whose asynchronous row-band schedule (same results bit for bit)
# is also timed in the per-workload block, with its band count
PER_CONFIG_BANDS = {"mnist_mlp_8x8": 4}
_DATA = {}


def run_workload(L, torch, name, steps, warmup, eval_reps, data_n=0, bands=0):
    """Time `steps` generations of workload `name` after `warmup` untimed ones,
    the evaluation alone, and the matrix-core kernels in an instrumented pass."""
    import synth

    wl = synth.workload(name)
    if bands:
        wl["bands"] = bands
    n_data = data_n or (8192 if wl["net"] == "dcgan" else wl["data"]["n"])
    wl["data"] = dict(wl["data"], n=n_data)
    key = json.dumps(wl["data"], sort_keys=True)
    if key not in _DATA:
        _DATA.clear()
        _DATA[key] = synth.make_dataset(wl["data"])
    data_np = _DATA[key]
    dev = "cuda"
    data = torch.from_numpy(data_np).to(dev)
    cfg = L.config_from_dict(wl)
    nb = L.lipz_workspace_bytes(cfg, len(data_np))
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    g = L.lipz_grid_create(cfg, ws.data_ptr(), nb, data.data_ptr(), len(data_np), stream.cuda_stream)
    C = wl["rows"] * wl["cols"]
    S = wl["steps"]

    def generation(gen):
        L.lipz_eval_neighborhoods(g, gen)
        L.lipz_select_replace(g, gen)
        L.lipz_train_step(g, gen, 0, S)
        if wl.get("elitism", 0):
            L.lipz_elitist_replace(g, gen)
        if wl["mix_enable"]:
            L.lipz_mixture_update(g, gen)

    gen = 0
    for _ in range(warmup):
        generation(gen)
        gen += 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if bands:  # one call: the bands run ahead of each other across generations
        L.lipz_run_generations(g, gen, steps, S)
        gen += steps
    else:
        for _ in range(steps):
            generation(gen)
            gen += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert L.lipz_sync(g) in (L.LIPZ_OK, L.LIPZ_E_NONFINITE)
    ms_per_gen = 1e3 * elapsed / steps

    # evaluation alone
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for r in range(eval_reps):
        L.lipz_eval_neighborhoods(g, gen + r)
    torch.cuda.synchronize()
    t_eval = (time.perf_counter() - t0) / eval_reps
    nbh = 5 * wl.get("pop_size", 1)
    pair_evals = C * nbh * nbh / t_eval

    # grouped-GEMM kernel timing with HIP events on the grid's stream
    # one instrumented generation first, so the timed ones reuse its event pairs
    L.lipz_set_gemm_timing(g, 1)
    generation(gen)
    gen += 1
    L.lipz_gemm_timing(g)  # reset
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        generation(gen)
        gen += 1
    torch.cuda.synchronize()
    inst_ms = 1e3 * (time.perf_counter() - t0) / steps
    gemm_ms, launches, gemm_flops, gemm_bytes = L.lipz_gemm_timing(g)
    L.lipz_set_gemm_timing(g, 0)

    cfg_desc = {"workload": name, "grid": f"{wl['rows']}x{wl['cols']}", "cells": C,
                "pairings_per_eval": nbh * nbh * C, "batch": wl["batch"], "steps_per_generation": S,
                "mixture_es": bool(wl["mix_enable"]), "bands": bands}
    if wl["net"] == "mlp":
        cfg_desc.update(g=[wl["z_dim"]] + wl["g_hidden"] + [wl["x_dim"]], d=[wl["x_dim"]] + wl["d_hidden"] + [1])
        data_desc = (f"synthetic (seeded MNIST-shaped blobs, {len(data_np)} x {wl['x_dim']}); "
                     "random-init MLPs")
        kernel = "grouped GEMM (gemm_fast_kernel + gemm_wave_kernel)"
    else:
        cfg_desc.update(image=list(wl["img"]), z=wl["z_dim"], g_channels=wl["g_hidden"],
                        d_channels=wl["d_hidden"], net="dcgan")
        data_desc = (f"synthetic (seeded colour fields + blobs, {len(data_np)} x {wl['img'][0]}x{wl['img'][1]}"
                     f"x{wl['img'][2]} NHWC); random-init DCGAN-style conv nets")
        kernel = "implicit-GEMM convolution (conv_kernel) + grouped GEMM"
    f_ev, f_tr, f_mix = gemm_flops_per_generation(wl)
    f_gen = f_ev + f_tr + f_mix
    avg_ms = gemm_ms / max(launches, 1)
    achieved = (gemm_flops / max(launches, 1)) / (avg_ms * 1e-3) if launches else 0.0
    L.lipz_grid_destroy(g)
    del ws, data
    torch.cuda.empty_cache()
    return {"wl": wl, "data": data_np, "data_desc": data_desc, "config": cfg_desc, "ms_per_gen": ms_per_gen,
            "pair_evals_per_s": pair_evals, "eval_ms": t_eval * 1e3, "gflop_per_gen": f_gen / 1e9,
            "mfma_frac": f_gen / (ms_per_gen * 1e-3) / FP32_MFMA_PEAK, "eval_mfma_frac": f_ev / t_eval / FP32_MFMA_PEAK,
            "roofline": {"kernel": kernel, "bound": "mfma", "achieved": achieved / 1e12,
                         "peak": FP32_MFMA_PEAK / 1e12, "unit": "TFLOP/s",
                         "frac": achieved / FP32_MFMA_PEAK, "traffic": None,
                         "launches": launches, "avg_launch_us": avg_ms * 1e3,
                         "flop_per_launch": gemm_flops / max(launches, 1),
                         "algorithmic_bytes_per_launch": gemm_bytes / max(launches, 1),
                         "instrumented_ms_per_step": inst_ms}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed generations")
    ap.add_argument("--warmup", type=int, default=1, help="untimed generations")
    ap.add_argument("--workload", default="mnist_mlp_4x4_mix")
    ap.add_argument("--data-n", type=int, default=0,
                    help="dataset rows (default: the workload's; 8192 for the 64x64 image workload, "
                         "whose 200000 rows take minutes to synthesise; minibatches are drawn "
                         "uniformly, so the work per step does not depend on it)")
    ap.add_argument("--eval-reps", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-config", action="store_true",
                    help="skip the one-generation measurements of the other workloads")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the large-GEMM measurement of the fp32 matrix-core ceiling")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--bands", type=int, default=0,
                    help="run the timed generations with lipz_run_generations on this many row bands "
                         "(asynchronous cells; MLP workloads without the mixture step)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (calibrates HBM byte counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * 1024 * 1024 // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n}), flush=True)
        return
    if args.gpus != 1:
        print("bench.py: the library runs a grid on one GPU; it is not sharded across GPUs "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_1811_12843_amd as L

    if not os.path.exists(L.LIB_PATH):
        from paper_1811_12843_amd import build as _b
        _b.build()
    r = run_workload(L, torch, args.workload, args.steps, args.warmup, args.eval_reps, args.data_n, args.bands)
    wl, data_np = r["wl"], r["data"]
    traffic = stored_gemm_traffic(args.workload)
    out = {
        "metric": METRIC,
        "value": 1e3 / r["ms_per_gen"],
        "unit": "generations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_gen"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": r["data_desc"],
        "config": r["config"],
        "pair_evals_per_s": r["pair_evals_per_s"],
        "eval_ms": r["eval_ms"],
        "gemm_gflop_per_generation": r["gflop_per_gen"],
        "mfma_frac": r["mfma_frac"],
        "eval_mfma_frac": r["eval_mfma_frac"],
        "roofline": dict(r["roofline"], traffic=traffic),
    }
    achieved = r["roofline"]["achieved"] * 1e12
    f_gen = r["gflop_per_gen"] * 1e9
    ms_per_gen = r["ms_per_gen"]
    if not args.no_per_config:
        # every other workload of the benchmark: one warm-up and one timed
        # generation each, the matrix-core kernels' rate from a second,
        # instrumented generation
        out["per_config"] = {}
        for name in PER_CONFIG:
            if name == args.workload:
                continue
            q = run_workload(L, torch, name, 1, 1, 3, PER_CONFIG[name], 0)
            out["per_config"][name] = {
                "generations_per_s": 1e3 / q["ms_per_gen"], "ms_per_gen": q["ms_per_gen"],
                "pair_evals_per_s": q["pair_evals_per_s"], "gflop_per_gen": q["gflop_per_gen"],
                "mfma_frac": q["mfma_frac"], "eval_mfma_frac": q["eval_mfma_frac"],
                "kernel": q["roofline"]["kernel"], "kernel_tflops": q["roofline"]["achieved"],
                "kernel_frac": q["roofline"]["frac"], "config": q["config"]}
            del q
            if name in PER_CONFIG_BANDS:
                # the generation rate only: with the bands' launches overlapping on
                # several streams, per-launch kernel times do not add up to a rate
                qb = run_workload(L, torch, name, 1, 1, 1, PER_CONFIG[name], PER_CONFIG_BANDS[name])
                out["per_config"][name]["row_bands"] = {
                    "bands": PER_CONFIG_BANDS[name], "generations_per_s": 1e3 / qb["ms_per_gen"],
                    "ms_per_gen": qb["ms_per_gen"], "mfma_frac": qb["mfma_frac"]}
                del qb
    if not args.no_ceiling:
        ceil = mfma_ceiling(torch, L)
        ceil["gen_frac_of_vendor"] = f_gen / (ms_per_gen * 1e-3) / (ceil["vendor_tflops"] * 1e12)
        ceil["gemm_frac_of_vendor"] = achieved / (ceil["vendor_tflops"] * 1e12)
        out["mfma_ceiling"] = ceil
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, data_np, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
