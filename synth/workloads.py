"""Workload descriptions for the grid-coevolution hot path.

The five workloads mirror the experiment settings table of the paper (Table 1,
Section 4: population size 1 per cell, tournament size 2, Adam, initial
learning rate, mutation rate 1e-4 with probability 0.5, MLP 64-256-256-784 /
DCGAN, batch size) at the grid sizes the paper sweeps.  Datasets are seeded
synthetic stand-ins with the shapes of MNIST and CelebA (Section 4), which are
not available here.

Every field is plain data.  Fields:
  rows, cols           grid shape (toroidal)
  net                  "mlp" or "dcgan"
  z_dim, x_dim         latent width, flat sample width
  img                  (h, w, c) for dcgan, else None
  g_hidden, d_hidden   hidden widths (MLP) / channel widths (DCGAN)
  g_hidden_act, g_out_act, d_hidden_act   "relu" | "lrelu" | "tanh" | "linear"
  lrelu_slope
  batch, steps, gens   minibatch size, training steps per generation, generations
  lr0_g, lr0_d, beta1, beta2, eps
  lr_mutation, lr_mut_std, lr_mut_prob
  tournament_size, fitness_mode (0: paper's single-objective fitness)
  loss                 "bce" (the paper's GAN objective) or "wasserstein" (the
                       WGAN trainer the paper names as the next one to add)
  wgan_clip            weight-clipping bound of the Wasserstein critic
  trainer              "gradient" (backpropagation + Adam, the paper's experiments)
                       or "nes" (the gradient-free NES trainer, oracle/nes.py)
                       or "es" (the gradient-free (1+lambda)-ES trainer, oracle/es.py)
  nes_pairs, nes_sigma antithetic direction pairs and perturbation scale of NES
                       and of the ES trainer's mutants
  pop_size             individuals per role and cell (Table 1: 1)
  elitism              1: post-training re-evaluation and elitist replacement
  mix_enable, mix_sigma, mix_samples, mix_feat_dim
  seed
  data                 dataset recipe name + size (see datasets.py)
"""
import copy

_BASE = dict(
    net="mlp", img=None,
    g_hidden_act="relu", g_out_act="tanh", d_hidden_act="lrelu", lrelu_slope=0.2,
    lr0_g=2e-4, lr0_d=2e-4, beta1=0.9, beta2=0.999, eps=1e-8,
    lr_mutation=1, lr_mut_std=1e-4, lr_mut_prob=0.5,
    tournament_size=2, fitness_mode=0,
    loss="bce", wgan_clip=0.01,
    trainer="gradient", nes_pairs=8, nes_sigma=0.01,
    pop_size=1, elitism=0,
    mix_enable=0, mix_sigma=0.01, mix_samples=1024, mix_feat_dim=64,
    seed=0,
)


def _w(**kw):
    d = copy.deepcopy(_BASE)
    d.update(kw)
    return d


WORKLOADS = {
    # 2x2 torus, ring of 8 Gaussians, tiny MLPs (duplicate neighbours: N==S, W==E)
    "ring8_mlp_2x2": _w(rows=2, cols=2, z_dim=8, x_dim=2,
                        g_hidden=[64, 64], d_hidden=[64, 64],
                        g_out_act="linear", d_hidden_act="relu",
                        batch=64, steps=20, gens=1,
                        data=dict(kind="ring8", n=65536, seed=0)),
    # 3x3 torus, MNIST-shaped MLPs
    "mnist_mlp_3x3": _w(rows=3, cols=3, z_dim=64, x_dim=784,
                        g_hidden=[256, 256], d_hidden=[256, 256],
                        batch=100, steps=100, gens=1,
                        data=dict(kind="mnist_like", n=60000, seed=0)),
    # 4x4 torus, MNIST-shaped MLPs, mixture weights evolved by a (1+1)-ES
    "mnist_mlp_4x4_mix": _w(rows=4, cols=4, z_dim=64, x_dim=784,
                            g_hidden=[256, 256], d_hidden=[256, 256],
                            batch=100, steps=100, gens=10,
                            mix_enable=1, mix_sigma=0.01,
                            data=dict(kind="mnist_like", n=60000, seed=0)),
    # 4x4 torus, MNIST-shaped MLPs, Wasserstein critic with weight clipping
    "mnist_mlp_4x4_wgan": _w(rows=4, cols=4, z_dim=64, x_dim=784,
                             g_hidden=[256, 256], d_hidden=[256, 256],
                             batch=100, steps=100, gens=10,
                             loss="wasserstein", wgan_clip=0.01,
                             data=dict(kind="mnist_like", n=60000, seed=0)),
    # 3x3 torus, MNIST-shaped MLPs trained by NES (8 antithetic pairs) instead of backpropagation
    "mnist_mlp_3x3_nes": _w(rows=3, cols=3, z_dim=64, x_dim=784,
                            g_hidden=[256, 256], d_hidden=[256, 256],
                            batch=100, steps=100, gens=1,
                            trainer="nes", nes_pairs=8, nes_sigma=0.01,
                            data=dict(kind="mnist_like", n=60000, seed=0)),
    # 3x3 torus, MNIST-shaped MLPs trained by a (1+16)-ES (8 antithetic mutant pairs)
    "mnist_mlp_3x3_es": _w(rows=3, cols=3, z_dim=64, x_dim=784,
                           g_hidden=[256, 256], d_hidden=[256, 256],
                           batch=100, steps=100, gens=1,
                           trainer="es", nes_pairs=8, nes_sigma=0.01,
                           data=dict(kind="mnist_like", n=60000, seed=0)),
    # 4x4 torus, MNIST-shaped MLPs, two individuals per role and cell, elitist replacement
    "mnist_mlp_4x4_pop2": _w(rows=4, cols=4, z_dim=64, x_dim=784,
                             g_hidden=[256, 256], d_hidden=[256, 256],
                             batch=100, steps=100, gens=10, pop_size=2, elitism=1,
                             data=dict(kind="mnist_like", n=60000, seed=0)),
    # 8x8 torus, MNIST-shaped MLPs
    "mnist_mlp_8x8": _w(rows=8, cols=8, z_dim=64, x_dim=784,
                        g_hidden=[256, 256], d_hidden=[256, 256],
                        batch=100, steps=100, gens=5,
                        data=dict(kind="mnist_like", n=60000, seed=0)),
    # 4x4 torus, DCGAN-style conv nets on 64x64x3 images
    "celeba_dcgan_4x4": _w(rows=4, cols=4, net="dcgan", z_dim=100, x_dim=64 * 64 * 3,
                           img=(64, 64, 3),
                           g_hidden=[512, 256, 128, 64], d_hidden=[64, 128, 256, 512],
                           g_hidden_act="relu", g_out_act="tanh", d_hidden_act="lrelu",
                           lr0_g=5e-5, lr0_d=5e-5,
                           batch=64, steps=50, gens=2,
                           data=dict(kind="celeba_like", n=200000, seed=0)),
}

# The workload the throughput metric is quoted on.
BENCH_WORKLOAD = "mnist_mlp_4x4_mix"


def workload(name):
    """Deep copy of a named workload."""
    return copy.deepcopy(WORKLOADS[name])


def small_workload(name, **overrides):
    """A named workload with fields overridden (used for reduced test sizes)."""
    w = workload(name)
    if "data" in overrides and isinstance(overrides["data"], dict):
        d = dict(w["data"])
        d.update(overrides.pop("data"))
        w["data"] = d
    w.update(overrides)
    return w
