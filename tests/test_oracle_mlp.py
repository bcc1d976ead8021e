"""Pins of the oracle's MLP forward / manual backward and initialisation."""
import numpy as np
import pytest
import torch

from oracle import mlp


def _tiny(acts, sizes, seed=0):
    g = np.random.default_rng(seed)
    _, P = mlp.layout(sizes)
    p = g.normal(0, 0.7, P)
    x = g.normal(0, 1.0, (4, sizes[0]))
    return p, x


def _loss(p, sizes, acts, x, r, slope):
    pre, post = mlp.forward(p, sizes, acts, x, slope)
    return float((post[-1] * r).sum())


@pytest.mark.parametrize("acts", [("relu", "relu", "linear"), ("lrelu", "lrelu", "linear"),
                                  ("relu", "relu", "tanh"), ("tanh", "lrelu", "tanh")])
def test_backward_matches_central_differences(acts):
    sizes = [3, 5, 4, 2]
    slope = 0.2
    p, x = _tiny(acts, sizes)
    r = np.random.default_rng(1).normal(size=(4, 2))
    pre, post = mlp.forward(p, sizes, acts, x, slope)
    g, dx = mlp.backward(p, sizes, acts, pre, post, r, slope, want_input_grad=True)
    h = 1e-6
    fd = np.zeros_like(p)
    for k in range(len(p)):
        e = np.zeros_like(p)
        e[k] = h
        fd[k] = (_loss(p + e, sizes, acts, x, r, slope) - _loss(p - e, sizes, acts, x, r, slope)) / (2 * h)
    assert np.allclose(g, fd, rtol=1e-6, atol=1e-7)
    fdx = np.zeros_like(x)
    for i in range(x.shape[0]):
        for j in range(x.shape[1]):
            e = np.zeros_like(x)
            e[i, j] = h
            fdx[i, j] = (_loss(p, sizes, acts, x + e, r, slope) - _loss(p, sizes, acts, x - e, r, slope)) / (2 * h)
    assert np.allclose(dx, fdx, rtol=1e-6, atol=1e-7)


def _torch_net(p, sizes, acts, x, slope):
    pt = torch.tensor(p, dtype=torch.float64, requires_grad=True)
    h = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    inp = h
    for (off, fi, fo), a in zip(mlp.layout(sizes)[0], acts):
        W = pt[off:off + fi * fo].view(fi, fo)
        b = pt[off + fi * fo: off + (fi + 1) * fo]
        h = torch.nn.functional.linear(h, W.t(), b)
        if a == "relu":
            h = torch.relu(h)
        elif a == "lrelu":
            h = torch.nn.functional.leaky_relu(h, slope)
        elif a == "tanh":
            h = torch.tanh(h)
    return pt, inp, h


@pytest.mark.parametrize("sizes,acts", [([64, 256, 256, 784], ("relu", "relu", "tanh")),
                                        ([784, 256, 256, 1], ("lrelu", "lrelu", "linear")),
                                        ([8, 64, 64, 2], ("relu", "relu", "linear"))])
def test_matches_torch_fp64_autograd(sizes, acts):
    g = np.random.default_rng(5)
    _, P = mlp.layout(sizes)
    p = mlp.init(sizes, 3, 1, "INIT_G")
    x = g.normal(0, 1, (7, sizes[0]))
    r = g.normal(0, 1, (7, sizes[-1]))
    pre, post = mlp.forward(p, sizes, acts, x, 0.2)
    grad, dx = mlp.backward(p, sizes, acts, pre, post, r, 0.2, want_input_grad=True)
    pt, xt, out = _torch_net(p, sizes, acts, x, 0.2)
    (out * torch.tensor(r)).sum().backward()
    assert np.allclose(post[-1], out.detach().numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(grad, pt.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_layout_blocks():
    lay, P = mlp.layout([64, 256, 256, 784])
    assert P == 65 * 256 + 257 * 256 + 257 * 784 == 283920
    assert [l[0] for l in lay] == [0, 65 * 256, 65 * 256 + 257 * 256]
    assert mlp.layout([784, 256, 256, 1])[1] == 267009


def test_init_uniform_in_fan_in_bounds():
    sizes = [64, 256, 256, 784]
    p = mlp.init(sizes, 0, 2, "INIT_G")
    for (off, fi, fo) in mlp.layout(sizes)[0]:
        blk = p[off:off + (fi + 1) * fo]
        bound = 1.0 / np.sqrt(fi)
        assert np.all(np.abs(blk) < bound)
        # U(-b, b): mean 0, variance b^2 / 3
        assert abs(blk.mean()) < 0.02 * bound
        assert abs(blk.var() / (bound ** 2 / 3) - 1) < 0.05
    # different cells and roles draw different streams
    assert not np.array_equal(p, mlp.init(sizes, 0, 3, "INIT_G"))
    assert not np.array_equal(p, mlp.init(sizes, 0, 2, "INIT_D"))
