"""Fully connected generator / discriminator networks in fp64 with manual
back-propagation (the "neural network model" component of Section 3; layer
widths from the experiment settings table: 64-256-256-784 for MNIST).

Flat parameter layout of a network with widths n_0 .. n_L: for each layer l,
W_l as an [n_{l-1}, n_l] row-major matrix followed by its bias b_l [n_l], so
that (W_l; b_l) is one [(n_{l-1} + 1), n_l] block.  y = act(x W_l + b_l).

Initialisation (Section 3, step 1: random weights): every element of layer l,
weights and bias alike, is U(-1/sqrt(n_{l-1}), +1/sqrt(n_{l-1})), element e of
the role's flat vector taking word e of the Philox stream (cell, 0, 0, tag).
"""
import numpy as np

from . import rng


def layout(sizes):
    """List of (offset_W, fan_in, fan_out) and the total parameter count."""
    out, off = [], 0
    for l in range(1, len(sizes)):
        fi, fo = sizes[l - 1], sizes[l]
        out.append((off, fi, fo))
        off += (fi + 1) * fo
    return out, off


def unpack(p, sizes):
    """Views (W_l, b_l) into the flat vector p."""
    lay, _ = layout(sizes)
    res = []
    for off, fi, fo in lay:
        W = p[off:off + fi * fo].reshape(fi, fo)
        b = p[off + fi * fo: off + (fi + 1) * fo]
        res.append((W, b))
    return res


def init(sizes, seed, cell, tag):
    lay, total = layout(sizes)
    u = rng.uniforms(seed, total, cell, 0, 0, tag)
    p = np.empty(total)
    for off, fi, fo in lay:
        n = (fi + 1) * fo
        p[off:off + n] = (2.0 * u[off:off + n] - 1.0) / np.sqrt(fi)
    return p


def act(name, x, slope):
    if name == "linear":
        return x
    if name == "relu":
        return np.maximum(x, 0.0)
    if name == "lrelu":
        return np.where(x > 0.0, x, slope * x)
    if name == "tanh":
        return np.tanh(x)
    raise ValueError(name)


def act_deriv(name, pre, slope):
    """Derivative at the pre-activation; at 0, ReLU' = 0 and LeakyReLU' = slope."""
    if name == "linear":
        return np.ones_like(pre)
    if name == "relu":
        return (pre > 0.0).astype(np.float64)
    if name == "lrelu":
        return np.where(pre > 0.0, 1.0, slope)
    if name == "tanh":
        t = np.tanh(pre)
        return 1.0 - t * t
    raise ValueError(name)


def forward(p, sizes, acts, x, slope):
    """Returns (pre, post) lists; post[0] = x, post[l] = act_l(pre[l])."""
    pre, post = [None], [np.asarray(x, dtype=np.float64)]
    for l, (W, b) in enumerate(unpack(p, sizes), start=1):
        z = post[-1] @ W + b
        pre.append(z)
        post.append(act(acts[l - 1], z, slope))
    return pre, post


def backward(p, sizes, acts, pre, post, d_out, slope, want_input_grad=False):
    """Back-propagate dLoss/d(post[L]) = d_out.

    Returns (flat gradient of p, dLoss/d(post[0]) or None).
    """
    params = unpack(p, sizes)
    grad = np.zeros_like(p)
    gparts = unpack(grad, sizes)
    L = len(params)
    delta = d_out * act_deriv(acts[L - 1], pre[L], slope)
    d_in = None
    for l in range(L, 0, -1):
        W, _ = params[l - 1]
        gW, gb = gparts[l - 1]
        gW[...] = post[l - 1].T @ delta
        gb[...] = delta.sum(axis=0)
        if l > 1:
            delta = (delta @ W.T) * act_deriv(acts[l - 2], pre[l - 1], slope)
        elif want_input_grad:
            d_in = delta @ W.T
    return grad, d_in
