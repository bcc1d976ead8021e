"""DCGAN-style convolutional generator / discriminator in fp64 with manual
back-propagation (the CelebA network of the experiment settings table,
Section 4: "DCGAN").  THIS IS TEST INFRASTRUCTURE (see the package header).

Images are NHWC.  With n stride-2 stages the image side is 4 * 2**n.

Generator, channel widths g[0..n-1] (outputs of layers 1..n):
  layer 1       dense z -> 4x4xg[0] (no bias), batch norm, ReLU.  This is the
                stride-1, pad-0, 4x4 transposed convolution of a 1x1 input;
                its weight is stored as the [z][(y, x, c)] matrix.
  layers 2..n   4x4 transposed convolution, stride 2, pad 1 (no bias),
                batch norm, ReLU
  layer n+1     4x4 transposed convolution, stride 2, pad 1, to the image
                channels, with bias, tanh
Discriminator, channel widths d[0..n-1]:
  layers 1..n   4x4 convolution, stride 2, pad 1, with bias, LeakyReLU
  layer n+1     the 4x4, stride-1, pad-0 convolution of the 4x4xd[n-1] map
                to one logit: a dense layer over the flattened (y, x, c) map,
                with bias

Readings (the paper names the architecture only): convolutions carry a bias
exactly when no batch norm follows; batch norm uses the statistics of the
batch it normalises (biased variance, eps 1e-5), never running averages; the
discriminator has no batch norm.

Flat parameter layout, layer after layer: the weight block [(taps * c_in)][c_out]
row-major with rows ordered (kh, kw, c_in) (dense layers: [fan_in][fan_out]),
then the bias row [c_out] if the layer has one, then gamma [c_out] and beta
[c_out] if it has batch norm.

Initialisation (Section 3 step 1 asks only for random weights; the usual
DCGAN reading): weights N(0, 0.02^2), gamma N(1, 0.02^2), bias and beta 0.
Element e of the role's flat vector uses normal number e of the Philox stream
(cell, 0, 0, tag).
"""
import numpy as np

from . import rng

BN_EPS = 1e-5
INIT_STD = 0.02


def n_stages(img_hw):
    n, s = 0, 4
    while s < img_hw:
        s *= 2
        n += 1
    if s != img_hw:
        raise ValueError("image side must be 4 * 2**n")
    return n


class Arch:
    """Layer list of one role.  Each layer: dict(kind, cin, cout, hin, hout,
    bias, bn, act, off_w, off_b, off_g, off_be, n_w)."""

    def __init__(self, role, z_dim, img, g_ch, d_ch):
        h, w, c = img
        if h != w:
            raise ValueError("square images only")
        n = n_stages(h)
        self.layers = []
        off = 0

        def add(kind, cin, cout, hin, hout, bias, bn, act):
            nonlocal off
            taps = 1 if kind == "dense" else 16
            L = dict(kind=kind, cin=cin, cout=cout, hin=hin, hout=hout, bias=bias, bn=bn, act=act,
                     taps=taps)
            L["off_w"] = off
            L["n_w"] = taps * cin * cout
            off += L["n_w"]
            L["off_b"] = off if bias else None
            off += cout if bias else 0
            nb = cout // 16 if kind == "dense" else cout
            L["off_g"] = off if bn else None
            L["off_be"] = off + nb if bn else None
            off += 2 * nb if bn else 0
            self.layers.append(L)

        if role == "G":
            if len(g_ch) != n:
                raise ValueError("generator needs one channel width per stage")
            add("dense", z_dim, 16 * g_ch[0], 1, 4, False, True, "relu")
            for k in range(1, n):
                add("convT", g_ch[k - 1], g_ch[k], 4 << (k - 1), 4 << k, False, True, "relu")
            add("convT", g_ch[n - 1], c, 4 << (n - 1), h, True, False, "tanh")
        else:
            if len(d_ch) != n:
                raise ValueError("discriminator needs one channel width per stage")
            cin = c
            for k in range(n):
                add("conv", cin, d_ch[k], h >> k, h >> (k + 1), True, False, "lrelu")
                cin = d_ch[k]
            add("dense", 16 * d_ch[n - 1], 1, 4, 1, True, False, "linear")
        self.P = off
        self.role = role
        self.out_ch = c if role == "G" else 1


def init(arch, seed, cell, tag):
    n = rng.normals(seed, arch.P, cell, 0, 0, tag)
    p = np.zeros(arch.P)
    for L in arch.layers:
        s = slice(L["off_w"], L["off_w"] + L["n_w"])
        p[s] = INIT_STD * n[s]
        if L["bn"]:
            c = bn_channels(L)
            s = slice(L["off_g"], L["off_g"] + c)
            p[s] = 1.0 + INIT_STD * n[s]
    return p


def bn_channels(L):
    """Channels normalised by a layer's batch norm (the dense layer 1 of G
    normalises its 4x4 map per channel)."""
    return L["cout"] // 16 if L["kind"] == "dense" else L["cout"]


def weights(p, L):
    W = p[L["off_w"]:L["off_w"] + L["n_w"]]
    if L["kind"] == "dense":
        return W.reshape(L["cin"], L["cout"])
    return W.reshape(4, 4, L["cin"], L["cout"])


# ---------------------------------------------------------------------------
# Convolutions by their definitions, one kernel tap at a time
# ---------------------------------------------------------------------------
def conv_s2(x, W):
    """y[n, oh, ow] = sum over taps (kh, kw) of x[n, 2 oh - 1 + kh, 2 ow - 1 + kw] @ W[kh, kw],
    input positions outside the image contributing zero (stride 2, pad 1)."""
    N, H, Wd, _ = x.shape
    OH, OW = H // 2, Wd // 2
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    y = np.zeros((N, OH, OW, W.shape[3]))
    for kh in range(4):
        for kw in range(4):
            y += xp[:, kh:kh + 2 * OH:2, kw:kw + 2 * OW:2, :] @ W[kh, kw]
    return y


def conv_s2_backward(x, W, dy):
    """Gradients of conv_s2 with respect to x and W."""
    N, H, Wd, _ = x.shape
    OH, OW = H // 2, Wd // 2
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    dxp = np.zeros_like(xp)
    dW = np.zeros_like(W)
    dyf = dy.reshape(-1, dy.shape[3])
    for kh in range(4):
        for kw in range(4):
            xs = xp[:, kh:kh + 2 * OH:2, kw:kw + 2 * OW:2, :]
            dW[kh, kw] = xs.reshape(-1, xs.shape[3]).T @ dyf
            dxp[:, kh:kh + 2 * OH:2, kw:kw + 2 * OW:2, :] += dy @ W[kh, kw].T
    return dxp[:, 1:H + 1, 1:Wd + 1, :], dW


def convT_s2(x, W):
    """Transposed convolution, stride 2, pad 1: every input position (ih, iw)
    adds x[n, ih, iw] @ W[kh, kw] to output position (2 ih - 1 + kh, 2 iw - 1 + kw);
    outputs that land outside the 2H x 2W image are dropped."""
    N, H, Wd, _ = x.shape
    yf = np.zeros((N, 2 * H + 2, 2 * Wd + 2, W.shape[3]))
    for kh in range(4):
        for kw in range(4):
            yf[:, kh:kh + 2 * H:2, kw:kw + 2 * Wd:2, :] += x @ W[kh, kw]
    return yf[:, 1:2 * H + 1, 1:2 * Wd + 1, :]


def convT_s2_backward(x, W, dy):
    """Gradients of convT_s2 with respect to x and W."""
    N, H, Wd, _ = x.shape
    dyf = np.pad(dy, ((0, 0), (1, 1), (1, 1), (0, 0)))
    dx = np.zeros_like(x)
    dW = np.zeros_like(W)
    xf = x.reshape(-1, x.shape[3])
    for kh in range(4):
        for kw in range(4):
            ds = dyf[:, kh:kh + 2 * H:2, kw:kw + 2 * Wd:2, :]
            dx += ds @ W[kh, kw].T
            dW[kh, kw] = xf.T @ ds.reshape(-1, ds.shape[3])
    return dx, dW


# ---------------------------------------------------------------------------
# Batch norm over every position of the batch, per channel
# ---------------------------------------------------------------------------
def bn_forward(x, gamma, beta):
    """x [..., C]: statistics over all leading axes.  Returns (y, xhat, rstd)."""
    axes = tuple(range(x.ndim - 1))
    mu = x.mean(axis=axes)
    var = ((x - mu) ** 2).mean(axis=axes)
    rstd = 1.0 / np.sqrt(var + BN_EPS)
    xhat = (x - mu) * rstd
    return gamma * xhat + beta, xhat, rstd


def bn_backward(dy, xhat, rstd, gamma):
    """Returns (dx, dgamma, dbeta) for y = gamma * xhat + beta with batch statistics."""
    axes = tuple(range(dy.ndim - 1))
    dbeta = dy.sum(axis=axes)
    dgamma = (dy * xhat).sum(axis=axes)
    M = dy.size // dy.shape[-1]
    dx = gamma * rstd * (dy - dbeta / M - xhat * (dgamma / M))
    return dx, dgamma, dbeta


def act(name, x, slope):
    if name == "relu":
        return np.maximum(x, 0.0)
    if name == "lrelu":
        return np.where(x > 0.0, x, slope * x)
    if name == "tanh":
        return np.tanh(x)
    if name == "linear":
        return x
    raise ValueError(name)


def act_deriv(name, pre, slope):
    if name == "relu":
        return (pre > 0.0).astype(np.float64)
    if name == "lrelu":
        return np.where(pre > 0.0, 1.0, slope)
    if name == "tanh":
        t = np.tanh(pre)
        return 1.0 - t * t
    if name == "linear":
        return np.ones_like(pre)
    raise ValueError(name)


# ---------------------------------------------------------------------------
# Whole networks
# ---------------------------------------------------------------------------
def forward(arch, p, x, slope):
    """x: [N, z] for G, [N, h*w*c] (flat NHWC) for D.  Returns (cache, out) with
    out [N, h*w*c] (G) or logits [N] (D)."""
    N = x.shape[0]
    h = np.asarray(x, dtype=np.float64)
    if arch.role == "D":
        L0 = arch.layers[0]
        h = h.reshape(N, L0["hin"], L0["hin"], L0["cin"])
    cache = []
    for L in arch.layers:
        W = weights(p, L)
        inp = h
        if L["kind"] == "dense":
            z = inp.reshape(N, -1) @ W
            if arch.role == "G":
                z = z.reshape(N, 4, 4, L["cout"] // 16)
        elif L["kind"] == "conv":
            z = conv_s2(inp, W)
        else:
            z = convT_s2(inp, W)
        if L["bias"]:
            z = z + p[L["off_b"]:L["off_b"] + L["cout"]]
        rec = dict(inp=inp, pre_bn=None, xhat=None, rstd=None)
        if L["bn"]:
            c = bn_channels(L)
            g = p[L["off_g"]:L["off_g"] + c]
            be = p[L["off_be"]:L["off_be"] + c]
            rec["pre_bn"] = z
            z, rec["xhat"], rec["rstd"] = bn_forward(z, g, be)
        rec["pre"] = z
        h = act(L["act"], z, slope)
        cache.append(rec)
    out = h.reshape(N, -1) if arch.role == "G" else h.reshape(N)
    return cache, out


def backward(arch, p, cache, d_out, slope, want_input_grad=False):
    """Back-propagate dLoss/d(out) (G: [N, h*w*c]; D: [N] per logit).

    Returns (flat gradient of p, dLoss/d(input) or None)."""
    grad = np.zeros_like(p)
    N = d_out.shape[0]
    last = arch.layers[-1]
    if arch.role == "G":
        dh = d_out.reshape(N, last["hout"], last["hout"], last["cout"])
    else:
        dh = d_out.reshape(N, 1)
    d_in = None
    for li in range(len(arch.layers) - 1, -1, -1):
        L, rec = arch.layers[li], cache[li]
        W = weights(p, L)
        dz = dh * act_deriv(L["act"], rec["pre"], slope)
        if L["bn"]:
            c = bn_channels(L)
            g = p[L["off_g"]:L["off_g"] + c]
            dz, dg, dbe = bn_backward(dz, rec["xhat"], rec["rstd"], g)
            grad[L["off_g"]:L["off_g"] + c] = dg
            grad[L["off_be"]:L["off_be"] + c] = dbe
        if L["bias"]:
            grad[L["off_b"]:L["off_b"] + L["cout"]] = dz.reshape(-1, L["cout"]).sum(axis=0)
        need_dx = li > 0 or want_input_grad
        inp = rec["inp"]
        if L["kind"] == "dense":
            x2 = inp.reshape(N, -1)
            dz2 = dz.reshape(N, -1)
            grad[L["off_w"]:L["off_w"] + L["n_w"]] = (x2.T @ dz2).ravel()
            dx = (dz2 @ W.T).reshape(inp.shape) if need_dx else None
        elif L["kind"] == "conv":
            dx, dW = conv_s2_backward(inp, W, dz)
            grad[L["off_w"]:L["off_w"] + L["n_w"]] = dW.ravel()
        else:
            dx, dW = convT_s2_backward(inp, W, dz)
            grad[L["off_w"]:L["off_w"] + L["n_w"]] = dW.ravel()
        if li > 0:
            dh = dx
        elif want_input_grad:
            d_in = dx.reshape(N, -1)
    return grad, d_in
