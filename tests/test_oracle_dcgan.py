"""Pins of the oracle's convolutional networks: each convolution, transposed
convolution and batch norm against torch's CPU fp64 library routines, whole
networks and their gradients against torch autograd, finite differences, the
parameter count of the 64x64 workload, initial statistics, the BCE closed
form and, on a 1x1 grid, a textbook torch GAN + Adam loop."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import coevo, dcgan, rng


def _t(a):
    return torch.tensor(a, dtype=torch.float64)


def _nchw(x):
    return _t(x).permute(0, 3, 1, 2)


def _nhwc(x):
    return x.permute(0, 2, 3, 1).detach().numpy()


def test_conv_s2_is_torch_conv2d():
    r = np.random.default_rng(0)
    x = r.normal(size=(3, 8, 8, 5))
    W = r.normal(size=(4, 4, 5, 7))
    ref = F.conv2d(_nchw(x), _t(W).permute(3, 2, 0, 1), stride=2, padding=1)
    assert np.allclose(dcgan.conv_s2(x, W), _nhwc(ref), rtol=1e-12, atol=1e-12)


def test_convT_s2_is_torch_conv_transpose2d():
    r = np.random.default_rng(1)
    x = r.normal(size=(2, 4, 4, 6))
    W = r.normal(size=(4, 4, 6, 3))
    ref = F.conv_transpose2d(_nchw(x), _t(W).permute(2, 3, 0, 1), stride=2, padding=1)
    assert ref.shape[2:] == (8, 8)
    assert np.allclose(dcgan.convT_s2(x, W), _nhwc(ref), rtol=1e-12, atol=1e-12)


def test_conv_backward_matches_autograd():
    r = np.random.default_rng(2)
    for conv, tfn, wperm, shape in (
            (dcgan.conv_s2_backward, lambda a, w: F.conv2d(a, w, stride=2, padding=1), (3, 2, 0, 1), (2, 8, 8, 3)),
            (dcgan.convT_s2_backward, lambda a, w: F.conv_transpose2d(a, w, stride=2, padding=1), (2, 3, 0, 1),
             (2, 4, 4, 3))):
        x = r.normal(size=shape)
        W = r.normal(size=(4, 4, 3, 5))
        xt = _nchw(x).requires_grad_(True)
        Wt = _t(W).requires_grad_(True)
        y = tfn(xt, Wt.permute(*wperm))
        dy = r.normal(size=tuple(y.shape))
        y.backward(_t(dy))
        dx, dW = conv(x, W, _nhwc(_t(dy)))
        assert np.allclose(dx, _nhwc(xt.grad), rtol=1e-11, atol=1e-12)
        assert np.allclose(dW, Wt.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_dense_first_generator_layer_is_a_4x4_transposed_convolution():
    """G's layer 1, stored as a [z][(y, x, c)] matrix, is the stride-1, pad-0
    4x4 transposed convolution of the 1x1 latent map."""
    r = np.random.default_rng(3)
    z = r.normal(size=(3, 6))
    W = r.normal(size=(6, 4 * 4 * 5))
    y = (z @ W).reshape(3, 4, 4, 5)
    Wt = _t(W).view(6, 4, 4, 5).permute(0, 3, 1, 2)          # [ci][co][kh][kw]
    ref = F.conv_transpose2d(_t(z).view(3, 6, 1, 1), Wt, stride=1, padding=0)
    assert np.allclose(y, _nhwc(ref), rtol=1e-12, atol=1e-12)


def test_dense_last_discriminator_layer_is_a_4x4_convolution():
    r = np.random.default_rng(4)
    h = r.normal(size=(3, 4, 4, 5))
    W = r.normal(size=(4 * 4 * 5, 1))
    ref = F.conv2d(_nchw(h), _t(W).view(4, 4, 5, 1).permute(3, 2, 0, 1))
    assert np.allclose(h.reshape(3, -1) @ W, ref.view(3, 1).numpy(), rtol=1e-12, atol=1e-12)


def test_batch_norm_is_torch_batch_norm_with_batch_statistics():
    r = np.random.default_rng(5)
    x = r.normal(2.0, 3.0, size=(4, 3, 3, 6))
    g, b = r.normal(size=6), r.normal(size=6)
    y, xhat, rstd = dcgan.bn_forward(x, g, b)
    ref = F.batch_norm(_nchw(x), None, None, _t(g), _t(b), training=True, eps=dcgan.BN_EPS)
    assert np.allclose(y, _nhwc(ref), rtol=1e-12, atol=1e-12)
    # backward against autograd
    xt = _nchw(x).requires_grad_(True)
    gt, bt = _t(g).requires_grad_(True), _t(b).requires_grad_(True)
    yt = F.batch_norm(xt, None, None, gt, bt, training=True, eps=dcgan.BN_EPS)
    dy = r.normal(size=tuple(yt.shape))
    yt.backward(_t(dy))
    dx, dg, db = dcgan.bn_backward(_nhwc(_t(dy)), xhat, rstd, g)
    assert np.allclose(dx, _nhwc(xt.grad), rtol=1e-10, atol=1e-12)
    assert np.allclose(dg, gt.grad.numpy(), rtol=1e-11) and np.allclose(db, bt.grad.numpy(), rtol=1e-11)


def _small_wl(**kw):
    base = dict(rows=2, cols=2, img=(16, 16, 3), x_dim=16 * 16 * 3, z_dim=8,
                g_hidden=[16, 8], d_hidden=[8, 16], batch=4, steps=2,
                data=dict(n=256, h=16, w=16))
    base.update(kw)
    return synth.small_workload("celeba_dcgan_4x4", **base)


def test_parameter_count_of_the_64x64_networks():
    wl = synth.workload("celeba_dcgan_4x4")
    G = dcgan.Arch("G", 100, (64, 64, 3), wl["g_hidden"], wl["d_hidden"])
    D = dcgan.Arch("D", 100, (64, 64, 3), wl["g_hidden"], wl["d_hidden"])
    # G: 100*8192 + 2*512 | 16*512*256 + 2*256 | 16*256*128 + 2*128 | 16*128*64 + 2*64 | 16*64*3 + 3
    assert G.P == 819200 + 1024 + 2097152 + 512 + 524288 + 256 + 131072 + 128 + 3072 + 3
    # D: 16*3*64 + 64 | 16*64*128 + 128 | 16*128*256 + 256 | 16*256*512 + 512 | 8192 + 1
    assert D.P == 3136 + 131200 + 524544 + 2097664 + 8193
    assert G.P + D.P == 6341444


def test_init_statistics():
    wl = synth.workload("celeba_dcgan_4x4")
    G = dcgan.Arch("G", 100, (64, 64, 3), wl["g_hidden"], wl["d_hidden"])
    p = dcgan.init(G, 0, 1, "INIT_G")
    L2 = G.layers[1]
    W = p[L2["off_w"]:L2["off_w"] + L2["n_w"]]
    assert abs(W.mean()) < 1e-4 and abs(W.std() - 0.02) < 2e-4
    g = p[L2["off_g"]:L2["off_g"] + L2["cout"]]
    assert abs(g.mean() - 1.0) < 0.01 and np.all(p[L2["off_be"]:L2["off_be"] + L2["cout"]] == 0)
    L5 = G.layers[-1]
    assert np.all(p[L5["off_b"]:L5["off_b"] + L5["cout"]] == 0)
    # element e is normal number e of the role's stream
    n = rng.normals(0, 16, 1, 0, 0, "INIT_G")
    assert np.allclose(p[:16], 0.02 * n, rtol=0, atol=0)


def _torch_net(arch, pt, x, slope):
    """The same network written with torch's own layers (NCHW)."""
    N = x.shape[0]
    h = x
    if arch.role == "D":
        L0 = arch.layers[0]
        h = h.view(N, L0["hin"], L0["hin"], L0["cin"]).permute(0, 3, 1, 2)
    for L in arch.layers:
        W = pt[L["off_w"]:L["off_w"] + L["n_w"]]
        b = pt[L["off_b"]:L["off_b"] + L["cout"]] if L["bias"] else None
        if L["kind"] == "dense" and arch.role == "G":
            Wt = W.view(L["cin"], 4, 4, L["cout"] // 16).permute(0, 3, 1, 2).contiguous()
            h = F.conv_transpose2d(h.view(N, L["cin"], 1, 1), Wt, b)
        elif L["kind"] == "dense":
            Wc = W.view(4, 4, L["cin"] // 16, 1).permute(3, 2, 0, 1).contiguous()
            h = F.conv2d(h, Wc, b).view(N)
        elif L["kind"] == "conv":
            h = F.conv2d(h, W.view(4, 4, L["cin"], L["cout"]).permute(3, 2, 0, 1).contiguous(), b,
                         stride=2, padding=1)
        else:
            h = F.conv_transpose2d(h, W.view(4, 4, L["cin"], L["cout"]).permute(2, 3, 0, 1).contiguous(),
                                   b, stride=2, padding=1)
        if L["bn"]:
            c = dcgan.bn_channels(L)
            h = F.batch_norm(h, None, None, pt[L["off_g"]:L["off_g"] + c], pt[L["off_be"]:L["off_be"] + c],
                             training=True, eps=dcgan.BN_EPS)
        if L["act"] == "relu":
            h = torch.relu(h)
        elif L["act"] == "lrelu":
            h = F.leaky_relu(h, slope)
        elif L["act"] == "tanh":
            h = torch.tanh(h)
    if arch.role == "G":
        h = h.permute(0, 2, 3, 1).reshape(N, -1)
    return h


@pytest.mark.parametrize("role", ["G", "D"])
def test_network_forward_and_gradients_match_torch(role):
    wl = _small_wl()
    S = coevo.Setup(wl, 10)
    net = S.Gnet if role == "G" else S.Dnet
    r = np.random.default_rng(6)
    p = net.init(0, 1, "INIT_" + role)
    p += 0.05 * r.normal(size=p.shape)          # non-zero biases and betas
    x = r.normal(size=(5, wl["z_dim"] if role == "G" else wl["x_dim"]))
    cache, out = net.forward(p, x)
    pt = _t(p).requires_grad_(True)
    xt = _t(x).requires_grad_(True)
    ref = _torch_net(net.arch, pt, xt, wl["lrelu_slope"])
    assert np.allclose(out, ref.detach().numpy(), rtol=1e-10, atol=1e-12)
    d_out = r.normal(size=out.shape)
    ref.backward(_t(d_out))
    grad, d_in = net.backward(p, cache, d_out, want_input_grad=True)
    assert np.allclose(grad, pt.grad.numpy(), rtol=1e-9, atol=1e-11)
    assert np.allclose(d_in, xt.grad.numpy(), rtol=1e-9, atol=1e-11)


def test_gradients_match_central_differences():
    wl = _small_wl(g_hidden=[4, 4], d_hidden=[4, 4], z_dim=3)
    S = coevo.Setup(wl, 10)
    r = np.random.default_rng(7)
    for net in (S.Gnet, S.Dnet):
        p = net.init(0, 0, "INIT_" + net.role) + 0.05 * r.normal(size=net.P)
        x = r.normal(size=(3, wl["z_dim"] if net.role == "G" else wl["x_dim"]))
        _, out = net.forward(p, x)
        w = r.normal(size=out.shape)
        cache, _ = net.forward(p, x)
        grad, _ = net.backward(p, cache, w)
        # one index in every parameter section of every layer
        idx = []
        for L in net.arch.layers:
            idx.append(L["off_w"] + L["n_w"] // 3)
            for k in ("off_b", "off_g", "off_be"):
                if L[k] is not None:
                    idx.append(L[k] + 1 if L["cout"] > 1 else L[k])
        h = 1e-6
        for i in idx:
            pp, pm = p.copy(), p.copy()
            pp[i] += h
            pm[i] -= h
            fd = ((net.forward(pp, x)[1] * w).sum() - (net.forward(pm, x)[1] * w).sum()) / (2 * h)
            assert abs(fd - grad[i]) <= 1e-6 * max(1.0, abs(fd)), (net.role, i, fd, grad[i])


def test_bce_closed_form_at_half():
    wl = _small_wl()
    data = synth.make_dataset(wl["data"])
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    last = S.Dnet.arch.layers[-1]
    st.Dp[:, last["off_w"]:] = 0.0
    L, Lg, fg, fd = coevo.evaluate(S, st, data, 0)
    assert np.allclose(L, 2 * math.log(2), rtol=0, atol=1e-15)
    assert np.allclose(Lg, math.log(2), rtol=0, atol=1e-15)


@pytest.mark.parametrize("loss", ["bce", "wasserstein"])
def test_one_by_one_grid_is_plain_gan_training(loss):
    """On a 1x1 torus a generation is textbook alternating GAN training (for
    the Wasserstein trainer: critic loss mean D(fake) - mean D(real), the
    critic clamped after its step, generator loss -mean D(fake))."""
    wl = _small_wl(rows=1, cols=1, lr_mutation=0, steps=3, lr0_g=2e-3, lr0_d=2e-3, loss=loss, wgan_clip=0.05)
    wgan = loss == "wasserstein"
    data = synth.make_dataset(wl["data"])
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    new, rec = coevo.generation(S, st, data, 1)
    Gp = _t(st.Gp[0]).requires_grad_(True)
    Dp = _t(st.Dp[0]).requires_grad_(True)
    b = (wl["beta1"], wl["beta2"])
    og = torch.optim.Adam([Gp], lr=float(st.Glr[0]), betas=b, eps=wl["eps"])
    od = torch.optim.Adam([Dp], lr=float(st.Dlr[0]), betas=b, eps=wl["eps"])
    bce = F.binary_cross_entropy_with_logits
    slope = wl["lrelu_slope"]
    for s in range(wl["steps"]):
        idx = rng.indices(S.seed, S.B, S.N, 0, 1, s + 1)
        z = _t(rng.normals(S.seed, S.B * S.zd, 0, 1, s + 1, "Z").reshape(S.B, S.zd))
        x = _t(data[idx])
        xf = _torch_net(S.Gnet.arch, Gp, z, slope)
        ar = _torch_net(S.Dnet.arch, Dp, x, slope)
        af = _torch_net(S.Dnet.arch, Dp, xf.detach(), slope)
        ld = af.mean() - ar.mean() if wgan else bce(ar, torch.ones_like(ar)) + bce(af, torch.zeros_like(af))
        od.zero_grad()
        ld.backward()
        od.step()
        if wgan:
            with torch.no_grad():
                Dp.clamp_(-0.05, 0.05)
        af2 = _torch_net(S.Dnet.arch, Dp, xf, slope)
        lg = -af2.mean() if wgan else bce(af2, torch.ones_like(af2))
        og.zero_grad()
        lg.backward()
        og.step()
        assert np.isclose(rec["losses"][s, 0, 0], ld.item(), rtol=1e-10)
        assert np.isclose(rec["losses"][s, 0, 1], lg.item(), rtol=1e-10)
    assert np.allclose(new.Gp[0], Gp.detach().numpy(), rtol=1e-9, atol=1e-12)
    assert np.allclose(new.Dp[0], Dp.detach().numpy(), rtol=1e-9, atol=1e-12)


def test_wasserstein_constant_critic_closed_form():
    """A critic whose weights are all zero outputs its output bias b for every
    image: the critic loss is exactly 0 and the generator loss exactly -b."""
    wl = _small_wl(loss="wasserstein")
    data = synth.make_dataset(wl["data"])
    S = coevo.Setup(wl, len(data))
    st = coevo.create(S)
    last = S.Dnet.arch.layers[-1]
    st.Dp[...] = 0.0
    st.Dp[:, last["off_b"]] = 0.37
    L, Lg, fg, fd = coevo.evaluate(S, st, data, 0)
    assert np.all(L == 0.0) and np.all(Lg == -0.37)
    assert np.all(fd == 0.0)
