"""Pins of the CPU oracle against things other than itself.

Each test fixes a part of the oracle with an independent statement of the
same mathematics: a brute-force loop, a closed form, an invariant, or a
library routine (torch, float64) that computes the same operator.  A dropped
term, a wrong sign or index, or a transposed operand in the oracle fails at
least one of them.
"""
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2401_16757_amd import workloads as W

RNG = np.random.default_rng(1234)


def brute_conv(x, w, b, stride, pad, dil):
    """Seven nested loops over the definition of 2-D cross-correlation."""
    ci, h, wd = x.shape
    co, _, kh, kw = w.shape
    ho = (h + 2 * pad - dil * (kh - 1) - 1) // stride + 1
    wo = (wd + 2 * pad - dil * (kw - 1) - 1) // stride + 1
    out = np.zeros((co, ho, wo))
    for o in range(co):
        for y in range(ho):
            for xx in range(wo):
                acc = b[o]
                for c in range(ci):
                    for r in range(kh):
                        for s in range(kw):
                            iy = y * stride - pad + r * dil
                            ix = xx * stride - pad + s * dil
                            if 0 <= iy < h and 0 <= ix < wd:
                                acc += w[o, c, r, s] * x[c, iy, ix]
                out[o, y, xx] = acc
    return out


@pytest.mark.parametrize("k,stride,dil,pad", [
    (1, 1, 1, 0), (1, 2, 1, 0), (3, 1, 1, 1), (3, 2, 1, 1), (3, 1, 2, 2), (3, 1, 4, 4),
    (3, 2, 2, 1), (7, 2, 1, 3), (2, 1, 1, 0), (3, 1, 1, 0),
])
def test_conv_matches_brute_force(k, stride, dil, pad):
    ci, co, h, w = 3, 4, 9, 8
    x = RNG.standard_normal((ci, h, w))
    wt = RNG.standard_normal((co, ci, k, k))
    b = RNG.standard_normal(co)
    ref = brute_conv(x, wt, b, stride, pad, dil)
    got = oracle.conv2d(x, wt, b, stride, pad, dil)
    assert got.shape == ref.shape
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("k,stride,dil,pad", [(3, 1, 1, 1), (3, 2, 1, 1), (3, 1, 2, 2),
                                              (3, 1, 4, 4), (7, 2, 1, 3), (1, 2, 1, 0)])
def test_conv_matches_torch_float64(k, stride, dil, pad):
    ci, co, h, w = 8, 16, 17, 15
    x = RNG.standard_normal((ci, h, w))
    wt = RNG.standard_normal((co, ci, k, k))
    b = RNG.standard_normal(co)
    ref = F.conv2d(torch.from_numpy(x)[None], torch.from_numpy(wt), torch.from_numpy(b),
                   stride=stride, padding=pad, dilation=dil)[0].numpy()
    np.testing.assert_allclose(oracle.conv2d(x, wt, b, stride, pad, dil), ref, rtol=0, atol=1e-11)


def test_conv_identity_and_delta_kernels():
    x = RNG.standard_normal((5, 7, 6))
    eye1 = np.eye(5).reshape(5, 5, 1, 1)
    np.testing.assert_array_equal(oracle.conv2d(x, eye1, np.zeros(5)), x)
    delta3 = np.zeros((5, 5, 3, 3))
    delta3[range(5), range(5), 1, 1] = 1.0
    np.testing.assert_array_equal(oracle.conv2d(x, delta3, np.zeros(5), 1, 1, 1), x)
    # dilated centre delta is still the identity
    np.testing.assert_array_equal(oracle.conv2d(x, delta3, np.zeros(5), 1, 2, 2), x)


@pytest.mark.parametrize("r,s", [(0, 0), (0, 2), (2, 1), (1, 0)])
def test_conv_one_hot_tap_is_a_shift(r, s):
    """A single tap (r, s) of a 3x3, pad 1 conv copies the input shifted by
    (r-1, s-1) with zeros entering at the border."""
    x = RNG.standard_normal((1, 6, 7))
    w = np.zeros((1, 1, 3, 3))
    w[0, 0, r, s] = 1.0
    out = oracle.conv2d(x, w, np.zeros(1), 1, 1, 1)
    exp = np.zeros_like(x)
    dy, dx = r - 1, s - 1
    for y in range(6):
        for xx in range(7):
            if 0 <= y + dy < 6 and 0 <= xx + dx < 7:
                exp[0, y, xx] = x[0, y + dy, xx + dx]
    np.testing.assert_array_equal(out, exp)


def test_conv_all_ones_on_constant_counts_taps():
    """All-ones 3x3 (pad 1) on a constant c: c * Cin * (#in-bounds taps), i.e.
    4 at corners, 6 on edges, 9 inside."""
    c, cin = 1.5, 3
    x = np.full((cin, 5, 6), c)
    out = oracle.conv2d(x, np.ones((2, cin, 3, 3)), np.zeros(2), 1, 1, 1)
    taps = np.full((5, 6), 9.0)
    taps[0, :] = taps[-1, :] = 6
    taps[:, 0] = taps[:, -1] = 6
    taps[0, 0] = taps[0, -1] = taps[-1, 0] = taps[-1, -1] = 4
    np.testing.assert_array_equal(out[0], c * cin * taps)
    np.testing.assert_array_equal(out[1], c * cin * taps)


def test_linear_identity_and_one_hot_rows():
    x = RNG.standard_normal(9)
    np.testing.assert_array_equal(oracle.linear(x, np.eye(9)), x)
    w = np.zeros((3, 9))
    w[0, 4] = w[1, 0] = w[2, 8] = 1.0
    np.testing.assert_array_equal(oracle.linear(x, w, np.array([0.0, 1.0, -2.0])),
                                  [x[4], x[0] + 1.0, x[8] - 2.0])
    wr = RNG.standard_normal((4, 9))
    np.testing.assert_allclose(oracle.linear(x, wr), [sum(wr[i, j] * x[j] for j in range(9))
                                                      for i in range(4)], atol=1e-13)


@pytest.mark.parametrize("k,stride,pad", [(3, 2, 1), (2, 2, 0), (3, 1, 1)])
def test_maxpool_matches_torch(k, stride, pad):
    x = RNG.standard_normal((4, 11, 10))
    ref = F.max_pool2d(torch.from_numpy(x)[None], k, stride, pad)[0].numpy()
    np.testing.assert_array_equal(oracle.maxpool(x, k, stride, pad), ref)


def test_maxpool_never_selects_padding():
    x = -np.ones((1, 4, 4)) * 5.0
    assert (oracle.maxpool(x, 3, 2, 1) == -5.0).all()


def test_gavgpool_constant_and_torch():
    np.testing.assert_array_equal(oracle.gavgpool(np.full((3, 7, 7), 2.5)), [2.5] * 3)
    x = RNG.standard_normal((6, 7, 7))
    ref = F.adaptive_avg_pool2d(torch.from_numpy(x)[None], 1)[0, :, 0, 0].numpy()
    np.testing.assert_allclose(oracle.gavgpool(x), ref, atol=1e-14)


@pytest.mark.parametrize("scale,h,w", [(8, 8, 8), (2, 5, 3), (4, 3, 7)])
def test_upsample_matches_torch_bilinear(scale, h, w):
    x = RNG.standard_normal((3, h, w))
    ref = F.interpolate(torch.from_numpy(x)[None], scale_factor=scale, mode="bilinear",
                        align_corners=False)[0].numpy()
    np.testing.assert_allclose(oracle.upsample_bilinear(x, scale), ref, atol=1e-13)


def test_upsample_constant_and_ramp():
    np.testing.assert_allclose(oracle.upsample_bilinear(np.full((2, 4, 4), 3.0), 8), 3.0)
    # an affine ramp in the input grid is reproduced exactly away from the border
    h = w = 6
    yy, xx = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    x = (0.5 * yy - 0.25 * xx + 1.0)[None].astype(np.float64)
    out = oracle.upsample_bilinear(x, 4)
    oy, ox = np.meshgrid(np.arange(4 * h), np.arange(4 * w), indexing="ij")
    sy, sx = (oy + 0.5) / 4 - 0.5, (ox + 0.5) / 4 - 0.5
    inner = (sy >= 0) & (sy <= h - 1) & (sx >= 0) & (sx <= w - 1)
    np.testing.assert_allclose(out[0][inner], (0.5 * sy - 0.25 * sx + 1.0)[inner], atol=1e-13)


def test_bn_fold_equals_explicit_batch_norm():
    """conv(x; W', b') with the folded parameters equals BN(conv(x; W)) with
    the raw statistics (inference batch norm)."""
    net = W.resnet50(res=32)
    li = 5
    layer = net.layers[li]
    wraw = W.conv_weight_raw(net.cfg, li, layer)
    g, beta, mean, var = W.bn_raw(net.cfg, li, layer)
    x = RNG.standard_normal((layer.c_in, 6, 6))
    y = oracle.conv2d(x, wraw, np.zeros(layer.c_out), layer.stride, layer.pad, layer.dilation)
    bn = (y - mean[:, None, None]) / np.sqrt(var[:, None, None] + W.BN_EPS) * g[:, None, None] \
        + beta[:, None, None]
    s = g / np.sqrt(var + W.BN_EPS)
    wf, bf = wraw * s[:, None, None, None], beta - mean * s
    np.testing.assert_allclose(oracle.conv2d(x, wf, bf, layer.stride, layer.pad, layer.dilation),
                               bn, atol=1e-12)
    p = W.layer_params(net, li)
    np.testing.assert_array_equal(p["weight"], wf.astype(np.float16))
    np.testing.assert_array_equal(p["bias"], bf.astype(np.float16))


# ---------------------------------------------------------------------------
# Composition: independent torch float64 builds of each CNN
# ---------------------------------------------------------------------------

def _t(a):
    return torch.from_numpy(np.asarray(a, np.float64))


def _by_name(net, weights):
    return {l.name: weights[i] for i, l in enumerate(net.layers)}


def torch_resnet(x, P, depths, dilate):
    """torchvision-style ResNet v1.5 body in torch float64, wired by hand."""
    def cbr(x, n, stride=1, pad=0, dil=1, relu=True):
        y = F.conv2d(x, _t(P[n]["weight"]), _t(P[n]["bias"]), stride=stride, padding=pad,
                     dilation=dil)
        return F.relu(y) if relu else y
    x = cbr(x, "stem", 2, 3)
    x = F.max_pool2d(x, 3, 2, 1)
    dil = 1
    for si, n in enumerate(depths):
        stride = 1 if si == 0 else 2
        prev = dil
        if dilate[si]:
            dil, stride = dil * stride, 1
        for bi in range(n):
            t = f"s{si + 1}b{bi}"
            d = prev if bi == 0 else dil
            s = stride if bi == 0 else 1
            y = cbr(x, t + "_c1")
            y = cbr(y, t + "_c2", s, d, d)
            y = cbr(y, t + "_c3", relu=False)
            sc = cbr(x, t + "_down", s, relu=False) if bi == 0 else x
            x = F.relu(y + sc)
    return x


def torch_build(net, weights, x):
    P = _by_name(net, weights)
    x = _t(x)[None]
    if net.name == "tiny_cnn":
        for n, s in (("conv1", 1), ("conv2", 2), ("conv3", 2)):
            x = F.relu(F.conv2d(x, _t(P[n]["weight"]), _t(P[n]["bias"]), stride=s, padding=1))
        x = x.mean(dim=(2, 3))[0]
        return (x @ _t(P["fc"]["weight"]).T + _t(P["fc"]["bias"])).numpy()
    if net.name == "resnet50":
        x = torch_resnet(x, P, (3, 4, 6, 3), (False,) * 4)
        x = x.mean(dim=(2, 3))[0]
        return (x @ _t(P["fc"]["weight"]).T + _t(P["fc"]["bias"])).numpy()
    if net.name == "vgg16":
        i = 0
        for v in [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
                  512, 512, 512, "M"]:
            if v == "M":
                x = F.max_pool2d(x, 2, 2)
            else:
                i += 1
                x = F.relu(F.conv2d(x, _t(P[f"conv{i}"]["weight"]), _t(P[f"conv{i}"]["bias"]),
                                    padding=1))
        x = torch.flatten(x, 1)[0]          # (C, H, W) order, as torchvision flattens
        x = F.relu(x @ _t(P["fc1"]["weight"]).T + _t(P["fc1"]["bias"]))
        x = F.relu(x @ _t(P["fc2"]["weight"]).T + _t(P["fc2"]["bias"]))
        return (x @ _t(P["fc3"]["weight"]).T + _t(P["fc3"]["bias"])).numpy()
    if net.name == "fcn_resnet101":
        h = x.shape[-1]
        x = torch_resnet(x, P, (3, 4, 23, 3), (False, False, True, True))
        x = F.conv2d(x, _t(P["classifier"]["weight"]), _t(P["classifier"]["bias"]))
        return F.interpolate(x, size=(h, h), mode="bilinear", align_corners=False)[0].numpy()
    raise KeyError(net.name)


@pytest.mark.parametrize("name,kw", [("tiny_cnn", {}), ("resnet50", {"res": 64}),
                                     ("vgg16", {"res": 32}), ("fcn_resnet101", {"res": 64})])
def test_network_composition_matches_torch_build(name, kw):
    net = W.get_network(name, **kw)
    wts = W.make_weights(net)
    x = W.make_input(net)
    got = oracle.forward(net, wts, x)
    ref = torch_build(net, wts, x)
    assert got.shape == ref.shape
    scale = np.abs(ref).max()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10 * max(scale, 1.0))


def test_vgg_flatten_order_matters():
    """The torch build flattens (C, H, W); a plant of (H, W, C) order in the
    oracle would be caught: the two orders differ on this input."""
    net = W.vgg16(res=64)   # 2x2 spatial before fc1, so the order is visible
    wts = W.make_weights(net)
    x = W.make_input(net)
    ref = torch_build(net, wts, x)
    np.testing.assert_allclose(oracle.forward(net, wts, x), ref, atol=1e-10 * np.abs(ref).max())
    slots = {0: np.asarray(x, np.float64)}
    feat = None
    for li, layer in enumerate(net.layers):
        if layer.name == "fc1":
            feat = slots[layer.src]
        oracle.run_layer(layer, wts[li], slots)
    hwc = np.transpose(feat, (1, 2, 0)).reshape(-1)
    assert not np.allclose(hwc, feat.reshape(-1))


@pytest.mark.parametrize("name,kw", [("tiny_cnn", {}), ("resnet50", {"res": 64})])
def test_block_partition_invariance(name, kw):
    net = W.get_network(name, **kw)
    wts = W.make_weights(net)
    x = W.make_input(net)
    whole = oracle.forward(net, wts, x)
    L = len(net.layers)
    for parts in (net.blocks, [[0, 1], [1, L]], [[i, i + 1] for i in range(L)]):
        np.testing.assert_array_equal(oracle.forward_blocks(net, wts, x, parts), whole)


# ---------------------------------------------------------------------------
# Decoder pieces
# ---------------------------------------------------------------------------

def test_rmsnorm_unit_rms_and_gain():
    h = RNG.standard_normal((5, 64)) * 3.0
    y = oracle.rmsnorm(h, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt((y * y).mean(axis=1)), 1.0, atol=1e-14)
    g = RNG.standard_normal(64)
    np.testing.assert_allclose(oracle.rmsnorm(h, g, 1e-5), oracle.rmsnorm(h, np.ones(64), 1e-5) * g)


def test_rope_closed_forms():
    x = RNG.standard_normal((4, 3, 16))
    # position 0 is the identity
    np.testing.assert_allclose(oracle.rope(x, np.zeros(4), 10000.0), x, atol=0)
    # rotations preserve the norm of every head vector
    y = oracle.rope(x, np.arange(4) * 7, 10000.0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)
    # complex form: (a + i b) * exp(i p theta^(-2j/hd))
    hd, half = 16, 8
    p = np.arange(4) * 7.0
    z = x[..., :half] + 1j * x[..., half:]
    rot = np.exp(1j * p[:, None, None] * 10000.0 ** (-2.0 * np.arange(half) / hd))
    zr = z * rot
    np.testing.assert_allclose(y, np.concatenate([zr.real, zr.imag], -1), atol=1e-12)


def test_attention_single_key_returns_value_and_matches_torch():
    q = RNG.standard_normal((1, 2, 8))
    k = RNG.standard_normal((1, 2, 8))
    v = RNG.standard_normal((1, 2, 8))
    np.testing.assert_allclose(oracle.causal_attention(q, k, v), v, atol=1e-15)
    t, h, d = 9, 3, 16
    q, k, v = (RNG.standard_normal((t, h, d)) for _ in range(3))
    ref = F.scaled_dot_product_attention(*(torch.from_numpy(a).transpose(0, 1)[None]
                                           for a in (q, k, v)), is_causal=True)
    ref = ref[0].transpose(0, 1).numpy()
    np.testing.assert_allclose(oracle.causal_attention(q, k, v), ref, atol=1e-13)


def small_decoder():
    return W.decoder7b(n_layers=2, d=64, heads=4, ffn=96, vocab=50, max_seq=24, prompt=12, gen=4)


def torch_decoder(net, wts, ids):
    """Independent torch float64 decoder forward (Llama-style)."""
    P = _by_name(net, wts)
    E = net.extra
    d, nh = E["d"], E["heads"]
    hd = d // nh
    T = len(ids)
    h = _t(P["embed"]["table"])[torch.as_tensor(ids, dtype=torch.long)]

    def norm(v, g):
        return v * torch.rsqrt(v.pow(2).mean(-1, keepdim=True) + 1e-5) * _t(g)
    inv = 1.0 / (10000.0 ** (torch.arange(0, hd, 2, dtype=torch.float64) / hd))
    ang = torch.arange(T, dtype=torch.float64)[:, None] * inv[None]
    cos, sin = ang.cos()[:, None], ang.sin()[:, None]

    def rot(x):
        a, b = x[..., :hd // 2], x[..., hd // 2:]
        return torch.cat([a * cos - b * sin, a * sin + b * cos], -1)
    for l in range(E["n_layers"]):
        p = f"l{l}_"
        a = norm(h, P[p + "attn_norm"]["gain"])
        qkv = P[p + "qkv"]
        q = rot((a @ _t(qkv["wq"]).T).view(T, nh, hd))
        k = rot((a @ _t(qkv["wk"]).T).view(T, nh, hd))
        v = (a @ _t(qkv["wv"]).T).view(T, nh, hd)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1),
                                           v.transpose(0, 1), is_causal=True)
        h = h + o.transpose(0, 1).reshape(T, d) @ _t(P[p + "wo"]["weight"]).T
        m = norm(h, P[p + "ffn_norm"]["gain"])
        g = P[p + "gateup"]
        h = h + (F.silu(m @ _t(g["w1"]).T) * (m @ _t(g["w3"]).T)) @ _t(P[p + "w2"]["weight"]).T
    return (norm(h, P["final_norm"]["gain"]) @ _t(P["lm_head"]["weight"]).T).numpy()


def test_decoder_matches_torch_build():
    net = small_decoder()
    wts = W.make_weights(net)
    ids = W.make_input(net)
    got = oracle.decoder_forward(net, wts, ids)
    ref = torch_decoder(net, wts, ids)
    np.testing.assert_allclose(got, ref, atol=1e-10 * np.abs(ref).max())


def test_decoder_prefix_invariance():
    """Causality: the logits of position t depend only on ids[0..t], so the
    pass over a prefix reproduces the first rows of the pass over the whole
    sequence (decode step == prefill row)."""
    net = small_decoder()
    wts = W.make_weights(net)
    ids = W.make_input(net)
    full = oracle.decoder_forward(net, wts, ids)
    for t in (1, 5, len(ids)):
        np.testing.assert_allclose(oracle.decoder_forward(net, wts, ids[:t]), full[:t],
                                   atol=1e-12 * np.abs(full).max())


# ---------------------------------------------------------------------------
# Generator
# ---------------------------------------------------------------------------

def test_generator_statistics_and_determinism():
    net = W.resnet50(res=32)
    li = 10
    layer = net.layers[li]
    w = W.conv_weight_raw(net.cfg, li, layer)
    std = math.sqrt(2.0 / (layer.c_in * layer.k * layer.k))
    n = w.size
    assert abs(w.mean()) < 4 * std / math.sqrt(n)
    assert abs(w.std() / std - 1.0) < 4 / math.sqrt(2 * n)
    a = W.layer_params(net, li)
    b = W.layer_params(net, li)
    for k in a:
        assert a[k].dtype == np.float16
        np.testing.assert_array_equal(a[k], b[k])
    x = W.make_input(net)
    assert abs(float(x.astype(np.float64).mean())) < 4 / math.sqrt(x.size)
    np.testing.assert_array_equal(x, W.make_input(net))


def test_workload_sizes():
    """Parameter counts and byte totals of the five workloads (fp16, batch
    norm folded into one bias per channel)."""
    exp = {"tiny_cnn": (24234, 29081), "resnet50": (25530472, 22009028),
           "vgg16": (138357544, 47627382), "fcn_resnet101": (42490517, 28327011),
           "decoder7b": (6738415616, 1619066880)}
    for name, (params, budget) in exp.items():
        net = W.get_network(name)
        assert net.param_count() == params, name
        assert net.weight_bytes() == 2 * params
        assert net.budget_bytes() == budget, name
