"""Seeded synthetic workloads: network descriptions, weights and inputs.

This module describes the five networks the swap engine is measured on and
draws their parameters and inputs from fixed seeds.  It holds no forward-pass
arithmetic: the engine (through ``swapnet``) and the CPU oracle both consume
the arrays made here and compute on their own.

The networks are shaped like the workloads of the paper's evaluation (Sec. 7:
VGG, ResNet and FCN classification/segmentation models) plus a 7B-shaped
decoder, which the paper names as outside its design (Sec. 9).  No trained
weights or datasets are used: every tensor is synthetic.

Seeding (one stream per tensor, so any tensor can be regenerated alone):
  weights of layer ``li``, tensor ``ti``  -> SeedSequence([cfg, 0, li, ti])
  network input                            -> SeedSequence([cfg, 1])
Draws are fp64 (the decoder's N(0, 0.02) tensors: fp32, to keep the 6.7B
generator near a minute); folding of batch-norm statistics is done in fp64;
every stored tensor is then rounded once to fp16 (round-to-nearest-even).

Batch-norm statistics are data-independent (running mean ~ N(0, 0.1),
running variance ~ U(0.5, 1.5), gamma ~ U(0.5, 1.5), beta ~ N(0, 0.1)); the
gamma of the last batch-norm in every residual branch is multiplied by
1/sqrt(L), L = number of residual blocks, so that the residual stream stays
O(1) at depth 33 instead of overflowing fp16.
"""
from __future__ import annotations

import concurrent.futures
import math
import os
from dataclasses import dataclass, field

import numpy as np

BN_EPS = 1e-5

# Config indices used as the first seed word.
CFG_TINY, CFG_RESNET50, CFG_VGG16, CFG_FCN_R101, CFG_DECODER7B = 1, 2, 3, 4, 5


@dataclass
class LayerSpec:
    """One layer in execution order.

    ``src``/``dst``/``res`` are activation slot ids.  Slot 0 holds the network
    input.  ``res`` (>= 0) is added before the fused ReLU.
    Canonical parameter layouts (what the engine receives):
      conv2d : weight [c_out][c_in][k][k], bias [c_out]
      linear : weight [c_out][c_in],       bias [c_out] (optional)
      rmsnorm: gain [c_in]
      qkv    : wq, wk, wv [d][d]  (engine sees them row-stacked)
      gateup : w1, w3 [f][d]      (engine sees them row-stacked, SwiGLU output)
      embed  : table [vocab][d]
    """
    name: str
    op: str
    src: int
    dst: int
    res: int = -1
    c_in: int = 0
    c_out: int = 0
    h_in: int = 1
    w_in: int = 1
    k: int = 1
    stride: int = 1
    pad: int = 0
    dilation: int = 1
    relu: bool = False
    flatten_chw: bool = False   # linear over a CHW-flattened spatial input
    scale: int = 1              # upsample factor
    heads: int = 0
    head_dim: int = 0
    kv_layer: int = -1
    eps: float = 0.0
    theta: float = 0.0
    out_f32: bool = False
    # generator recipe (not used by the compute side)
    bn: bool = False            # conv followed by batch-norm (folded)
    bn_damp: float = 1.0        # multiplier on that batch-norm's gamma
    bias_std: float = 0.1       # std of a plain (non-BN) bias; 0 -> no bias
    w_std: float = 0.0          # 0 -> He-normal, else N(0, w_std)

    def out_hw(self):
        if self.op == "conv2d":
            ho = (self.h_in + 2 * self.pad - self.dilation * (self.k - 1) - 1) // self.stride + 1
            wo = (self.w_in + 2 * self.pad - self.dilation * (self.k - 1) - 1) // self.stride + 1
            return ho, wo
        if self.op == "maxpool":
            ho = (self.h_in + 2 * self.pad - self.k) // self.stride + 1
            wo = (self.w_in + 2 * self.pad - self.k) // self.stride + 1
            return ho, wo
        if self.op == "upsample_bilinear":
            return self.h_in * self.scale, self.w_in * self.scale
        return 1, 1

    def param_shapes(self):
        """Canonical parameter shapes in the order the tensors are seeded."""
        if self.op == "conv2d":
            return {"weight": (self.c_out, self.c_in, self.k, self.k), "bias": (self.c_out,)}
        if self.op == "linear":
            d = {"weight": (self.c_out, self.c_in)}
            if self.bias_std > 0:
                d["bias"] = (self.c_out,)
            return d
        if self.op == "rmsnorm":
            return {"gain": (self.c_in,)}
        if self.op == "qkv":
            d = self.c_in
            return {"wq": (d, d), "wk": (d, d), "wv": (d, d)}
        if self.op == "gateup":
            return {"w1": (self.c_out, self.c_in), "w3": (self.c_out, self.c_in)}
        if self.op == "embed":
            return {"table": (self.c_out, self.c_in)}
        return {}

    def weight_bytes(self):
        return sum(2 * int(np.prod(s)) for s in self.param_shapes().values())


@dataclass
class Network:
    name: str
    cfg: int
    layers: list
    blocks: list                # list of [first, last) layer index ranges
    input_shape: tuple          # (C, H, W) for images; (T,) for token ids
    out_slot: int
    budget_fraction: float = 1.0
    budget_bytes_fixed: int = 0
    kind: str = "cnn"           # "cnn" or "decoder"
    extra: dict = field(default_factory=dict)

    def weight_bytes(self):
        return sum(l.weight_bytes() for l in self.layers)

    def streamed_weight_bytes(self):
        """Bytes of the weights that live in blocks (the embedding table is
        gathered row by row and is not a block)."""
        return sum(l.weight_bytes() for l in self.layers if l.op != "embed")

    def budget_bytes(self):
        if self.budget_bytes_fixed:
            return self.budget_bytes_fixed
        return int(round(self.weight_bytes() * self.budget_fraction))

    def param_count(self):
        return sum(int(np.prod(s)) for l in self.layers for s in l.param_shapes().values())


class _Builder:
    def __init__(self):
        self.layers = []
        self.nslots = 1  # slot 0 = input

    def new_slot(self):
        s = self.nslots
        self.nslots += 1
        return s

    def add(self, **kw):
        kw.setdefault("dst", self.new_slot())
        self.layers.append(LayerSpec(**kw))
        return self.layers[-1].dst


# ----------------------------------------------------------------------------
# Network descriptions
# ----------------------------------------------------------------------------

def tiny_cnn():
    """Three 3x3 convs (pad 1, folded BN, ReLU), global average pool, linear 64->10."""
    b = _Builder()
    x = b.add(name="conv1", op="conv2d", src=0, c_in=3, c_out=16, h_in=32, w_in=32,
              k=3, stride=1, pad=1, relu=True, bn=True)
    x = b.add(name="conv2", op="conv2d", src=x, c_in=16, c_out=32, h_in=32, w_in=32,
              k=3, stride=2, pad=1, relu=True, bn=True)
    x = b.add(name="conv3", op="conv2d", src=x, c_in=32, c_out=64, h_in=16, w_in=16,
              k=3, stride=2, pad=1, relu=True, bn=True)
    x = b.add(name="pool", op="gavgpool", src=x, c_in=64, c_out=64, h_in=8, w_in=8)
    x = b.add(name="fc", op="linear", src=x, c_in=64, c_out=10)
    return Network("tiny_cnn", CFG_TINY, b.layers, [[0, 2], [2, 5]], (3, 32, 32), x,
                   budget_fraction=0.6)


def _resnet_body(b, depths, res, dilate, n_res_blocks):
    """Stem + bottleneck stages (v1.5: stride on the 3x3).  ``dilate[s]``
    replaces stage s's stride by dilation (torchvision convention: the first
    3x3 of a dilated stage keeps the previous dilation).  Returns (slot, C, H,
    W, list of (stage, block, first layer index))."""
    damp = 1.0 / math.sqrt(n_res_blocks)
    x = b.add(name="stem", op="conv2d", src=0, c_in=3, c_out=64, h_in=res, w_in=res,
              k=7, stride=2, pad=3, relu=True, bn=True)
    h = (res + 6 - 7) // 2 + 1
    x = b.add(name="maxpool", op="maxpool", src=x, c_in=64, c_out=64, h_in=h, w_in=h,
              k=3, stride=2, pad=1)
    h = (h + 2 - 3) // 2 + 1
    cin, dil = 64, 1
    starts = []
    for si, (n, w) in enumerate(zip(depths, (64, 128, 256, 512))):
        stride = 1 if si == 0 else 2
        prev_dil = dil
        if dilate[si]:
            dil *= stride
            stride = 1
        for bi in range(n):
            starts.append((si, bi, len(b.layers)))
            s = stride if bi == 0 else 1
            d = prev_dil if bi == 0 else dil
            tag = f"s{si + 1}b{bi}"
            y = b.add(name=tag + "_c1", op="conv2d", src=x, c_in=cin, c_out=w, h_in=h, w_in=h,
                      k=1, relu=True, bn=True)
            y = b.add(name=tag + "_c2", op="conv2d", src=y, c_in=w, c_out=w, h_in=h, w_in=h,
                      k=3, stride=s, pad=d, dilation=d, relu=True, bn=True)
            ho = (h + 2 * d - d * 2 - 1) // s + 1
            if bi == 0:
                sc = b.add(name=tag + "_down", op="conv2d", src=x, c_in=cin, c_out=4 * w,
                           h_in=h, w_in=h, k=1, stride=s, relu=False, bn=True)
            else:
                sc = x
            x = b.add(name=tag + "_c3", op="conv2d", src=y, res=sc, c_in=w, c_out=4 * w,
                      h_in=ho, w_in=ho, k=1, relu=True, bn=True, bn_damp=damp)
            cin, h = 4 * w, ho
    return x, cin, h, starts


def resnet50(res=224):
    b = _Builder()
    x, c, h, starts = _resnet_body(b, (3, 4, 6, 3), res, (False,) * 4, 16)
    x = b.add(name="avgpool", op="gavgpool", src=x, c_in=c, c_out=c, h_in=h, w_in=h)
    x = b.add(name="fc", op="linear", src=x, c_in=c, c_out=1000)
    first = {(s, bi): li for s, bi, li in starts}
    cuts = [0, first[(1, 0)], first[(2, 0)], first[(2, 3)], first[(3, 0)], first[(3, 1)],
            first[(3, 2)], len(b.layers) - 2, len(b.layers)]
    blocks = [[cuts[i], cuts[i + 1]] for i in range(8)]
    return Network("resnet50", CFG_RESNET50, b.layers, blocks, (3, res, res), x,
                   budget_fraction=1 / 2.32)


def vgg16(res=224):
    b = _Builder()
    cfg = [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
           512, 512, 512, "M"]
    x, c, h, n = 0, 3, res, 0
    block_ends = []
    for v in cfg:
        if v == "M":
            x = b.add(name=f"pool{len(block_ends) + 1}", op="maxpool", src=x, c_in=c, c_out=c,
                      h_in=h, w_in=h, k=2, stride=2)
            h //= 2
            block_ends.append(len(b.layers))
        else:
            n += 1
            x = b.add(name=f"conv{n}", op="conv2d", src=x, c_in=c, c_out=v, h_in=h, w_in=h,
                      k=3, pad=1, relu=True)
            c = v
    x = b.add(name="fc1", op="linear", src=x, c_in=c * h * h, c_out=4096, h_in=h, w_in=h,
              relu=True, flatten_chw=True)
    x = b.add(name="fc2", op="linear", src=x, c_in=4096, c_out=4096, relu=True)
    x = b.add(name="fc3", op="linear", src=x, c_in=4096, c_out=1000)
    L = len(b.layers)
    # conv1_1..conv3_3 (+pools) | conv4 | conv5 | fc1 | fc2 | fc3
    cuts = [0, block_ends[2], block_ends[3], block_ends[4], L - 2, L - 1, L]
    blocks = [[cuts[i], cuts[i + 1]] for i in range(len(cuts) - 1)]
    return Network("vgg16", CFG_VGG16, b.layers, blocks, (3, res, res), x,
                   budget_fraction=1 / 5.81)


def fcn_resnet101(res=512):
    b = _Builder()
    x, c, h, starts = _resnet_body(b, (3, 4, 23, 3), res, (False, False, True, True), 33)
    x = b.add(name="classifier", op="conv2d", src=x, c_in=c, c_out=21, h_in=h, w_in=h, k=1,
              bn=False, bias_std=0.1)
    x = b.add(name="upsample", op="upsample_bilinear", src=x, c_in=21, c_out=21, h_in=h,
              w_in=h, scale=8)
    first = {(s, bi): li for s, bi, li in starts}
    cuts = [0, first[(2, 0)]]
    for r in (3, 6, 9, 12, 15, 18, 21):
        cuts.append(first[(2, r)])
    cuts += [first[(3, 0)], first[(3, 1)], first[(3, 2)], len(b.layers)]
    blocks = [[cuts[i], cuts[i + 1]] for i in range(len(cuts) - 1)]
    return Network("fcn_resnet101", CFG_FCN_R101, b.layers, blocks, (3, res, res), x,
                   budget_fraction=1 / 3)


def decoder7b(n_layers=32, d=4096, heads=32, ffn=11008, vocab=32000, max_seq=640,
              prompt=512, gen=128):
    """Llama-shaped decoder.  Slot 0 = residual stream h [T][d] (updated in
    place), 1 = normed, 2 = qkv, 3 = attention output, 4 = SwiGLU output,
    5 = logits (fp32)."""
    L = []
    hd = d // heads
    L.append(LayerSpec(name="embed", op="embed", src=-1, dst=0, c_in=d, c_out=vocab,
                       w_std=0.02))
    for l in range(n_layers):
        p = f"l{l}_"
        L.append(LayerSpec(name=p + "attn_norm", op="rmsnorm", src=0, dst=1, c_in=d, c_out=d,
                           eps=1e-5))
        L.append(LayerSpec(name=p + "qkv", op="qkv", src=1, dst=2, c_in=d, c_out=3 * d,
                           w_std=0.02))
        L.append(LayerSpec(name=p + "attn", op="attention", src=2, dst=3, c_in=3 * d, c_out=d,
                           heads=heads, head_dim=hd, kv_layer=l, theta=10000.0))
        L.append(LayerSpec(name=p + "wo", op="linear", src=3, dst=0, res=0, c_in=d, c_out=d,
                           w_std=0.02, bias_std=0.0))
        L.append(LayerSpec(name=p + "ffn_norm", op="rmsnorm", src=0, dst=1, c_in=d, c_out=d,
                           eps=1e-5))
        L.append(LayerSpec(name=p + "gateup", op="gateup", src=1, dst=4, c_in=d, c_out=ffn,
                           w_std=0.02))
        L.append(LayerSpec(name=p + "w2", op="linear", src=4, dst=0, res=0, c_in=ffn, c_out=d,
                           w_std=0.02, bias_std=0.0))
    L.append(LayerSpec(name="final_norm", op="rmsnorm", src=0, dst=1, c_in=d, c_out=d, eps=1e-5))
    L.append(LayerSpec(name="lm_head", op="linear", src=1, dst=5, c_in=d, c_out=vocab,
                       w_std=0.02, bias_std=0.0, out_f32=True))
    per = 7
    blocks = [[0, 1 + per]]
    for l in range(1, n_layers):
        blocks.append([1 + per * l, 1 + per * (l + 1)])
    blocks.append([1 + per * n_layers, len(L)])
    layer_bytes = sum(x.weight_bytes() for x in L[1:1 + per])
    return Network("decoder7b", CFG_DECODER7B, L, blocks, (prompt,), 5, kind="decoder",
                   budget_bytes_fixed=4 * layer_bytes,
                   extra=dict(d=d, heads=heads, ffn=ffn, vocab=vocab, max_seq=max_seq,
                              prompt=prompt, gen=gen, n_layers=n_layers))


NETWORKS = {
    "tiny_cnn": tiny_cnn,
    "resnet50": resnet50,
    "vgg16": vgg16,
    "fcn_resnet101": fcn_resnet101,
    "decoder7b": decoder7b,
}


def get_network(name, **kw):
    return NETWORKS[name](**kw)


# ----------------------------------------------------------------------------
# Generators
# ----------------------------------------------------------------------------

def rng_for(cfg, *words):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg, *words])))


def _fold_bn(w, rng_g, rng_b, rng_m, rng_v, damp):
    """Batch-norm folded into the preceding conv (inference form):
    W' = W * g / sqrt(v + eps), b' = beta - mean * g / sqrt(v + eps)."""
    co = w.shape[0]
    g = rng_g.uniform(0.5, 1.5, co) * damp
    beta = rng_b.normal(0.0, 0.1, co)
    mean = rng_m.normal(0.0, 0.1, co)
    var = rng_v.uniform(0.5, 1.5, co)
    s = g / np.sqrt(var + BN_EPS)
    return w * s.reshape(-1, *([1] * (w.ndim - 1))), beta - mean * s


def bn_raw(cfg, li, layer):
    """Unfolded batch-norm parameters (gamma, beta, mean, var) of layer li, as
    drawn before folding; used to check the fold against an explicit BN."""
    co = layer.c_out
    g = rng_for(cfg, 0, li, 1).uniform(0.5, 1.5, co) * layer.bn_damp
    beta = rng_for(cfg, 0, li, 2).normal(0.0, 0.1, co)
    mean = rng_for(cfg, 0, li, 3).normal(0.0, 0.1, co)
    var = rng_for(cfg, 0, li, 4).uniform(0.5, 1.5, co)
    return g, beta, mean, var


def conv_weight_raw(cfg, li, layer):
    """Unfolded conv weight of layer li (fp64, He-normal)."""
    fan_in = layer.c_in * layer.k * layer.k
    shape = (layer.c_out, layer.c_in, layer.k, layer.k)
    return rng_for(cfg, 0, li, 0).normal(0.0, math.sqrt(2.0 / fan_in), shape)


def layer_params(net, li):
    """fp16 canonical parameters of layer ``li`` (dict name -> ndarray)."""
    layer = net.layers[li]
    cfg = net.cfg
    out = {}
    if layer.op == "conv2d":
        w = conv_weight_raw(cfg, li, layer)
        if layer.bn:
            w, b = _fold_bn(w, rng_for(cfg, 0, li, 1), rng_for(cfg, 0, li, 2),
                            rng_for(cfg, 0, li, 3), rng_for(cfg, 0, li, 4), layer.bn_damp)
        else:
            b = rng_for(cfg, 0, li, 5).normal(0.0, layer.bias_std, layer.c_out)
        out["weight"] = w.astype(np.float16)
        out["bias"] = b.astype(np.float16)
    elif layer.op == "linear":
        if layer.w_std:
            # decoder projections: float32 draws (see the other decoder tensors)
            a = rng_for(cfg, 0, li, 0).standard_normal((layer.c_out, layer.c_in), dtype=np.float32)
            a *= np.float32(layer.w_std)
            out["weight"] = a.astype(np.float16)
        else:
            std = math.sqrt(2.0 / layer.c_in)
            out["weight"] = rng_for(cfg, 0, li, 0).normal(0.0, std, (layer.c_out, layer.c_in)
                                                          ).astype(np.float16)
        if layer.bias_std > 0:
            out["bias"] = rng_for(cfg, 0, li, 5).normal(0.0, layer.bias_std, layer.c_out
                                                        ).astype(np.float16)
    elif layer.op == "rmsnorm":
        out["gain"] = np.ones(layer.c_in, np.float16)
    else:
        for ti, (name, shape) in enumerate(layer.param_shapes().items()):
            r = rng_for(cfg, 0, li, ti)
            # float32 draws keep the 7B generator to ~a minute; still one RNE round to fp16
            a = r.standard_normal(shape, dtype=np.float32)
            a *= np.float32(layer.w_std)
            out[name] = a.astype(np.float16)
    return out


def layers_params(net, indices, threads=None):
    """{li: params} for the given layers, generated on a thread pool (every
    tensor has its own seed, so the result does not depend on the order)."""
    indices = list(indices)
    threads = threads or min(16, os.cpu_count() or 1)
    if threads <= 1 or len(indices) <= 1:
        return {li: layer_params(net, li) for li in indices}
    with concurrent.futures.ThreadPoolExecutor(threads) as ex:
        return dict(zip(indices, ex.map(lambda li: layer_params(net, li), indices)))


def make_weights(net, threads=None):
    """List (per layer) of dicts of fp16 canonical parameter arrays."""
    p = layers_params(net, range(len(net.layers)), threads)
    return [p[li] for li in range(len(net.layers))]


def make_input(net, seed_word=1):
    """fp16 network input: CHW image ~ N(0,1), or int32 token ids."""
    r = rng_for(net.cfg, seed_word)
    if net.kind == "decoder":
        return r.integers(0, net.extra["vocab"], net.input_shape[0]).astype(np.int32)
    return r.standard_normal(net.input_shape).astype(np.float16)
