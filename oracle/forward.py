"""CPU oracle for block-swapped inference: the plain forward pass, in fp64.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this module;
only the tests, the package smoke check and the CPU-baseline leg of the bench
call it.  It shares no code with the HIP engine.

What is computed.  Swapping changes where weights live, never what is
computed: the paper's design goals (Sec. 3, "Lossless") state that the model
architecture and parameters are untouched, and Sec. 3 "Basic Idea" runs the
blocks one by one in order, each block's output feeding the next (Sec. 6.2.2,
partition of blocks).  The result of an n-block swapped inference is
therefore the ordinary forward pass of the whole network.  This module writes
that forward pass out directly, layer by layer, in float64 on the fp16
weights and inputs given to it (upcast exactly, no intermediate rounding).
Blocks appear only in ``forward_blocks``, which runs the same layers grouped
by a partition, to state the partition invariance explicitly.

Operator definitions (standard; the paper uses stock framework operators):
  conv2d   : cross-correlation with zero padding, stride and dilation
  maxpool  : max over the window, padding never selected (-inf)
  gavgpool : mean over H x W
  linear   : y = W x + b
  upsample : bilinear, half-pixel centres, edge-clamped (align_corners=False)
  rmsnorm  : v / sqrt(mean(v^2) + eps) * gain
  attention: RoPE (rotate-half, theta), causal softmax(q k^T / sqrt(hd)) v
  gateup   : silu(W1 x) * (W3 x)

Pins (the tests of the oracle, independent of this code): brute-force loops
on tiny shapes, torch float64 operators, closed forms (identity / one-hot
kernels, tap counts, constants and ramps, RoPE as a complex rotation, unit
RMS), BN folding against explicit batch norm, independent torch builds of
every network, and partition invariance.  Whole-network output values
against the paper: parity unpinned (the paper prints no forward-pass
values, weights or inputs).
"""
from __future__ import annotations

import numpy as np


# ---------------------------------------------------------------------------
# CNN operators (CHW float64)
# ---------------------------------------------------------------------------

def conv2d(x, w, b, stride=1, pad=0, dilation=1):
    """out[co, y, x] = b[co] + sum_{ci,r,s} w[co,ci,r,s] * xp[ci, y*st + r*dil, x*st + s*dil]
    where xp is x zero-padded by ``pad`` on each side.  The sum over (ci, r, s)
    is one matrix product over the gathered input patches (im2col)."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    ci, h, wd = x.shape
    co, ci2, kh, kw = w.shape
    assert ci == ci2, (ci, ci2)
    ho = (h + 2 * pad - dilation * (kh - 1) - 1) // stride + 1
    wo = (wd + 2 * pad - dilation * (kw - 1) - 1) // stride + 1
    xp = np.zeros((ci, h + 2 * pad, wd + 2 * pad), np.float64)
    xp[:, pad:pad + h, pad:pad + wd] = x
    cols = np.empty((ci, kh, kw, ho, wo), np.float64)
    for r in range(kh):
        for s in range(kw):
            y0, x0 = r * dilation, s * dilation
            cols[:, r, s] = xp[:, y0:y0 + stride * (ho - 1) + 1:stride,
                               x0:x0 + stride * (wo - 1) + 1:stride]
    out = w.reshape(co, ci * kh * kw) @ cols.reshape(ci * kh * kw, ho * wo)
    if b is not None:
        out += np.asarray(b, np.float64)[:, None]
    return out.reshape(co, ho, wo)


def maxpool(x, k, stride, pad=0):
    x = np.asarray(x, np.float64)
    c, h, w = x.shape
    ho = (h + 2 * pad - k) // stride + 1
    wo = (w + 2 * pad - k) // stride + 1
    xp = np.full((c, h + 2 * pad, w + 2 * pad), -np.inf)
    xp[:, pad:pad + h, pad:pad + w] = x
    out = np.full((c, ho, wo), -np.inf)
    for r in range(k):
        for s in range(k):
            out = np.maximum(out, xp[:, r:r + stride * (ho - 1) + 1:stride,
                                     s:s + stride * (wo - 1) + 1:stride])
    return out


def gavgpool(x):
    x = np.asarray(x, np.float64)
    return x.reshape(x.shape[0], -1).mean(axis=1)


def linear(x, w, b=None):
    y = np.asarray(w, np.float64) @ np.asarray(x, np.float64).reshape(-1)
    if b is not None:
        y = y + np.asarray(b, np.float64)
    return y


def _bilinear_index(n_out, n_in, scale):
    o = np.arange(n_out, dtype=np.float64)
    src = np.maximum((o + 0.5) / scale - 0.5, 0.0)
    i0 = np.floor(src).astype(np.int64)
    i0 = np.minimum(i0, n_in - 1)
    i1 = np.minimum(i0 + 1, n_in - 1)
    lam = src - i0
    return i0, i1, lam


def upsample_bilinear(x, scale):
    """Bilinear resize by an integer factor with half-pixel centres:
    source coordinate (o + 0.5) / scale - 0.5, clamped at 0; the upper
    neighbour is clamped to the last row/column."""
    x = np.asarray(x, np.float64)
    c, h, w = x.shape
    y0, y1, ly = _bilinear_index(h * scale, h, scale)
    x0, x1, lx = _bilinear_index(w * scale, w, scale)
    top = x[:, y0, :] * (1 - ly)[None, :, None] + x[:, y1, :] * ly[None, :, None]
    return top[:, :, x0] * (1 - lx)[None, None, :] + top[:, :, x1] * lx[None, None, :]


def relu(x):
    return np.maximum(x, 0.0)


# ---------------------------------------------------------------------------
# Decoder operators (token-major [T][d] float64)
# ---------------------------------------------------------------------------

def rmsnorm(h, gain, eps):
    h = np.asarray(h, np.float64)
    return h / np.sqrt((h * h).mean(axis=-1, keepdims=True) + eps) * np.asarray(gain, np.float64)


def rope(x, positions, theta):
    """Rotary position embedding, rotate-half pairing: for head dim hd, pair
    (i, i + hd/2) is rotated by angle p * theta^(-2i/hd).  x: [T][H][hd]."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(positions, np.float64)[:, None] * inv[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def causal_attention(q, k, v):
    """q, k, v: [T][H][hd] (already rotated).  Row t attends to keys 0..t."""
    t, nh, hd = q.shape
    out = np.empty_like(q)
    mask = np.triu(np.ones((t, t), bool), 1)
    for hh in range(nh):
        s = q[:, hh, :] @ k[:, hh, :].T / np.sqrt(hd)
        s[mask] = -np.inf
        s -= s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, hh, :] = p @ v[:, hh, :]
    return out


def silu(x):
    return x / (1.0 + np.exp(-x))


# ---------------------------------------------------------------------------
# Whole networks
# ---------------------------------------------------------------------------

def _f64(a):
    return np.asarray(a, np.float64)


def run_layer(layer, params, slots):
    """Apply one CNN layer: reads slots[layer.src] (and slots[layer.res]),
    writes slots[layer.dst]."""
    x = slots[layer.src]
    op = layer.op
    if op == "conv2d":
        y = conv2d(x, params["weight"], params["bias"], layer.stride, layer.pad, layer.dilation)
    elif op == "maxpool":
        y = maxpool(x, layer.k, layer.stride, layer.pad)
    elif op == "gavgpool":
        y = gavgpool(x)
    elif op == "linear":
        y = linear(x.reshape(-1), params["weight"], params.get("bias"))
    elif op == "upsample_bilinear":
        y = upsample_bilinear(x, layer.scale)
    else:
        raise ValueError("oracle: op %r is not a CNN op" % op)
    if layer.res >= 0:
        y = y + slots[layer.res]
    if layer.relu:
        y = relu(y)
    slots[layer.dst] = y


def forward(net, weights, x):
    """Forward pass of a CNN-kind network on input x (CHW fp16); fp64 result."""
    return forward_blocks(net, weights, x, [[0, len(net.layers)]])


def forward_blocks(net, weights, x, blocks):
    """Run the network block by block, in order; each block's layers read
    their inputs from the activations left by the previous blocks (Sec. 3,
    "Basic Idea": the blocks execute one by one; Sec. 6, partition of
    blocks: the output of one block feeds the next)."""
    assert net.kind == "cnn"
    assert blocks[0][0] == 0 and blocks[-1][1] == len(net.layers)
    assert all(blocks[i][1] == blocks[i + 1][0] for i in range(len(blocks) - 1))
    slots = {0: _f64(x)}
    for a, b in blocks:
        for li in range(a, b):
            run_layer(net.layers[li], weights[li], slots)
    return slots[net.out_slot]


def decoder_forward(net, weights, ids):
    """Causal pass of the decoder over token ids (positions 0..T-1); returns
    fp64 logits [T][vocab].  ``weights`` may be a list of dicts or a callable
    li -> dict (so the 7B weights can be generated layer by layer)."""
    get = weights if callable(weights) else (lambda li: weights[li])
    ids = np.asarray(ids, np.int64)
    t = len(ids)
    pos = np.arange(t)
    slots = {}
    for li, layer in enumerate(net.layers):
        p = get(li)
        op = layer.op
        if op == "embed":
            y = _f64(p["table"][ids])
        elif op == "rmsnorm":
            y = rmsnorm(slots[layer.src], p["gain"], layer.eps)
        elif op == "qkv":
            a = slots[layer.src]
            y = (a @ _f64(p["wq"]).T, a @ _f64(p["wk"]).T, a @ _f64(p["wv"]).T)
        elif op == "attention":
            nh, hd = layer.heads, layer.head_dim
            q, k, v = (m.reshape(t, nh, hd) for m in slots[layer.src])
            q = rope(q, pos, layer.theta)
            k = rope(k, pos, layer.theta)
            y = causal_attention(q, k, v).reshape(t, nh * hd)
        elif op == "linear":
            y = slots[layer.src] @ _f64(p["weight"]).T
            if "bias" in p:
                y = y + _f64(p["bias"])
        elif op == "gateup":
            a = slots[layer.src]
            y = silu(a @ _f64(p["w1"]).T) * (a @ _f64(p["w3"]).T)
        else:
            raise ValueError("oracle: op %r is not a decoder op" % op)
        if layer.res >= 0:
            y = y + slots[layer.res]
        slots[layer.dst] = y
    return slots[net.out_slot]
