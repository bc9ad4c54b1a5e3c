"""Python binding of libswapnet.so (ctypes).  Argument marshalling only: every
step of inference runs in the library's HIP kernels.

    eng = SwapNet(budget_bytes)
    eng.add_block(layers, weights_blob)      # repeated, in order
    eng.plan()
    y = eng.infer(x)                         # host numpy in/out
    eng.infer_dev(x_ptr, y_ptr, stream_ptr)  # device pointers (e.g. torch tensors)

``build_engine(net, weights, budget)`` turns a network description from
``workloads`` into descriptors and weight blobs, one block per user block.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libswapnet.so")

SN_OK, SN_E_INVALID, SN_E_STATE, SN_E_INFEASIBLE, SN_E_NOMEM, SN_E_HIP, SN_E_UNSUPPORTED = \
    0, -1, -2, -3, -4, -5, -6
OP = {"conv2d": 1, "linear": 2, "maxpool": 3, "gavgpool": 4, "upsample_bilinear": 5,
      "embed": 6, "rmsnorm": 7, "attention": 8}
FLAG_RELU, FLAG_FLATTEN_CHW, FLAG_SWIGLU, FLAG_OUT_F32, FLAG_LAST_ROW = 1, 2, 4, 8, 16
CREATE_HOST_ONLY = 1
OPT_SPLIT_BUDGET, OPT_TIMING, OPT_MAX_SLAB, OPT_GRAPH, OPT_SWAPIN, OPT_SWAPIN_BLOCKS = 1, 2, 3, 4, 5, 6
OPT_COPY_STREAMS = 7
OPT_PARTITION = 8
OPT_SYNC = 9
OPT_NAIVE = 10
OPT_CONV_KERNEL = 11
OPT_GATE_LIMIT_US = 12
NAIVE_SEQUENTIAL, NAIVE_ALLOC, NAIVE_PAGEABLE, NAIVE_COPY_ASSEMBLY = 1, 2, 4, 8

EXPORTS = ["sn_create", "sn_create_ex", "sn_add_block", "sn_plan", "sn_set_option", "sn_infer",
           "sn_infer_dev", "sn_infer_tokens", "sn_reset", "sn_get_stats", "sn_get_slab",
           "sn_get_piece", "sn_get_image", "sn_kernel_name", "sn_last_error", "sn_destroy",
           "sn_set_cost_model", "sn_get_cost_model", "sn_calibrate", "sn_predict", "sn_replan",
           "sn_tune", "sn_split_budget", "sn_save_image", "sn_attach_image_file"]
COST_KEYS = ("alpha", "beta", "gamma", "kappa", "gate", "wake", "slab_ex")


class SnLayer(C.Structure):
    _fields_ = [("op", C.c_int32), ("src", C.c_int32), ("res", C.c_int32), ("dst", C.c_int32),
                ("c_in", C.c_int32), ("c_out", C.c_int32), ("h_in", C.c_int32),
                ("w_in", C.c_int32), ("k", C.c_int32), ("stride", C.c_int32),
                ("pad", C.c_int32), ("dilation", C.c_int32), ("scale", C.c_int32),
                ("heads", C.c_int32), ("head_dim", C.c_int32), ("kv_layer", C.c_int32),
                ("max_tokens", C.c_int32), ("max_seq", C.c_int32), ("flags", C.c_int32),
                ("eps", C.c_float), ("theta", C.c_float),
                ("w_off", C.c_int64), ("w_bytes", C.c_int64),
                ("b_off", C.c_int64), ("b_bytes", C.c_int64)]


class SnStats(C.Structure):
    _fields_ = [("budget_bytes", C.c_int64), ("image_bytes", C.c_int64),
                ("arena_high_water", C.c_int64), ("streamed_bytes", C.c_int64),
                ("activation_bytes", C.c_int64), ("kv_bytes", C.c_int64),
                ("table_bytes", C.c_int64), ("n_slabs", C.c_int32), ("n_pieces", C.c_int32),
                ("n_layers", C.c_int32), ("resident", C.c_int32), ("n_infers", C.c_int64),
                ("last_ms", C.c_double), ("input_bytes", C.c_int64), ("output_bytes", C.c_int64),
                ("host_weight_bytes", C.c_int64), ("file_backed", C.c_int32),
                ("direct_io", C.c_int32), ("read_ms", C.c_double)]


class SnSlabInfo(C.Structure):
    _fields_ = [("image_off", C.c_int64), ("arena_off", C.c_int64), ("bytes", C.c_int64),
                ("first_piece", C.c_int32), ("n_pieces", C.c_int32),
                ("t_in_ms", C.c_float), ("t_ex_ms", C.c_float),
                ("t_in_start_ms", C.c_float), ("t_ex_start_ms", C.c_float),
                ("wait_slab", C.c_int32), ("wrap_slab", C.c_int32)]


class SnPieceInfo(C.Structure):
    _fields_ = [("layer", C.c_int32), ("c0", C.c_int32), ("c1", C.c_int32),
                ("kernel", C.c_int32), ("w_off", C.c_int64), ("b_off", C.c_int64),
                ("w_bytes", C.c_int64), ("b_bytes", C.c_int64), ("t_ms", C.c_float),
                ("ksplit", C.c_int32), ("t_main_ms", C.c_float)]


class SnCostModel(C.Structure):
    _fields_ = [(k, C.c_double) for k in COST_KEYS] + \
               [("layer_ex", C.POINTER(C.c_float)), ("n_layers", C.c_int32)]


_lib = None


def load_library(path=LIB_PATH):
    """Load libswapnet.so.  Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libswapnet.so not built (%s); run python -m paper_2401_16757_amd.build"
                           % path)
    lib = C.CDLL(path)
    P, I, I64, S = C.c_void_p, C.c_int, C.c_int64, C.c_size_t
    sig = {
        "sn_create": (P, [S]), "sn_create_ex": (P, [S, I]),
        "sn_add_block": (I, [P, C.POINTER(SnLayer), I, P, S]),
        "sn_plan": (I, [P]), "sn_set_option": (I, [P, I, I64]),
        "sn_infer": (I, [P, P, P]), "sn_infer_dev": (I, [P, P, P, P]),
        "sn_infer_tokens": (I, [P, P, I, P]), "sn_reset": (I, [P]),
        "sn_get_stats": (I, [P, C.POINTER(SnStats)]),
        "sn_get_slab": (I, [P, I, C.POINTER(SnSlabInfo)]),
        "sn_get_piece": (I, [P, I, C.POINTER(SnPieceInfo)]),
        "sn_get_image": (I, [P, C.POINTER(C.c_void_p), C.POINTER(C.c_size_t)]),
        "sn_kernel_name": (C.c_char_p, [I]),
        "sn_set_cost_model": (I, [P, C.POINTER(SnCostModel)]),
        "sn_get_cost_model": (I, [P, C.POINTER(SnCostModel), P, I]),
        "sn_calibrate": (I, [P, I]),
        "sn_replan": (I, [P, S]),
        "sn_tune": (I, [P, I, C.POINTER(C.c_double)]),
        "sn_split_budget": (I, [I, C.POINTER(C.c_int64), C.POINTER(C.c_double),
                                C.POINTER(C.c_double), C.c_int64, C.POINTER(C.c_int64)]),
        "sn_predict": (I, [P, C.POINTER(C.c_double), C.POINTER(C.c_double)]),
        "sn_save_image": (I, [P, C.c_char_p]), "sn_attach_image_file": (I, [P, C.c_char_p]),
        "sn_last_error": (C.c_char_p, [P]), "sn_destroy": (None, [P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def conv_kernel_count():
    """Number of convolution kernel variants (valid SN_OPT_CONV_KERNEL values
    are 0 .. this count)."""
    n = 0
    while kernel_name(n) != "?":
        n += 1
    return n


def kernel_name(kernel_id):
    return load_library().sn_kernel_name(int(kernel_id)).decode()


def split_budget(need, latency_s, urgency, total):
    """Budgets of several models sharing ``total`` bytes (sn_split_budget)."""
    lib = load_library()
    n = len(need)
    a_need = (C.c_int64 * n)(*[int(v) for v in need])
    a_lat = (C.c_double * n)(*[float(v) for v in latency_s])
    a_urg = (C.c_double * n)(*[float(v) for v in urgency])
    out = (C.c_int64 * n)()
    rc = lib.sn_split_budget(n, a_need, a_lat, a_urg, int(total), out)
    if rc != SN_OK:
        raise SwapNetError(rc, "invalid arguments to sn_split_budget")
    return list(out)


class SwapNetError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("swapnet error %d: %s" % (code, msg))
        self.code = code


class SwapNet:
    """One engine context: a budget-sized HBM arena plus its plan."""

    def __init__(self, budget_bytes, host_only=False):
        self.lib = load_library()
        self.ctx = self.lib.sn_create_ex(int(budget_bytes), CREATE_HOST_ONLY if host_only else 0)
        if not self.ctx:
            raise SwapNetError(SN_E_HIP, self.lib.sn_last_error(None).decode())
        self.budget = int(budget_bytes)
        self.out_shape = None
        self.out_dtype = np.float16
        self.in_shape = None

    def _check(self, rc):
        if rc != SN_OK:
            raise SwapNetError(rc, self.lib.sn_last_error(self.ctx).decode())
        return rc

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.sn_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def set_option(self, opt, value):
        return self._check(self.lib.sn_set_option(self.ctx, opt, int(value)))

    def add_block(self, layers, blob):
        arr = (SnLayer * len(layers))(*layers)
        buf = np.ascontiguousarray(np.frombuffer(blob, np.uint8)) if len(blob) else np.zeros(1, np.uint8)
        return self._check(self.lib.sn_add_block(self.ctx, arr, len(layers),
                                                 buf.ctypes.data_as(C.c_void_p), len(blob)))

    def plan(self):
        return self._check(self.lib.sn_plan(self.ctx))

    def _host_buffers(self, x, dtype):
        # the library reads / writes exactly input_bytes / output_bytes
        st = self.stats()
        if x is not None and x.nbytes != st["input_bytes"]:
            raise ValueError("input has %d bytes, the network takes %d" % (x.nbytes, st["input_bytes"]))
        shape = self.out_shape if self.out_shape is not None else \
            (st["output_bytes"] // np.dtype(dtype).itemsize,)
        out = np.empty(shape, dtype)
        if out.nbytes != st["output_bytes"]:
            raise ValueError("output shape %s holds %d bytes, the network writes %d"
                             % (shape, out.nbytes, st["output_bytes"]))
        return out

    def infer(self, x):
        x = np.ascontiguousarray(x, np.float16)
        out = self._host_buffers(x, self.out_dtype)
        self._check(self.lib.sn_infer(self.ctx, x.ctypes.data_as(C.c_void_p),
                                      out.ctypes.data_as(C.c_void_p)))
        return out

    def infer_dev(self, d_in, d_out, stream=None):
        """Device pointers (ints); ``stream``: a hipStream_t as int, or None."""
        return self._check(self.lib.sn_infer_dev(self.ctx, C.c_void_p(d_in), C.c_void_p(d_out),
                                                 C.c_void_p(stream or 0)))

    def infer_tokens(self, ids):
        ids = np.ascontiguousarray(ids, np.int32)
        out = self._host_buffers(None, np.float32)
        self._check(self.lib.sn_infer_tokens(self.ctx, ids.ctypes.data_as(C.c_void_p), len(ids),
                                             out.ctypes.data_as(C.c_void_p)))
        return out

    def reset(self):
        return self._check(self.lib.sn_reset(self.ctx))

    def stats(self):
        s = SnStats()
        self._check(self.lib.sn_get_stats(self.ctx, C.byref(s)))
        return {k: getattr(s, k) for k, _ in SnStats._fields_}

    def slabs(self):
        out = []
        for i in range(self.stats()["n_slabs"]):
            s = SnSlabInfo()
            self._check(self.lib.sn_get_slab(self.ctx, i, C.byref(s)))
            out.append({k: getattr(s, k) for k, _ in SnSlabInfo._fields_})
        return out

    def pieces(self):
        out = []
        for j in range(self.stats()["n_pieces"]):
            p = SnPieceInfo()
            self._check(self.lib.sn_get_piece(self.ctx, j, C.byref(p)))
            out.append({k: getattr(p, k) for k, _ in SnPieceInfo._fields_})
        return out

    def set_cost_model(self, model):
        """``model``: dict with the coefficient keys of sn_cost_model (missing
        ones keep the context's values) and optionally ``layer_ex`` (seconds
        per layer, < 0 = not measured)."""
        cur = self.cost_model()
        m = SnCostModel()
        for k in COST_KEYS:
            setattr(m, k, float(model.get(k, cur[k])))
        ex = model.get("layer_ex")
        if ex is not None:
            ex = np.ascontiguousarray(ex, np.float32)
            m.layer_ex = ex.ctypes.data_as(C.POINTER(C.c_float))
            m.n_layers = len(ex)
        return self._check(self.lib.sn_set_cost_model(self.ctx, C.byref(m)))

    def cost_model(self):
        n = self.stats()["n_layers"]
        ex = np.zeros(max(n, 1), np.float32)
        m = SnCostModel()
        self._check(self.lib.sn_get_cost_model(self.ctx, C.byref(m),
                                               ex.ctypes.data_as(C.c_void_p) if n else None, n))
        out = {k: getattr(m, k) for k in COST_KEYS}
        out["layer_ex"] = ex[:n].copy()
        return out

    def replan(self, budget=0):
        """Re-plan in place for ``budget`` bytes (0: keep) and the current
        options."""
        r = self._check(self.lib.sn_replan(self.ctx, int(budget)))
        if budget:
            self.budget = int(budget)
        return r

    def tune(self, reps=3):
        """Measure partitions 0, 1 and 2 and keep the fastest; returns the
        measured seconds per inference of each (0: infeasible)."""
        t = (C.c_double * 3)()
        self._check(self.lib.sn_tune(self.ctx, int(reps), t))
        return list(t)

    def calibrate(self, reps=3):
        return self._check(self.lib.sn_calibrate(self.ctx, int(reps)))

    def predict(self):
        """(latency_s, period_s) of the plan under the context's delay model."""
        lat, per = C.c_double(), C.c_double()
        self._check(self.lib.sn_predict(self.ctx, C.byref(lat), C.byref(per)))
        return lat.value, per.value

    def save_image(self, path):
        """Write the planned image to ``path`` (sn_save_image)."""
        return self._check(self.lib.sn_save_image(self.ctx, os.fsencode(path)))

    def attach_image_file(self, path):
        """Swap in from the image file at ``path`` (sn_attach_image_file)."""
        return self._check(self.lib.sn_attach_image_file(self.ctx, os.fsencode(path)))

    def image(self):
        ptr, n = C.c_void_p(), C.c_size_t()
        self._check(self.lib.sn_get_image(self.ctx, C.byref(ptr), C.byref(n)))
        return np.ctypeslib.as_array(C.cast(ptr, C.POINTER(C.c_uint8)), shape=(n.value,)).copy() \
            if n.value else np.zeros(0, np.uint8)


# ---------------------------------------------------------------------------
# Network description -> descriptors and canonical weight blobs
# ---------------------------------------------------------------------------

def _layer_tensors(spec, params):
    """Canonical tensors the engine takes for one layer: (weight, bias)."""
    op = spec.op
    if op in ("conv2d", "linear"):
        return params["weight"], params.get("bias")
    if op == "qkv":
        return np.concatenate([params["wq"], params["wk"], params["wv"]], axis=0), None
    if op == "gateup":
        return np.concatenate([params["w1"], params["w3"]], axis=0), None
    if op == "rmsnorm":
        return params["gain"], None
    if op == "embed":
        return params["table"], None
    return None, None


def layer_descriptor(spec, net=None):
    d = SnLayer()
    op = {"qkv": "linear", "gateup": "linear"}.get(spec.op, spec.op)
    d.op = OP[op]
    d.src, d.res, d.dst = spec.src, spec.res, spec.dst
    d.c_in, d.c_out = spec.c_in, spec.c_out
    d.h_in, d.w_in = spec.h_in, spec.w_in
    d.k, d.stride, d.pad, d.dilation = spec.k, spec.stride, spec.pad, spec.dilation
    d.scale = spec.scale
    d.heads, d.head_dim, d.kv_layer = spec.heads, spec.head_dim, spec.kv_layer
    d.eps, d.theta = spec.eps, spec.theta
    flags = 0
    if spec.relu:
        flags |= FLAG_RELU
    if spec.flatten_chw:
        flags |= FLAG_FLATTEN_CHW
    if spec.op == "gateup":
        flags |= FLAG_SWIGLU
    if spec.out_f32:
        flags |= FLAG_OUT_F32
    if net is not None and net.kind == "decoder":
        if spec.op == "embed":
            d.max_tokens = net.extra.get("max_tokens", net.extra["prompt"])
        if spec.op == "attention":
            d.max_seq = net.extra["max_seq"]
        if spec.op == "linear" and spec.out_f32:
            flags |= FLAG_LAST_ROW
    d.flags = flags
    return d


def block_payload(net, weights, first, last):
    """Descriptors and one canonical weight blob for layers [first, last)."""
    descs, parts, off = [], [], 0
    for li in range(first, last):
        spec = net.layers[li]
        d = layer_descriptor(spec, net)
        params = weights(li) if callable(weights) else weights[li]
        w, b = _layer_tensors(spec, params)
        for t, which in ((w, "w"), (b, "b")):
            if t is None:
                continue
            t = np.ascontiguousarray(t, np.float16)
            setattr(d, which + "_off", off)
            setattr(d, which + "_bytes", t.nbytes)
            parts.append(t.reshape(-1).view(np.uint8))
            off += t.nbytes
        descs.append(d)
    blob = np.concatenate(parts) if parts else np.zeros(0, np.uint8)
    return descs, blob


def output_shape(net):
    last = net.layers[-1]
    if net.kind == "decoder":
        return (last.c_out,), np.float32
    if last.op in ("conv2d", "maxpool", "upsample_bilinear"):
        h, w = last.out_hw()
        return (last.c_out, h, w), np.float16
    return (last.c_out,), (np.float32 if last.out_f32 else np.float16)


def build_engine(net, weights, budget=None, blocks=None, split_budget=None, host_only=False,
                 timing=False, max_slab=0, partition=0, cost_model=None, conv_kernel=0):
    """Create, register and plan an engine for ``net``.  ``weights`` is a list
    of per-layer parameter dicts or a callable li -> dict.  ``cost_model``
    (a dict as returned by ``SwapNet.cost_model``) is set before planning;
    with ``partition=2`` it decides the slab partition."""
    eng = SwapNet(budget if budget is not None else net.budget_bytes(), host_only=host_only)
    if split_budget is not None:
        eng.set_option(OPT_SPLIT_BUDGET, split_budget)
    if max_slab:
        eng.set_option(OPT_MAX_SLAB, max_slab)
    if partition:
        eng.set_option(OPT_PARTITION, partition)
    if timing:
        eng.set_option(OPT_TIMING, int(timing))
    if conv_kernel:
        eng.set_option(OPT_CONV_KERNEL, conv_kernel)
    for a, b in (blocks or net.blocks):
        descs, blob = block_payload(net, weights, a, b)
        eng.add_block(descs, blob)
    if cost_model is not None:
        eng.set_cost_model(cost_model)
    eng.plan()
    eng.out_shape, eng.out_dtype = output_shape(net)
    eng.in_shape = net.input_shape
    return eng
