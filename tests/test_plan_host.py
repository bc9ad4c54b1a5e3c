"""Host-side tests of the C ABI (no GPU): exported symbols, the planner's
invariants, the prepacked image layout and the error/state machine.  They use
host-only contexts, which make no device calls."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2401_16757_amd import swapnet as S
from paper_2401_16757_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(S.LIB_PATH):
        from paper_2401_16757_amd import build
        build.build()
    S.load_library()


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "swapnet.h")).read()
    declared = set(re.findall(r"\b(sn_[a-z_]+)\s*\(", hdr))
    declared -= {"sn_ctx"}
    assert declared == set(S.EXPORTS)
    lib = C.CDLL(S.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name


def test_struct_sizes_match_header_layout():
    # sn_layer: 19 int32 + 2 float + 4 int64 = 76 + 8 + 32 -> 120 with alignment
    assert C.sizeof(S.SnLayer) == 120
    assert C.sizeof(S.SnStats) == 7 * 8 + 4 * 4 + 8 + 8 + 2 * 8 + 8 + 2 * 4 + 8


def plan_of(name, budget=None, **kw):
    net = W.get_network(name, **kw)
    wts = W.make_weights(net)
    eng = S.build_engine(net, wts, budget=budget, host_only=True)
    return net, wts, eng


def check_plan(net, eng, budget):
    st = eng.stats()
    slabs, pieces = eng.slabs(), eng.pieces()
    B = budget // 256 * 256
    # every weighted layer's output units covered exactly once, in order
    cover = {}
    order = []
    for s in slabs:
        for j in range(s["first_piece"], s["first_piece"] + s["n_pieces"]):
            p = pieces[j]
            order.append(p["layer"])
            cover.setdefault(p["layer"], []).append((p["c0"], p["c1"]))
    assert order == sorted(order)
    for li, spec in enumerate(net.layers):
        if spec.op in ("conv2d", "linear", "qkv", "gateup"):
            rngs = cover[li]
            assert rngs[0][0] == 0 and rngs[-1][1] == spec.c_out
            assert all(rngs[i][1] == rngs[i + 1][0] for i in range(len(rngs) - 1))
    # alignment, arena bounds, pair constraint, consecutive slabs disjoint
    total = 0
    for i, s in enumerate(slabs):
        assert s["bytes"] % 256 == 0 and s["arena_off"] % 256 == 0 and s["image_off"] == total
        total += s["bytes"]
        if not st["resident"]:
            assert 0 <= s["arena_off"] and s["arena_off"] + s["bytes"] <= B
        if i + 1 < len(slabs) and not st["resident"]:
            t = slabs[i + 1]
            assert s["bytes"] + t["bytes"] <= B
            a0, a1 = s["arena_off"], s["arena_off"] + s["bytes"]
            b0, b1 = t["arena_off"], t["arena_off"] + t["bytes"]
            assert a1 <= b0 or b1 <= a0
        if not st["resident"]:
            # the swap-in of slab i waits for the compute of slab `wait`; every
            # slab after that one may still be in use, so none may overlap
            w = s["wait_slab"]
            assert w == -1 or 0 <= w <= i - 2
            for j in range(w + 1, i):
                t = slabs[j]
                assert (s["arena_off"] + s["bytes"] <= t["arena_off"] or
                        t["arena_off"] + t["bytes"] <= s["arena_off"]), (i, j)
            if w >= 0:
                t = slabs[w]
                assert not (s["arena_off"] + s["bytes"] <= t["arena_off"] or
                            t["arena_off"] + t["bytes"] <= s["arena_off"])
            # the next inference's swap-in of a slab without an earlier
            # overlapping slab waits for the last overlapping slab of this one
            def over(u, v):
                return not (u["arena_off"] + u["bytes"] <= v["arena_off"] or
                            v["arena_off"] + v["bytes"] <= u["arena_off"])
            later = [j for j in range(i + 1, len(slabs)) if over(s, slabs[j])]
            expect = (later[-1] if later else -1) if w == -1 else -1
            assert s["wrap_slab"] == expect, (i, s["wrap_slab"], expect)
    assert total == st["image_bytes"]
    # streamed bytes: the weights plus alignment padding only
    assert st["image_bytes"] >= net.streamed_weight_bytes()


@pytest.mark.parametrize("name,kw", [("tiny_cnn", {}), ("resnet50", {}), ("vgg16", {}),
                                     ("fcn_resnet101", {})])
@pytest.mark.parametrize("frac", [None, 1 / 2.32, 1 / 3, 1 / 4, 1 / 5.81])
@pytest.mark.parametrize("partition", [0, 1, 2])
def test_plan_invariants(name, kw, frac, partition):
    net = W.get_network(name, **kw)
    budget = net.budget_bytes() if frac is None else int(net.weight_bytes() * frac)
    wts = W.make_weights(net)
    try:
        eng = S.build_engine(net, wts, budget=budget, host_only=True, partition=partition)
    except S.SwapNetError as e:
        # only the tiny network is too small to meet 1/5.81 with 256-byte slabs
        assert e.code == S.SN_E_INFEASIBLE and name == "tiny_cnn", e
        return
    check_plan(net, eng, budget)
    assert eng.stats()["resident"] == 0
    if partition == 1 and name != "tiny_cnn":
        # Sec. 6 with m = 2: n = ceil(2 s / B) slabs (rounded up to even) of
        # near-equal size, each at most half the budget
        sl = eng.slabs()
        total = sum(s["bytes"] for s in sl)
        n = -(-2 * total // (budget // 256 * 256))
        n += n % 2
        assert len(sl) in (n - 1, n, n + 1), (len(sl), n)
        assert max(s["bytes"] for s in sl) <= budget // 2
        assert max(s["bytes"] for s in sl[:-1]) - min(s["bytes"] for s in sl[:-1]) <= 0.02 * total / len(sl) + 4096


def test_slab_counts_of_the_workloads():
    exp = {"tiny_cnn": 4, "resnet50": 8, "vgg16": 15, "fcn_resnet101": 12}
    for name, n in exp.items():
        _, _, eng = plan_of(name)
        assert eng.stats()["n_slabs"] == n, name
    for name, n in (("resnet50", 16), ("fcn_resnet101", 14)):
        net = W.get_network(name)
        _, _, eng = plan_of(name, budget=int(net.weight_bytes() / 5.81))
        assert eng.stats()["n_slabs"] == n, name


def test_resident_when_budget_covers_image():
    net = W.get_network("resnet50", res=32)
    wts = W.make_weights(net)
    eng = S.build_engine(net, wts, budget=net.weight_bytes() * 2, host_only=True)
    st = eng.stats()
    assert st["resident"] == 1 and st["n_slabs"] == len(net.blocks)
    # same slabs as a swapped plan when a split budget is given
    eng2 = S.build_engine(net, wts, budget=net.weight_bytes() * 2, host_only=True,
                          split_budget=net.budget_bytes())
    eng3 = S.build_engine(net, wts, budget=net.budget_bytes(), host_only=True)
    assert [s["bytes"] for s in eng2.slabs()] == [s["bytes"] for s in eng3.slabs()]
    assert eng2.stats()["resident"] == 1 and eng3.stats()["resident"] == 0


def test_image_holds_device_layout():
    """The pinned image holds conv weights as [c_out][kh][kw][cin_pad8] and
    bias after them, FC1 columns permuted from (C,H,W) to (H,W,C), all at the
    offsets the piece table reports."""
    net = W.get_network("vgg16", res=32)
    wts = W.make_weights(net)
    eng = S.build_engine(net, wts, budget=net.weight_bytes() // 3, host_only=True)
    img = eng.image()
    slabs, pieces = eng.slabs(), eng.pieces()
    seen = set()
    for s in slabs:
        for j in range(s["first_piece"], s["first_piece"] + s["n_pieces"]):
            p = pieces[j]
            spec = net.layers[p["layer"]]
            if spec.op not in ("conv2d", "linear"):
                continue
            c0, c1 = p["c0"], p["c1"]
            wb = img[s["image_off"] + p["w_off"]: s["image_off"] + p["w_off"] + p["w_bytes"]]
            w = wb.view(np.float16)
            canon = wts[p["layer"]]["weight"]
            if spec.op == "conv2d":
                cp = (spec.c_in + 7) // 8 * 8
                dev = np.zeros((spec.c_out, spec.k, spec.k, cp), np.float16)
                dev[..., :spec.c_in] = canon.transpose(0, 2, 3, 1)
                exp = dev[c0:c1].reshape(-1)
            elif spec.flatten_chw:
                C_, H, Wd = spec.c_in // (spec.h_in * spec.w_in), spec.h_in, spec.w_in
                exp = canon.reshape(spec.c_out, C_, H, Wd).transpose(0, 2, 3, 1)[c0:c1].reshape(-1)
            else:
                exp = canon[c0:c1].reshape(-1)
            np.testing.assert_array_equal(w.view(np.uint16), exp.view(np.uint16))
            bb = img[s["image_off"] + p["b_off"]: s["image_off"] + p["b_off"] + p["b_bytes"]]
            np.testing.assert_array_equal(bb.view(np.uint16),
                                          wts[p["layer"]]["bias"][c0:c1].view(np.uint16))
            seen.add(spec.op)
    assert seen == {"conv2d", "linear"}


def test_swiglu_rows_interleaved_in_image():
    net = W.decoder7b(n_layers=1, d=64, heads=4, ffn=96, vocab=40, max_seq=16, prompt=8)
    wts = W.make_weights(net)
    eng = S.build_engine(net, wts, budget=1 << 24, host_only=True)
    img, slabs, pieces = eng.image(), eng.slabs(), eng.pieces()
    li = [i for i, l in enumerate(net.layers) if l.op == "gateup"][0]
    for s in slabs:
        for j in range(s["first_piece"], s["first_piece"] + s["n_pieces"]):
            p = pieces[j]
            if p["layer"] != li:
                continue
            w = img[s["image_off"] + p["w_off"]:][:p["w_bytes"]].view(np.float16).reshape(-1, 64)
            w1, w3 = wts[li]["w1"], wts[li]["w3"]
            np.testing.assert_array_equal(w[0::2], w1[p["c0"]:p["c1"]])
            np.testing.assert_array_equal(w[1::2], w3[p["c0"]:p["c1"]])
    st = eng.stats()
    # the embedding table is not part of any slab
    assert st["image_bytes"] < net.weight_bytes()


def test_infeasible_budget_reports_error():
    net = W.get_network("vgg16", res=32)
    wts = W.make_weights(net)
    with pytest.raises(S.SwapNetError) as e:
        S.build_engine(net, wts, budget=4096, host_only=True)
    assert e.value.code == S.SN_E_INFEASIBLE
    assert "infeasible" in str(e.value)


def test_state_machine_and_argument_errors():
    lib = S.load_library()
    assert lib.sn_create_ex(16, S.CREATE_HOST_ONLY) is None
    assert b"budget" in lib.sn_last_error(None)
    eng = S.SwapNet(1 << 20, host_only=True)
    # plan before any block
    assert lib.sn_plan(eng.ctx) == S.SN_E_STATE
    net = W.get_network("tiny_cnn")
    wts = W.make_weights(net)
    descs, blob = S.block_payload(net, wts, 0, 2)
    # weight bytes that do not match the descriptor
    bad = S.SnLayer.from_buffer_copy(descs[0])
    bad.w_bytes -= 2
    with pytest.raises(S.SwapNetError) as e:
        eng.add_block([bad, descs[1]], blob)
    assert e.value.code == S.SN_E_INVALID
    # offsets beyond the buffer
    with pytest.raises(S.SwapNetError) as e:
        eng.add_block(descs, blob[:100])
    assert e.value.code == S.SN_E_INVALID
    # reading a slot nobody wrote
    bad = S.SnLayer.from_buffer_copy(descs[1])
    bad.src = 77
    with pytest.raises(S.SwapNetError):
        eng.add_block([descs[0], bad], blob)
    # a failed add leaves the context usable
    eng.add_block(descs, blob)
    d2, b2 = S.block_payload(net, wts, 2, 5)
    eng.add_block(d2, b2)
    eng.plan()
    with pytest.raises(S.SwapNetError) as e:
        eng.add_block(d2, b2)
    assert e.value.code == S.SN_E_STATE
    assert lib.sn_plan(eng.ctx) == S.SN_E_STATE
    x = np.zeros((3, 32, 32), np.float16)
    out = np.zeros(10, np.float16)
    assert lib.sn_infer(eng.ctx, x.ctypes.data_as(C.c_void_p),
                        out.ctypes.data_as(C.c_void_p)) == S.SN_E_UNSUPPORTED
    assert lib.sn_infer(None, None, None) == S.SN_E_INVALID
    lib.sn_destroy(None)
    eng.close()


def test_token_network_errors():
    lib = S.load_library()
    eng = S.SwapNet(1 << 20, host_only=True)
    net = W.get_network("tiny_cnn")
    wts = W.make_weights(net)
    d, b = S.block_payload(net, wts, 0, 5)
    eng.add_block(d, b)
    eng.plan()
    ids = np.zeros(4, np.int32)
    lg = np.zeros(10, np.float32)
    assert lib.sn_infer_tokens(eng.ctx, ids.ctypes.data_as(C.c_void_p), 4,
                               lg.ctypes.data_as(C.c_void_p)) in (S.SN_E_UNSUPPORTED,)


def test_host_buffers_sized_from_the_library():
    # sn_stats reports the bytes sn_infer reads and writes; the binding sizes
    # its buffers from them and refuses mismatched inputs before any call
    net = W.tiny_cnn()
    eng = S.build_engine(net, lambda li: W.layer_params(net, li), host_only=True)
    st = eng.stats()
    assert st["input_bytes"] == 3 * 32 * 32 * 2
    assert st["output_bytes"] == 10 * 2
    with pytest.raises(ValueError):
        eng.infer(np.zeros((3, 16, 16), np.float16))
    eng.out_shape = (3,)
    with pytest.raises(ValueError):
        eng.infer(np.zeros((3, 32, 32), np.float16))
    eng.out_shape = None   # unknown shape: a flat buffer of output_bytes
    with pytest.raises(S.SwapNetError):   # host-only contexts cannot run
        eng.infer(np.zeros((3, 32, 32), np.float16))
    eng.close()
    dec = W.decoder7b(n_layers=1, d=64, heads=2, ffn=96, vocab=100, max_seq=16, prompt=4, gen=2)
    eng = S.build_engine(dec, lambda li: W.layer_params(dec, li), host_only=True)
    st = eng.stats()
    assert st["input_bytes"] == 0 and st["output_bytes"] == 100 * 4
    eng.close()
