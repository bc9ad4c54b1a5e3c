"""GPU parity: the HIP engine (through the C ABI) against the fp64 oracle.

Bar: max|gpu - ref| <= 1e-2 * max|ref| on the final output of each network
(per step for the decoder); swapped runs bit-identical to all-resident runs
and to runs with a different slab partition.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2401_16757_amd import swapnet as S
from paper_2401_16757_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 1e-2


def rel_err(got, ref):
    ref = np.asarray(ref, np.float64)
    return float(np.abs(np.asarray(got, np.float64) - ref).max() / np.abs(ref).max())


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    S.load_library()


_cache = {}


def net_case(name, **kw):
    key = (name, tuple(sorted(kw.items())))
    if key not in _cache:
        net = W.get_network(name, **kw)
        wts = W.make_weights(net)
        x = W.make_input(net)
        ref = oracle.forward(net, wts, x)
        _cache[key] = (net, wts, x, ref)
    return _cache[key]


def run(net, wts, x, **kw):
    with S.build_engine(net, wts, **kw) as eng:
        st = eng.stats()
        y = eng.infer(x)
        y2 = eng.infer(x)
    assert np.array_equal(y.view(np.uint16), y2.view(np.uint16)), "repeat run not bit-identical"
    return y, st


CNN_CASES = [("tiny_cnn", {}), ("resnet50", {}), ("vgg16", {}), ("fcn_resnet101", {}),
             ("resnet50", {"res": 96}), ("fcn_resnet101", {"res": 128}), ("vgg16", {"res": 64})]


@pytest.mark.parametrize("name,kw", CNN_CASES)
def test_swapped_matches_oracle_and_resident(name, kw):
    print(f"[case] {name} {kw}", flush=True)
    net, wts, x, ref = net_case(name, **kw)
    budget = net.budget_bytes()
    y, st = run(net, wts, x, budget=budget)
    assert st["resident"] == 0 and st["n_slabs"] >= 2
    assert st["arena_high_water"] <= budget
    err = rel_err(y, ref)
    print(f"  swapped slabs={st['n_slabs']} err={err:.2e}", flush=True)
    assert err <= TOL
    big = st["image_bytes"] + 4096
    # all-resident with the same slabs, all-resident unsplit, and a stricter partition
    y_res_same, st1 = run(net, wts, x, budget=big, split_budget=budget)
    y_res, st2 = run(net, wts, x, budget=big)
    assert st1["resident"] == 1 and st2["resident"] == 1
    for other in (y_res_same, y_res):
        assert np.array_equal(y.view(np.uint16), other.view(np.uint16))
    tight = max(int(net.weight_bytes() / 5.81), 4 * 1024)
    try:
        y_tight, st3 = run(net, wts, x, budget=tight)
    except S.SwapNetError as e:
        assert e.code == S.SN_E_INFEASIBLE
    else:
        assert st3["n_slabs"] >= st["n_slabs"]
        assert np.array_equal(y.view(np.uint16), y_tight.view(np.uint16))


def single_layer_net(spec, cfg=90):
    spec.src, spec.dst = 0, 1
    net = W.Network("one_" + spec.op, cfg, [spec], [[0, 1]], (spec.c_in, spec.h_in, spec.w_in), 1)
    return net


CONV_SHAPES = [
    # c_in, c_out, h, w, k, stride, pad, dil
    (3, 16, 32, 32, 3, 1, 1, 1), (3, 64, 37, 29, 7, 2, 3, 1), (16, 40, 17, 19, 3, 2, 1, 1),
    (64, 72, 9, 11, 3, 1, 2, 2), (32, 24, 13, 13, 3, 1, 4, 4), (256, 520, 7, 7, 1, 1, 0, 1),
    (24, 200, 15, 15, 1, 2, 0, 1), (512, 96, 7, 7, 3, 1, 1, 1), (64, 21, 40, 40, 1, 1, 0, 1),
    (128, 256, 56, 56, 1, 1, 0, 1), (64, 64, 56, 56, 3, 1, 1, 1),
    # K-split with 16 tiles and a ragged last tile (partials added in-kernel)
    (1024, 200, 14, 14, 3, 1, 1, 1),
]


@pytest.mark.parametrize("shape", CONV_SHAPES)
def test_conv_kernel_parity_and_slice_invariance(shape):
    ci, co, h, w, k, st, pad, dil = shape
    print(f"[case] conv {shape}", flush=True)
    spec = W.LayerSpec(name="c", op="conv2d", src=0, dst=1, c_in=ci, c_out=co, h_in=h, w_in=w,
                       k=k, stride=st, pad=pad, dilation=dil, relu=True, bn=True)
    net = single_layer_net(spec)
    wts = W.make_weights(net)
    x = W.make_input(net)
    ref = oracle.forward(net, wts, x)
    y, _ = run(net, wts, x, budget=1 << 30)
    assert rel_err(y, ref) <= TOL
    # split the layer by output channels: every output bit must be unchanged
    wbytes = net.weight_bytes()
    for parts in (2, 3, 5):
        y2, st2 = run(net, wts, x, budget=1 << 30, split_budget=max(2 * wbytes // (parts + 1), 2048))
        assert st2["n_slabs"] >= 2
        assert np.array_equal(y.view(np.uint16), y2.view(np.uint16)), parts


# every tile variant of the conv kernels, forced (SN_OPT_CONV_KERNEL) on the
# shapes of its kind: strided and ragged 1x1, dilated and strided taps with
# Cin_p a multiple of 64, K shorter than the stages in flight, output
# channels not a multiple of the tile, weight rows outnumbering pixels
FORCED_SHAPES = {
    "1x1": [(64, 96, 9, 9, 1, 1, 0, 1), (40, 70, 11, 13, 1, 2, 0, 1), (512, 200, 7, 7, 1, 1, 0, 1),
            (48, 40, 5, 3, 1, 1, 0, 1)],
    "tap": [(64, 72, 11, 13, 3, 1, 2, 2), (128, 64, 7, 7, 3, 1, 1, 1), (64, 24, 6, 5, 3, 2, 1, 1),
            (256, 300, 4, 4, 3, 1, 1, 1)],
    "gen": [(3, 16, 13, 11, 3, 1, 1, 1), (16, 40, 9, 9, 3, 2, 1, 1), (8, 70, 12, 12, 7, 2, 3, 1)],
}


def _variant_kind(name):
    return "1x1" if name.endswith("_1x1") else "tap" if name.endswith("_tap") else "gen"


@pytest.mark.parametrize("variant", range(S.conv_kernel_count()))
def test_forced_conv_variants(variant):
    name = S.kernel_name(variant)
    for shape in FORCED_SHAPES[_variant_kind(name)]:
        ci, co, h, w, k, st, pad, dil = shape
        print(f"[case] conv variant {name} shape {shape}", flush=True)
        spec = W.LayerSpec(name="c", op="conv2d", src=0, dst=1, c_in=ci, c_out=co, h_in=h, w_in=w,
                           k=k, stride=st, pad=pad, dilation=dil, relu=True, bn=True)
        net = single_layer_net(spec)
        wts = W.make_weights(net)
        x = W.make_input(net)
        ref = oracle.forward(net, wts, x)
        y, _ = run(net, wts, x, budget=1 << 30, conv_kernel=variant + 1)
        assert rel_err(y, ref) <= TOL, shape
        wbytes = net.weight_bytes()
        for parts in (2, 3):
            y2, st2 = run(net, wts, x, budget=1 << 30, conv_kernel=variant + 1,
                          split_budget=max(2 * wbytes // (parts + 1), 2048))
            assert st2["n_slabs"] >= 2
            assert np.array_equal(y.view(np.uint16), y2.view(np.uint16)), (shape, parts)


def _random_conv_shapes(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        k = int(rng.choice([1, 3, 3, 5, 7]))
        ci = int(rng.choice([3, 8, 13, 32, 64, 72, 128, 200, 256]))
        co = int(rng.choice([5, 16, 33, 64, 100, 128, 257]))
        h, w = int(rng.integers(3, 30)), int(rng.integers(3, 30))
        st = int(rng.choice([1, 1, 2]))
        dil = int(rng.choice([1, 1, 2])) if k > 1 else 1
        pad = int(rng.integers(0, dil * (k // 2) + 1))
        if (h + 2 * pad - dil * (k - 1) - 1) < 0 or (w + 2 * pad - dil * (k - 1) - 1) < 0:
            pad = dil * (k // 2)
        out.append((ci, co, h, w, k, st, pad, dil))
    return out


@pytest.mark.parametrize("shape", _random_conv_shapes(16, 2024))
def test_random_conv_shapes(shape):
    # seeded random convolutions (ragged channels and sizes, any padding,
    # strides, dilations): parity with the oracle and bit-identity of the
    # layer cut into two and three channel slices
    ci, co, h, w, k, st, pad, dil = shape
    print(f"[case] random conv {shape}", flush=True)
    spec = W.LayerSpec(name="c", op="conv2d", src=0, dst=1, c_in=ci, c_out=co, h_in=h, w_in=w,
                       k=k, stride=st, pad=pad, dilation=dil, relu=bool(co % 2), bn=True)
    net = single_layer_net(spec)
    wts = W.make_weights(net)
    x = W.make_input(net)
    ref = oracle.forward(net, wts, x)
    y, _ = run(net, wts, x, budget=1 << 30)
    assert rel_err(y, ref) <= TOL
    wbytes = net.weight_bytes()
    for parts in (2, 3):
        y2, st2 = run(net, wts, x, budget=1 << 30, split_budget=max(2 * wbytes // (parts + 1), 2048))
        assert np.array_equal(y.view(np.uint16), y2.view(np.uint16)), parts


LINEAR_SHAPES = [(256, 10, False), (2048, 1000, True), (25088, 4096, True), (4096, 37, False),
                 (520, 1003, True)]


@pytest.mark.parametrize("k_in,n_out,relu", LINEAR_SHAPES)
def test_linear_kernel_parity_and_slice_invariance(k_in, n_out, relu):
    print(f"[case] linear {k_in}->{n_out}", flush=True)
    spec = W.LayerSpec(name="fc", op="linear", src=0, dst=1, c_in=k_in, c_out=n_out, relu=relu)
    net = W.Network("one_linear", 91, [spec], [[0, 1]], (k_in, 1, 1), 1)
    wts = W.make_weights(net)
    x = W.make_input(net)
    ref = oracle.forward(net, wts, x)
    y, _ = run(net, wts, x, budget=1 << 30)
    assert rel_err(y, ref) <= TOL
    y2, st2 = run(net, wts, x, budget=1 << 30, split_budget=max(int(0.7 * net.weight_bytes()), 4096))
    assert st2["n_slabs"] >= 2
    assert np.array_equal(y.view(np.uint16), y2.view(np.uint16))


def test_infer_dev_on_torch_stream_matches_host_path():
    net, wts, x, ref = net_case("resnet50", res=96)
    with S.build_engine(net, wts) as eng:
        y_host = eng.infer(x)
        xd = torch.from_numpy(x).cuda()
        yd = torch.empty(eng.out_shape, dtype=torch.float16, device="cuda")
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            for _ in range(3):
                eng.infer_dev(xd.data_ptr(), yd.data_ptr(), s.cuda_stream)
        s.synchronize()
        assert np.array_equal(yd.cpu().numpy().view(np.uint16), y_host.view(np.uint16))


@pytest.mark.parametrize("name,kw,frac", [("resnet50", {"res": 96}, 1 / 5.81),
                                          ("fcn_resnet101", {"res": 128}, 1 / 3),
                                          ("vgg16", {"res": 64}, 1 / 4)])
def test_balanced_partition_matches_resident(name, kw, frac):
    # the balanced partition (layers re-cut into equal slabs, layers split by
    # output channels at slab boundaries) computes the same bits as the
    # all-resident run and matches the oracle
    net, wts, x, ref = net_case(name, **kw)
    budget = int(net.weight_bytes() * frac)
    with S.build_engine(net, wts, budget=budget, partition=1) as eng:
        assert not eng.stats()["resident"]
        y = eng.infer(x)
        y2 = eng.infer(x)
    with S.build_engine(net, wts, budget=1 << 33) as res:
        yr = res.infer(x)
    assert np.array_equal(y.view(np.uint16), yr.view(np.uint16))
    assert np.array_equal(y2.view(np.uint16), yr.view(np.uint16))
    assert rel_err(y, ref) <= TOL


@pytest.mark.parametrize("name,kw,frac", [("resnet50", {"res": 96}, 1 / 5.81),
                                         ("fcn_resnet101", {"res": 128}, 1 / 4)])
def test_calibrated_searched_partition_matches_resident(name, kw, frac):
    # the delay model measured on one plan (sn_calibrate) drives the search
    # of another (partition 2); calibration leaves its engine computing the
    # same bits, and the searched plan computes the all-resident bits
    net, wts, x, ref = net_case(name, **kw)
    budget = int(net.weight_bytes() * frac)
    with S.build_engine(net, wts, budget=budget) as cal:
        y0 = cal.infer(x)
        cal.calibrate(3)
        m = cal.cost_model()
        y1 = cal.infer(x)
    assert np.array_equal(y0.view(np.uint16), y1.view(np.uint16))
    assert 10e9 < 1 / m["alpha"] < 100e9 and 0 <= m["beta"] < 200e-6, m
    assert 0 <= m["gate"] < 1e-3 and 0 <= m["wake"] < 1e-3 and 0 <= m["slab_ex"] < 1e-3, m
    ex = m["layer_ex"]
    assert len(ex) == len(net.layers) and np.all(np.isfinite(ex)) and np.all(ex > 0) and ex.sum() < 0.1
    with S.build_engine(net, wts, budget=budget, partition=2, cost_model=m) as eng:
        assert not eng.stats()["resident"]
        y = eng.infer(x)
        lat, per = eng.predict()
        assert 0 < per < 2 * lat and 0 < lat
    with S.build_engine(net, wts, budget=1 << 33) as res:
        yr = res.infer(x)
        res.calibrate(2)   # rewrites the resident arena with its own bytes
        yr2 = res.infer(x)
    assert np.array_equal(y.view(np.uint16), yr.view(np.uint16))
    assert np.array_equal(yr2.view(np.uint16), yr.view(np.uint16))
    assert rel_err(y, ref) <= TOL


@pytest.mark.parametrize("modes", [((2, 0),), ((2, 1),), ((2, 2),), ((1, 0),), ((0, 0),),
                                   ((2, 0, 2),), ((2, 1, 2),),
                                   ((2, 1), (1, 0), (2, 0), (0, 0), (2, 1)),
                                   ((2, 2), (2, 0), (1, 0), (2, 2), (2, 1), (2, 2)),
                                   ((2, 0, 2), (2, 1, 2), (2, 0, 1), (2, 0, 2), (1, 0, 2))])
def test_back_to_back_inferences_with_cross_inference_prefetch(modes):
    # Several inferences queued without a host synchronisation: the next
    # inference's swap-ins of slabs that no earlier slab shares start while
    # the previous one still computes (waiting only for its `wrap` slabs).
    # Every output must equal a one-at-a-time inference of the same input,
    # bit for bit, in every swap-in mode (the copy thread with either kind of
    # stream ordering, SN_OPT_SYNC 0 and 1, or ROCr copies with gate kernels,
    # SN_OPT_SYNC 2; one DMA queue or slabs alternating between two) and when
    # the modes alternate.
    net, wts, x0, _ = net_case("resnet50", res=96)
    rng = np.random.default_rng(7)
    xs = [x0] + [rng.standard_normal(x0.shape).astype(np.float16) for _ in range(3)]
    with S.build_engine(net, wts) as eng:
        assert eng.stats()["n_slabs"] >= 4 and not eng.stats()["resident"]
        assert any(s["wrap_slab"] >= 0 for s in eng.slabs())
        want = [eng.infer(x) for x in xs]
        xd = [torch.from_numpy(x).cuda() for x in xs]
        s = torch.cuda.Stream()
        for mode, sync, *queues in modes:
            eng.set_option(S.OPT_SWAPIN, mode)
            eng.set_option(S.OPT_SYNC, sync)
            eng.set_option(S.OPT_COPY_STREAMS, queues[0] if queues else 1)
            yd = [torch.empty(eng.out_shape, dtype=torch.float16, device="cuda") for _ in xs]
            with torch.cuda.stream(s):
                for rep in range(2):
                    for i in range(len(xs)):
                        eng.infer_dev(xd[i].data_ptr(), yd[i].data_ptr(), s.cuda_stream)
            s.synchronize()
            for i in range(len(xs)):
                assert np.array_equal(yd[i].cpu().numpy().view(np.uint16), want[i].view(np.uint16)), (mode, i)


@pytest.mark.parametrize("name,kw,div", [("tiny_cnn", {}, 1.0), ("resnet50", {"res": 96}, 5.81),
                                         ("vgg16", {"res": 64}, 5.81)])
def test_rocr_swapin_gates(tmp_path, name, kw, div):
    # SN_OPT_SYNC 2: every swap-in is a ROCr SDMA copy with its own completion
    # signal, and a gate kernel on the compute stream polls that signal before
    # the slab's kernels.  Outputs equal the all-resident ones bit for bit,
    # host and device paths, after sn_tune and sn_replan in that mode, and
    # with an image file attached (which uses the event ordering).
    net, wts, x0, ref = net_case(name, **kw)
    rng = np.random.default_rng(5)
    xs = [x0] + [rng.standard_normal(x0.shape).astype(np.float16) for _ in range(2)]
    with S.build_engine(net, wts, budget=1 << 33) as res:
        want = [res.infer(x) for x in xs]
    budget = int(net.weight_bytes() * (0.6 if div == 1.0 else 1.0 / div))
    with S.build_engine(net, wts, budget=budget) as eng:
        eng.set_option(S.OPT_SYNC, 2)
        st = eng.stats()
        print(f"[case] {name}: {st['n_slabs']} slabs, budget {budget}", flush=True)
        assert not st["resident"] and st["n_slabs"] >= 2
        for x, w in zip(xs, want):
            assert np.array_equal(eng.infer(x).view(np.uint16), w.view(np.uint16))
        assert rel_err(eng.infer(x0), ref) <= TOL
        t = eng.tune(2)
        assert max(t) > 0
        xd = [torch.from_numpy(x).cuda() for x in xs]
        yd = [torch.empty(eng.out_shape, dtype=torch.float16, device="cuda") for _ in xs]
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            for rep in range(3):
                for i in range(len(xs)):
                    eng.infer_dev(xd[i].data_ptr(), yd[i].data_ptr(), s.cuda_stream)
        s.synchronize()
        for i in range(len(xs)):
            assert np.array_equal(yd[i].cpu().numpy().view(np.uint16), want[i].view(np.uint16)), i
        eng.replan(int(budget * 0.8))
        assert eng.stats()["n_slabs"] >= 2
        for x, w in zip(xs, want):
            assert np.array_equal(eng.infer(x).view(np.uint16), w.view(np.uint16))
        path = str(tmp_path / "image.bin")
        eng.save_image(path)
        eng.attach_image_file(path)
        for sync in (2, 0, 2):
            eng.set_option(S.OPT_SYNC, sync)
            for x, w in zip(xs, want):
                assert np.array_equal(eng.infer(x).view(np.uint16), w.view(np.uint16)), sync


def test_gate_time_out_is_reported():
    # Failure path of the device-side gates (SN_OPT_SYNC 2), forced from the
    # host: with a 1 us bound every gate that starts before its slab has
    # landed gives up at once.  VGG-16 at 1/5.81 is link-bound (12 slabs of
    # ~23 MB, ~0.4 ms each, little compute), so gates do start early.  The
    # call reports SN_E_HIP (its output is undefined), the error is reported
    # once, and with the bound restored the outputs are bit-identical again.
    net, wts, x0, _ = net_case("vgg16")
    with S.build_engine(net, wts, budget=int(net.weight_bytes() / 5.81)) as eng:
        st = eng.stats()
        print(f"[case] vgg16 gate time-out: {st['n_slabs']} slabs", flush=True)
        want = eng.infer(x0)
        eng.set_option(S.OPT_GATE_LIMIT_US, 1)
        with pytest.raises(S.SwapNetError) as e:
            for _ in range(3):
                eng.infer(x0)
        assert e.value.code == S.SN_E_HIP and "gate" in str(e.value)
        eng.set_option(S.OPT_GATE_LIMIT_US, 0)
        for _ in range(2):
            assert np.array_equal(eng.infer(x0).view(np.uint16), want.view(np.uint16))


@pytest.mark.parametrize("name,kw", [("tiny_cnn", {}), ("resnet50", {"res": 96})])
def test_image_file_swapin_matches_memory(tmp_path, name, kw):
    # Storage tier (direct block fetch): after sn_attach_image_file every
    # swap-in reads its slab from the file into a staging slot, then DMAs it.
    # Outputs must equal the in-memory image's bit for bit: host path, device
    # path, several inferences queued back to back.
    net, wts, x0, ref = net_case(name, **kw)
    rng = np.random.default_rng(11)
    xs = [x0] + [rng.standard_normal(x0.shape).astype(np.float16) for _ in range(2)]
    path = str(tmp_path / "image.bin")
    with S.build_engine(net, wts) as eng:
        st0 = eng.stats()
        assert not st0["resident"] and st0["n_slabs"] >= 2
        want = [eng.infer(x) for x in xs]
        eng.save_image(path)
        eng.attach_image_file(path)
        st = eng.stats()
        print(f"[case] {name}: {st['n_slabs']} slabs, direct_io={st['direct_io']}, "
              f"host weight bytes {st['host_weight_bytes']} of {st['image_bytes']}", flush=True)
        assert st["file_backed"] == 1
        # two read slots and two pinned slots of the largest slab (4 KiB pages)
        slot = -(-max(s["bytes"] for s in eng.slabs()) // 4096) * 4096
        assert st["host_weight_bytes"] == 4 * slot
        for rep in range(2):
            for x, w in zip(xs, want):
                assert np.array_equal(eng.infer(x).view(np.uint16), w.view(np.uint16)), rep
        xd = [torch.from_numpy(x).cuda() for x in xs]
        yd = [torch.empty(eng.out_shape, dtype=torch.float16, device="cuda") for _ in xs]
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            for rep in range(2):
                for i in range(len(xs)):
                    eng.infer_dev(xd[i].data_ptr(), yd[i].data_ptr(), s.cuda_stream)
        s.synchronize()
        for i in range(len(xs)):
            assert np.array_equal(yd[i].cpu().numpy().view(np.uint16), want[i].view(np.uint16)), i
        assert eng.stats()["read_ms"] > 0
        # calls that need the in-memory image are refused
        for call in (lambda: eng.replan(), lambda: eng.tune(1), lambda: eng.calibrate(1),
                     lambda: eng.image(), lambda: eng.set_option(S.OPT_SWAPIN, 1),
                     lambda: eng.set_option(S.OPT_NAIVE, 1), lambda: eng.attach_image_file(path)):
            with pytest.raises(S.SwapNetError) as e:
                call()
            assert e.value.code == S.SN_E_STATE
        # still running from the file afterwards
        assert np.array_equal(eng.infer(x0).view(np.uint16), want[0].view(np.uint16))
    assert rel_err(want[0], ref) <= TOL
    # a file of another plan, and a file whose slab bytes differ, are refused;
    # the engine keeps swapping from memory
    with S.build_engine(net, wts, budget=int(st0["image_bytes"] * 0.3)) as other:
        assert other.stats()["n_slabs"] != st0["n_slabs"]
        with pytest.raises(S.SwapNetError) as e:
            other.attach_image_file(path)
        assert e.value.code == S.SN_E_INVALID
    raw = bytearray(open(path, "rb").read())
    raw[-5000] ^= 0x5A if len(raw) > 5000 else 0
    raw[4096 + 17] ^= 0x01
    bad = str(tmp_path / "bad.bin")
    open(bad, "wb").write(bytes(raw))
    with S.build_engine(net, wts) as eng:
        with pytest.raises(S.SwapNetError) as e:
            eng.attach_image_file(bad)
        assert e.value.code == S.SN_E_INVALID
        assert eng.stats()["file_backed"] == 0
        assert np.array_equal(eng.infer(x0).view(np.uint16), want[0].view(np.uint16))


def small_decoder(**kw):
    a = dict(n_layers=2, d=128, heads=4, ffn=160, vocab=300, max_seq=48, prompt=24, gen=8)
    a.update(kw)
    return W.decoder7b(**a)


def test_decoder_teacher_forced_parity():
    net = small_decoder()
    wts = W.make_weights(net)
    prompt = W.make_input(net)
    gen = net.extra["gen"]
    lb = sum(l.weight_bytes() for l in net.layers[1:8])
    for budget, split, sync in ((2 * lb, None, 0), (2 * lb, None, 1), (2 * lb, None, 2), (1 << 30, 2 * lb, 0)):
        eng = S.build_engine(net, wts, budget=budget, split_budget=split)
        eng.set_option(S.OPT_SYNC, sync)
        rows, fed = [], []
        logits = eng.infer_tokens(prompt)
        rows.append(logits)
        for _ in range(gen - 1):
            nxt = int(np.argmax(logits))
            fed.append(nxt)
            logits = eng.infer_tokens(np.array([nxt], np.int32))
            rows.append(logits)
        eng.close()
        seq = np.concatenate([prompt, np.array(fed, np.int32)])
        ref = oracle.decoder_forward(net, wts, seq)
        got = np.stack(rows)
        want = ref[len(prompt) - 1:]
        for t in range(gen):
            assert rel_err(got[t], want[t]) <= TOL, t
        if split is None and sync == 0:
            first = got
        else:
            assert np.array_equal(first.view(np.uint32), got.view(np.uint32))


def test_decoder_calibration_keeps_generation():
    # calibrating a token network runs one token at the current position
    # without advancing it: the generation that follows is unchanged
    net = small_decoder()
    wts = W.make_weights(net)
    prompt = W.make_input(net)
    lb = sum(l.weight_bytes() for l in net.layers[1:8])
    runs = []
    for calibrate in (False, True):
        with S.build_engine(net, wts, budget=2 * lb) as eng:
            rows = [eng.infer_tokens(prompt)]
            if calibrate:
                eng.calibrate(2)
                assert np.all(eng.cost_model()["layer_ex"] > 0)
            for _ in range(4):
                rows.append(eng.infer_tokens(np.array([int(np.argmax(rows[-1]))], np.int32)))
            runs.append(np.stack(rows))
    assert np.array_equal(runs[0].view(np.uint32), runs[1].view(np.uint32))


def test_replan_in_place_keeps_results():
    # one context re-planned for a smaller budget, for a budget above its
    # arena (resident: a new arena) and for the balanced partition computes
    # the same bits every time
    net, wts, x, ref = net_case("resnet50", res=96)
    B = net.weight_bytes()
    with S.build_engine(net, wts, budget=int(B / 2.32)) as eng:
        y0 = eng.infer(x)
        for budget, partition, resident in ((int(B / 5.81), 0, 0), (2 * B, 0, 1), (int(B / 3), 1, 0)):
            eng.set_option(S.OPT_PARTITION, partition)
            eng.replan(budget)
            assert eng.stats()["resident"] == resident
            y = eng.infer(x)
            assert np.array_equal(y.view(np.uint16), y0.view(np.uint16)), (budget, partition)
    assert rel_err(y0, ref) <= TOL


@pytest.mark.parametrize("flags", [1, 3, 5, 9, 15])
def test_naive_swapping_modes_compute_the_same(flags):
    # the measurement-only naive modes (sequential, per-swap allocation,
    # pageable source, copy-based assembly) run the same kernels on the same
    # bytes: bit-identical to the engine's own path
    net, wts, x, _ = net_case("resnet50", res=96)
    with S.build_engine(net, wts, budget=int(net.weight_bytes() / 5.81)) as eng:
        y0 = eng.infer(x)
        eng.set_option(S.OPT_NAIVE, flags)
        y1 = eng.infer(x)
        y2 = eng.infer(x)
        eng.set_option(S.OPT_NAIVE, 0)
        y3 = eng.infer(x)
    for y in (y1, y2, y3):
        assert np.array_equal(y.view(np.uint16), y0.view(np.uint16)), flags


def test_tune_keeps_the_fastest_partition():
    net, wts, x, _ = net_case("fcn_resnet101", res=128)
    with S.build_engine(net, wts, budget=int(net.weight_bytes() / 4)) as eng:
        y0 = eng.infer(x)
        t = eng.tune(2)
        assert all(v >= 0 for v in t) and sum(1 for v in t if v > 0) >= 2, t
        y = eng.infer(x)
        assert np.array_equal(y.view(np.uint16), y0.view(np.uint16))


def test_two_models_share_a_budget_and_adapt():
    # Eq. 1 splits one budget between two models; when the total shrinks,
    # both are re-planned in place and compute the same bits
    cases = [net_case("resnet50", res=96), net_case("fcn_resnet101", res=128)]
    need = [c[0].weight_bytes() for c in cases]
    engines, outs = [], []
    budgets = S.split_budget(need, [1e-3, 2e-3], [1.0, 1.0], sum(need) // 2)
    for (net, wts, x, ref), b in zip(cases, budgets):
        eng = S.build_engine(net, wts, budget=b)
        assert not eng.stats()["resident"]
        y = eng.infer(x)
        assert rel_err(y, ref) <= TOL
        engines.append(eng)
        outs.append(y)
    smaller = S.split_budget(need, [1e-3, 2e-3], [1.0, 1.0], int(sum(need) * 0.35))
    assert all(a < b for a, b in zip(smaller, budgets))
    for eng, b, (net, wts, x, _), y0 in zip(engines, smaller, cases, outs):
        eng.replan(b)
        assert eng.stats()["budget_bytes"] == b
        y = eng.infer(x)
        assert np.array_equal(y.view(np.uint16), y0.view(np.uint16))
        eng.close()


def test_decoder_replan_mid_generation():
    # a token network re-planned between tokens keeps its KV cache and
    # position: the generation continues as if nothing happened
    net = small_decoder()
    wts = W.make_weights(net)
    prompt = W.make_input(net)
    lb = sum(l.weight_bytes() for l in net.layers[1:8])
    runs = []
    for replan in (False, True):
        with S.build_engine(net, wts, budget=2 * lb) as eng:
            rows = [eng.infer_tokens(prompt)]
            for k in range(5):
                if replan and k == 2:
                    eng.replan(3 * lb)
                if replan and k == 4:
                    eng.set_option(S.OPT_PARTITION, 1)
                    eng.replan(2 * lb)
                rows.append(eng.infer_tokens(np.array([int(np.argmax(rows[-1]))], np.int32)))
            runs.append(np.stack(rows))
    assert np.array_equal(runs[0].view(np.uint32), runs[1].view(np.uint32))


def test_decoder_generation_from_image_file(tmp_path):
    # the storage tier under a token network: prefill and decode steps with
    # every layer block read from the image file give the same logits bits
    net = small_decoder()
    wts = W.make_weights(net)
    prompt = W.make_input(net)
    lb = sum(l.weight_bytes() for l in net.layers[1:8])
    path = str(tmp_path / "decoder.img")
    runs = []
    for from_file in (False, True):
        with S.build_engine(net, wts, budget=2 * lb) as eng:
            assert not eng.stats()["resident"]
            if from_file:
                eng.save_image(path)
                eng.attach_image_file(path)
                assert eng.stats()["file_backed"] == 1
            rows = [eng.infer_tokens(prompt)]
            for _ in range(5):
                rows.append(eng.infer_tokens(np.array([int(np.argmax(rows[-1]))], np.int32)))
            runs.append(np.stack(rows))
    assert np.array_equal(runs[0].view(np.uint32), runs[1].view(np.uint32))


def test_decoder_long_context_split_attention():
    # 200-token prompt: single-token steps attend over 200+ cached positions,
    # which the attention kernel splits over several blocks (per-chunk
    # partials merged in order); teacher-forced against the oracle
    net = small_decoder(max_seq=224, prompt=200, gen=6)
    wts = W.make_weights(net)
    prompt = W.make_input(net)
    gen = net.extra["gen"]
    with S.build_engine(net, wts, budget=1 << 30) as eng:
        rows, fed = [eng.infer_tokens(prompt)], []
        for _ in range(gen - 1):
            nxt = int(np.argmax(rows[-1]))
            fed.append(nxt)
            rows.append(eng.infer_tokens(np.array([nxt], np.int32)))
    seq = np.concatenate([prompt, np.array(fed, np.int32)])
    want = oracle.decoder_forward(net, wts, seq)[len(prompt) - 1:]
    for t in range(gen):
        assert rel_err(rows[t], want[t]) <= TOL, t


def test_decoder_prefill_uses_mfma_path_and_decode_matches_prefix():
    """Logits of a prompt processed in one call equal (to the bar) the logits
    of the same tokens fed one by one (GEMM path vs GEMV path)."""
    net = small_decoder()
    wts = W.make_weights(net)
    prompt = W.make_input(net)[:10]
    with S.build_engine(net, wts, budget=1 << 30) as eng:
        a = eng.infer_tokens(prompt)
        eng.reset()
        for t in prompt:
            b = eng.infer_tokens(np.array([t], np.int32))
    ref = oracle.decoder_forward(net, wts, prompt)[-1]
    assert rel_err(a, ref) <= TOL
    assert rel_err(b, ref) <= TOL


@pytest.mark.slow
def test_decoder_full_width_two_layers():
    """Full 7B layer shapes (d 4096, 32 heads, SwiGLU 11008, vocab 32000), two
    layers, a 512-token prompt (prefill on the MFMA GEMM path) and four decode
    steps (GEMV path), swapped at a budget of one layer's weights plus change,
    teacher-forced against the oracle."""
    net = W.decoder7b(n_layers=2, max_seq=520, prompt=512, gen=4)
    print("[case] decoder full width, generating weights", flush=True)
    wts = W.make_weights(net)
    prompt = W.make_input(net)
    layer_bytes = sum(l.weight_bytes() for l in net.layers[1:8])
    eng = S.build_engine(net, wts, budget=int(layer_bytes * 1.2))
    st = eng.stats()
    assert st["resident"] == 0 and st["n_slabs"] >= 3
    rows, fed = [eng.infer_tokens(prompt)], []
    for _ in range(3):
        nxt = int(np.argmax(rows[-1]))
        fed.append(nxt)
        rows.append(eng.infer_tokens(np.array([nxt], np.int32)))
    eng.close()
    print("[case] decoder full width, oracle", flush=True)
    seq = np.concatenate([prompt, np.array(fed, np.int32)])
    ref = oracle.decoder_forward(net, wts, seq)[len(prompt) - 1:]
    for t in range(4):
        e = rel_err(rows[t], ref[t])
        print(f"  step {t}: rel err {e:.2e}", flush=True)
        assert e <= TOL
