"""Host-side tests of the delay model and the partition search (no GPU):
the predicted time of a plan against closed forms that hold whatever the
partition (link only, compute only, resident), the search against the other
partitions and against brute force over every layer-boundary partition of a
small network, and the cost-model C API."""
import itertools
import math

import numpy as np
import pytest

from paper_2401_16757_amd import swapnet as S
from paper_2401_16757_amd import workloads as W


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import os
    if not os.path.exists(S.LIB_PATH):
        from paper_2401_16757_amd import build
        build.build()
    S.load_library()


_WEIGHTS = {}


def weights_of(name):
    if name not in _WEIGHTS:
        net = W.get_network(name)
        _WEIGHTS[name] = (net, W.make_weights(net))
    return _WEIGHTS[name]


def model_for(net, **kw):
    """A delay model with seeded per-layer times in [2, 32) us (any positive
    times will do)."""
    rng = np.random.default_rng(5)
    ex = np.array([2e-6 + rng.uniform(0, 30e-6) for _ in net.layers], np.float32)
    m = dict(alpha=1 / 50e9, beta=10e-6, gamma=0.0, kappa=4e-6, gate=20e-6, wake=5e-6,
             slab_ex=5e-6, layer_ex=ex)
    m.update(kw)
    return m


def plan(net, wts, budget, partition, model, blocks=None):
    return S.build_engine(net, wts, budget=budget, host_only=True, partition=partition,
                          cost_model=model, blocks=blocks)


@pytest.mark.parametrize("name", ["resnet50", "fcn_resnet101", "vgg16"])
@pytest.mark.parametrize("partition", [0, 1, 2])
def test_predicted_time_closed_forms(name, partition):
    net, wts = weights_of(name)
    budget = int(net.weight_bytes() / 4)
    base = model_for(net)
    ex = np.asarray(base["layer_ex"], np.float64)
    with plan(net, wts, budget, partition, base) as eng:
        sl = eng.slabs()
        nz = sum(1 for s in sl if s["bytes"])
        n = len(sl)
        image = sum(s["bytes"] for s in sl)
        # link only: the DMAs run back to back (no compute to wait for)
        eng.set_cost_model(dict(alpha=base["alpha"], beta=base["beta"], gamma=0, kappa=0, gate=0,
                                wake=0, slab_ex=0, layer_ex=np.zeros(len(net.layers))))
        lat, per = eng.predict()
        link = base["alpha"] * image + base["beta"] * nz
        assert math.isclose(lat, link, rel_tol=1e-12) and math.isclose(per, link, rel_tol=1e-12)
        # compute only: slab overheads plus every layer once (a layer cut into
        # slices costs its whole time when kappa = 0)
        eng.set_cost_model(dict(alpha=0, beta=0, gamma=0, kappa=0, gate=0, wake=0,
                                slab_ex=base["slab_ex"], layer_ex=ex))
        lat, per = eng.predict()
        comp = n * base["slab_ex"] + ex.sum()
        assert math.isclose(lat, comp, rel_tol=1e-9) and math.isclose(per, comp, rel_tol=1e-9)
        # both: never faster than either resource alone
        eng.set_cost_model(base)
        lat, per = eng.predict()
        # (slices of a layer only add time when kappa > 0)
        assert per >= max(link, comp) * (1 - 1e-12)
        assert lat >= max(link, comp) * (1 - 1e-12)


def test_resident_prediction_is_the_sum_of_execution():
    net, wts = weights_of("resnet50")
    m = model_for(net)
    with plan(net, wts, net.weight_bytes() * 2, 0, m) as eng:
        assert eng.stats()["resident"] == 1
        lat, per = eng.predict()
        want = eng.stats()["n_slabs"] * m["slab_ex"] + float(np.sum(np.asarray(m["layer_ex"], np.float64)))
        assert math.isclose(lat, want, rel_tol=1e-9) and lat == per


@pytest.mark.parametrize("name", ["resnet50", "fcn_resnet101", "vgg16"])
@pytest.mark.parametrize("frac", [1 / 2.32, 1 / 3, 1 / 4, 1 / 5.81])
def test_search_never_loses_to_the_other_partitions(name, frac):
    net, wts = weights_of(name)
    budget = int(net.weight_bytes() * frac)
    m = model_for(net)
    per = {}
    for p in (0, 1, 2):
        with plan(net, wts, budget, p, m) as eng:
            per[p] = eng.predict()[1]
            assert eng.stats()["resident"] == 0
    assert per[2] <= min(per[0], per[1]) * (1 + 1e-9), per


def chain_net():
    """Eight 1x1 convolutions of different widths on a 4x4 input: small
    enough to enumerate every partition at layer boundaries."""
    b = W._Builder()
    widths = [64, 96, 160, 128, 224, 96, 192, 64, 128]
    x = 0
    for i in range(8):
        x = b.add(name="c%d" % i, op="conv2d", src=x, c_in=widths[i], c_out=widths[i + 1],
                  h_in=4, w_in=4, k=1, relu=True, bn=True)
    return W.Network("chain8", 1, b.layers, [[0, 8]], (64, 4, 4), x)


@pytest.mark.parametrize("frac", [0.7, 0.55, 0.46])
def test_search_matches_brute_force_over_layer_cuts(frac):
    net = chain_net()
    wts = W.make_weights(net)
    budget = int(net.weight_bytes() * frac)
    rng = np.random.default_rng(11)
    m = dict(alpha=1 / 50e9, beta=3e-6, gamma=0.0, kappa=1e-6, gate=4e-6, wake=1e-6, slab_ex=1e-6,
             layer_ex=rng.uniform(1e-6, 12e-6, len(net.layers)).astype(np.float32))
    best = None
    for k in range(1, 8):
        for cuts in itertools.combinations(range(1, 8), k):
            edges = (0,) + cuts + (8,)
            blocks = [[edges[i], edges[i + 1]] for i in range(len(edges) - 1)]
            try:
                eng = plan(net, wts, budget, 0, m, blocks=blocks)
            except S.SwapNetError:
                continue
            # only plans that kept the given cuts (no channel splits) count
            if eng.stats()["n_slabs"] == len(blocks):
                per = eng.predict()[1]
                best = per if best is None else min(best, per)
            eng.close()
    assert best is not None
    with plan(net, wts, budget, 2, m) as eng:
        per = eng.predict()[1]
    assert per <= best * (1 + 1e-9), (per, best)


def test_cost_model_api_round_trip_and_errors():
    net, wts = weights_of("resnet50")
    m = model_for(net)
    eng = S.SwapNet(int(net.weight_bytes() / 3), host_only=True)
    with pytest.raises(S.SwapNetError) as e:
        eng.predict()
    assert e.value.code == S.SN_E_STATE
    for a, b in net.blocks:
        eng.add_block(*S.block_payload(net, wts, a, b))
    eng.set_cost_model(m)
    got = eng.cost_model()
    for k in S.COST_KEYS:
        assert got[k] == m[k]
    assert np.array_equal(got["layer_ex"], m["layer_ex"])
    for bad in (dict(alpha=-1.0), dict(beta=float("nan")), dict(gate=float("inf")),
                dict(layer_ex=np.zeros(3, np.float32))):
        with pytest.raises(S.SwapNetError) as e:
            eng.set_cost_model(dict(m, **bad))
        assert e.value.code == S.SN_E_INVALID
    assert np.array_equal(eng.cost_model()["layer_ex"], m["layer_ex"])   # unchanged
    eng.set_option(S.OPT_PARTITION, 2)
    with pytest.raises(S.SwapNetError):
        eng.set_option(S.OPT_PARTITION, 3)
    # swap-in ordering modes 0..2 (2: ROCr copies + gate kernels; a host-only
    # context sets it up nothing)
    for v in (2, 1, 0):
        eng.set_option(S.OPT_SYNC, v)
    for bad in (-1, 3):
        with pytest.raises(S.SwapNetError) as e:
            eng.set_option(S.OPT_SYNC, bad)
        assert e.value.code == S.SN_E_INVALID
    for v in (1, 0):
        eng.set_option(S.OPT_GATE_LIMIT_US, v)
    for bad in (-1, 3600 * 10**6 + 1):
        with pytest.raises(S.SwapNetError) as e:
            eng.set_option(S.OPT_GATE_LIMIT_US, bad)
        assert e.value.code == S.SN_E_INVALID
    eng.plan()
    lat, per = eng.predict()
    assert 0 < per <= lat * 1.5
    with pytest.raises(S.SwapNetError) as e:
        eng.calibrate(3)
    assert e.value.code == S.SN_E_UNSUPPORTED
    eng.close()


@pytest.mark.parametrize("name", ["resnet50", "fcn_resnet101"])
def test_replan_in_place_equals_a_fresh_plan(name):
    # re-forming the slabs from the registered layers (no re-registration)
    # gives the very image a fresh plan at that budget / partition gives
    net, wts = weights_of(name)
    B1, B2 = int(net.weight_bytes() / 2.32), int(net.weight_bytes() / 5.81)
    eng = S.build_engine(net, wts, budget=B1, host_only=True)
    img1 = eng.image()
    eng.replan(B2)
    with S.build_engine(net, wts, budget=B2, host_only=True) as fresh:
        assert np.array_equal(eng.image(), fresh.image())
        assert eng.slabs() == fresh.slabs()
    eng.set_option(S.OPT_PARTITION, 1)
    eng.replan()
    with S.build_engine(net, wts, budget=B2, host_only=True, partition=1) as fresh:
        assert np.array_equal(eng.image(), fresh.image())
    eng.set_option(S.OPT_PARTITION, 0)
    eng.replan(B1)
    assert np.array_equal(eng.image(), img1)
    assert eng.stats()["budget_bytes"] == B1
    eng.close()


def test_replan_errors_leave_the_context_unchanged():
    net, wts = weights_of("resnet50")
    eng = S.SwapNet(int(net.weight_bytes() / 3), host_only=True)
    with pytest.raises(S.SwapNetError) as e:
        eng.replan(1 << 20)
    assert e.value.code == S.SN_E_STATE
    for a, b in net.blocks:
        eng.add_block(*S.block_payload(net, wts, a, b))
    eng.plan()
    img, sl = eng.image(), eng.slabs()
    with pytest.raises(S.SwapNetError) as e:
        eng.replan(4096)            # no layer fits half of it
    assert e.value.code == S.SN_E_INFEASIBLE
    with pytest.raises(S.SwapNetError) as e:
        eng.replan(100)
    assert e.value.code == S.SN_E_INVALID
    assert np.array_equal(eng.image(), img) and eng.slabs() == sl
    eng.close()


def test_split_budget_follows_eq1():
    GB = 1 << 30
    # the paper's example: 1.5 GB of demand in 1 GB; with equal scores the
    # first term gives each model 2/3 of its demand times (1 - 1/n), the
    # reserved 1/n is shared equally
    out = S.split_budget([GB // 2, GB], [1.0, 2.0], [1.0, 1.0], GB)
    # PS = latency / memory: 1/(GB/2) and 2/GB are equal
    want = [(1 / 3) * 0.5 * GB + 0.5 * 0.5 * GB, (2 / 3) * 0.5 * GB + 0.5 * 0.5 * GB]
    assert all(abs(o - w) < 256 for o, w in zip(out, want)), (out, want)
    assert all(o % 256 == 0 for o in out) and sum(out) <= GB
    # scores proportional to demand: both terms proportional, shares = demand share
    need = [3 * GB, 5 * GB, 8 * GB]
    lat = [n * n / GB for n in need]          # PS = latency / memory = need / GB
    out = S.split_budget(need, lat, [1, 1, 1], 4 * GB)
    for o, n in zip(out, need):
        assert abs(o - n / sum(need) * 4 * GB) < 256
    # one model: all of it; demands that fit: the demands
    assert S.split_budget([5 * GB], [0.1], [1.0], GB) == [GB]
    assert S.split_budget([GB, GB], [1, 1], [1, 1], 3 * GB) == [GB, GB]
    # urgency moves the reserved share only
    a = S.split_budget([GB, GB], [1, 1], [1, 0], GB)
    assert abs(a[0] - (0.25 + 0.5) * GB) < 256 and abs(a[1] - 0.25 * GB) < 256
    with pytest.raises(S.SwapNetError):
        S.split_budget([0, GB], [1, 1], [1, 1], GB)
