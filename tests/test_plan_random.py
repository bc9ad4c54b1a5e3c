"""Randomised planning on the host (no GPU): seeded random chains of
convolutions, pools and linear layers, random user blocks, budgets from
the smallest feasible one up to beyond the image, every partition mode and
slab caps.  Every plan must satisfy the invariants of the swap engine's
plan (each output channel of each layer in exactly one piece, in order;
256-byte alignment; Eq. 3's pair constraint; a swap-in never overwrites a
slab that may still be in use; `wrap` slabs) and every budget below the
feasibility limit must be refused with SN_E_INFEASIBLE, never a bad plan."""
import numpy as np
import pytest

from paper_2401_16757_amd import swapnet as S
from paper_2401_16757_amd import workloads as W

from test_plan_host import check_plan


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import os
    if not os.path.exists(S.LIB_PATH):
        from paper_2401_16757_amd import build
        build.build()
    S.load_library()


def random_cnn(rng):
    """A chain: convs (k 1/3, stride 1/2, some with a residual), an optional
    max-pool, then global pooling and one or two linear layers."""
    c, h = int(rng.choice([3, 8, 16])), int(rng.choice([8, 12, 16]))
    layers, slot = [], 0
    n_conv = int(rng.integers(2, 9))
    for i in range(n_conv):
        k = int(rng.choice([1, 3]))
        st = int(rng.choice([1, 1, 2])) if h >= 4 else 1
        co = int(rng.choice([8, 16, 24, 40, 64, 96]))
        pad = k // 2
        spec = W.LayerSpec(name="c%d" % i, op="conv2d", src=slot, dst=slot + 1, c_in=c, c_out=co,
                           h_in=h, w_in=h, k=k, stride=st, pad=pad, relu=True, bn=True)
        ho = spec.out_hw()[0]
        if st == 1 and co == c and i > 0 and rng.random() < 0.5:
            spec.res = slot
        layers.append(spec)
        slot += 1
        c, h = co, ho
        if i == 1 and h >= 4 and rng.random() < 0.5:
            layers.append(W.LayerSpec(name="mp", op="maxpool", src=slot, dst=slot + 1, c_in=c,
                                      c_out=c, h_in=h, w_in=h, k=2, stride=2))
            slot += 1
            h = layers[-1].out_hw()[0]
    layers.append(W.LayerSpec(name="gap", op="gavgpool", src=slot, dst=slot + 1, c_in=c, c_out=c,
                              h_in=h, w_in=h))
    slot += 1
    for j in range(int(rng.integers(1, 3))):
        co = int(rng.choice([10, 37, 64, 100]))
        layers.append(W.LayerSpec(name="fc%d" % j, op="linear", src=slot, dst=slot + 1, c_in=c,
                                  c_out=co, relu=j == 0))
        slot += 1
        c = co
    # random user blocks: cut points between layers
    n = len(layers)
    cuts = sorted(set(int(x) for x in rng.integers(1, n, size=int(rng.integers(0, 4)))))
    bounds = [0] + cuts + [n]
    blocks = [[bounds[i], bounds[i + 1]] for i in range(len(bounds) - 1)]
    return W.Network("random", 97, layers, blocks, (layers[0].c_in, layers[0].h_in, layers[0].w_in),
                     slot)


@pytest.mark.parametrize("seed", range(24))
def test_random_networks_plan_invariants(seed):
    rng = np.random.default_rng(1000 + seed)
    net = random_cnn(rng)
    wts = W.make_weights(net)
    image = None
    with S.build_engine(net, wts, budget=1 << 30, host_only=True) as eng:
        image = eng.stats()["image_bytes"]
        assert eng.stats()["resident"] == 1
    for frac in (1.2, 0.8, 0.5, 0.3, 0.15, 0.05):
        budget = max(int(image * frac), 512)
        for partition in (0, 1, 2):
            max_slab = int(rng.choice([0, 0, budget // 3]))
            try:
                eng = S.build_engine(net, wts, budget=budget, host_only=True, partition=partition,
                                     max_slab=max_slab)
            except S.SwapNetError as e:
                assert e.code == S.SN_E_INFEASIBLE, (seed, frac, partition, e)
                continue
            with eng:
                check_plan(net, eng, budget)
                st = eng.stats()
                # everything fits: one upload, nothing swapped per inference
                if budget // 256 * 256 >= image and not max_slab:
                    assert st["resident"] == 1 and st["streamed_bytes"] == 0
                if budget < image:
                    # every slab streamed; a plan that cuts layers into
                    # channel slices pads each slice's tensors to 256 bytes
                    assert st["resident"] == 0 and st["streamed_bytes"] == st["image_bytes"]
                    assert image <= st["image_bytes"] <= image + 512 * len(eng.pieces())
                if max_slab and not st["resident"]:
                    assert max(s["bytes"] for s in eng.slabs()) <= max(max_slab, 256)
