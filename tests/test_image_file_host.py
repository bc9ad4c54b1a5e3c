"""Storage tier on the host (no GPU): the image file written by
sn_save_image, read back and parsed here independently of the library.

The file holds the plan's image in device layout (Sec. 4.2.1: blocks kept
in external storage, fetched with direct I/O), so every slab must sit at a
4 KiB-aligned offset with its exact bytes and the checksum recorded for it
(FNV-1a 64, computed here from its published definition), and nothing else
may differ from the in-memory image.  Attaching a file needs a device;
error paths are checked here."""
import os
import struct

import numpy as np
import pytest

from paper_2401_16757_amd import swapnet as S
from paper_2401_16757_amd import workloads as W


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(S.LIB_PATH):
        from paper_2401_16757_amd import build
        build.build()
    S.load_library()


def fnv1a64(data):
    """FNV-1a, 64-bit: offset basis 0xcbf29ce484222325, prime 0x100000001b3."""
    h = 0xcbf29ce484222325
    for b in bytes(data):
        h ^= b
        h = (h * 0x100000001b3) & 0xFFFFFFFFFFFFFFFF
    return h


def parse(path):
    raw = open(path, "rb").read()
    magic, ver, n, img, hb = struct.unpack_from("<8sIIQQ", raw, 0)
    slabs = [struct.unpack_from("<QQQQ", raw, 32 + 32 * i) for i in range(n)]
    return raw, magic, ver, n, img, hb, slabs


@pytest.mark.parametrize("name,kw,frac", [("tiny_cnn", {}, None), ("resnet50", {"res": 64}, 1 / 4)])
def test_saved_image_layout_and_checksums(tmp_path, name, kw, frac):
    net = W.get_network(name, **kw)
    wts = W.make_weights(net)
    budget = None if frac is None else int(net.weight_bytes() * frac)
    with S.build_engine(net, wts, budget=budget, host_only=True) as eng:
        img = eng.image()
        sl = eng.slabs()
        st = eng.stats()
        path = str(tmp_path / "image.bin")
        eng.save_image(path)
        assert st["file_backed"] == 0 and st["host_weight_bytes"] == st["image_bytes"]
        with pytest.raises(S.SwapNetError) as e:
            eng.attach_image_file(path)
        assert e.value.code == S.SN_E_UNSUPPORTED
    raw, magic, ver, n, img_bytes, hb, slabs = parse(path)
    assert magic == b"SNIMAGE1" and ver == 1 and n == len(sl) and img_bytes == img.size
    assert hb % 4096 == 0 and hb >= 32 + 32 * n
    prev_end = hb
    for i, (image_off, nbytes, file_off, csum) in enumerate(slabs):
        assert image_off == sl[i]["image_off"] and nbytes == sl[i]["bytes"]
        assert file_off % 4096 == 0 and file_off >= prev_end
        data = raw[file_off:file_off + nbytes]
        assert data == img[image_off:image_off + nbytes].tobytes(), i
        assert csum == fnv1a64(data), i
        pad_end = file_off + (nbytes + 4095) // 4096 * 4096
        assert set(raw[file_off + nbytes:pad_end]) <= {0}
        prev_end = pad_end
    assert len(raw) == prev_end


def test_fnv1a64_reference_values():
    # published test vectors of FNV-1a 64
    assert fnv1a64(b"") == 0xcbf29ce484222325
    assert fnv1a64(b"a") == 0xaf63dc4c8601ec8c
    assert fnv1a64(b"foobar") == 0x85944171f73967e8


def test_save_image_errors(tmp_path):
    net = W.get_network("tiny_cnn")
    wts = W.make_weights(net)
    eng = S.SwapNet(1 << 20, host_only=True)
    with pytest.raises(S.SwapNetError) as e:
        eng.save_image(str(tmp_path / "x.bin"))
    assert e.value.code == S.SN_E_STATE
    eng.close()
    with S.build_engine(net, wts, host_only=True) as eng:
        with pytest.raises(S.SwapNetError) as e:
            eng.save_image(str(tmp_path / "no_such_dir" / "x.bin"))
        assert e.value.code == S.SN_E_INVALID
