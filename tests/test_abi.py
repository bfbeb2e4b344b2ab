"""Host-side checks of the C ABI: the library loads, exports every declared entry point, and
rejects bad arguments before touching the device (these calls never reach a kernel)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2011_13824_amd import lirpa
from paper_2011_13824_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lirpa.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lirpa.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return lirpa.load()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lirpa_[a-z_0-9]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(names) == set(lirpa.SYMBOLS)
    for n in names:
        assert hasattr(L, n), n


def _fake_layers(arch):
    # distinct non-null fake device addresses: creation only records them
    out = []
    for i, t in enumerate(arch):
        out.append(lirpa.lirpa_layer(t["kind"], t["in_c"], t["in_h"], t["in_w"], t["out_c"],
                                     t["out_h"], t["out_w"], t["k"], t["stride"], t["pad"],
                                     0x1000 * (2 * i + 1), 0x1000 * (2 * i + 2)))
    return out


def _create(L, layers):
    arr = (lirpa.lirpa_layer * len(layers))(*layers)
    h = ctypes.c_void_p()
    rc = L.lirpa_net_create(arr, len(layers), ctypes.byref(h))
    return rc, h


@pytest.mark.parametrize("arch,n_relu", [("tiny", 64), ("base", 3172), ("wide", 6244),
                                         ("deep", 6756)])
def test_create_and_num_relu(L, arch, n_relu):
    rc, h = _create(L, _fake_layers(wl.ARCHS[arch]))
    assert rc == 0
    assert L.lirpa_net_num_relu(h) == n_relu
    assert L.lirpa_workspace_bytes(h, 9, 4, 0) > 0
    assert L.lirpa_workspace_bytes(h, 9, 8, 0) > L.lirpa_workspace_bytes(h, 9, 4, 0)
    assert L.lirpa_workspace_bytes(h, 0, 4, 0) == 0
    L.lirpa_net_destroy(h)


def test_create_rejects_bad_chains(L):
    good = _fake_layers(wl.ARCHS["base"])
    bad = list(good)
    bad[2] = lirpa.lirpa_layer(0, 1000, 1, 1, 100, 1, 1, 0, 1, 0, 0x9000, 0xA000)
    rc, h = _create(L, bad)
    assert rc == lirpa.LIRPA_EINVAL and not h.value
    assert "input size" in lirpa.lirpa_last_error()
    bad = list(good)
    bad[0] = lirpa.lirpa_layer(1, 3, 32, 32, 8, 15, 16, 4, 2, 1, 0x9000, 0xA000)
    rc, _ = _create(L, bad)
    assert rc == lirpa.LIRPA_EINVAL and "output size" in lirpa.lirpa_last_error()
    bad = list(good)
    bad[1] = lirpa.lirpa_layer(1, 8, 16, 16, 16, 8, 8, 4, 2, 1, 0, 0xA000)
    rc, _ = _create(L, bad)
    assert rc == lirpa.LIRPA_EINVAL and "null" in lirpa.lirpa_last_error()
    rc, _ = _create(L, [])
    assert rc == lirpa.LIRPA_EINVAL
    big = lirpa.lirpa_layer(1, 3, 32, 32, 8, 12, 12, 9, 2, 0, 0x9000, 0xA000)
    rc, _ = _create(L, [big])
    assert rc == lirpa.LIRPA_EUNSUPPORTED


def test_bound_validates_before_launching(L):
    rc, h = _create(L, _fake_layers(wl.ARCHS["tiny"]))
    assert rc == 0
    P = 0x10000
    need = L.lirpa_workspace_bytes(h, 1, 1, 0)

    def call(**kw):
        a = dict(x0=P, eps=0.1, C=P, S=1, B=4, split=P, alpha=None, lb=P, l=None, u=None,
                 ws=P, ws_bytes=need * 4)
        a.update(kw)
        return L.lirpa_bound(h, a["x0"], a["eps"], a["C"], a["S"], a["B"], a["split"],
                             a["alpha"], a["lb"], a["l"], a["u"], None, a["ws"], a["ws_bytes"],
                             None)

    assert call(S=0) == lirpa.LIRPA_EINVAL
    assert call(B=0) == lirpa.LIRPA_EINVAL
    assert call(eps=-1.0) == lirpa.LIRPA_EINVAL
    assert call(eps=float("inf")) == lirpa.LIRPA_EINVAL
    assert call(eps=float("nan")) == lirpa.LIRPA_EINVAL
    assert call(x0=None) == lirpa.LIRPA_EINVAL
    assert call(C=None) == lirpa.LIRPA_EINVAL
    assert call(lb=None) == lirpa.LIRPA_EINVAL
    assert call(ws=None) == lirpa.LIRPA_EINVAL
    assert call(l=P) == lirpa.LIRPA_EINVAL          # l without u
    assert call(ws_bytes=need - 1) == lirpa.LIRPA_ENOMEM
    assert "workspace" in lirpa.lirpa_last_error()
    assert L.lirpa_bound(None, P, 0.1, P, 1, 1, None, None, P, None, None, None, P, need,
                         None) == lirpa.LIRPA_EINVAL
    L.lirpa_net_destroy(h)


def test_workspace_chunking_is_monotone(L):
    rc, h = _create(L, _fake_layers(wl.ARCHS["wide"]))
    sizes = [L.lirpa_workspace_bytes(h, 9, b, 0) for b in (1, 2, 3, 64, 1024)]
    assert all(x < y for x, y in zip(sizes, sizes[1:]))
    L.lirpa_net_destroy(h)


@pytest.mark.parametrize("arch,B", [("base", 400), ("wide", 1024), ("deep", 1024),
                                    ("wide", 2048)])
def test_full_batches_fit_one_chunk(L, arch, B):
    # bound mode reserves no bound-matrix slab for the passes that run on chip (receptive-field
    # and fused pass kernels), so every full batch of the benchmark runs as one chunk
    rc, h = _create(L, _fake_layers(wl.ARCHS[arch]))
    need = L.lirpa_workspace_bytes(h, 9, B, 0)
    assert 0 < need < 8 << 30, need
    L.lirpa_net_destroy(h)


def test_workspace_sentinel_for_unaddressable_chunks(L):
    # gradient mode of the deep net at B = 1024 needs a tape slab over 2^31 floats: the
    # documented SIZE_MAX, while smaller chunks have a real size
    rc, h = _create(L, _fake_layers(wl.ARCHS["deep"]))
    assert L.lirpa_workspace_bytes(h, 9, 1024, 1) == 2**64 - 1
    assert 0 < L.lirpa_workspace_bytes(h, 9, 64, 1) < 2**40
    L.lirpa_net_destroy(h)
