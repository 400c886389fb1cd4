"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol declared in include/gdn_tree.h, computes the metadata size, and
rejects bad arguments on the host before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2607_06763_amd import gdn_tree as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gdn_tree.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(G.LIB_PATH):
        from paper_2607_06763_amd import build
        build.build()
    return G.lib()


def _declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\w[\w\s\*]*?\b(gdn_\w+)\s*\(", txt, re.M)))


def test_header_declarations_are_exported(L):
    names = _declared()
    assert set(names) == set(G.EXPORTS), names
    for n in names:
        assert hasattr(L, n), n


def test_exported_symbols_match_nm(L):
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", G.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    gdn = {n for n in exported if n.startswith("gdn_")}
    assert gdn == set(G.EXPORTS)


def test_meta_bytes_layout(L):
    assert G.meta_bytes(0, 5) == 0 and G.meta_bytes(3, 0) == 0
    for B, T in [(1, 1), (1, 7), (8, 64), (32, 128), (3, 65), (5, 33)]:
        off = G.meta_layout(B, T)
        end = off["ppos"] + 4 * B * T
        assert G.meta_bytes(B, T) == (end + 255) // 256 * 256
        for k in ("depth", "order", "pos", "parent", "status", "nvalid", "pdep", "ppos"):
            assert off[k] % 16 == 0
        assert off["depth"] >= 8 * B * T * off["W"]


def test_version(L):
    assert b"gfx950" in L.gdn_version()


def _call_verify(L, d, ptr=1):
    p = ctypes.c_void_p(ptr) if ptr else None
    return L.gdn_tree_verify(ctypes.byref(d), p, p, p, p, p, p, p, p, p, p, None)


def test_host_validation_errors(L):
    ok = G.make_dims(1, 7, 2, 2, 16, 16, "f32")
    cases = [
        (G.make_dims(1, 7, 2, 3, 16, 16), G.GDN_EINVAL),         # Hv % Hk
        (G.make_dims(1, 7, 0, 2, 16, 16), G.GDN_EINVAL),         # Hk < 1
        (G.make_dims(-1, 7, 2, 2, 16, 16), G.GDN_EINVAL),        # B < 0
        (G.make_dims(1, 7, 2, 2, 24, 16), G.GDN_EUNSUPPORTED),   # dk
        (G.make_dims(1, 7, 2, 2, 16, 256), G.GDN_EUNSUPPORTED),  # dv
        (G.make_dims(1, 513, 2, 2, 16, 16), G.GDN_EUNSUPPORTED),  # T > 512
        (G.Dims(1, 7, 2, 2, 16, 16, 5, 0.0), G.GDN_EINVAL),      # dtype
        (G.Dims(1, 7, 2, 2, 16, 16, 0, -1.0), G.GDN_EINVAL),     # scale
    ]
    for d, want in cases:
        assert _call_verify(L, d) == want, d
        assert G.last_error()
    # NULL tensor pointers are rejected before any device work
    assert _call_verify(L, ok, ptr=0) == G.GDN_EINVAL
    assert "NULL" in G.last_error()
    assert L.gdn_tree_commit(ctypes.byref(ok), *([None] * 12)) == G.GDN_EINVAL
    assert L.gdn_tree_prepare(None, None, None, None, None) == G.GDN_EINVAL
    assert L.gdn_tree_prepare(ctypes.byref(G.make_dims(1, 7, 1, 1, 16, 16)), None, None, None,
                              None) == G.GDN_EINVAL
    # empty problems are no-ops that succeed without touching pointers
    empty = G.make_dims(0, 7, 2, 2, 16, 16)
    assert _call_verify(L, empty, ptr=0) == G.GDN_OK
    assert L.gdn_tree_prepare(ctypes.byref(empty), None, None, None, None) == G.GDN_OK


def _call_step(L, d, ptrs):
    return L.gdn_tree_step(ctypes.byref(d), *[ctypes.c_void_p(x) if x else None for x in ptrs],
                           None)


def test_step_host_validation(L):
    d = G.make_dims(2, 7, 2, 2, 16, 16, "f32")
    good = [0x1000 * (i + 1) for i in range(19)]   # never dereferenced on these paths
    for i in range(19):
        if i == 7:          # commit_status may be NULL
            continue
        ptrs = list(good)
        ptrs[i] = 0
        assert _call_step(L, d, ptrs) == G.GDN_EINVAL, i
        assert "NULL" in G.last_error()
    # conv_state (index 15) and conv_state_out (16) must not overlap
    cs_bytes = 2 * 3 * d.C * 4
    ptrs = list(good)
    ptrs[15], ptrs[16] = 0x100000, 0x100000 + cs_bytes - 16
    assert _call_step(L, d, ptrs) == G.GDN_EINVAL
    assert "overlap" in G.last_error()
    # shape errors come first; empty problems succeed without touching pointers
    assert _call_step(L, G.make_dims(1, 7, 2, 3, 16, 16), good) == G.GDN_EINVAL
    assert _call_step(L, G.make_dims(1, 513, 2, 2, 16, 16), good) == G.GDN_EUNSUPPORTED
    assert _call_step(L, G.make_dims(0, 7, 2, 2, 16, 16), [0] * 19) == G.GDN_OK


def test_chunked_host_validation(L):
    p = [ctypes.c_void_p(0x1000)] * 10   # never dereferenced: refused on the host
    # trees above GDN_MAX_T and unsupported head dims are refused before any device work
    assert L.gdn_tree_verify_chunked(ctypes.byref(G.make_dims(1, 513, 2, 2, 32, 32)), *p,
                                     None) == G.GDN_EUNSUPPORTED
    assert L.gdn_tree_verify_chunked(ctypes.byref(G.make_dims(1, 7, 2, 2, 48, 32)), *p,
                                     None) == G.GDN_EUNSUPPORTED
    d2 = G.make_dims(1, 7, 2, 2, 16, 16, "f32")
    assert L.gdn_tree_verify_chunked(ctypes.byref(d2), *([None] * 10), None) == G.GDN_EINVAL
    assert L.gdn_tree_verify_chunked(ctypes.byref(G.make_dims(0, 7, 2, 2, 32, 32)), *([None] * 10),
                                     None) == G.GDN_OK


def test_binding_rejects_host_tensors(L):
    import torch
    d = G.make_dims(1, 7, 2, 2, 16, 16, "f32")
    with pytest.raises(ValueError):
        G.prepare(d, torch.zeros(1, 7, dtype=torch.int32), torch.zeros(G.meta_bytes(1, 7),
                                                                       dtype=torch.uint8))
