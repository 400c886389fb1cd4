"""GPU parity of the chunked-form verification (gdn_tree_verify_chunked,
Sec. 3.4.1-3.4.2 Eq. 9-13: sub-blocks of 32 positions, diagonal blocks
inverted by repeated squaring) against the CPU oracle, for trees of 1..512
slots.

Bars: max|o - o_ref| <= 2e-3 max|o_ref|; invalid trees and padding slots give
zero rows; S0 and the conv state stay bit-identical."""
import numpy as np
import pytest

from paper_2607_06763_amd import workloads as W

pytestmark = pytest.mark.gpu

O_TOL = 2e-3


@pytest.fixture(scope="module")
def G():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_06763_amd import gdn_tree as G
    G.lib()
    return G


def _announce(msg):
    print(f"[gpu] {msg}", flush=True)


def _out_err(got, ref):
    return np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30)


def _run(G, w, chunked=True):
    import torch
    dt = G.DeviceTree(w)
    dt.prepare()
    dt.verify(chunked=chunked)
    torch.cuda.synchronize()
    return dt, dt.out.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("cfg", [0, 1, 2, 3])
def test_chunked_named_full(G, orc, cfg):
    w = W.make_config(cfg)
    _announce(f"chunked cfg={cfg} B={w.B} T={w.T}")
    _dt, got = _run(G, w)
    err = _out_err(got, orc.verify(w))
    _announce(f"  err {err:.3e}")
    assert err <= O_TOL


def test_chunked_large_full(G, orc):
    w = W.make_config(4)
    _announce("chunked cfg=4 (all nodes)")
    _dt, got = _run(G, w)
    err = _out_err(got, orc.verify(w))
    _announce(f"  err {err:.3e}")
    assert err <= O_TOL


SHAPES = [
    # (B, T, Hk, Hv, dk, dv, dtype, n_valid or None, max_depth)
    (2, 1, 1, 1, 32, 32, "f32", None, None),           # one node
    (3, 9, 2, 6, 32, 64, "bf16", [9, 5, 1], None),     # ragged, padding
    (2, 33, 1, 3, 64, 128, "bf16", [33, 20], 4),
    (1, 64, 2, 4, 128, 32, "f32", None, None),
    (2, 100, 3, 3, 64, 64, "bf16", [100, 71], 12),
    (2, 128, 1, 2, 128, 128, "bf16", [128, 97], None),
    (4, 17, 4, 8, 64, 64, "bf16", [17, 0, 3, 16], 3),  # includes an empty tree
    (1, 128, 2, 2, 32, 128, "f32", None, None),
    (2, 40, 1, 2, 16, 16, "f32", [40, 33], None),        # 16 x 16 heads
    (2, 256, 2, 4, 128, 128, "bf16", [256, 200], None),
    (3, 384, 3, 3, 16, 64, "bf16", [384, 0, 5], 12),    # includes an empty tree
    (2, 512, 1, 2, 128, 128, "bf16", [512, 301], None),
    (1, 500, 2, 2, 64, 32, "f32", None, None),           # ragged last block
]


@pytest.mark.parametrize("idx", range(len(SHAPES)))
def test_chunked_random_shapes(G, orc, idx):
    B, T, Hk, Hv, dk, dv, dt_, nv, md = SHAPES[idx]
    w = W.make_random(8000 + idx, B, T, Hk, Hv, dk, dv, dt_, n_valid=nv, shuffle=True, max_depth=md)
    _announce(f"chunked random shape {SHAPES[idx]}")
    _dt, got = _run(G, w)
    err = _out_err(got, orc.verify(w))
    _announce(f"  err {err:.3e}")
    assert err <= O_TOL
    assert (got[w.parent == W.PAD] == 0).all()


@pytest.mark.parametrize("T", [128, 512])
def test_chunked_deep_chain(G, orc, T):
    """Chains (depth T - 1): the case the block solve is for; at T = 512 every
    earlier block holds ancestors of every later one."""
    w = W.make_random(8100 + T, 2, T, 1, 2, 128, 128, "bf16", parent=np.stack([W.chain_tree(T)] * 2))
    _announce(f"chunked chain T={T}")
    _dt, got = _run(G, w)
    err = _out_err(got, orc.verify(w))
    _announce(f"  err {err:.3e}")
    assert err <= O_TOL


def test_chunked_tiny_alpha(G, orc):
    """Decays of 1e-30 and exactly 0 on some nodes: the log-decay ratios stay
    finite (log alpha floored at the smallest normal float)."""
    w = W.make_random(8150, 2, 64, 1, 2, 32, 32, "f32", shuffle=True)
    a = w.alpha.copy()
    a[0, ::5, 0] = 1e-30
    a[1, ::7, 1] = 0.0
    w.alpha = a
    _announce("chunked tiny alpha")
    _dt, got = _run(G, w)
    assert np.isfinite(got).all()
    err = _out_err(got, orc.verify(w))
    _announce(f"  err {err:.3e}")
    assert err <= O_TOL


def test_chunked_invalid_trees_read_only_deterministic(G, orc):
    import torch
    T = 8
    par = np.array([
        [-1, 0, 0, 1, 1, 2, 2, 3],
        [-1, 0, 9, 1, 1, 2, 2, 3],
        [1, 0, -2, -2, -2, -2, -2, -2],
        [-2] * 8,
    ], np.int32)
    w = W.make_random(8200, 4, T, 2, 2, 32, 32, "bf16", parent=par)
    dt = G.DeviceTree(w)
    S0 = dt.S0.clone()
    cs = dt.conv_state.clone()
    dt.prepare()
    dt.verify(chunked=True)
    o1 = dt.out.clone()
    dt.verify(chunked=True)
    torch.cuda.synchronize()
    got = o1.cpu().numpy().astype(np.float64)
    assert _out_err(got, orc.verify(w)) <= O_TOL
    assert (got[1:] == 0).all()
    assert torch.equal(o1.view(torch.int32), dt.out.view(torch.int32))
    assert torch.equal(S0.view(torch.int32), dt.S0.view(torch.int32))
    assert torch.equal(cs.view(torch.int32), dt.conv_state.view(torch.int32))
