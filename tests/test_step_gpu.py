"""GPU parity of the fused decode step (gdn_tree_step): the commit of the
previous step's accepted node followed by the verification of the current
tree, in one launch.

Reference: the oracle's commit of the previous step, then the oracle's verify
of the current tree on the committed state and conv state (Sec. 3.4-3.4.2).
Bars as for the separate entry points: statuses and the conv state
bit-exact, outputs within 2e-3 max|o_ref|, the committed state within 1e-4
relative Frobenius per (sequence, value head), on every node.
"""
import numpy as np
import pytest

from paper_2607_06763_amd import workloads as W

pytestmark = pytest.mark.gpu

O_TOL = 2e-3
S_TOL = 1e-4


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
    scale = max(np.max(np.abs(ref)), 1e-30)
    return np.max(np.abs(got - ref)) / scale


def _state_err(S_got, S_ref):
    num = np.sqrt(np.sum((S_got.astype(np.float64) - S_ref) ** 2, axis=(2, 3)))
    den = np.sqrt(np.sum(S_ref ** 2, axis=(2, 3)))
    return np.max(num / np.maximum(den, 1e-30))


def _pair(seed, B, T, Hk, Hv, dk, dv, dt, prev_parent=None, cur_parent=None, **kw):
    """Two consecutive steps of one layer: same shapes and conv weights."""
    wp = W.make_random(seed, B, T, Hk, Hv, dk, dv, dt, parent=prev_parent, **kw)
    wc = W.make_random(seed + 500, B, T, Hk, Hv, dk, dv, dt, parent=cur_parent, **kw)
    wc.conv_w = wp.conv_w
    return wp, wc


def _run_step(G, wp, wc):
    """Fused step on the device; returns host copies and the device trees."""
    import torch
    dp, dc = G.DeviceTree(wp), G.DeviceTree(wc)
    dp.prepare()
    dc.prepare()
    S = dp.S0.clone()
    cs_in = dp.conv_state.clone()
    cs_out = torch.full_like(cs_in, float("nan"))
    dc.step_from(dp, S, cs_in, cs_out)
    torch.cuda.synchronize()
    assert torch.equal(cs_in.view(torch.int32), dp.conv_state.view(torch.int32))  # read-only
    return dict(S=S.cpu().numpy(), cs=cs_out.cpu().numpy(), out=dc.out.cpu().numpy(),
                status=dp.commit_status.cpu().numpy(), dp=dp, dc=dc)


def _reference(orc, wp, wc, node_mask=None):
    S_ref, cs_ref, st = orc.commit(wp)
    wc.S0 = S_ref
    wc.conv_state = cs_ref
    out_ref = orc.verify(wc, node_mask=node_mask)
    return S_ref, cs_ref, st, out_ref


def _check(got, ref, mask=None):
    S_ref, cs_ref, st, out_ref = ref
    np.testing.assert_array_equal(got["status"], st)
    np.testing.assert_array_equal(got["cs"], cs_ref.astype(np.float32))
    serr = _state_err(got["S"], S_ref)
    sel = np.ones(got["out"].shape[:2], bool) if mask is None else mask.astype(bool)
    oerr = _out_err(got["out"][sel].astype(np.float64), out_ref[sel])
    _announce(f"  state err {serr:.3e}  out err {oerr:.3e}")
    assert serr <= S_TOL
    assert oerr <= O_TOL
    assert np.isfinite(got["out"]).all()


def test_step_large(G, orc):
    """32 sequences, 16 key / 48 value heads, d = 128, 128-node trees: the
    previous step is the large named workload, the current one a fresh tree
    set of the same recipe; every node of every head is checked."""
    wp = W.make_config(4)
    rng = np.random.default_rng(77)
    par = np.stack([W.random_depth_capped_tree(rng, 128, 15, spine=16, max_children=8)
                    for _ in range(32)])
    wc = W.make_random(4077, 32, 128, 16, 48, 128, 128, "bf16", parent=par)
    wc.conv_w = wp.conv_w
    _announce("step large B=32 T=128 Hk=16 Hv=48 d=128 (all nodes)")
    got = _run_step(G, wp, wc)
    _check(got, _reference(orc, wp, wc))


STEP_SHAPES = [
    # (B, T, Hk, Hv, dk, dv, dtype, n_valid or None, max_depth)
    (2, 1, 1, 1, 16, 16, "f32", None, None),          # one node, 16 x 16 heads
    (3, 9, 2, 6, 32, 16, "bf16", [9, 5, 1], None),
    (2, 33, 1, 3, 64, 128, "bf16", [33, 20], 4),      # dv split into slices
    (1, 64, 2, 4, 128, 32, "f32", None, None),
    (2, 100, 3, 3, 16, 64, "bf16", [100, 71], 12),
    (2, 128, 1, 2, 128, 128, "bf16", [128, 97], None),
    (4, 17, 4, 8, 64, 64, "bf16", [17, 0, 3, 16], 3),  # includes an empty tree
    (128, 20, 2, 6, 32, 32, "bf16", [20, 0] + [20 - (i % 7) for i in range(126)], None),
]


@pytest.mark.parametrize("idx", range(len(STEP_SHAPES)))
def test_step_random_shapes(G, orc, idx):
    B, T, Hk, Hv, dk, dv, dt, nv, md = STEP_SHAPES[idx]
    wp, wc = _pair(6000 + 10 * idx, B, T, Hk, Hv, dk, dv, dt, n_valid=nv, max_depth=md,
                   shuffle=True)
    _announce(f"step random shape {STEP_SHAPES[idx]}")
    got = _run_step(G, wp, wc)
    _check(got, _reference(orc, wp, wc))
    assert (got["out"][wc.parent == W.PAD] == 0).all()


def test_step_path_lengths(G, orc):
    """Accepted paths of 1, 2, 3, 4 nodes (the committed conv slots mix old
    slots and path inputs) and of 32, 33, 64 and 128 nodes (one, two, two and
    four feature chunks), on 128-node chains."""
    depths = [0, 1, 2, 3, 31, 32, 63, 127]
    B = len(depths)
    chain = np.stack([W.chain_tree(128)] * B)
    wp, wc = _pair(6500, B, 128, 1, 2, 64, 64, "bf16", prev_parent=chain)
    wp.accepted[:] = depths
    _announce(f"step path lengths {[d + 1 for d in depths]}")
    got = _run_step(G, wp, wc)
    _check(got, _reference(orc, wp, wc))


@pytest.mark.parametrize("T,dk,dv", [(8, 32, 32), (200, 32, 32), (200, 16, 16)])
def test_step_errors(G, orc, T, dk, dv):
    """Nothing to commit (accepted -1, out of range, padding, invalid previous
    tree) keeps S and copies the conv state; an invalid current tree still
    commits and gets zero outputs.  T = 8: one fused launch; T = 200: the
    commit inside the pull-back (32 x 32 heads) or the commit kernels before
    the verification (16 x 16 heads)."""
    prev8 = np.array([
        [-1, 0, 0, 1, 1, 2, 2, 3],       # accepted -1
        [-1, 0, 0, 1, 1, 2, 2, 3],       # accepted out of range
        [-1, 0, -2, -2, -2, -2, -2, -2],  # accepted padding
        [-1, 0, 9, 1, 1, 2, 2, 3],       # invalid previous tree
        [-1, 0, 0, 1, 1, 2, 2, 3],       # ok, current tree invalid
        [-1, 0, 0, 1, 1, 2, 2, 3],       # ok, current tree empty
        [-1, 0, 0, 1, 1, 2, 2, 3],       # ok
    ], np.int32)
    prev = np.full((7, T), W.PAD, np.int32)
    prev[:, :8] = prev8
    cur = np.array([W.heap_tree(T)] * 7, np.int32)
    cur[4] = W.PAD
    cur[4, :4] = [-1, -1, 0, 1]
    cur[5] = W.PAD
    wp, wc = _pair(6700 + T + dk, 7, T, 2, 4, dk, dv, "bf16", prev_parent=prev, cur_parent=cur)
    wp.accepted[:] = [-1, T, 3, 3, 7, 5, 6]
    got = _run_step(G, wp, wc)
    ref = _reference(orc, wp, wc)
    assert ref[2].tolist() == [0, 5, 5, 3, 0, 0, 0]
    _check(got, ref)
    S0 = wp.S0
    for b in range(4):
        assert np.array_equal(got["S"][b].view(np.int32), S0[b].view(np.int32))
        assert np.array_equal(got["cs"][b].view(np.int32), wp.conv_state[b].view(np.int32))
    assert not np.array_equal(got["S"][4], S0[4])
    assert (got["out"][4:6] == 0).all()


def test_step_multi(G, orc):
    """Four decode steps chained through the fused entry point (the conv state
    ping-pongs between two buffers); every step's outputs and the state after
    every commit match the oracle chained through the same steps."""
    import torch
    conv_w = None
    S = cs_a = cs_b = None
    S_ref = cs_ref = None
    prev_w = prev_d = None
    for step in range(4):
        w = W.make_random(6900 + step, 3, 40, 2, 4, 64, 64, "bf16", shuffle=True)
        if conv_w is None:
            conv_w = w.conv_w
        w.conv_w = conv_w
        d = G.DeviceTree(w)
        d.prepare()
        if prev_d is None:
            S, cs_a = d.S0.clone(), d.conv_state.clone()
            cs_b = torch.empty_like(cs_a)
            S_ref = w.S0.astype(np.float64)
            cs_ref = w.conv_state.astype(np.float64)
            w.S0, w.conv_state = S_ref, cs_ref
            d.verify(S0=S, conv_state=cs_a)
        else:
            prev_w.S0, prev_w.conv_state = S_ref, cs_ref
            S_ref, cs_ref, st = orc.commit(prev_w)
            d.step_from(prev_d, S, cs_a, cs_b)
            cs_a, cs_b = cs_b, cs_a
            torch.cuda.synchronize()
            np.testing.assert_array_equal(prev_d.commit_status.cpu().numpy(), st)
            assert _state_err(S.cpu().numpy(), S_ref) <= S_TOL
            np.testing.assert_array_equal(cs_a.cpu().numpy(), cs_ref.astype(np.float32))
            # keep the oracle on the device's fp32 state so errors do not compound
            S_ref = S.cpu().numpy().astype(np.float64)
            cs_ref = cs_a.cpu().numpy().astype(np.float64)
            w.S0, w.conv_state = S_ref, cs_ref
        torch.cuda.synchronize()
        err = _out_err(d.out.cpu().numpy().astype(np.float64), orc.verify(w))
        _announce(f"  step {step}: out err {err:.3e}")
        assert err <= O_TOL
        prev_w, prev_d = w, d


def test_step_tiny_alpha(G, orc):
    """The fused step's commit with decays of 1e-30 and exactly 0 on the
    accepted paths (128-node chains)."""
    chain = np.stack([W.chain_tree(128)] * 2)
    wp, wc = _pair(6900, 2, 128, 1, 2, 64, 64, "f32", prev_parent=chain)
    a = wp.alpha.copy()
    a[0, ::3, :] = 1e-30
    a[1, ::4, 1] = 0.0
    wp.alpha = a
    wp.accepted[:] = [127, 90]
    _announce("step tiny alpha")
    got = _run_step(G, wp, wc)
    assert np.isfinite(got["S"]).all()
    _check(got, _reference(orc, wp, wc))
