"""GPU parity for trees of 129..512 slots (feature workspace + gathered
pull-back verify, commit over paths of up to 512 nodes, and the step as
commit then verify), through the C ABI against the CPU oracle.

Bars as for smaller trees: metadata, statuses and the conv state
bit-exact; outputs within 2e-3 max|o_ref| on every node; committed state
within 1e-4 relative Frobenius per (sequence, value head).  Every output,
state and conv-state buffer sits between guard bands that must survive.
"""
import numpy as np
import pytest

from paper_2607_06763_amd import workloads as W
from tests.guard import check_guards, guarded

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


def _verify_commit(G, orc, w, tag):
    import torch
    dt = G.DeviceTree(w)
    dt.prepare()
    ref_meta = orc.prepare(w.parent)
    got_meta = dt.meta_arrays()
    for key in ("depth", "order", "anc", "nvalid", "status"):
        np.testing.assert_array_equal(got_meta[key], ref_meta[key], err_msg=key)
    out, out_full = guarded(tuple(dt.out.shape))
    S0_before = dt.S0.clone()
    dt.verify(out=out)
    torch.cuda.synchronize()
    check_guards(out_full, "out")
    assert torch.equal(dt.S0.view(torch.int32), S0_before.view(torch.int32))
    got = out.cpu().numpy().astype(np.float64)
    ref = orc.verify(w)
    err = _out_err(got, ref)
    _announce(f"  {tag} verify err {err:.3e}")
    assert err <= O_TOL
    assert (got[w.parent == W.PAD] == 0).all()
    S, S_full = guarded(tuple(dt.S0.shape), fill=dt.S0)
    cs, cs_full = guarded(tuple(dt.conv_state.shape), fill=dt.conv_state)
    dt.commit(S, cs)
    torch.cuda.synchronize()
    check_guards(S_full, "S")
    check_guards(cs_full, "conv_state")
    S_ref, cs_ref, st_ref = orc.commit(w)
    np.testing.assert_array_equal(dt.commit_status.cpu().numpy(), st_ref)
    serr = _state_err(S.cpu().numpy(), S_ref)
    _announce(f"  {tag} state err {serr:.3e}")
    assert serr <= S_TOL
    np.testing.assert_array_equal(cs.cpu().numpy(), cs_ref.astype(np.float32))


LARGE_SHAPES = [
    # (B, T, Hk, Hv, dk, dv, dtype, n_valid per seq or None, max_depth)
    (2, 129, 1, 2, 64, 64, "bf16", [129, 77], None),
    (2, 256, 2, 4, 128, 128, "bf16", [256, 200], None),
    (1, 256, 1, 3, 32, 16, "f32", None, 40),
    (2, 512, 1, 2, 128, 128, "bf16", [512, 301], None),
    (3, 384, 3, 3, 16, 64, "bf16", [384, 0, 5], 12),    # includes an empty tree
]


@pytest.mark.parametrize("idx", range(len(LARGE_SHAPES)))
def test_large_random_verify_commit(G, orc, idx):
    B, T, Hk, Hv, dk, dv, dt_, nv, md = LARGE_SHAPES[idx]
    w = W.make_random(7000 + idx, B, T, Hk, Hv, dk, dv, dt_, n_valid=nv, shuffle=True,
                      max_depth=md)
    _announce(f"large-T random shape {LARGE_SHAPES[idx]}")
    _verify_commit(G, orc, w, f"shape {idx}")


def _deep_tree(rng, T):
    """Random tree of depth about T / 2 (each node hangs 1..3 slots back),
    relabelled by a random permutation."""
    par = np.full(T, -1, np.int32)
    for i in range(1, T):
        par[i] = max(0, i - 1 - int(rng.integers(0, 3)))
    perm = rng.permutation(T)
    out = np.full(T, -1, np.int32)
    for i in range(T):
        out[perm[i]] = -1 if par[i] < 0 else perm[par[i]]
    return out


def test_deep_random_512(G, orc):
    rng = np.random.default_rng(7150)
    par = np.stack([_deep_tree(rng, 512), _deep_tree(rng, 512)])
    w = W.make_random(7150, 2, 512, 2, 2, 64, 32, "f32", parent=par)
    _announce("deep random trees T=512 (depth ~256), fp32 inputs")
    _verify_commit(G, orc, w, "deep512")


def test_shallow_wide_trees(G, orc):
    """Every node within two levels of the root (a star of 300 nodes and a
    root with 15 children of 20 children each): the conv taps above the
    root are taken from the conv state in every position block."""
    star = np.full(300, 0, np.int32)
    star[0] = -1
    two = np.full(300, -1, np.int32)
    two[1:16] = 0
    two[16:] = 1 + (np.arange(16, 300) - 16) % 15
    w = W.make_random(7170, 2, 300, 2, 4, 64, 32, "bf16", parent=np.stack([star, two]))
    assert np.any(w.conv_state != 0)
    _announce("shallow wide trees T=300 (depth 1 and 2)")
    _verify_commit(G, orc, w, "wide300")


def test_chain_512(G, orc):
    """A single 512-node path (depth 511): the longest walks and a commit of
    the whole chain (16 feature chunks)."""
    w = W.make_random(7100, 1, 512, 1, 2, 64, 64, "bf16", parent=W.chain_tree(512)[None])
    w.accepted[:] = 511
    _announce("chain of 512 nodes, commit of the whole path")
    _verify_commit(G, orc, w, "chain512")


@pytest.mark.parametrize("T", [256, 512])
def test_large_recipe(G, orc, T):
    """The large workload's recipe (16 key / 48 value heads, d = 128, bf16,
    depth <= 16, at most 8 children) at T = 256 and 512, 4 sequences."""
    w = W.make_sweep(T, B=4)
    _announce(f"large recipe T={T} B=4")
    _verify_commit(G, orc, w, f"recipe T={T}")


def _pair(seed, B, T, Hk, Hv, dk, dv, dt, prev_parent=None, **kw):
    wp = W.make_random(seed, B, T, Hk, Hv, dk, dv, dt, parent=prev_parent, **kw)
    wc = W.make_random(seed + 500, B, T, Hk, Hv, dk, dv, dt, **kw)
    wc.conv_w = wp.conv_w
    return wp, wc


def _step_check(G, orc, wp, wc):
    import torch
    dp, dc = G.DeviceTree(wp), G.DeviceTree(wc)
    dp.prepare()
    dc.prepare()
    S, S_full = guarded(tuple(dp.S0.shape), fill=dp.S0)
    cs_in = dp.conv_state.clone()
    cs_out, cs_full = guarded(tuple(cs_in.shape), fill=torch.full_like(cs_in, float("nan")))
    out, out_full = guarded(tuple(dc.out.shape))
    dc.step_from(dp, S, cs_in, cs_out, out=out)
    torch.cuda.synchronize()
    for f, n in ((S_full, "S"), (cs_full, "conv_state_out"), (out_full, "out")):
        check_guards(f, n)
    assert torch.equal(cs_in.view(torch.int32), dp.conv_state.view(torch.int32))
    S_ref, cs_ref, st = orc.commit(wp)
    wc.S0 = S_ref
    wc.conv_state = cs_ref
    out_ref = orc.verify(wc)
    np.testing.assert_array_equal(dp.commit_status.cpu().numpy(), st)
    np.testing.assert_array_equal(cs_out.cpu().numpy(), cs_ref.astype(np.float32))
    serr = _state_err(S.cpu().numpy(), S_ref)
    oerr = _out_err(out.cpu().numpy().astype(np.float64), out_ref)
    _announce(f"  step state err {serr:.3e}  out err {oerr:.3e}")
    assert serr <= S_TOL
    assert oerr <= O_TOL


@pytest.mark.parametrize("shape", [
    (2, 256, 2, 4, 128, 128, "bf16", [256, 180], None),
    (3, 512, 1, 3, 64, 32, "bf16", [512, 0, 400], None),  # includes an empty tree
    (2, 200, 2, 4, 16, 32, "f32", [200, 150], 6),        # one state element per thread
    (3, 160, 1, 1, 32, 16, "bf16", [160, 1, 129], None),  # 32 lanes per state row, one-node tree
    (2, 300, 1, 2, 16, 16, "bf16", [300, 257], None),    # tiny heads: commit kernels first
])
def test_large_step(G, orc, shape):
    B, T, Hk, Hv, dk, dv, dt_, nv, md = shape
    wp, wc = _pair(7200 + T, B, T, Hk, Hv, dk, dv, dt_, n_valid=nv, max_depth=md, shuffle=True)
    _announce(f"large-T step {shape}")
    _step_check(G, orc, wp, wc)


def test_large_step_path_lengths(G, orc):
    """Commits of 1, 2, 129, 256, 300 and 512 path nodes on 512-node chains
    (path extraction over 8 ancestor words), then the verify of a random
    tree against the committed state."""
    depths = [0, 1, 128, 255, 299, 511]
    chain = np.stack([W.chain_tree(512)] * len(depths))
    wp, wc = _pair(7300, len(depths), 512, 1, 2, 32, 32, "bf16", prev_parent=chain)
    wp.accepted[:] = depths
    _announce(f"large-T step path lengths {[d + 1 for d in depths]}")
    _step_check(G, orc, wp, wc)


def test_two_streams_share_nothing(G, orc):
    """Trees above 128 slots on two streams at once, different sizes: each
    stream gets its own cached workspace, so the results equal the oracle's
    (and are the same as when run one after the other)."""
    import torch
    wa = W.make_random(7400, 2, 300, 1, 2, 64, 64, "bf16", shuffle=True)
    wb = W.make_random(7401, 3, 180, 2, 4, 32, 32, "bf16", shuffle=True)
    da, db = G.DeviceTree(wa), G.DeviceTree(wb)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    for s, d in ((sa, da), (sb, db)):
        s.wait_stream(torch.cuda.current_stream())
    for _ in range(3):   # interleaved launches on the two streams
        with torch.cuda.stream(sa):
            da.prepare(stream=sa)
            da.verify(stream=sa)
        with torch.cuda.stream(sb):
            db.prepare(stream=sb)
            db.verify(stream=sb)
    torch.cuda.synchronize()
    for w, d in ((wa, da), (wb, db)):
        ref = orc.verify(w)
        got = d.out.cpu().numpy().astype(np.float64)
        assert np.max(np.abs(got - ref)) <= O_TOL * np.max(np.abs(ref))


@pytest.mark.parametrize("vscale", [1e5, 1e-6])
def test_value_range_through_fp16_workspace(G, orc, vscale):
    """The workspace above 128 slots holds v~ in fp16 with a power-of-two
    scale per (position, head): raw values (and their conv-state slots)
    scaled by 1e5 put v~ far above the fp16 range, by 1e-6 below its
    normal range.  With S0 = 0 the outputs are the value terms alone, so
    the 2e-3 max|o_ref| bar measures them."""
    import torch
    w = W.make_random(9300, 2, 256, 1, 2, 128, 128, "bf16", n_valid=[256, 200], shuffle=True)
    v = W.bf16_bits_to_f32(w.v).astype(np.float64) * vscale
    w.v = W.f32_to_bf16_bits(v.astype(np.float32))
    cs = w.conv_state.copy()
    cs[:, :, 2 * w.Hk * w.dk:] *= vscale
    w.conv_state = cs
    w.S0 = np.zeros_like(w.S0)
    _announce(f"value range x{vscale:g} through the fp16 workspace (T=256)")
    dt = G.DeviceTree(w)
    dt.prepare()
    dt.verify()
    torch.cuda.synchronize()
    got = dt.out.cpu().numpy().astype(np.float64)
    ref = orc.verify(w)
    assert np.isfinite(got).all()
    # the post-conv values really leave fp16's normal range (65504 / 2^-14)
    vt = orc.features(w)[..., 2 * w.Hk * w.dk:][w.parent != W.PAD]
    assert np.max(np.abs(vt)) > 65504.0 if vscale > 1 else np.max(np.abs(vt)) < 2.0 ** -14
    err = _out_err(got, ref)
    _announce(f"  err {err:.3e}  max|o_ref| {np.max(np.abs(ref)):.3e}")
    assert err <= O_TOL
