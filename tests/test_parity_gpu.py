"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: tree metadata, statuses and the conv state are bit-exact; verify
outputs satisfy max|o - o_ref| <= 2e-3 * max|o_ref|; the committed fp32
state satisfies ||S - S_ref||_F <= 1e-4 ||S_ref||_F for every
(sequence, value head).  The large workload (32 x 128-node trees, 48 value
heads) is checked on every node.
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


def _check_meta(G, dt, w, orc):
    ref = orc.prepare(w.parent)
    got = dt.meta_arrays()
    for key in ("depth", "order", "anc", "nvalid", "status"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    ok = ref["status"] == 0
    if ok.any():
        pos = np.argsort(ref["order"], axis=1)
        np.testing.assert_array_equal(got["pos"][ok], pos[ok])
    # per-position copies: depth of the node at position p, parent's position
    B, T = w.parent.shape
    for b in range(B):
        if ref["status"][b] != 0:
            assert (got["pdep"][b] == -1).all() and (got["ppos"][b] == -1).all()
            continue
        pos = np.argsort(ref["order"][b])
        for p_ in range(T):
            node = ref["order"][b, p_]
            assert got["pdep"][b, p_] == ref["depth"][b, node]
            par = w.parent[b, node]
            assert got["ppos"][b, p_] == (pos[par] if par >= 0 else -1)
    np.testing.assert_array_equal(got["parent"], w.parent)
    np.testing.assert_array_equal(dt.tree_status.cpu().numpy(), ref["status"])


def _run_verify(G, w, dt=None):
    import torch
    dt = dt or G.DeviceTree(w)
    dt.prepare()
    dt.verify()
    torch.cuda.synchronize()
    return dt, dt.out.cpu().numpy().astype(np.float64)


def _out_err(got, ref):
    scale = max(np.max(np.abs(ref)), 1e-30)
    return np.max(np.abs(got - ref)) / scale


def _state_err(S_got, S_ref):
    B, H = S_ref.shape[:2]
    num = np.sqrt(np.sum((S_got.astype(np.float64) - S_ref) ** 2, axis=(2, 3)))
    den = np.sqrt(np.sum(S_ref ** 2, axis=(2, 3)))
    return np.max(num / np.maximum(den, 1e-30))


def _sample_mask(w, per_seq, seed):
    rng = np.random.default_rng(seed)
    mask = np.zeros((w.B, w.T), np.uint8)
    for b in range(w.B):
        real = np.nonzero(w.parent[b] != W.PAD)[0]
        depth = np.zeros(w.T, int)
        for i in range(w.T):  # parent[i] < i in the named workloads
            p = w.parent[b, i]
            depth[i] = 0 if p < 0 else depth[p] + 1
        pick = {int(w.accepted[b]), int(real[np.argmax(depth[real])]), int(real[0])}
        pick |= set(int(x) for x in rng.choice(real, size=min(per_seq, len(real)), replace=False))
        mask[b, sorted(pick)] = 1
    return mask


# ---------------------------------------------------------------------------
# named workloads
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_prepare_bit_exact(G, orc, cfg):
    w = W.make_config(cfg)
    _announce(f"prepare cfg={cfg} B={w.B} T={w.T}")
    dt = G.DeviceTree(w)
    dt.prepare()
    _check_meta(G, dt, w, orc)


@pytest.mark.parametrize("T", [1, 63, 64, 65, 128, 129, 192, 193, 256, 257, 320, 384, 448, 511, 512])
def test_prepare_word_count_boundaries(G, orc, T):
    """The prepare kernel is built for 1, 2, 4 and 8 ancestor words per node;
    trees of 129-192 slots use 3 of the 4-word build.  At every boundary: a
    relabelled random tree, a padded one, a chain (the longest pointer
    jumping) and a tree with a cycle, bit-exact against the oracle."""
    rng = np.random.default_rng(4200 + T)
    par = np.stack([W.random_tree(rng, T, None, True),
                    W.random_tree(rng, T, T // 2 + 1, True),
                    W.chain_tree(T),
                    W.random_tree(rng, T, None, True)])
    if T >= 4:  # close a cycle among three non-root nodes of the last tree
        nodes = [i for i in range(T) if par[3, i] != -1][:3]
        par[3, nodes[0]], par[3, nodes[1]], par[3, nodes[2]] = nodes[1], nodes[2], nodes[0]
    w = W.make_random(4300 + T, 4, T, 1, 1, 16, 16, "bf16", parent=par)
    _announce(f"prepare boundaries T={T}")
    dt = G.DeviceTree(w)
    dt.prepare()
    _check_meta(G, dt, w, orc)
    if T >= 4:
        assert orc.prepare(w.parent)["status"][3] != 0


@pytest.mark.parametrize("cfg", [0, 1, 2, 3])
def test_verify_named_full(G, orc, cfg):
    w = W.make_config(cfg)
    _announce(f"verify cfg={cfg} B={w.B} T={w.T} Hk={w.Hk} Hv={w.Hv} d={w.dk}")
    _dt, got = _run_verify(G, w)
    ref = orc.verify(w)
    err = _out_err(got, ref)
    _announce(f"  max|err|/max|ref| = {err:.3e}")
    assert err <= O_TOL


def test_verify_large_full(G, orc):
    """The large workload (32 trees x 128 nodes, 16 key / 48 value heads,
    d = 128): every node of every head against the oracle.  This is the
    grouped grid (all value heads of a key head in one workgroup)."""
    w = W.make_config(4)
    _announce(f"verify cfg=4 B={w.B} T={w.T} Hv={w.Hv} (all nodes)")
    _dt, got = _run_verify(G, w)
    ref = orc.verify(w)
    err = _out_err(got, ref)
    _announce(f"  max|err|/max|ref| = {err:.3e}")
    assert err <= O_TOL
    assert np.isfinite(got).all()


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_commit_named(G, orc, cfg):
    import torch
    w = W.make_config(cfg)
    _announce(f"commit cfg={cfg}")
    dt = G.DeviceTree(w)
    dt.prepare()
    S = dt.S0.clone()
    cs = dt.conv_state.clone()
    dt.commit(S, cs)
    torch.cuda.synchronize()
    S_ref, cs_ref, st_ref = orc.commit(w)
    np.testing.assert_array_equal(dt.commit_status.cpu().numpy(), st_ref)
    err = _state_err(S.cpu().numpy(), S_ref)
    _announce(f"  max per-head rel Frobenius = {err:.3e}")
    assert err <= S_TOL
    np.testing.assert_array_equal(cs.cpu().numpy(), cs_ref.astype(np.float32))


def test_verify_is_read_only_and_deterministic(G):
    import torch
    w = W.make_config(3)
    dt = G.DeviceTree(w)
    S0_before = dt.S0.clone()
    cs_before = dt.conv_state.clone()
    dt.prepare()
    dt.verify()
    o1 = dt.out.clone()
    dt.verify()
    torch.cuda.synchronize()
    assert torch.equal(dt.S0.view(torch.int32), S0_before.view(torch.int32))
    assert torch.equal(dt.conv_state.view(torch.int32), cs_before.view(torch.int32))
    assert torch.equal(o1.view(torch.int32), dt.out.view(torch.int32))


# ---------------------------------------------------------------------------
# random shapes, padding, relabelling
# ---------------------------------------------------------------------------
SHAPES = [
    # (B, T, Hk, Hv, dk, dv, dtype, n_valid per seq or None, max_depth)
    (2, 1, 1, 1, 16, 16, "f32", None, None),
    (3, 9, 2, 6, 32, 16, "bf16", [9, 5, 1], None),
    (2, 33, 1, 3, 64, 128, "bf16", [33, 20], 4),
    (1, 64, 2, 4, 128, 32, "f32", None, None),
    (2, 100, 3, 3, 16, 64, "bf16", [100, 71], 12),
    (2, 128, 1, 2, 128, 128, "bf16", [128, 97], None),
    (1, 128, 1, 1, 32, 32, "f32", None, None),   # deep random tree
    (4, 17, 4, 8, 64, 64, "bf16", [17, 0, 3, 16], 3),  # includes an empty tree
    # B * Hk >= 256: every value head of a key head in one workgroup
    (128, 20, 2, 6, 32, 32, "bf16", [20, 0] + [20 - (i % 7) for i in range(126)], None),
]


@pytest.mark.parametrize("idx", range(len(SHAPES)))
def test_random_shapes_verify_commit(G, orc, idx):
    import torch
    B, T, Hk, Hv, dk, dv, dt_, nv, md = SHAPES[idx]
    w = W.make_random(1000 + idx, B, T, Hk, Hv, dk, dv, dt_, n_valid=nv, shuffle=True,
                      max_depth=md)
    _announce(f"random shape {SHAPES[idx]}")
    dt = G.DeviceTree(w)
    dt.prepare()
    _check_meta(G, dt, w, orc)
    dt.verify()
    torch.cuda.synchronize()
    got = dt.out.cpu().numpy().astype(np.float64)
    ref = orc.verify(w)
    err = _out_err(got, ref)
    _announce(f"  verify err {err:.3e}")
    assert err <= O_TOL
    pad = w.parent == W.PAD
    assert (got[pad] == 0).all()
    S = dt.S0.clone()
    cs = dt.conv_state.clone()
    dt.commit(S, cs)
    torch.cuda.synchronize()
    S_ref, cs_ref, st_ref = orc.commit(w)
    np.testing.assert_array_equal(dt.commit_status.cpu().numpy(), st_ref)
    assert _state_err(S.cpu().numpy(), S_ref) <= S_TOL
    np.testing.assert_array_equal(cs.cpu().numpy(), cs_ref.astype(np.float32))


def test_chain_deep_and_custom_scale(G, orc):
    import torch
    w = W.make_random(2000, 1, 128, 2, 4, 64, 32, "bf16", parent=W.chain_tree(128)[None])
    dt = G.DeviceTree(w, scale=0.25)
    dt.prepare()
    dt.verify()
    torch.cuda.synchronize()
    err = _out_err(dt.out.cpu().numpy(), orc.verify(w, scale=0.25))
    assert err <= O_TOL


def test_invalid_trees(G, orc):
    import torch
    T = 8
    par = np.array([
        [-1, 0, 0, 1, 1, 2, 2, 3],      # ok
        [-1, 0, 9, 1, 1, 2, 2, 3],      # out of range
        [1, 0, -2, -2, -2, -2, -2, -2],  # no root
        [-1, -1, 0, 1, -2, -2, -2, -2],  # two roots
        [-1, 2, 1, 0, -2, -2, -2, -2],  # cycle
        [-1, 0, -2, 2, -2, -2, -2, -2],  # parent is padding
        [-2] * 8,                       # empty
    ], np.int32)
    w = W.make_random(3000, par.shape[0], T, 2, 2, 16, 32, "bf16", parent=par)
    w.accepted[:] = [3, 0, 0, 0, 0, 0, -1]
    dt = G.DeviceTree(w)
    dt.prepare()
    _check_meta(G, dt, w, orc)
    dt.verify()
    S = dt.S0.clone()
    cs = dt.conv_state.clone()
    dt.commit(S, cs)
    torch.cuda.synchronize()
    got = dt.out.cpu().numpy()
    ref = orc.verify(w)
    assert _out_err(got, ref) <= O_TOL
    assert (got[1:] == 0).all()
    S_ref, cs_ref, st_ref = orc.commit(w)
    np.testing.assert_array_equal(dt.commit_status.cpu().numpy(), st_ref)
    assert st_ref.tolist() == [0, 3, 1, 2, 4, 3, 0]
    assert torch.equal(S[1:], dt.S0[1:])
    assert _state_err(S.cpu().numpy(), S_ref) <= S_TOL
    np.testing.assert_array_equal(cs.cpu().numpy(), cs_ref.astype(np.float32))


def test_bad_accepted(G, orc):
    import torch
    par = np.stack([W.chain_tree(6)] * 4)
    par[3, 5] = W.PAD
    w = W.make_random(3100, 4, 6, 1, 2, 32, 16, "f32", parent=par)
    w.accepted[:] = [-1, 6, -5, 5]   # skip, out of range, out of range, padding
    dt = G.DeviceTree(w)
    dt.prepare()
    S = dt.S0.clone()
    cs = dt.conv_state.clone()
    dt.commit(S, cs)
    torch.cuda.synchronize()
    assert dt.commit_status.cpu().numpy().tolist() == [0, 5, 5, 5]
    assert torch.equal(S, dt.S0) and torch.equal(cs, dt.conv_state)


def test_multi_step_resume(G, orc):
    """Three decode steps of (prepare, verify, commit) with fresh trees each step:
    the device state and conv state after every commit match the oracle chained
    through the same steps, and so does every step's verify."""
    import torch
    S = cs = S_ref = cs_ref = conv_w = None
    for step in range(3):
        w = W.make_random(4000 + step, 3, 40, 2, 4, 64, 64, "bf16", shuffle=True)
        conv_w = w.conv_w.copy() if conv_w is None else conv_w
        w.conv_w = conv_w                      # one layer: same weights every step
        dt = G.DeviceTree(w)
        if S is None:
            S, cs = dt.S0.clone(), dt.conv_state.clone()
            S_ref, cs_ref = w.S0.astype(np.float64), w.conv_state.astype(np.float64)
        w.S0 = S_ref
        w.conv_state = cs_ref
        dt.prepare()
        dt.verify(S0=S, conv_state=cs)
        dt.commit(S, cs)
        torch.cuda.synchronize()
        ref_out = orc.verify(w)
        assert _out_err(dt.out.cpu().numpy(), ref_out) <= O_TOL
        S_ref, cs_ref, st = orc.commit(w)
        assert _state_err(S.cpu().numpy(), S_ref) <= S_TOL
        np.testing.assert_array_equal(cs.cpu().numpy(), cs_ref.astype(np.float32))
        # keep the oracle on the device's fp32 state so errors do not compound
        S_ref = S.cpu().numpy().astype(np.float64)
        cs_ref = cs.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("T", [64, 200])
def test_tiny_alpha_verify_commit(G, orc, T):
    """Decays of 1e-30, 1e-25 and exactly 0 along committed chains: the commit
    replay never divides by an underflowed decay product, and outputs and
    state stay finite and within the bars (T = 64: on-chip kernels, T = 200:
    the workspace path)."""
    import torch
    par = np.stack([W.chain_tree(T)] * 2)
    w = W.make_random(3500 + T, 2, T, 1, 2, 64, 64, "f32", parent=par)
    a = w.alpha.copy()
    a[0, ::3, :] = 1e-30
    a[0, 1::3, :] = 1e-25
    a[1, ::4, 0] = 0.0
    w.alpha = a
    w.accepted[:] = [T - 1, T // 2]
    _announce(f"tiny alpha T={T}")
    dt = G.DeviceTree(w)
    dt.prepare()
    dt.verify()
    S = dt.S0.clone()
    cs = dt.conv_state.clone()
    dt.commit(S, cs)
    torch.cuda.synchronize()
    got = dt.out.cpu().numpy().astype(np.float64)
    assert np.isfinite(got).all()
    err = _out_err(got, orc.verify(w))
    S_ref, cs_ref, st_ref = orc.commit(w)
    S_got = S.cpu().numpy()
    assert np.isfinite(S_got).all()
    serr = _state_err(S_got, S_ref)
    _announce(f"  verify err {err:.3e}  state err {serr:.3e}")
    assert err <= O_TOL
    assert serr <= S_TOL
    np.testing.assert_array_equal(cs.cpu().numpy(), cs_ref.astype(np.float32))


def _wide_state(w, seed):
    """S0 rows scaled by 2^e, e uniform in [-60, 60], one element per row
    made 16 times larger: every row has its own binade range."""
    rng = np.random.default_rng(seed)
    B, H, dv, dk = w.S0.shape
    S = w.S0.astype(np.float64) * np.exp2(rng.integers(-60, 61, size=(B, H, dv)))[..., None]
    S[np.arange(B)[:, None, None], np.arange(H)[None, :, None], np.arange(dv)[None, None, :],
      rng.integers(0, dk, size=(B, H, dv))] *= 16.0
    return S.astype(np.float32)


def _per_channel_err(got, ref):
    """max over (sequence, head, value channel) of the channel's largest
    error over the nodes / the channel's largest reference magnitude."""
    num = np.max(np.abs(got - ref), axis=1)
    den = np.maximum(np.max(np.abs(ref), axis=1), 1e-300)
    return np.max(num / den)


def _per_row_err(S, S_ref):
    num = np.sqrt(((S.astype(np.float64) - S_ref) ** 2).sum(-1))
    den = np.maximum(np.sqrt((S_ref ** 2).sum(-1)), 1e-300)
    return np.max(num / den)


# Per-channel bar of the wide-range tests.  The readout rounds both operands
# of each product to fp16 (RNE, relative 2^-12 each), so a channel's error is
# at most about 2^-11 sum_k |s_k x_k| <= 2^-11 |s| |x|, which exceeds 2e-3 of
# the channel's own largest output when the products cancel; 1e-2 covers
# that.  Without the row scaling, rows above the fp16 range would read as
# inf and rows below it as 0 (errors of 100 %).
WIDE_TOL = 1e-2


@pytest.mark.parametrize("T", [64, 200])
def test_wide_dynamic_range_state(G, orc, T):
    """Rows of S0 spread over 2^-60..2^64 keep their relative accuracy: with
    v = 0 every output channel is the S0 readout alone, and each is checked
    against its own largest reference magnitude; each committed state row
    within 1e-4 relative (T = 64: on-chip kernels, T = 200: the workspace
    path)."""
    import torch
    w = W.make_random(3600 + T, 2, T, 2, 4, 64, 64, "f32", shuffle=True)
    w.S0 = _wide_state(w, T)
    w.v = np.zeros_like(w.v)
    rows = np.abs(w.S0).max(-1)
    assert rows.max() > 65504.0 and rows.min() < 6.1e-5   # beyond fp16 on both sides
    _announce(f"wide dynamic range S0, T={T}")
    dt = G.DeviceTree(w)
    dt.prepare()
    dt.verify()
    S = dt.S0.clone()
    cs = dt.conv_state.clone()
    dt.commit(S, cs)
    torch.cuda.synchronize()
    got = dt.out.cpu().numpy().astype(np.float64)
    ref = orc.verify(w)
    err = _per_channel_err(got, ref)
    S_ref, _cs_ref, _st = orc.commit(w)
    serr = _per_row_err(S.cpu().numpy(), S_ref)
    _announce(f"  per-channel out err {err:.3e}  per-row state err {serr:.3e}")
    assert np.isfinite(got).all()
    assert err <= WIDE_TOL
    assert serr <= S_TOL


def test_wide_dynamic_range_step(G, orc):
    """The fused step converts the committed rows to fp16 with their own
    scales before verifying: same per-channel / per-row bars."""
    import torch
    wp = W.make_random(3700, 2, 64, 2, 4, 64, 64, "f32", shuffle=True)
    wc = W.make_random(3701, 2, 64, 2, 4, 64, 64, "f32", shuffle=True)
    wc.conv_w = wp.conv_w
    wp.S0 = _wide_state(wp, 5)
    wp.v = np.zeros_like(wp.v)   # the commit keeps the rows' spread
    wc.v = np.zeros_like(wc.v)
    dp, dc = G.DeviceTree(wp), G.DeviceTree(wc)
    dp.prepare()
    dc.prepare()
    S = dp.S0.clone()
    cs_out = torch.empty_like(dp.conv_state)
    dc.step_from(dp, S, dp.conv_state.clone(), cs_out)
    torch.cuda.synchronize()
    S_ref, cs_ref, _st = orc.commit(wp)
    rows = np.abs(S_ref).max(-1)
    assert rows.max() > 65504.0 and rows.min() < 6.1e-5
    wc.S0, wc.conv_state = S_ref, cs_ref
    err = _per_channel_err(dc.out.cpu().numpy().astype(np.float64), orc.verify(wc))
    serr = _per_row_err(S.cpu().numpy(), S_ref)
    _announce(f"wide dynamic range step: per-channel out err {err:.3e}  per-row state err {serr:.3e}")
    assert err <= WIDE_TOL
    assert serr <= S_TOL


@pytest.mark.parametrize("T", [60, 300])
def test_nan_reaches_only_descendants(G, orc, T):
    """Failure containment: a NaN in the raw value of node j (one value
    head) reaches the outputs of j's descendants (and j) in that head only;
    every other output is bit-identical to the clean run (on-chip kernel at
    T = 60, workspace path at T = 300)."""
    import torch
    w = W.make_random(3800 + T, 2, T, 1, 2, 32, 32, "f32", shuffle=True)
    ref = orc.prepare(w.parent)
    b, j, h = 1, int(np.nonzero(w.parent[1] >= 0)[0][3]), 1
    dt = G.DeviceTree(w)
    dt.prepare()
    dt.verify()
    torch.cuda.synchronize()
    clean = dt.out.clone()
    v = dt.v.clone()
    v[b, j, h, 5] = float("nan")
    dt.v = v
    dt.verify()
    torch.cuda.synchronize()
    got = dt.out.cpu().numpy()
    base = clean.cpu().numpy()
    desc = np.zeros(T, bool)
    for i in range(T):
        anc = [(int(ref["anc"][b, i, t // 64]) >> (t % 64)) & 1 for t in range(T)]
        desc[i] = i == j or anc[j] == 1
    bad = ~np.isfinite(got).all(axis=-1)           # [B][T][Hv]
    assert bad[b, j, h]
    assert not bad[:, :, 1 - h].any() and not bad[1 - b].any()
    assert not (bad[b, :, h] & ~desc).any()
    keep = np.ones(got.shape[:3], bool)
    keep[b, desc, h] = False
    np.testing.assert_array_equal(got[keep].view(np.int32), base[keep].view(np.int32))
