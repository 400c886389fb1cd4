"""HIP graph capture of a decode step (Sec. 3.4.2: with fixed tree shapes the
launches of a step do not change from step to step, so they can be recorded
as a graph and replayed).

One decode step = prepare of the current tree, the fused commit-then-verify
launch, and the copy of the committed conv state back into the input buffer.
The step is captured once and replayed three times, with eager work and
synchronisations between the replays; every replay must reproduce, bit for
bit, the same step run eagerly on separate buffers (the kernels are
deterministic)."""
import numpy as np
import pytest

from paper_2607_06763_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_06763_amd import gdn_tree as G
    G.lib()
    return G


def _bits(t):
    import torch
    return t.view(torch.int32).cpu().numpy()


@pytest.mark.parametrize("T", [40, 200])
def test_graph_replay_matches_eager(G, T):
    """Prepare + fused step captured once and replayed three times, each
    replay bit-identical to the eager sequence.  At T = 200 the step is the
    conv-state shift, the features and the committing pull-back, through a
    workspace that an uncaptured call on the capture stream sized first."""
    import torch
    w = W.make_random(7100 + T, 4, T, 2, 4, 64, 64, "bf16", shuffle=True)
    wp = W.make_random(7101 + T, 4, T, 2, 4, 64, 64, "bf16", shuffle=True)
    wp.conv_w = w.conv_w
    print(f"[gpu] graph replay B=4 T={T} Hk=2 Hv=4 d=64", flush=True)
    dp, dc = G.DeviceTree(wp), G.DeviceTree(w)
    dp.prepare()

    def make_state():
        return dict(S=dp.S0.clone(), cs=dp.conv_state.clone(), cs_out=torch.empty_like(dp.conv_state),
                    out=torch.empty_like(dc.out))

    def one_step(st):
        dc.prepare()
        dc.step_from(dp, st["S"], st["cs"], st["cs_out"], out=st["out"])
        st["cs"].copy_(st["cs_out"])

    # eager reference: three steps
    ref = make_state()
    snaps = []
    for _ in range(3):
        one_step(ref)
        torch.cuda.synchronize()
        snaps.append({k: _bits(v) for k, v in ref.items() if k != "cs_out"})

    # capture one step on fresh buffers (after a warm-up launch on the side
    # stream, which is then undone by restoring the initial state)
    cap = make_state()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        one_step(cap)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    cap["S"].copy_(dp.S0)
    cap["cs"].copy_(dp.conv_state)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        one_step(cap)
    # capturing does not run the kernels: the state is still the initial one
    torch.cuda.synchronize()
    assert np.array_equal(_bits(cap["S"]), _bits(dp.S0))
    for r in range(3):
        g.replay()
        torch.cuda.synchronize()
        got = {k: _bits(v) for k, v in cap.items() if k != "cs_out"}
        for k in ("S", "cs", "out"):
            assert np.array_equal(got[k], snaps[r][k]), (r, k)
        # unrelated eager work between replays
        junk = torch.randn(1 << 16, device="cuda").sum()
        torch.cuda.synchronize()
        assert torch.isfinite(junk)


@pytest.mark.parametrize("T", [40, 200])
def test_graph_multilayer_shared_meta(G, orc, T):
    """A decode step of an L = 3 layer stack captured as one HIP graph:
    prepare of the tree once, then verify of every layer against the same
    metadata blob, then the commit of the accepted node in every layer
    (Sec. 3.4.2: the metadata is built once per step and shared by all
    layers).  Replayed three times with eager work in between; each replay
    must equal the same sequence run eagerly, bit for bit, and the first
    replay must match the oracle layer by layer.  At T = 200 the verify runs
    through the feature workspace, which an uncaptured call on the capture
    stream sized beforehand."""
    import torch
    L = 3
    base = W.make_random(7200 + T, 3, T, 2, 4, 64, 32, "bf16", shuffle=True)
    layers = [base] + [W.make_random(7200 + T + l, 3, T, 2, 4, 64, 32, "bf16", parent=base.parent)
                       for l in range(1, L)]
    for lw in layers[1:]:
        lw.accepted = base.accepted
    print(f"[gpu] graph {L} layers sharing one meta, T={T}", flush=True)
    dts = [G.DeviceTree(lw) for lw in layers]
    meta = dts[0].meta   # the one metadata blob of the step

    def make_state():
        return [dict(S=d.S0.clone(), cs=d.conv_state.clone(), out=torch.empty_like(d.out)) for d in dts]

    def one_step(st):
        G.prepare(dts[0].dims, dts[0].parent, meta, dts[0].tree_status)
        for d, s in zip(dts, st):
            G.verify(d.dims, meta, d.q, d.k, d.v, d.alpha, d.beta, d.conv_w, s["cs"], s["S"], s["out"])
        for d, s in zip(dts, st):
            G.commit(d.dims, meta, d.accepted, d.q, d.k, d.v, d.alpha, d.beta, d.conv_w, s["cs"], s["S"],
                     d.commit_status)

    def snap(st):
        return [{k: _bits(v) for k, v in s.items()} for s in st]

    ref = make_state()
    snaps = []
    for _ in range(3):
        one_step(ref)
        torch.cuda.synchronize()
        snaps.append(snap(ref))

    cap = make_state()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):   # sizes the workspace of this stream, then undone
        one_step(cap)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    for d, s in zip(dts, cap):
        s["S"].copy_(d.S0)
        s["cs"].copy_(d.conv_state)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        one_step(cap)
    torch.cuda.synchronize()
    for r in range(3):
        g.replay()
        torch.cuda.synchronize()
        got = snap(cap)
        for l in range(L):
            for k in ("S", "cs", "out"):
                assert np.array_equal(got[l][k], snaps[r][l][k]), (r, l, k)
        if r == 0:  # against the oracle, layer by layer
            for l, lw in enumerate(layers):
                out = cap[l]["out"].cpu().numpy().astype(np.float64)
                ref_o = orc.verify(lw)
                assert np.max(np.abs(out - ref_o)) <= 2e-3 * np.max(np.abs(ref_o))
                S_ref, cs_ref, _st = orc.commit(lw)
                Sg = cap[l]["S"].cpu().numpy().astype(np.float64)
                rel = np.sqrt(((Sg - S_ref) ** 2).sum((2, 3)) / (S_ref ** 2).sum((2, 3))).max()
                assert rel <= 1e-4
                np.testing.assert_array_equal(cap[l]["cs"].cpu().numpy(), cs_ref.astype(np.float32))
        junk = torch.randn(1 << 16, device="cuda").sum()
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
