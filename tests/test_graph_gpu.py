"""HIP graph capture of a decode step (Sec. 3.4.2: the tree shapes are fixed,
so the whole pass is captured once and replayed).

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


def test_graph_replay_matches_eager(G):
    import torch
    w = W.make_random(7100, 4, 40, 2, 4, 64, 64, "bf16", shuffle=True)
    wp = W.make_random(7101, 4, 40, 2, 4, 64, 64, "bf16", shuffle=True)
    wp.conv_w = w.conv_w
    print("[gpu] graph replay B=4 T=40 Hk=2 Hv=4 d=64", flush=True)
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
    with torch.cuda.graph(g):
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
