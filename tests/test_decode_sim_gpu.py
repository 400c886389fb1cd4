"""GPU decode loop driven by the simulated tree verification: per step, the
trees are built (best-first, Algorithm 1 order, or sampled), the accepted
slot of each sequence comes from the lossless tree acceptance rule, and one
gdn_tree_step launch commits the previous step's accepted node and verifies
the current trees.  Every step's outputs and the final state are compared
with the oracle's chain of commit -> verify on the same inputs."""
import numpy as np
import pytest

from paper_2607_06763_amd import decode_sim as D
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


@pytest.mark.parametrize("kind,T,B", [("best_first", 64, 4), ("sampled", 32, 3), ("best_first", 256, 2)])
def test_decode_loop_matches_oracle(G, orc, kind, T, B):
    import torch
    V, Hk, Hv, dk, dv = 32, 2, 4, 64, 64
    lm = D.SyntheticLM(vocab=V, seed=21, mismatch=0.6)
    emb = D.Embeddings(V, Hk, Hv, dk, dv, in_dtype=W.BF16, seed=21)
    rng = np.random.default_rng(77)
    C = 2 * Hk * dk + Hv * dv
    S_host = (0.1 * np.random.default_rng(5).standard_normal((B, Hv, dv, dk))).astype(np.float32)
    cs_host = np.random.default_rng(6).standard_normal((B, 3, C)).astype(np.float32)
    S = torch.from_numpy(S_host.copy()).cuda()
    cs = torch.from_numpy(cs_host.copy()).cuda()
    S_ref, cs_ref = S_host.astype(np.float64), cs_host.astype(np.float64)
    ctxs = [[int(x)] for x in rng.integers(0, V, B)]
    prev = None          # previous step's device tree (accepted slots set)
    prev_w = None
    for step in range(5):
        if kind == "best_first":
            trees = [D.build_tree_best_first(lm, c, budget=T, width=4, fanout=8) for c in ctxs]
        else:
            trees = [D.build_tree_sampled(lm, c, budget=T, fanout=3, rng=rng) for c in ctxs]
        acc = []
        for b, t in enumerate(trees):
            slot, _bonus, em = D.verify_tree(t, lm, rng)
            acc.append(slot)
            ctxs[b] = ctxs[b] + em
        w = D.layer_inputs(trees, T, emb, S_ref.astype(np.float32), cs_ref.astype(np.float32), acc)
        print(f"[gpu] decode {kind} T={T} B={B} step {step}: accepted {acc}", flush=True)
        dt = G.DeviceTree(w)
        dt.prepare()
        if prev is None:
            dt.verify(S0=S, conv_state=cs)
        else:
            cs_out = torch.empty_like(cs)
            dt.step_from(prev, S, cs, cs_out)
            cs = cs_out
        torch.cuda.synchronize()
        # oracle chain: commit of the previous step, then verify of this one
        if prev_w is not None:
            S_ref, cs_ref, st = orc.commit(prev_w, S=S_ref, conv_state=cs_ref)
            assert (st == 0).all()
            np.testing.assert_array_equal(prev.commit_status.cpu().numpy(), st)
        w.S0, w.conv_state = S_ref, cs_ref
        out_ref = orc.verify(w)
        got = dt.out.cpu().numpy().astype(np.float64)
        err = np.max(np.abs(got - out_ref)) / np.max(np.abs(out_ref))
        Sg = S.cpu().numpy().astype(np.float64)
        serr = np.sqrt(((Sg - S_ref) ** 2).sum((2, 3)) / (S_ref ** 2).sum((2, 3))).max()
        print(f"[gpu]   out err {err:.3e}  state err {serr:.3e}", flush=True)
        assert err <= O_TOL
        assert serr <= S_TOL
        np.testing.assert_array_equal(cs.cpu().numpy(), cs_ref.astype(np.float32))
        prev, prev_w = dt, w
