"""CPU tests of the decode-loop simulation: the tree acceptance rule is
lossless (every emitted token is distributed as the target given the tokens
before it), checked exactly on enumerated small trees and by sampling on
larger ones; the best-first construction follows Algorithm 1's order; and a
few simulated decode steps drive the oracle's commit / verify chain."""
import itertools

import numpy as np
import pytest

from paper_2607_06763_amd import decode_sim as D
from paper_2607_06763_amd import workloads as W


def _first_token_exact_sampled(q, p, kids):
    """Exact distribution of the first emitted token at a node whose children
    are the tokens `kids`, each drawn from p: speculative sampling with the
    residual max(r - p, 0) after each rejection, then the bonus from r."""
    out = np.zeros_like(q)
    r = q.copy()
    reach = 1.0
    for x in kids:
        a = min(1.0, r[x] / p[x])
        out[x] += reach * a
        reach *= 1.0 - a
        r = np.maximum(r - p, 0.0)
        if r.sum() == 0.0:
            return out
        r = r / r.sum()
    return out + reach * r


def test_multidraft_rule_is_exact_on_enumerated_children():
    """All ordered pairs / triples of i.i.d. children over a 3-token vocab:
    averaging the first emitted token's distribution over the draws gives q."""
    rng = np.random.default_rng(3)
    for _ in range(5):
        q = rng.dirichlet(np.ones(3))
        p = rng.dirichlet(np.ones(3))
        for m in (1, 2, 3):
            tot = np.zeros(3)
            for kids in itertools.product(range(3), repeat=m):
                tot += np.prod(p[list(kids)]) * _first_token_exact_sampled(q, p, kids)
            np.testing.assert_allclose(tot, q, rtol=0, atol=1e-12)


def test_verify_tree_matches_the_exact_rule():
    """verify_tree's first-token frequencies on a fixed one-level sampled tree
    agree with the exact distribution above (sampling error bound)."""
    lm = D.SyntheticLM(vocab=5, seed=1, mismatch=1.5)
    ctx = [2]
    p, q = lm.drafter(ctx), lm.target(ctx)
    tree = D._new_tree(ctx)
    for tok in (1, 1, 3):
        D._add(tree, 0, tok, p)
    want = _first_token_exact_sampled(q, p, [1, 1, 3])
    rng = np.random.default_rng(11)
    n = 40000
    cnt = np.zeros(5)
    for _ in range(n):
        cnt[D.verify_tree(tree, lm, rng)[2][0]] += 1
    sig = np.sqrt(want * (1 - want) / n)
    assert np.all(np.abs(cnt / n - want) <= 5 * sig + 1e-12)


@pytest.mark.parametrize("kind", ["best_first", "sampled"])
def test_lossless_by_sampling(kind):
    """Whole decode steps (tree built afresh each time for sampled trees):
    the first emitted token follows q(. | context), and after an accepted
    first token a the second follows q(. | context + a)."""
    lm = D.SyntheticLM(vocab=6, seed=5, mismatch=1.0)
    ctx = [0, 4]
    rng = np.random.default_rng(12)
    n = 30000
    first = np.zeros(lm.V)
    second = {}
    fixed = D.build_tree_best_first(lm, ctx, budget=12, width=2, fanout=3) if kind == "best_first" else None
    for _ in range(n):
        tree = fixed if fixed is not None else D.build_tree_sampled(lm, ctx, budget=10, fanout=3, rng=rng)
        slot, _bonus, em = D.verify_tree(tree, lm, rng)
        first[em[0]] += 1
        if len(em) >= 2:
            second.setdefault(em[0], np.zeros(lm.V))[em[1]] += 1
    q0 = lm.target(ctx)
    sig = np.sqrt(q0 * (1 - q0) / n)
    assert np.all(np.abs(first / n - q0) <= 5 * sig + 1e-12)
    checked = 0
    for a, c in second.items():
        m = c.sum()
        if m < 3000:
            continue
        qa = lm.target(ctx + [a])
        sig = np.sqrt(qa * (1 - qa) / m)
        assert np.all(np.abs(c / m - qa) <= 5 * sig + 1e-12), a
        checked += 1
    assert checked >= 1


def test_equal_distributions_accept_first_children():
    """p = q: every first child is accepted, so the walk ends at the leaf
    reached by first children, and the accepted slot is that leaf."""
    lm = D.SyntheticLM(vocab=8, seed=2, mismatch=0.0)
    rng = np.random.default_rng(4)
    for _ in range(20):
        tree = D.build_tree_sampled(lm, [1], budget=20, fanout=2, rng=rng)
        slot, _b, em = D.verify_tree(tree, lm, rng)
        node = 0
        while tree.children[node]:
            node = tree.children[node][0]
        assert slot == node
        assert len(em) == (0 if node == 0 else len(tree.ctx[node]) - 1) + 1


@pytest.mark.parametrize("width", [1, 4])
def test_best_first_order_and_shape(width):
    """Algorithm 1: each round adds the `width` most probable frontier nodes
    (in non-increasing path probability within the round; with width 1 the
    whole sequence is non-increasing), each parent precedes its children, no
    node has more than `fanout` children, and the tree has `budget` slots."""
    lm = D.SyntheticLM(vocab=12, seed=9, mismatch=0.7)
    tree = D.build_tree_best_first(lm, [3, 5], budget=41, width=width, fanout=8)
    assert len(tree) == 41
    prob = [1.0]
    for s in range(1, len(tree)):
        par = tree.parent[s]
        assert 0 <= par < s
        prob.append(prob[par] * float(lm.drafter(tree.ctx[par])[tree.tokens[s]]))
    for r0 in range(1, len(prob), width):
        rnd = prob[r0:r0 + width]
        assert all(rnd[i] >= rnd[i + 1] - 1e-15 for i in range(len(rnd) - 1))
    assert max(len(c) for c in tree.children) <= 8
    # each node's children in the tree are its most probable ones
    for s, kids in enumerate(tree.children):
        if kids:
            p = lm.drafter(tree.ctx[s])
            top = set(np.argsort(-p, kind="stable")[:len(kids)].tolist())
            assert set(tree.tokens[k] for k in kids) == top


def test_decode_loop_drives_oracle(orc):
    """Three simulated decode steps on the oracle: commit of the accepted
    node after each verify; the committed state equals the state after
    sequentially decoding all committed tokens, which are the root of each
    tree followed by its accepted path (a chain of the same layer inputs)."""
    lm = D.SyntheticLM(vocab=10, seed=3, mismatch=0.8)
    emb = D.Embeddings(10, Hk=1, Hv=2, dk=8, dv=6, in_dtype=W.F32, seed=3)
    rng = np.random.default_rng(8)
    B, T = 2, 12
    ctxs = [[1], [7]]
    C = 2 * 1 * 8 + 2 * 6
    S = 0.1 * np.random.default_rng(1).standard_normal((B, 2, 6, 8)).astype(np.float32)
    cs = np.random.default_rng(2).standard_normal((B, 3, C)).astype(np.float32)
    S0, cs0 = S.copy(), cs.copy()
    committed = [[], []]
    for _step in range(3):
        trees = [D.build_tree_best_first(lm, c, budget=T, width=2, fanout=3) for c in ctxs]
        acc = []
        for b, t in enumerate(trees):
            slot, _bonus, em = D.verify_tree(t, lm, rng)
            acc.append(slot)
            path = []
            node = slot
            while node >= 0:
                path.append(t.tokens[node])
                node = t.parent[node]
            committed[b] += path[::-1]
            ctxs[b] = ctxs[b] + em
        w = D.layer_inputs(trees, T, emb, S, cs, acc)
        S_new, cs_new, st = orc.commit(w)
        assert (st == 0).all()
        S, cs = S_new.astype(np.float32), cs_new.astype(np.float32)
    # the same commits as one chain per sequence
    for b in range(B):
        n = len(committed[b])
        chain = D.Tree(tokens=committed[b], parent=list(range(-1, n - 1)), ctx=[[]] * n)
        wb = D.layer_inputs([chain], n, emb, S0[b:b + 1], cs0[b:b + 1], [n - 1])
        Sc, csc, _ = orc.commit(wb)
        np.testing.assert_allclose(S[b], Sc[0], rtol=0, atol=1e-5)
        np.testing.assert_allclose(cs[b], csc[0], rtol=0, atol=0)
