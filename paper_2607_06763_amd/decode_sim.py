"""Decode-loop simulation around the tree verification path.

The GDN kernels take the accepted slot of each tree as an input; in a
speculative decoder it comes from the verification of the draft tree
against the target model's distributions (Sec. 2.2.3, Sec. 4.3).  Without
model weights, this module drives that loop with synthetic distributions:

* ``SyntheticLM``: a drafter p(. | context) and a target q(. | context) over a
  small vocabulary, pseudo-random but a deterministic function of the last
  two context tokens; p is q with its logits perturbed (``mismatch`` = 0
  gives p = q).
* Tree construction.  ``build_tree_best_first`` follows the best-first
  growth of the paper's Algorithm 1 (Appendix A): a max-heap of frontier
  nodes keyed by path probability, the ``width`` most probable popped per
  round and added to the tree, each expanded with its ``fanout`` most
  probable children under the drafter, until ``budget`` nodes.  Candidates
  are deterministic given the context (point-mass proposals).
  ``build_tree_sampled`` instead draws ``fanout`` children of every
  expanded node i.i.d. from the drafter, breadth first, until ``budget``.
* Acceptance: ``verify_tree`` walks the tree from the root with recursive
  rejection sampling over the children of the current node: child j,
  proposed from d_j (the drafter for sampled children, a point mass for
  deterministic ones), is accepted with probability min(1, r(x_j) / d_j(x_j))
  where r starts as q(. | node); a rejection replaces r by the normalised
  positive part of r - d_j.  An accepted child becomes the current node; when
  every child is rejected a bonus token is drawn from r.  Each emitted token
  is then distributed exactly as q given the tokens before it (lossless), and
  the last accepted node is the slot the commit writes.  The paper verifies
  sampled trees with traversal verification, whose steps it does not give;
  this rule is the lossless tree rule used here in its place (both pick one
  root-to-node path and a bonus token).
* ``layer_inputs``: the raw q, k, v, alpha, beta of one GDN layer for the
  tree's nodes, looked up per token from seeded embedding tables (the same
  token always gets the same inputs).

No GDN arithmetic lives here: the tree, the accepted slot and the inputs
feed the C ABI and the oracle alike.
"""
from __future__ import annotations

import heapq
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import workloads as W


# ---------------------------------------------------------------------------
# synthetic drafter / target
# ---------------------------------------------------------------------------
class SyntheticLM:
    def __init__(self, vocab: int = 16, seed: int = 0, mismatch: float = 1.0, sharpness: float = 2.0):
        self.V = int(vocab)
        self.seed = int(seed)
        self.mismatch = float(mismatch)
        self.sharpness = float(sharpness)
        self._cache = {}

    def _dists(self, ctx):
        key = tuple(int(t) for t in ctx[-2:])
        d = self._cache.get(key)
        if d is None:
            rng = np.random.default_rng([self.seed, 7919, len(key), *[t + 1 for t in key]])
            z = self.sharpness * rng.standard_normal(self.V)
            e = rng.standard_normal(self.V)
            q = np.exp(z - z.max())
            p = np.exp(z + self.mismatch * e - (z + self.mismatch * e).max())
            d = (p / p.sum(), q / q.sum())
            self._cache[key] = d
        return d

    def drafter(self, ctx) -> np.ndarray:
        return self._dists(ctx)[0]

    def target(self, ctx) -> np.ndarray:
        return self._dists(ctx)[1]


# ---------------------------------------------------------------------------
# draft trees
# ---------------------------------------------------------------------------
@dataclass
class Tree:
    tokens: List[int]                 # token of each slot (slot 0 = root)
    parent: List[int]                 # parent slot, -1 for the root
    ctx: List[List[int]]              # context (tokens up to and including the slot)
    proposal: List[Optional[np.ndarray]] = field(default_factory=list)  # distribution the slot was drawn from; None = point mass
    children: List[List[int]] = field(default_factory=list)

    def __len__(self):
        return len(self.tokens)


def _new_tree(context: List[int]) -> Tree:
    return Tree(tokens=[int(context[-1])], parent=[-1], ctx=[list(context)], proposal=[None], children=[[]])


def _add(tree: Tree, par: int, tok: int, prop) -> int:
    tree.tokens.append(int(tok))
    tree.parent.append(par)
    tree.ctx.append(tree.ctx[par] + [int(tok)])
    tree.proposal.append(prop)
    tree.children.append([])
    tree.children[par].append(len(tree.tokens) - 1)
    return len(tree.tokens) - 1


def build_tree_best_first(lm: SyntheticLM, context: List[int], budget: int, width: int = 4,
                          fanout: int = 8) -> Tree:
    """Best-first growth (Algorithm 1 with synthetic probabilities): the root
    is the last emitted token with path probability 1; each round pops the
    `width` most probable frontier entries, adds them to the tree and pushes
    their `fanout` most probable children (by the drafter) with path
    probability prob(parent) * p(child).  Ties break by insertion order."""
    tree = _new_tree(context)
    heap = []
    counter = 0

    def expand(slot):
        nonlocal counter
        p = lm.drafter(tree.ctx[slot])
        for tok in np.argsort(-p, kind="stable")[:fanout]:
            heapq.heappush(heap, (-prob[slot] * float(p[tok]), counter, slot, int(tok)))
            counter += 1

    prob = {0: 1.0}
    expand(0)
    while len(tree) < budget and heap:
        batch = [heapq.heappop(heap) for _ in range(min(width, budget - len(tree), len(heap)))]
        new = []
        for negp, _c, par, tok in batch:
            s = _add(tree, par, tok, None)
            prob[s] = -negp
            new.append(s)
        for s in new:
            expand(s)
    return tree


def build_tree_sampled(lm: SyntheticLM, context: List[int], budget: int, fanout: int,
                       rng: np.random.Generator) -> Tree:
    """Breadth-first tree whose expanded nodes get `fanout` children drawn
    i.i.d. from the drafter; the node count depends only on the order, never
    on the drawn values."""
    tree = _new_tree(context)
    frontier = 0
    while len(tree) < budget and frontier < len(tree):
        p = lm.drafter(tree.ctx[frontier])
        for _ in range(min(fanout, budget - len(tree))):
            _add(tree, frontier, int(rng.choice(lm.V, p=p)), p)
        frontier += 1
    return tree


# ---------------------------------------------------------------------------
# acceptance
# ---------------------------------------------------------------------------
def verify_tree(tree: Tree, lm: SyntheticLM, rng: np.random.Generator):
    """Recursive rejection sampling down the tree.  Returns (accepted slot,
    bonus token, emitted tokens: the accepted path below the root, then the
    bonus)."""
    node = 0
    emitted = []
    while True:
        r = lm.target(tree.ctx[node]).astype(np.float64).copy()
        nxt = None
        for c in tree.children[node]:
            tok = tree.tokens[c]
            d = tree.proposal[c]
            dj = float(d[tok]) if d is not None else 1.0
            acc = 1.0 if dj <= 0.0 else min(1.0, r[tok] / dj)
            if rng.random() < acc:
                nxt = c
                break
            if d is None:
                r[tok] = 0.0
            else:
                r = np.maximum(r - d, 0.0)
            tot = r.sum()
            if tot <= 0.0:  # r equalled d, whose acceptance probability is 1: only rounding gets here
                nxt = c
                break
            r /= tot
        if nxt is None:
            bonus = int(rng.choice(lm.V, p=r / r.sum()))
            emitted.append(bonus)
            return node, bonus, emitted
        node = nxt
        emitted.append(tree.tokens[node])


# ---------------------------------------------------------------------------
# GDN layer inputs for the nodes of a batch of trees
# ---------------------------------------------------------------------------
class Embeddings:
    """Seeded per-token raw inputs of one GDN layer (q, k, v ~ N(0, 1) with q
    and k L2-normalised per key head, beta = sigmoid(N(0, 1)), alpha =
    exp(-softplus(N(0, 1))), as for the named workloads), plus the layer's
    conv weights."""

    def __init__(self, vocab, Hk, Hv, dk, dv, in_dtype=W.BF16, seed=0):
        rng = np.random.default_rng([seed, 104729])
        self.Hk, self.Hv, self.dk, self.dv, self.in_dtype = Hk, Hv, dk, dv, in_dtype

        def unit(shape):
            x = rng.standard_normal(shape)
            return x / np.linalg.norm(x, axis=-1, keepdims=True)

        self.q = unit((vocab, Hk, dk))
        self.k = unit((vocab, Hk, dk))
        self.v = rng.standard_normal((vocab, Hv, dv))
        self.beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((vocab, Hv))))
        self.alpha = np.exp(-np.logaddexp(0.0, rng.standard_normal((vocab, Hv))))
        C = 2 * Hk * dk + Hv * dv
        self.conv_w = (0.5 * rng.standard_normal((C, 4))).astype(np.float32)


def layer_inputs(trees: List[Tree], T: int, emb: Embeddings, S: np.ndarray, conv_state: np.ndarray,
                 accepted: Optional[List[int]] = None) -> W.Workload:
    """One step's workload: the trees padded to T slots (parent -2), the raw
    inputs of every node looked up by token, the given state and conv state
    (float32), and the accepted slots (or -1)."""
    B = len(trees)
    parent = np.full((B, T), W.PAD, np.int32)
    tok = np.zeros((B, T), np.int64)
    for b, t in enumerate(trees):
        n = len(t)
        assert n <= T
        parent[b, :n] = t.parent
        tok[b, :n] = t.tokens

    def fin(a):
        return W.f32_to_bf16_bits(a.astype(np.float32)) if emb.in_dtype == W.BF16 else a.astype(np.float32)

    real = (parent != W.PAD)[..., None, None]
    q = np.where(real, emb.q[tok], 0.0)
    k = np.where(real, emb.k[tok], 0.0)
    v = np.where(real, emb.v[tok], 0.0)
    beta = np.where(real[..., 0], emb.beta[tok], 0.0)
    alpha = np.where(real[..., 0], emb.alpha[tok], 1.0)
    acc = np.full(B, -1, np.int32) if accepted is None else np.asarray(accepted, np.int32)
    return W.Workload(name="decode-sim", B=B, T=T, Hk=emb.Hk, Hv=emb.Hv, dk=emb.dk, dv=emb.dv,
                      in_dtype=emb.in_dtype, parent=parent, q=fin(q), k=fin(k), v=fin(v),
                      alpha=fin(alpha), beta=fin(beta), S0=np.asarray(S, np.float32),
                      conv_w=emb.conv_w, conv_state=np.asarray(conv_state, np.float32), accepted=acc)
