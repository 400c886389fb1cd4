"""Seeded synthetic draft-tree workloads for GDN tree verification.

This module only *generates inputs*: parent arrays, raw q/k/v, gates, the
cached recurrent state S0, the short-conv weights and conv state, and the
accepted node per sequence.  It contains none of the verification arithmetic
(no conv, no recurrence), so both the HIP path and the CPU oracle can be fed
from it without sharing any of the method.

Shapes and value distributions follow the problem statement of the paper's
rollback-free GDN tree verification (Sec. 3.4.1, Eq. 7-8; Sec. 3.4.2 for the
dense [N, T, H, d] tensors and the parent-pointer tree):

* q, k ~ N(0, 1), L2-normalised per (sequence, node, key head) over d_k
* v ~ N(0, 1)
* beta = sigmoid(N(0, 1)), alpha = exp(-softplus(N(0, 1)))  (both in (0, 1])
* S0 ~ 0.1 N(0, 1)   stored [B][Hv][dv][dk] fp32
* conv_w ~ N(0, 0.5^2)  [C][4] fp32,  C = 2 Hk dk + Hv dv
* conv_state ~ N(0, 1)  [B][3][C] fp32 (slot 2 is the most recent token)

Everything is drawn in float64, cast to float32, and for bf16 workloads
rounded to bfloat16 with round-to-nearest-even.  bf16 tensors are returned as
uint16 bit patterns (numpy has no bfloat16).  Each workload uses one
``numpy.random.SeedSequence`` whose children are spawned in the fixed order
tree, q, k, v, alpha, beta, S0, conv_w, conv_state, accepted.

The five named workloads (tiny heap tree, chain, top-K best-first tree,
batched random trees, large batched trees) are the synthetic stand-ins for the
paper's draft trees with budgets 64/128 (Table 1) on a Qwen-style GDN layer
(16 key heads, 32 or 48 value heads, head dim 128).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional

import numpy as np

PAD = -2   # parent value marking an absent (padding) node
ROOT = -1  # parent value of the root

F32 = "f32"
BF16 = "bf16"


# --------------------------------------------------------------------------
# dtype helpers (input marshalling only)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns the 16-bit patterns as uint16.  Inputs must be finite."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# workload container
# --------------------------------------------------------------------------
@dataclass
class Workload:
    name: str
    B: int
    T: int
    Hk: int
    Hv: int
    dk: int
    dv: int
    in_dtype: str                 # "f32" or "bf16": dtype of q, k, v, alpha, beta
    parent: np.ndarray            # int32 [B][T]; -1 root, -2 padding
    q: np.ndarray                 # [B][T][Hk][dk]  float32 or uint16 (bf16 bits)
    k: np.ndarray                 # [B][T][Hk][dk]
    v: np.ndarray                 # [B][T][Hv][dv]
    alpha: np.ndarray             # [B][T][Hv]
    beta: np.ndarray              # [B][T][Hv]
    S0: np.ndarray                # float32 [B][Hv][dv][dk]
    conv_w: np.ndarray            # float32 [C][4]
    conv_state: np.ndarray        # float32 [B][3][C]
    accepted: np.ndarray          # int32 [B]; -1 = commit nothing
    meta: Dict[str, object] = field(default_factory=dict)

    @property
    def C(self) -> int:
        return 2 * self.Hk * self.dk + self.Hv * self.dv

    def as_f32(self, name: str) -> np.ndarray:
        """Input tensor widened to float32 (exact for bf16)."""
        a = getattr(self, name)
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a)
        return np.asarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# tree generators
# --------------------------------------------------------------------------
def heap_tree(T: int) -> np.ndarray:
    """Complete binary tree in heap numbering: parent(i) = (i-1)//2."""
    p = np.array([(i - 1) // 2 for i in range(T)], dtype=np.int32)
    p[0] = ROOT
    return p


def chain_tree(T: int) -> np.ndarray:
    p = np.arange(-1, T - 1, dtype=np.int32)
    return p


def _depths(parent: List[int]) -> List[int]:
    d = []
    for i, p in enumerate(parent):
        d.append(0 if p < 0 else d[p] + 1)
    return d


def topk_best_first_tree(rng: np.random.Generator, T: int = 64, K: int = 4,
                         max_depth: int = 8) -> np.ndarray:
    """Best-first draft tree in the spirit of the paper's parallel best-first
    construction (Sec. 3.3, Algorithm 1), with Dirichlet(1) child scores.

    Spine: at each level 0..max_depth-1 the highest cumulative-score node of
    that level gets K children (1 + K*max_depth nodes, depth max_depth).
    Fill: the highest-scoring unexpanded node of depth < max_depth is expanded
    (children added in descending score) until T nodes exist.  Nodes are then
    renumbered breadth-first so that parent[i] < i."""
    par: List[int] = [ROOT]
    dep: List[int] = [0]
    score: List[float] = [1.0]
    expanded = [False]

    def expand(n: int) -> None:
        s = rng.dirichlet(np.ones(K))
        expanded[n] = True
        for c in np.argsort(-s, kind="stable"):
            if len(par) >= T:
                return
            par.append(n)
            dep.append(dep[n] + 1)
            score.append(score[n] * float(s[c]))
            expanded.append(False)

    for level in range(max_depth):
        cands = [i for i in range(len(par)) if dep[i] == level]
        best = max(cands, key=lambda i: (score[i], -i))
        expand(best)
    while len(par) < T:
        cands = [i for i in range(len(par)) if not expanded[i] and dep[i] < max_depth]
        best = max(cands, key=lambda i: (score[i], -i))
        expand(best)
    # breadth-first renumbering: stable by (depth, creation index)
    order = sorted(range(T), key=lambda i: (dep[i], i))
    new_of = {old: new for new, old in enumerate(order)}
    out = np.empty(T, dtype=np.int32)
    for new, old in enumerate(order):
        out[new] = ROOT if par[old] < 0 else new_of[par[old]]
    return out


def random_depth_capped_tree(rng: np.random.Generator, T: int, max_parent_depth: int,
                             spine: int = 0, max_children: Optional[int] = None) -> np.ndarray:
    """parent[i] uniform over {j < i : depth_j <= max_parent_depth
    (and children_j < max_children)}, after an optional forced spine
    0 -> 1 -> ... -> spine."""
    par = [ROOT]
    dep = [0]
    nch = [0]
    for i in range(1, T):
        if i <= spine:
            p = i - 1
        else:
            cands = [j for j in range(i) if dep[j] <= max_parent_depth
                     and (max_children is None or nch[j] < max_children)]
            p = cands[int(rng.integers(len(cands)))]
        par.append(p)
        dep.append(dep[p] + 1)
        nch.append(0)
        nch[p] += 1
    return np.array(par, dtype=np.int32)


# --------------------------------------------------------------------------
# tensor generators
# --------------------------------------------------------------------------
def _finish(x64: np.ndarray, dtype: str) -> np.ndarray:
    x32 = x64.astype(np.float32)
    return f32_to_bf16_bits(x32) if dtype == BF16 else x32


def _unit_normal(rng: np.random.Generator, shape) -> np.ndarray:
    x = rng.standard_normal(shape)
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True))


def make_inputs(name: str, parent: np.ndarray, Hk: int, Hv: int, dk: int, dv: int,
                in_dtype: str, children: List[np.random.SeedSequence],
                accepted_fn: Callable[[np.random.Generator, np.ndarray], np.ndarray],
                meta: Optional[dict] = None) -> Workload:
    """Draw every tensor of a workload from the spawned seed children
    (order: q, k, v, alpha, beta, S0, conv_w, conv_state, accepted)."""
    B, T = parent.shape
    C = 2 * Hk * dk + Hv * dv
    g = [np.random.default_rng(c) for c in children]
    q = _finish(_unit_normal(g[0], (B, T, Hk, dk)), in_dtype)
    k = _finish(_unit_normal(g[1], (B, T, Hk, dk)), in_dtype)
    v = _finish(g[2].standard_normal((B, T, Hv, dv)), in_dtype)
    alpha = _finish(np.exp(-np.logaddexp(0.0, g[3].standard_normal((B, T, Hv)))), in_dtype)
    beta = _finish(1.0 / (1.0 + np.exp(-g[4].standard_normal((B, T, Hv)))), in_dtype)
    S0 = (0.1 * g[5].standard_normal((B, Hv, dv, dk))).astype(np.float32)
    conv_w = (0.5 * g[6].standard_normal((C, 4))).astype(np.float32)
    conv_state = g[7].standard_normal((B, 3, C)).astype(np.float32)
    accepted = accepted_fn(g[8], parent).astype(np.int32)
    return Workload(name, B, T, Hk, Hv, dk, dv, in_dtype, np.ascontiguousarray(parent, np.int32),
                    q, k, v, alpha, beta, S0, conv_w, conv_state, accepted, meta or {})


def _uniform_valid_node(rng: np.random.Generator, parent: np.ndarray) -> np.ndarray:
    out = []
    for b in range(parent.shape[0]):
        valid = np.nonzero(parent[b] != PAD)[0]
        out.append(int(valid[int(rng.integers(len(valid)))]) if len(valid) else -1)
    return np.array(out, dtype=np.int32)


CONFIG_NAMES = ["tiny", "chain", "topk", "batched", "large"]


def make_config(cfg: int) -> Workload:
    """The five named workloads, seeded with SeedSequence(20260 + cfg)."""
    ss = np.random.SeedSequence(20260 + cfg)
    ch = ss.spawn(10)
    tree_rng = np.random.default_rng(ch[0])
    if cfg == 0:
        # B=1, 2 key / 2 value heads, d=16, complete binary tree of 7 nodes, fp32
        parent = heap_tree(7)[None, :]
        return make_inputs("tiny", parent, 2, 2, 16, 16, F32, ch[1:], _uniform_valid_node)
    if cfg == 1:
        # B=1, 16k/32v heads, d=128, 16-node chain, bf16 inputs
        parent = chain_tree(16)[None, :]
        return make_inputs("chain", parent, 16, 32, 128, 128, BF16, ch[1:], _uniform_valid_node)
    if cfg == 2:
        # B=1, 16k/32v, d=128, 64-node top-K (K=4) best-first tree of depth 8
        parent = topk_best_first_tree(tree_rng, 64, 4, 8)[None, :]
        return make_inputs("topk", parent, 16, 32, 128, 128, BF16, ch[1:], _uniform_valid_node)
    if cfg == 3:
        # B=8 independent 64-node trees, parent uniform over earlier nodes of depth <= 7
        parent = np.stack([random_depth_capped_tree(tree_rng, 64, 7) for _ in range(8)])
        return make_inputs("batched", parent, 16, 32, 128, 128, BF16, ch[1:], _uniform_valid_node)
    if cfg == 4:
        # B=32, 16k/48v, d=128, 128-node trees of depth 16 (forced spine, <= 8 children)
        parent = np.stack([random_depth_capped_tree(tree_rng, 128, 15, spine=16, max_children=8)
                           for _ in range(32)])
        return make_inputs("large", parent, 16, 48, 128, 128, BF16, ch[1:], _uniform_valid_node)
    raise ValueError(f"unknown workload {cfg}")


def random_tree(rng: np.random.Generator, T: int, n_valid: Optional[int] = None,
                shuffle: bool = True, max_depth: Optional[int] = None) -> np.ndarray:
    """A random valid tree over T slots with n_valid real nodes (the rest are
    padding), arbitrary node numbering when shuffle=True."""
    n = T if n_valid is None else n_valid
    par = np.full(T, PAD, dtype=np.int32)
    if n == 0:
        return par
    dep = [0]
    lp = [ROOT]
    for i in range(1, n):
        cands = [j for j in range(i) if max_depth is None or dep[j] < max_depth]
        p = cands[int(rng.integers(len(cands)))]
        lp.append(p)
        dep.append(dep[p] + 1)
    slots = rng.permutation(T)[:n] if shuffle else np.arange(n)
    for i in range(n):
        par[slots[i]] = ROOT if lp[i] < 0 else slots[lp[i]]
    return par


def make_random(seed: int, B: int, T: int, Hk: int, Hv: int, dk: int, dv: int,
                in_dtype: str = BF16, n_valid: Optional[List[int]] = None,
                shuffle: bool = True, max_depth: Optional[int] = None,
                parent: Optional[np.ndarray] = None) -> Workload:
    """Random trees (optionally padded / relabelled) with the same value
    distributions as the named workloads."""
    ss = np.random.SeedSequence(seed)
    ch = ss.spawn(10)
    tree_rng = np.random.default_rng(ch[0])
    if parent is None:
        parent = np.stack([random_tree(tree_rng, T, None if n_valid is None else n_valid[b],
                                       shuffle, max_depth) for b in range(B)])
    return make_inputs(f"random{seed}", np.asarray(parent, np.int32), Hk, Hv, dk, dv,
                       in_dtype, ch[1:], _uniform_valid_node)


def make_sweep(T: int, B: int = 32, shape: str = "large", seed: int = 0) -> Workload:
    """The large workload's recipe at another tree size T (16 key / 48 value
    heads, d = 128, bf16 inputs): shape "large" grows a forced spine of
    min(16, T - 1) edges, then attaches each further node to a uniformly
    chosen earlier node of depth <= 15 with fewer than 8 children (depth <= 16);
    shape "chain" makes every tree a single path of T nodes (depth T - 1)."""
    ss = np.random.SeedSequence([20270, T, B, 0 if shape == "large" else 1, seed])
    ch = ss.spawn(10)
    tree_rng = np.random.default_rng(ch[0])
    if shape == "large":
        parent = np.stack([random_depth_capped_tree(tree_rng, T, 15, spine=min(16, T - 1),
                                                    max_children=8) for _ in range(B)])
    elif shape == "chain":
        parent = np.stack([chain_tree(T)] * B)
    else:
        raise ValueError(f"unknown sweep shape {shape}")
    return make_inputs(f"{shape}-T{T}", parent, 16, 48, 128, 128, BF16, ch[1:], _uniform_valid_node)
