"""Pins for the oracle's arithmetic, each independent of the oracle's own code:

* the short convolution against torch.nn.functional.conv1d (a library routine),
  on chains and on every node's root-to-node path of random trees;
* verify against the paper's chunked tree form (Eq. 9-11: masked Gram
  matrices X, Y, the solves (I+X)U = beta V, (I+X)W = beta a K and
  O = (aQS0 + Y(U - WS0))/sqrt(dk)), written with dense numpy solves;
* commit against the end-of-path state of Eq. 12 (restricted to the path);
* closed forms: beta = 0 (pure decay, the diagonal case of Sec. 2.2.5),
  alpha = beta = 1 with q = k (delta-rule write: o = scale v);
* a chain tree equals sequential decoding written in the stored [dv][dk]
  orientation, including two verify/commit steps (conv-state shift);
* node locality and relabelling invariance of the tree semantics.

Shapes use dk != dv so that a transposed operand cannot pass unnoticed.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_2607_06763_amd import workloads as W

TOL = 1e-11


def _small(seed, parent, Hk=2, Hv=4, dk=8, dv=6, dtype=W.F32):
    parent = np.asarray(parent, np.int32)
    if parent.ndim == 1:
        parent = parent[None]
    return W.make_random(seed, parent.shape[0], parent.shape[1], Hk, Hv, dk, dv, dtype,
                         parent=parent)


def _f64(w, name):
    a = getattr(w, name)
    if a.dtype == np.uint16:
        return W.bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


def _path(parent_row, i):
    p = []
    while i >= 0:
        p.append(i)
        i = parent_row[i]
    return p[::-1]


def _raw_channels(w, b):
    """[T][C] raw inputs, channel order q | k | v."""
    T = w.T
    return np.concatenate([_f64(w, "q")[b].reshape(T, -1), _f64(w, "k")[b].reshape(T, -1),
                           _f64(w, "v")[b].reshape(T, -1)], axis=1)


def _torch_conv_seq(w, b, seq_nodes, conv_state=None):
    """Library reference: depthwise causal conv1d (left context = conv state)
    followed by SiLU, over the raw inputs of seq_nodes; returns [len][C]."""
    raw = _raw_channels(w, b)[seq_nodes]                        # [L][C]
    cs = _f64(w, "conv_state")[b] if conv_state is None else conv_state
    x = torch.from_numpy(np.concatenate([cs, raw], 0).T[None])  # [1][C][3+L]
    wt = torch.from_numpy(_f64(w, "conv_w"))[:, None, :]       # [C][1][4]
    y = F.conv1d(x, wt, groups=x.shape[1])                     # [1][C][L]
    return F.silu(y)[0].T.numpy()


def _normalize_qk(w, y):
    y = y.copy()
    nq = w.Hk * w.dk
    for part in range(2):
        for g in range(w.Hk):
            sl = slice(part * nq + g * w.dk, part * nq + (g + 1) * w.dk)
            y[..., sl] = y[..., sl] / np.sqrt(np.sum(y[..., sl] ** 2, -1, keepdims=True) + 1e-6)
    return y


# ----------------------------------------------------------------------------
# convolution
# ----------------------------------------------------------------------------
def test_conv_chain_matches_conv1d(orc):
    w = _small(1, W.chain_tree(9))
    feat = orc.features(w)[0]
    ref = _normalize_qk(w, _torch_conv_seq(w, 0, list(range(9))))
    np.testing.assert_allclose(feat, ref, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("seed", [2, 3, 4])
def test_conv_tree_paths_match_conv1d(orc, seed):
    rng = np.random.default_rng(seed)
    par = W.random_tree(rng, 20, 17, shuffle=True)
    w = _small(seed, par)
    feat = orc.features(w)[0]
    for i in range(20):
        if par[i] == W.PAD:
            assert not feat[i].any()
            continue
        path = _path(par, i)
        ref = _normalize_qk(w, _torch_conv_seq(w, 0, path))[-1]
        np.testing.assert_allclose(feat[i], ref, rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------
# chunked tree form, Eq. 9-11 and Eq. 12
# ----------------------------------------------------------------------------
def _closure(par):
    T = len(par)
    A = np.zeros((T, T), bool)
    for i, p in enumerate(par):
        if p >= 0:
            A[i, p] = True
    R = A.copy()
    for _ in range(8):
        R = R | ((R.astype(np.int64) @ R.astype(np.int64)) > 0)
    return R  # R[i, j]: j is a proper ancestor of i


def _chunk_quantities(w, feat, b, h):
    nq = w.Hk * w.dk
    g = h * w.Hk // w.Hv
    valid = np.nonzero(w.parent[b] != W.PAD)[0]
    R = _closure(w.parent[b])[np.ix_(valid, valid)]
    Rs = R | np.eye(len(valid), dtype=bool)                 # j ancestor-or-self of i
    Q = feat[b, valid, g * w.dk:(g + 1) * w.dk]
    K = feat[b, valid, nq + g * w.dk: nq + (g + 1) * w.dk]
    V = feat[b, valid, 2 * nq + h * w.dv: 2 * nq + (h + 1) * w.dv]
    al = _f64(w, "alpha")[b, valid, h]
    be = _f64(w, "beta")[b, valid, h]
    a = np.prod(np.where(Rs, al[None, :], 1.0), axis=1)     # a_i = prod_{t <= i} alpha_t
    ratio = a[:, None] / a[None, :]
    X = np.where(R, ratio * be[:, None] * (K @ K.T), 0.0)   # Eq. 9
    Y = np.where(Rs, ratio * (Q @ K.T), 0.0)
    I = np.eye(len(valid))
    U = np.linalg.solve(I + X, be[:, None] * V)             # Eq. 10
    Wm = np.linalg.solve(I + X, (be * a)[:, None] * K)
    S0 = _f64(w, "S0")[b, h].T                              # paper orientation dk x dv
    return valid, Rs, Q, K, a, U, Wm, S0, Y


@pytest.mark.parametrize("seed", range(5))
def test_verify_equals_chunked_tree_form(orc, seed):
    rng = np.random.default_rng(10 + seed)
    T = 24
    par = W.random_tree(rng, T, 21 if seed % 2 else T, shuffle=bool(seed % 2))
    w = _small(20 + seed, np.stack([par, W.random_tree(rng, T, T)]))
    feat = orc.features(w)
    out = orc.verify(w)
    scale = 1.0 / np.sqrt(w.dk)
    for b in range(w.B):
        for h in range(w.Hv):
            valid, Rs, Q, K, a, U, Wm, S0, Y = _chunk_quantities(w, feat, b, h)
            O = scale * (a[:, None] * (Q @ S0) + Y @ (U - Wm @ S0))   # Eq. 11
            got = out[b, valid, h]
            assert np.max(np.abs(got - O)) <= TOL * max(1.0, np.max(np.abs(O)))
        pad = w.parent[b] == W.PAD
        assert not out[b, pad].any()


@pytest.mark.parametrize("seed", range(4))
def test_commit_equals_path_restricted_eq12(orc, seed):
    rng = np.random.default_rng(30 + seed)
    T = 18
    par = W.random_tree(rng, T, T, shuffle=True)
    w = _small(40 + seed, par)
    feat = orc.features(w)
    S_new, _cs, st = orc.commit(w)
    assert st[0] == 0
    n = int(w.accepted[0])
    for h in range(w.Hv):
        valid, Rs, Q, K, a, U, Wm, S0, _Y = _chunk_quantities(w, feat, 0, h)
        ni = int(np.nonzero(valid == n)[0][0])
        on_path = Rs[ni]                                  # j <= n
        r = np.where(on_path, a[ni] / a, 0.0)
        Sn = a[ni] * S0 + K.T @ (r[:, None] * (U - Wm @ S0))   # Eq. 12, rows j <= n
        np.testing.assert_allclose(S_new[0, h], Sn.T, rtol=0, atol=TOL * max(1, np.abs(Sn).max()))


# ----------------------------------------------------------------------------
# closed forms
# ----------------------------------------------------------------------------
def test_beta_zero_is_pure_decay(orc):
    rng = np.random.default_rng(5)
    par = W.random_tree(rng, 15, 15, shuffle=True)
    w = _small(50, par)
    w.beta[:] = 0.0
    feat = orc.features(w)
    out = orc.verify(w)
    al = _f64(w, "alpha")
    scale = 1.0 / np.sqrt(w.dk)
    for i in range(w.T):
        path = _path(par, i)
        for h in range(w.Hv):
            g = h * w.Hk // w.Hv
            a = np.prod(al[0, path, h])
            q = feat[0, i, g * w.dk:(g + 1) * w.dk]
            want = scale * a * (_f64(w, "S0")[0, h] @ q)
            np.testing.assert_allclose(out[0, i, h], want, rtol=1e-13, atol=1e-15)


def test_delta_write_returns_value(orc):
    """alpha = beta = 1 and q_hat = k_hat at node i: the step writes v along k,
    so S_i k = v and o_i = scale v_hat, whatever S0 and the ancestors were."""
    rng = np.random.default_rng(6)
    par = W.random_tree(rng, 12, 12, shuffle=True)
    w = _small(60, par, Hk=2, Hv=2, dk=16, dv=5)
    nq = w.Hk * w.dk
    w.k[:] = 20.0 * w.q          # large raw inputs: ||k_hat||^2 = 1 - O(1e-9)
    w.q[:] = w.k
    w.conv_w[nq:2 * nq] = w.conv_w[:nq]
    w.conv_state[:, :, nq:2 * nq] = w.conv_state[:, :, :nq]
    w.alpha[:] = 1.0
    w.beta[:] = 1.0
    feat = orc.features(w)
    np.testing.assert_array_equal(feat[..., :nq], feat[..., nq:2 * nq])
    out = orc.verify(w)
    scale = 1.0 / np.sqrt(w.dk)
    for h in range(w.Hv):
        v = feat[0, :, 2 * nq + h * w.dv: 2 * nq + (h + 1) * w.dv]
        np.testing.assert_allclose(out[0, :, h], scale * v, rtol=0, atol=1e-7)
    # commit: the accepted node's write is exact as well: S k_hat = v_hat
    S_new, _cs, _st = orc.commit(w)
    a = int(w.accepted[0])
    for h in range(w.Hv):
        g = h * w.Hk // w.Hv
        kk = feat[0, a, nq + g * w.dk: nq + (g + 1) * w.dk]
        v = feat[0, a, 2 * nq + h * w.dv: 2 * nq + (h + 1) * w.dv]
        np.testing.assert_allclose(S_new[0, h] @ kk, v, rtol=0, atol=1e-7)


def test_zero_decay_forgets_the_past(orc):
    """alpha = 0 at node j (Eq. 7): the state after j is beta_j v_j k_j^T
    whatever came before, so the commit of j equals that rank-1 matrix and
    the output of j is scale beta_j (k_j . q_j) v_j; tiny decays (1e-30)
    elsewhere on the path keep everything finite."""
    rng = np.random.default_rng(61)
    par = W.random_tree(rng, 14, 14, shuffle=True)
    w = _small(61, par, Hk=1, Hv=2, dk=8, dv=6)
    a = int(w.accepted[0])
    w.alpha[0, :, :] = 1e-30
    w.alpha[0, a, :] = 0.0
    feat = orc.features(w)
    nq = w.Hk * w.dk
    S_new, _cs, _st = orc.commit(w)
    out = orc.verify(w)
    scale = 1.0 / np.sqrt(w.dk)
    for h in range(w.Hv):
        kk = feat[0, a, nq: nq + w.dk]
        qq = feat[0, a, :w.dk]
        v = feat[0, a, 2 * nq + h * w.dv: 2 * nq + (h + 1) * w.dv]
        be = _f64(w, "beta")[0, a, h]
        np.testing.assert_allclose(S_new[0, h], be * np.outer(v, kk), rtol=0, atol=1e-14)
        np.testing.assert_allclose(out[0, a, h], scale * be * (kk @ qq) * v, rtol=0, atol=1e-14)
    assert np.isfinite(out).all() and np.isfinite(S_new).all()


# ----------------------------------------------------------------------------
# chains = sequential decoding in the stored orientation
# ----------------------------------------------------------------------------
def _decode(S, feats, al, be, w, h):
    """Sequential GDN decode, stored orientation S in R^{dv x dk}:
    S <- alpha S (I - beta k k^T) + beta v k^T;  o = scale S q."""
    nq = w.Hk * w.dk
    g = h * w.Hk // w.Hv
    scale = 1.0 / np.sqrt(w.dk)
    S = S.copy()
    outs = []
    for t in range(len(feats)):
        q = feats[t, g * w.dk:(g + 1) * w.dk]
        k = feats[t, nq + g * w.dk: nq + (g + 1) * w.dk]
        v = feats[t, 2 * nq + h * w.dv: 2 * nq + (h + 1) * w.dv]
        S = al[t] * (S - be[t] * np.outer(S @ k, k)) + be[t] * np.outer(v, k)
        outs.append(scale * (S @ q))
    return np.array(outs), S


def test_chain_equals_sequential_decode(orc):
    w = _small(70, W.chain_tree(11))
    feat = orc.features(w)
    out = orc.verify(w)
    for h in range(w.Hv):
        o, _ = _decode(_f64(w, "S0")[0, h], feat[0], _f64(w, "alpha")[0, :, h],
                       _f64(w, "beta")[0, :, h], w, h)
        np.testing.assert_allclose(out[0, :, h], o, rtol=1e-12, atol=1e-14)


def test_two_steps_equal_sequential_decode(orc):
    """verify/commit on chain 1 (accept node 3), then verify on chain 2 from the
    committed state and conv state == decoding the 4 + 6 tokens in sequence."""
    w1 = _small(80, W.chain_tree(7))
    w1.accepted[:] = 3
    w2 = _small(81, W.chain_tree(6))
    S1, cs1, st = orc.commit(w1)
    assert st[0] == 0
    w2.conv_w = w1.conv_w.copy()   # same layer weights in both steps
    w2.S0 = S1.astype(np.float64)
    w2.conv_state = cs1
    out2 = orc.verify(w2)
    # reference: conv over the concatenated raw stream, then decode
    raw = np.concatenate([_raw_channels(w1, 0)[:4], _raw_channels(w2, 0)], 0)
    x = np.concatenate([_f64(w1, "conv_state")[0], raw], 0)
    wt = torch.from_numpy(_f64(w1, "conv_w"))[:, None, :]
    y = F.silu(F.conv1d(torch.from_numpy(x.T[None]), wt, groups=x.shape[1]))[0].T.numpy()
    feats = _normalize_qk(w1, y)
    for h in range(w1.Hv):
        al = np.concatenate([_f64(w1, "alpha")[0, :4, h], _f64(w2, "alpha")[0, :, h]])
        be = np.concatenate([_f64(w1, "beta")[0, :4, h], _f64(w2, "beta")[0, :, h]])
        o, _ = _decode(_f64(w1, "S0")[0, h], feats, al, be, w1, h)
        np.testing.assert_allclose(out2[0, :, h], o[4:], rtol=1e-11, atol=1e-13)
    # conv state after the first step = raw inputs of chain nodes 1, 2, 3
    np.testing.assert_array_equal(cs1[0], _raw_channels(w1, 0)[1:4])


@pytest.mark.parametrize("acc,want", [(0, "s1 s2 x0"), (1, "s2 x0 x1"), (2, "x0 x1 x2"),
                                      (5, "x3 x4 x5")])
def test_conv_state_shift_closed_form(orc, acc, want):
    w = _small(90, W.chain_tree(6))
    w.accepted[:] = acc
    _S, cs, st = orc.commit(w)
    raw = _raw_channels(w, 0)
    old = _f64(w, "conv_state")[0]
    for slot, tok in enumerate(want.split()):
        ref = old[int(tok[1])] if tok[0] == "s" else raw[int(tok[1])]
        np.testing.assert_array_equal(cs[0, slot], ref)


def test_commit_skip_and_bad_accepted(orc):
    par = np.stack([W.chain_tree(5), W.chain_tree(5), W.chain_tree(5)])
    par[2, 4] = W.PAD
    w = _small(91, par)
    for acc, st_want in [([-1, 7, 4], [0, 5, 5]), ([-1, -3, -1], [0, 5, 0])]:
        S, cs, st = orc.commit(w, accepted=np.array(acc, np.int32))
        assert st.tolist() == st_want
        np.testing.assert_array_equal(S, _f64(w, "S0"))
        np.testing.assert_array_equal(cs, _f64(w, "conv_state"))


# ----------------------------------------------------------------------------
# tree semantics
# ----------------------------------------------------------------------------
def test_verify_commit_consistency(orc):
    rng = np.random.default_rng(7)
    par = np.stack([W.random_tree(rng, 30, 30, shuffle=True) for _ in range(2)])
    w = _small(100, par)
    feat = orc.features(w)
    out = orc.verify(w)
    S_new, _cs, _st = orc.commit(w)
    scale = 1.0 / np.sqrt(w.dk)
    for b in range(2):
        a = int(w.accepted[b])
        for h in range(w.Hv):
            g = h * w.Hk // w.Hv
            q = feat[b, a, g * w.dk:(g + 1) * w.dk]
            np.testing.assert_allclose(scale * S_new[b, h] @ q, out[b, a, h], rtol=1e-12,
                                       atol=1e-14)


def test_node_locality(orc):
    rng = np.random.default_rng(8)
    par = W.random_tree(rng, 25, 25, shuffle=True)
    w = _small(110, par)
    out = orc.verify(w)
    R = _closure(par) | np.eye(25, dtype=bool)
    # a non-root node with the most descendants
    ndesc = np.where(par >= 0, R.sum(0), -1)
    j = int(np.argmax(ndesc))
    assert 1 < ndesc[j] < 25
    # perturb node j's raw inputs and gates
    w2 = _small(110, par)
    w2.q[0, j] += 0.5
    w2.k[0, j] -= 0.25
    w2.v[0, j] *= -1.0
    w2.alpha[0, j] *= 0.5
    w2.beta[0, j] *= 0.5
    out2 = orc.verify(w2)
    for i in range(25):
        if R[i, j]:
            assert not np.array_equal(out[0, i], out2[0, i])
        else:
            np.testing.assert_array_equal(out[0, i], out2[0, i])


def test_relabelled_tree_permutes_outputs(orc):
    rng = np.random.default_rng(9)
    T = 20
    par = W.random_tree(rng, T, T, shuffle=False)
    w = _small(120, par)
    perm = rng.permutation(T)
    w2 = _small(120, par)
    par2 = np.empty(T, np.int32)
    for i in range(T):
        par2[perm[i]] = par[i] if par[i] < 0 else perm[par[i]]
    w2.parent = par2[None]
    for name in ("q", "k", "v", "alpha", "beta"):
        a = getattr(w, name)
        b = np.empty_like(a)
        b[0, perm] = a[0]
        setattr(w2, name, b)
    out, out2 = orc.verify(w), orc.verify(w2)
    np.testing.assert_array_equal(out2[0, perm], out[0])


def test_verify_leaves_inputs_untouched(orc):
    w = _small(130, W.heap_tree(9))
    before = {n: getattr(w, n).copy() for n in ("q", "k", "v", "alpha", "beta", "S0",
                                                  "conv_w", "conv_state", "parent")}
    orc.verify(w)
    for n, a in before.items():
        np.testing.assert_array_equal(getattr(w, n), a)


def test_node_mask_and_invalid_sequence(orc):
    par = np.stack([W.heap_tree(7), np.array([-1, -1, 0, 0, 1, 1, 2], np.int32)])
    w = _small(140, par)
    full = orc.verify(w)
    assert not full[1].any()       # two roots: status 2, zero output
    mask = np.zeros((2, 7), np.uint8)
    mask[0, [1, 5]] = 1
    part = orc.verify(w, node_mask=mask)
    np.testing.assert_array_equal(part[0, [1, 5]], full[0, [1, 5]])
    assert not part[0, [0, 2, 3, 4, 6]].any()


def test_custom_scale(orc):
    w = _small(150, W.heap_tree(5))
    o1 = orc.verify(w)
    o2 = orc.verify(w, scale=0.5)
    np.testing.assert_allclose(o2, o1 * 0.5 * np.sqrt(w.dk), rtol=1e-13, atol=1e-15)


def test_recurrence_exact_rationals(orc):
    """Eq. 7-8 in exact rational arithmetic on 7-node trees (dk = 4, so the
    readout scale 1/2 is exact, dv = 3): starting from the post-conv features
    the oracle uses, every node's output and the committed state agree with
    the exact values to rounding."""
    from fractions import Fraction as Fr
    for seed, par in ((71, [-1, 0, 0, 1, 1, 2, 2]), (72, [3, 3, -1, 2, 0, 4, 0])):
        w = _small(seed, par, Hk=1, Hv=2, dk=4, dv=3)
        feat = orc.features(w)
        out = orc.verify(w)
        S_new, _cs, _st = orc.commit(w)
        nq = w.Hk * w.dk
        al, be = _f64(w, "alpha"), _f64(w, "beta")

        def walk(i, h):
            S = [[Fr(float(x)) for x in row] for row in _f64(w, "S0")[0, h]]  # [dv][dk]
            for t in _path(w.parent[0].tolist(), i):
                k = [Fr(float(x)) for x in feat[0, t, nq: nq + w.dk]]
                v = [Fr(float(x)) for x in feat[0, t, 2 * nq + h * w.dv: 2 * nq + (h + 1) * w.dv]]
                a, b_ = Fr(float(al[0, t, h])), Fr(float(be[0, t, h]))
                Sk = [sum(S[r][c] * k[c] for c in range(w.dk)) for r in range(w.dv)]
                S = [[a * (S[r][c] - b_ * Sk[r] * k[c]) + b_ * v[r] * k[c] for c in range(w.dk)]
                     for r in range(w.dv)]
            return S

        for h in range(w.Hv):
            for i in range(w.T):
                S = walk(i, h)
                q = [Fr(float(x)) for x in feat[0, i, :w.dk]]
                o = [Fr(1, 2) * sum(S[r][c] * q[c] for c in range(w.dk)) for r in range(w.dv)]
                np.testing.assert_allclose(out[0, i, h], [float(x) for x in o], rtol=1e-13, atol=1e-15)
            S = walk(int(w.accepted[0]), h)
            np.testing.assert_allclose(S_new[0, h], [[float(x) for x in row] for row in S], rtol=1e-13,
                                       atol=1e-15)
