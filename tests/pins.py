"""Pins for the CPU oracle: checks against what the paper and the mathematics fix, independent of the oracle's
own code.  Each pin is a function of an ``oracle.Oracle`` instance so that the same checks can be run against
copies of the oracle with planted mistakes (tests/test_oracle_mutants.py) to show that they would catch them.

Sources of truth used here: brute-force dense masked softmax (numpy, fp64) with the ancestor relation built
as a transitive closure; library attention (torch scaled_dot_product_attention, fp64) for the chain and
single-node special cases; closed forms; invariants (non-ancestor perturbation, relabelling); exhaustive
enumeration of root-to-node paths for acceptance; the greedy rule's worked instances in tests/golden; the exact
expected acceptance length of the independent-agreement model; and a direct numpy gather for the commit.
"""
from __future__ import annotations

import os

import numpy as np
from scipy.special import logsumexp

from paper_2606_00535_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ------------------------------------------------------------------------------------------ helpers (numpy)
def ancestor_closure(parent: np.ndarray) -> np.ndarray:
    """C[i, j] = True iff node j is node i or one of its ancestors (reflexive-transitive closure of the
    child->parent relation, by repeated boolean matrix products)."""
    T = len(parent)
    A = np.zeros((T, T), dtype=bool)
    for i in range(1, T):
        A[i, parent[i]] = True
    C = np.eye(T, dtype=bool)
    for _ in range(T):
        C = C | ((C.astype(np.int64) @ A.astype(np.int64)) > 0)
    return C


def mask_bits_from_closure(C: np.ndarray) -> np.ndarray:
    T = C.shape[0]
    Wd = (T + 63) // 64
    bits = np.zeros((T, Wd), dtype=np.uint64)
    for i in range(T):
        for j in range(T):
            if C[i, j]:
                bits[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return bits


def dense_tree_attention(q, k, v, kv_len, parent, scale, Hkv):
    """Brute force: per (b, h) a dense [T, L+T] score matrix, -inf outside the visibility mask, softmax, @V."""
    q = q.astype(np.float64)
    B, Hq, T, D = q.shape
    G = Hq // Hkv
    out = np.zeros((B, Hq, T, D))
    lse = np.zeros((B, Hq, T))
    for b in range(B):
        L = int(kv_len[b])
        C = ancestor_closure(parent[b])
        vis = np.concatenate([np.ones((T, L), dtype=bool), C], axis=1)
        for h in range(Hq):
            g = h // G
            K = k[b, g, :L + T].astype(np.float64)
            V = v[b, g, :L + T].astype(np.float64)
            s = scale * (q[b, h] @ K.T)
            s[~vis] = -np.inf
            lse[b, h] = logsumexp(s, axis=1)
            out[b, h] = np.exp(s - lse[b, h][:, None]) @ V
    return out, lse


def random_inputs(rng, B, Hq, Hkv, T, D, L, extra=0, dtype=np.float32):
    S = L + T + extra
    q = rng.standard_normal((B, Hq, T, D)).astype(dtype)
    k = rng.standard_normal((B, Hkv, S, D)).astype(dtype)
    v = rng.standard_normal((B, Hkv, S, D)).astype(dtype)
    return q, k, v


def random_parent(rng, T, max_branch=3):
    if T == 1:
        return np.array([-1], dtype=np.int32)
    depth = int(rng.integers(1, T))
    b = max_branch
    while sum(b ** d for d in range(depth + 1)) < T:
        b += 1
    return W.random_tree(rng, T, depth, b)


# ---------------------------------------------------------------------------------------- attention pins
def pin_attn_bruteforce(orc):
    rng = np.random.default_rng(1234)
    for (B, Hq, Hkv, D) in [(1, 2, 2, 8), (2, 4, 2, 8), (1, 3, 1, 16)]:
        for L in (0, 1, 5, 17):
            for T in (1, 2, 5, 16):
                q, k, v = random_inputs(rng, B, Hq, Hkv, T, D, L, extra=3)
                parent = np.stack([random_parent(rng, T) for _ in range(B)])
                kv_len = np.full(B, L, dtype=np.int32)
                scale = 1.0 / np.sqrt(D)
                o, lse = orc.tree_attn(q, k, v, kv_len, parent, scale, Hkv)
                eo, else_ = dense_tree_attention(q, k, v, kv_len, parent, scale, Hkv)
                assert np.max(np.abs(o - eo)) <= 1e-12, (B, Hq, Hkv, D, L, T)
                assert np.max(np.abs(lse - else_)) <= 1e-12, (B, Hq, Hkv, D, L, T)
    # ragged prefix lengths inside one batch
    B, Hq, Hkv, D, T = 3, 2, 1, 8, 7
    q, k, v = random_inputs(rng, B, Hq, Hkv, T, D, 20)
    parent = np.stack([random_parent(rng, T) for _ in range(B)])
    kv_len = np.array([0, 20, 9], dtype=np.int32)
    o, lse = orc.tree_attn(q, k, v, kv_len, parent, 0.3, Hkv)
    eo, else_ = dense_tree_attention(q, k, v, kv_len, parent, 0.3, Hkv)
    assert np.max(np.abs(o - eo)) <= 1e-12 and np.max(np.abs(lse - else_)) <= 1e-12


def _torch_sdpa(q, k, v, mask, scale):
    import torch
    tq = torch.from_numpy(np.asarray(q, dtype=np.float64))
    tk = torch.from_numpy(np.asarray(k, dtype=np.float64))
    tv = torch.from_numpy(np.asarray(v, dtype=np.float64))
    tm = None if mask is None else torch.from_numpy(mask)
    return torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=tm, scale=scale).numpy()


def pin_attn_chain_is_causal(orc):
    """A chain-shaped tree is ordinary causal attention of T new tokens after an L-token prefix (explicit
    bottom-right-aligned causal mask: new token i sees the prefix and new tokens 0..i)."""
    rng = np.random.default_rng(7)
    for (L, T, D) in [(0, 6, 16), (11, 9, 16), (40, 16, 32)]:
        q, k, v = random_inputs(rng, 1, 2, 2, T, D, L)
        parent = W.chain_tree(T)[None]
        o, _ = orc.tree_attn(q, k, v, np.array([L], np.int32), parent, 1.0 / np.sqrt(D), 2)
        mask = np.zeros((T, L + T), dtype=bool)
        for i in range(T):
            mask[i, :L + i + 1] = True
        ref = _torch_sdpa(q[0], k[0, :, :L + T], v[0, :, :L + T], mask, 1.0 / np.sqrt(D))
        assert np.max(np.abs(o[0] - ref)) <= 1e-12, (L, T)


def pin_attn_single_node_is_decode(orc):
    """T = 1 is one decode step: plain softmax attention over the L prefix keys plus the node's own key."""
    rng = np.random.default_rng(8)
    for L in (0, 1, 33, 200):
        q, k, v = random_inputs(rng, 1, 4, 2, 1, 16, L)
        o, _ = orc.tree_attn(q, k, v, np.array([L], np.int32), np.array([[-1]], np.int32), 0.25, 2)
        kk = np.repeat(k[0, :, :L + 1], 2, axis=0)      # query head h reads KV head h // 2
        vv = np.repeat(v[0, :, :L + 1], 2, axis=0)
        ref = _torch_sdpa(q[0], kk, vv, None, 0.25)
        assert np.max(np.abs(o[0] - ref)) <= 1e-12, L


def pin_attn_star(orc):
    """Star tree: node i > 0 sees the prefix, the root and itself; the root sees the prefix and itself."""
    rng = np.random.default_rng(9)
    L, T, D = 13, 6, 8
    q, k, v = random_inputs(rng, 1, 1, 1, T, D, L)
    o, _ = orc.tree_attn(q, k, v, np.array([L], np.int32), W.star_tree(T)[None], 0.5, 1)
    for i in range(T):
        keys = list(range(L)) + [L] + ([L + i] if i > 0 else [])
        s = 0.5 * (k[0, 0, keys].astype(np.float64) @ q[0, 0, i].astype(np.float64))
        p = np.exp(s - s.max())
        ref = (p / p.sum()) @ v[0, 0, keys].astype(np.float64)
        assert np.max(np.abs(o[0, 0, i] - ref)) <= 1e-12, i


def pin_attn_nonancestor_perturbation(orc):
    """Changing K/V of tree nodes that are not ancestors-or-self of node i leaves row i bitwise unchanged;
    changing one of its ancestors changes it."""
    rng = np.random.default_rng(10)
    L, T, D, Hkv = 9, 12, 8, 2
    q, k, v = random_inputs(rng, 1, 2, Hkv, T, D, L)
    parent = W.random_tree(rng, T, 4, 3)[None]
    kv = np.array([L], np.int32)
    o, lse = orc.tree_attn(q, k, v, kv, parent, 0.35, Hkv)
    C = ancestor_closure(parent[0])
    for i in range(T):
        k2, v2 = k.copy(), v.copy()
        for j in range(T):
            if not C[i, j]:
                k2[0, :, L + j] = rng.standard_normal((Hkv, D))
                v2[0, :, L + j] = rng.standard_normal((Hkv, D))
        o2, lse2 = orc.tree_attn(q, k2, v2, kv, parent, 0.35, Hkv)
        assert np.array_equal(o2[0, :, i], o[0, :, i]) and np.array_equal(lse2[0, :, i], lse[0, :, i]), i
        anc = [j for j in range(T) if C[i, j]]
        j = anc[int(rng.integers(len(anc)))]
        v3 = v.copy()
        v3[0, :, L + j] += 1.0
        o3, _ = orc.tree_attn(q, k, v3, kv, parent, 0.35, Hkv)
        assert np.all(np.abs(o3[0, :, i] - o[0, :, i]) > 1e-9), (i, j)


def pin_attn_closed_forms(orc):
    """V constant => out equals that constant; K constant => out is the plain mean of the visible V rows and
    lse = scale*q.k + log(#visible)."""
    rng = np.random.default_rng(11)
    L, T, D = 21, 10, 8
    q, k, v = random_inputs(rng, 1, 2, 1, T, D, L)
    parent = W.random_tree(rng, T, 3, 4)[None]
    kv = np.array([L], np.int32)
    vc = np.full_like(v, 0.625)
    o, _ = orc.tree_attn(q, k, vc, kv, parent, 0.4, 1)
    assert np.max(np.abs(o - 0.625)) <= 1e-14
    kc = np.broadcast_to(k[:, :, :1], k.shape).copy()
    o, lse = orc.tree_attn(q, kc, v, kv, parent, 0.4, 1)
    C = ancestor_closure(parent[0])
    for h in range(2):
        for i in range(T):
            rows = list(range(L)) + [L + j for j in range(T) if C[i, j]]
            ref = v[0, 0, rows].astype(np.float64).mean(axis=0)
            assert np.max(np.abs(o[0, h, i] - ref)) <= 1e-12
            ref_lse = 0.4 * float(q[0, h, i].astype(np.float64) @ kc[0, 0, 0].astype(np.float64)) + np.log(len(rows))
            assert abs(lse[0, h, i] - ref_lse) <= 1e-12


def pin_attn_relabelling(orc):
    """Renumbering the tree in another topological order (children before ... any order with parents first)
    permutes the output rows the same way."""
    rng = np.random.default_rng(12)
    L, T, D = 15, 14, 8
    q, k, v = random_inputs(rng, 1, 2, 2, T, D, L)
    parent = W.random_tree(rng, T, 5, 3)
    o, lse = orc.tree_attn(q, k, v, np.array([L], np.int32), parent[None], 0.3, 2)
    # depth-first order (pre-order, last child first) is another valid topological numbering
    children = [[] for _ in range(T)]
    for i in range(1, T):
        children[parent[i]].append(i)
    order, stack = [], [0]
    while stack:
        n = stack.pop()
        order.append(n)
        stack.extend(children[n])
    new_of = {old: new for new, old in enumerate(order)}
    p2 = np.array([-1 if parent[old] < 0 else new_of[parent[old]] for old in order], dtype=np.int32)
    q2 = q[:, :, order]
    k2, v2 = k.copy(), v.copy()
    k2[:, :, L:L + T] = k[:, :, L + np.array(order)]
    v2[:, :, L:L + T] = v[:, :, L + np.array(order)]
    o2, lse2 = orc.tree_attn(q2, k2, v2, np.array([L], np.int32), p2[None], 0.3, 2)
    assert np.max(np.abs(o2 - o[:, :, order])) <= 1e-12
    assert np.max(np.abs(lse2 - lse[:, :, order])) <= 1e-12


def pin_attn_mask_input(orc):
    """An explicit ancestor-or-self bit mask gives the same result as the parent array; an all-zero mask row
    over an empty prefix has no visible key and is defined as a zero row with lse = -inf."""
    rng = np.random.default_rng(13)
    for T in (5, 64, 70):
        L, D = 6, 8
        q, k, v = random_inputs(rng, 1, 1, 1, T, D, L)
        parent = random_parent(rng, T)
        bits = mask_bits_from_closure(ancestor_closure(parent))[None]
        kv = np.array([L], np.int32)
        o1, l1 = orc.tree_attn(q, k, v, kv, parent[None], 0.3, 1)
        o2, l2 = orc.tree_attn(q, k, v, kv, None, 0.3, 1, tree_mask=bits)
        assert np.array_equal(o1, o2) and np.array_equal(l1, l2), T
    q, k, v = random_inputs(rng, 1, 1, 1, 3, 8, 0)
    bits = np.zeros((1, 3, 1), dtype=np.uint64)
    bits[0, 1, 0] = 0b011
    o, lse = orc.tree_attn(q, k, v, np.array([0], np.int32), None, 0.3, 1, tree_mask=bits)
    assert np.all(o[0, 0, 0] == 0) and lse[0, 0, 0] == -np.inf
    assert np.all(o[0, 0, 2] == 0) and lse[0, 0, 2] == -np.inf
    s = 0.3 * (k[0, 0, :2].astype(np.float64) @ q[0, 0, 1].astype(np.float64))
    p = np.exp(s - s.max())
    assert np.max(np.abs(o[0, 0, 1] - (p / p.sum()) @ v[0, 0, :2].astype(np.float64))) <= 1e-12


def pin_attn_rows_entry(orc):
    """The selected-rows entry point agrees exactly with the full one."""
    rng = np.random.default_rng(14)
    B, Hq, Hkv, T, D, L = 2, 4, 2, 9, 8, 12
    q, k, v = random_inputs(rng, B, Hq, Hkv, T, D, L)
    parent = np.stack([random_parent(rng, T) for _ in range(B)])
    kv = np.array([L, 5], np.int32)
    o, lse = orc.tree_attn(q, k, v, kv, parent, 0.3, Hkv)
    rows = np.array([[0, 0, 0], [1, 3, 8], [1, 2, 4], [0, 1, 7]], dtype=np.int32)
    orow, lrow = orc.tree_attn_rows(q, k, v, kv, parent, 0.3, Hkv, rows)
    for n, (b, h, i) in enumerate(rows):
        assert np.array_equal(orow[n], o[b, h, i]) and lrow[n] == lse[b, h, i]


ATTN_PINS = [pin_attn_bruteforce, pin_attn_chain_is_causal, pin_attn_single_node_is_decode, pin_attn_star,
             pin_attn_nonancestor_perturbation, pin_attn_closed_forms, pin_attn_relabelling,
             pin_attn_mask_input, pin_attn_rows_entry]


# ----------------------------------------------------------------------------------------- acceptance pins
def brute_force_accept(logits, tokens, parent):
    """Enumerate every node; it is acceptable iff each node on its root path (root excluded) carries the
    target's token at its parent (numpy argmax: first maximal index).  Take the deepest, smallest index."""
    T = len(parent)
    am = [int(np.argmax(logits[i])) for i in range(T)]
    best, best_depth = 0, 0
    for i in range(T):
        path = [i]
        while path[-1] != 0:
            path.append(int(parent[path[-1]]))
        path = path[::-1]
        if all(tokens[path[d]] == am[path[d - 1]] for d in range(1, len(path))):
            if len(path) - 1 > best_depth:
                best, best_depth = i, len(path) - 1
    path = [best]
    while path[-1] != 0:
        path.append(int(parent[path[-1]]))
    return best_depth, path[::-1], am[best], am


def pin_accept_bruteforce(orc):
    rng = np.random.default_rng(21)
    B = 256
    for V in (2, 3, 4, 7):
        for T in (1, 2, 5, 9, 16):
            parent = np.stack([random_parent(rng, T, max_branch=4) for _ in range(B)])
            # values from a tiny set force argmax ties, including -0.0 against +0.0
            logits = rng.choice(np.array([-1.0, -0.0, 0.0, 0.5, 1.0], dtype=np.float32), size=(B, T, V))
            tokens = rng.integers(0, V, size=(B, T)).astype(np.int32)
            alen, path, nxt, am = orc.tree_accept(logits, tokens, parent)
            for b in range(B):
                a, p, n, ref_am = brute_force_accept(logits[b], tokens[b], parent[b])
                assert alen[b] == a and nxt[b] == n, (V, T, b)
                assert list(path[b, :a + 1]) == p and np.all(path[b, a + 1:] == -1), (V, T, b)
                assert list(am[b]) == ref_am


def load_golden_chain_cases():
    cases = []
    with open(os.path.join(GOLDEN, "greedy_rule_chain.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, draft, target, emitted = [x.strip() for x in line.split("|")]
            cases.append((name, [int(x) for x in draft.split()], [int(x) for x in target.split()],
                          [int(x) for x in emitted.split()]))
    return cases


def pin_accept_golden_chain(orc):
    """The paper's greedy rule on its own terms (tests/golden/greedy_rule_chain.txt): a chain of drafts
    t_1..t_6 with the target's tokens t'_1..t'_7 planted as the unique row maxima."""
    V = 10
    for name, draft, target, emitted in load_golden_chain_cases():
        T = len(draft) + 1
        parent = W.chain_tree(T)[None]
        tokens = np.array([[0] + draft], dtype=np.int32)
        logits = np.zeros((1, T, V), dtype=np.float32)
        for r, t in enumerate(target):
            logits[0, r, t] = 1.0
        alen, path, nxt, _ = orc.tree_accept(logits, tokens, parent)
        got = [int(tokens[0, path[0, d]]) for d in range(1, alen[0] + 1)] + [int(nxt[0])]
        assert got == emitted, (name, got, emitted)


def pin_accept_chain_rule(orc):
    """On random chains the result equals a direct transcription of the sequential rule."""
    rng = np.random.default_rng(22)
    B, T, V = 500, 7, 5
    logits = rng.standard_normal((B, T, V)).astype(np.float32)
    tokens = rng.integers(0, V, size=(B, T)).astype(np.int32)
    tgt = np.argmax(logits, axis=2)
    tokens[rng.random((B, T)) < 0.6] = -1
    tokens = np.where(tokens < 0, np.roll(tgt, 1, axis=1), tokens).astype(np.int32)
    alen, path, nxt, _ = orc.tree_accept(logits, tokens, np.tile(W.chain_tree(T), (B, 1)))
    for b in range(B):
        emitted = []
        for i in range(1, T):
            if tokens[b, i] != tgt[b, i - 1]:
                emitted.append(int(tgt[b, i - 1]))
                break
            emitted.append(int(tokens[b, i]))
        else:
            emitted.append(int(tgt[b, T - 1]))
        got = [int(tokens[b, path[b, d]]) for d in range(1, alen[b] + 1)] + [int(nxt[b])]
        assert got == emitted, b
        assert 1 <= alen[b] + 1 <= T          # tau within [1, gamma + 1]


def pin_accept_special_cases(orc):
    """Every draft agrees => the deepest node with the smallest index is accepted (a = depth); no draft
    agrees => a = 0, path = [root] and the bonus token is the target's token at the root."""
    rng = np.random.default_rng(23)
    for _ in range(20):
        T, V = 30, 11
        parent = W.random_tree(rng, T, 5, 3)
        logits = rng.standard_normal((1, T, V)).astype(np.float32)
        am = np.argmax(logits[0], axis=1)
        depth = W.tree_depths_for_generator_checks(parent)
        tok = np.array([0] + [am[parent[i]] for i in range(1, T)], dtype=np.int32)[None]
        alen, path, nxt, _ = orc.tree_accept(logits, tok, parent[None])
        last = int(np.flatnonzero(depth == depth.max())[0])
        assert alen[0] == depth.max() and path[0, alen[0]] == last and nxt[0] == am[last]
        tok2 = np.array([0] + [(am[parent[i]] + 1) % V for i in range(1, T)], dtype=np.int32)[None]
        alen, path, nxt, _ = orc.tree_accept(logits, tok2, parent[None])
        assert alen[0] == 0 and path[0, 0] == 0 and np.all(path[0, 1:] == -1) and nxt[0] == am[0]


def pin_accept_signed_zero_ties(orc):
    logits = np.array([[[-0.0, 0.0, -1.0], [0.0, -0.0, -1.0], [-3.0, 0.0, -0.0]]], dtype=np.float32)
    tokens = np.array([[2, 0, 1]], dtype=np.int32)
    _, _, _, am = orc.tree_accept(logits, tokens, np.array([[-1, 0, 1]], np.int32))
    assert list(am[0]) == [0, 0, 1]


def expected_accept_length(parent: np.ndarray, p_eff: float) -> float:
    """E[a] when every non-root node independently carries its parent's target token with probability p_eff:
    with F_i(d) = P(consistent descendants of i reach at most d levels below i),
    F_i(d) = prod_{c child of i} (1 - p_eff + p_eff * F_c(d - 1)), F_c(-1) = 0, and E[a] = sum_{d>=1} (1 - F_0(d-1))."""
    T = len(parent)
    children = [[] for _ in range(T)]
    for i in range(1, T):
        children[parent[i]].append(i)
    maxd = T
    F = np.ones((T, maxd + 1))
    for i in reversed(range(T)):
        for d in range(maxd + 1):
            prod = 1.0
            for c in children[i]:
                Fc = F[c, d - 1] if d >= 1 else 0.0
                prod *= 1.0 - p_eff + p_eff * Fc
            F[i, d] = prod
    return float(sum(1.0 - F[0, d - 1] for d in range(1, maxd + 1)))


def pin_accept_expected_length(orc):
    """Statistical pin: the mean accepted length over many independent token draws matches the exact
    expectation of the independent-agreement model (within 4 standard errors)."""
    rng = np.random.default_rng(24)
    T, V, p, N = 16, 8, 0.7, 20000
    parent = W.random_tree(rng, T, 4, 3)
    row = rng.standard_normal((T, V)).astype(np.float32)
    am = np.argmax(row, axis=1)
    logits = np.broadcast_to(row, (N, T, V)).copy()
    hit = rng.random((N, T)) < p
    uni = rng.integers(0, V, size=(N, T))
    tokens = np.where(hit, am[np.maximum(parent, 0)][None, :], uni).astype(np.int32)
    alen, _, _, _ = orc.tree_accept(logits, tokens, np.tile(parent, (N, 1)))
    exact = expected_accept_length(parent, p + (1 - p) / V)
    se = alen.std() / np.sqrt(N)
    assert abs(alen.mean() - exact) <= 4 * se, (alen.mean(), exact, se)


ACCEPT_PINS = [pin_accept_bruteforce, pin_accept_golden_chain, pin_accept_chain_rule, pin_accept_special_cases,
               pin_accept_signed_zero_ties, pin_accept_expected_length]


# ---------------------------------------------------------------------------------------------- commit pins
def pin_commit_gather(orc):
    """Direct gather from a snapshot: slot L+k <- old slot L+path[k] for k <= a; everything else untouched;
    includes aliasing paths such as [0, 2, 5] (slot L+2 is both a source and a destination)."""
    rng = np.random.default_rng(31)
    for dtype in (np.uint16, np.float32):
        NL, B, Hkv, T, D = 3, 4, 2, 9, 8
        S = 64
        # paths of the tree with parent array [-1, 0, 0, 2, 1, 3, 5, 5, 6]
        paths = [[0, 2, 5, 7], [0], [0, 1, 4], [0, 2, 3]]
        kv_in = np.array([10, 0, 33, 54], np.int32)
        alen = np.array([len(p) - 1 for p in paths], np.int32)
        path = np.full((B, T), -1, np.int32)
        for b, p in enumerate(paths):
            path[b, :len(p)] = p
        if dtype == np.uint16:
            k = rng.integers(0, 65535, size=(NL, B, Hkv, S, D)).astype(np.uint16)
            v = rng.integers(0, 65535, size=(NL, B, Hkv, S, D)).astype(np.uint16)
        else:
            k = rng.standard_normal((NL, B, Hkv, S, D)).astype(np.float32)
            v = rng.standard_normal((NL, B, Hkv, S, D)).astype(np.float32)
        k0, v0 = k.copy(), v.copy()
        out = orc.kv_commit(k, v, kv_in, path, alen)
        ek, ev = k0.copy(), v0.copy()
        for b, p in enumerate(paths):
            L = kv_in[b]
            ek[:, b, :, L:L + len(p)] = k0[:, b][:, :, L + np.array(p)]
            ev[:, b, :, L:L + len(p)] = v0[:, b][:, :, L + np.array(p)]
        assert np.array_equal(k.view(np.uint8), ek.view(np.uint8)) and np.array_equal(v.view(np.uint8), ev.view(np.uint8))
        assert list(out) == [kv_in[b] + alen[b] + 1 for b in range(B)]


def pin_commit_composition(orc):
    """After commit, one decode step of the last accepted node's query over the committed cache (prefix of
    length L+a, then the node itself) equals that node's row of the tree attention before the commit."""
    rng = np.random.default_rng(32)
    for trial in range(6):
        T, D, Hkv, Hq, L = 20, 16, 2, 4, 25
        parent = W.random_tree(rng, T, 5, 3)
        q, k, v = random_inputs(rng, 1, Hq, Hkv, T, D, L, extra=5)
        logits = rng.standard_normal((1, T, 6)).astype(np.float32)
        am = np.argmax(logits[0], axis=1)
        tok = np.array([0] + [am[parent[i]] if rng.random() < 0.8 else rng.integers(6) for i in range(1, T)],
                       dtype=np.int32)[None]
        alen, path, _, _ = orc.tree_accept(logits, tok, parent[None])
        a, last = int(alen[0]), int(path[0, alen[0]])
        o_tree, lse_tree = orc.tree_attn(q, k, v, np.array([L], np.int32), parent[None], 0.25, Hkv)
        kc, vc = k[None].copy(), v[None].copy()
        out_len = orc.kv_commit(kc, vc, np.array([L], np.int32), path, alen)
        assert out_len[0] == L + a + 1
        o_dec, lse_dec = orc.tree_attn(q[:, :, last:last + 1], kc[0], vc[0], np.array([L + a], np.int32),
                                       np.array([[-1]], np.int32), 0.25, Hkv)
        assert np.max(np.abs(o_dec[0, :, 0] - o_tree[0, :, last])) <= 1e-12, trial
        assert np.max(np.abs(lse_dec[0, :, 0] - lse_tree[0, :, last])) <= 1e-12, trial


COMMIT_PINS = [pin_commit_gather, pin_commit_composition]


# ------------------------------------------------------------------------------------- attention entropy
def _visible_counts(parent, L):
    """Number of slots each node sees: the L prefix slots plus its ancestors-or-self."""
    C = ancestor_closure(parent)
    return L + C.sum(axis=1)


def pin_entropy_uniform_is_log_count(orc):
    """Equal keys make every visible score equal, so a row's attention is uniform over its n visible slots and
    its entropy is exactly ln n (the maximum); prefix-free rows of a chain see depth+1 slots."""
    rng = np.random.default_rng(41)
    for L, T in ((0, 1), (0, 9), (13, 12), (40, 33)):
        parent = W.random_tree(rng, T, max(1, min(5, T - 1)), 3)[None] if T > 1 else np.array([[-1]], np.int32)
        q, k, _ = random_inputs(rng, 1, 4, 2, T, 8, L)
        kc = np.broadcast_to(k[:, :, :1], k.shape).copy()
        ent = orc.tree_attn_entropy(q, kc, np.array([L], np.int32), parent, 0.3, 2)
        n = _visible_counts(parent[0], L)
        for h in range(4):
            assert np.max(np.abs(ent[0, h] - np.log(n))) <= 1e-12, (L, T, h)


def pin_entropy_two_slots_closed_form(orc):
    """A single node over one prefix slot sees two keys with score gap d: the binary entropy
    H = ln(1 + e^-d) + d e^-d / (1 + e^-d) (written for d >= 0 by symmetry)."""
    rng = np.random.default_rng(42)
    for trial in range(20):
        D = 8
        q, k, _ = random_inputs(rng, 1, 1, 1, 1, D, 1)
        q *= rng.uniform(0.1, 3.0)
        scale = 0.5
        ent = orc.tree_attn_entropy(q, k, np.array([1], np.int32), np.array([[-1]], np.int32), scale, 1)
        qd, kd = q[0, 0, 0].astype(np.float64), k[0, 0].astype(np.float64)
        d = abs(scale * (qd @ kd[1] - qd @ kd[0]))
        H = np.log1p(np.exp(-d)) + d * np.exp(-d) / (1.0 + np.exp(-d))
        assert abs(ent[0, 0, 0] - H) <= 1e-12, trial


def pin_entropy_one_slot_is_zero(orc):
    """A root with an empty prefix sees only itself: its attention is one-hot, entropy 0; a one-hot row also
    results when one score dominates all others by far."""
    rng = np.random.default_rng(43)
    q, k, _ = random_inputs(rng, 2, 2, 1, 5, 8, 0)
    parent = np.array([[-1, 0, 1, 2, 3]] * 2, np.int32)
    ent = orc.tree_attn_entropy(q, k, np.array([0, 0], np.int32), parent, 0.25, 1)
    assert np.all(ent[:, :, 0] == 0.0)
    kb = k.copy()
    kb[:, :, 3] = q[:, 0:1, 3] * 1000.0   # node 3's own key dominates its row
    ent = orc.tree_attn_entropy(q[:, :1], kb, np.array([0, 0], np.int32), parent, 1.0, 1)
    assert np.all(ent[:, 0, 3] <= 1e-200)


def pin_entropy_bruteforce_and_bounds(orc):
    """Dense masked softmax (closure-built mask, scipy logsumexp) then -sum p log p agrees to 1e-11; every
    entropy lies in [0, ln n]; the values V play no part."""
    rng = np.random.default_rng(44)
    for trial in range(4):
        B, Hq, Hkv, T, D = 2, 4, 2, int(rng.integers(1, 18)), 8
        Ls = [int(rng.integers(0, 30)), int(rng.integers(0, 30))]
        S = max(Ls) + T
        q = rng.standard_normal((B, Hq, T, D)).astype(np.float32)
        k = rng.standard_normal((B, Hkv, S, D)).astype(np.float32)
        parent = np.stack([random_parent(rng, T) for _ in range(B)])
        kv = np.array(Ls, np.int32)
        ent = orc.tree_attn_entropy(q, k, kv, parent, 0.45, Hkv)
        for b in range(B):
            L = Ls[b]
            C = ancestor_closure(parent[b])
            vis = np.concatenate([np.ones((T, L), dtype=bool), C], axis=1)
            n = vis.sum(axis=1)
            for h in range(Hq):
                sc = 0.45 * (q[b, h].astype(np.float64) @ k[b, h // (Hq // Hkv), :L + T].astype(np.float64).T)
                sc[~vis] = -np.inf
                logp = sc - logsumexp(sc, axis=1)[:, None]
                H = -np.sum(np.where(vis, np.exp(logp) * np.where(vis, logp, 0.0), 0.0), axis=1)
                assert np.max(np.abs(ent[b, h] - H)) <= 1e-11, (trial, b, h)
                assert np.all(ent[b, h] >= -1e-15) and np.all(ent[b, h] <= np.log(n) + 1e-12)


def pin_entropy_nonancestor_invariance(orc):
    """A row's entropy ignores every key it cannot see: changing a non-ancestor tree key leaves it bitwise
    unchanged, while changing an ancestor's key moves it."""
    rng = np.random.default_rng(45)
    L, T, D = 9, 15, 8
    q, k, _ = random_inputs(rng, 1, 2, 2, T, D, L)
    parent = W.random_tree(rng, T, 4, 3)[None]
    kv = np.array([L], np.int32)
    ent = orc.tree_attn_entropy(q, k, kv, parent, 0.5, 2)
    C = ancestor_closure(parent[0])
    for j in range(1, T):
        k2 = k.copy()
        k2[0, :, L + j] += 0.75
        ent2 = orc.tree_attn_entropy(q, k2, kv, parent, 0.5, 2)
        for i in range(T):
            if C[i, j]:
                assert np.all(ent2[0, :, i] != ent[0, :, i]), (i, j)
            else:
                assert np.array_equal(ent2[0, :, i], ent[0, :, i]), (i, j)


def pin_entropy_layer_choice(orc):
    """AE is the plain mean of the rows' entropies; the distillation layer minimises AE(l) + |AE(l) - AE(l-1)|
    over the layers that have a predecessor, the first such layer on ties (hand-worked cases)."""
    import oracle as O
    assert O.attn_entropy_mean([[1.0, 2.0], [3.0, 6.0]]) == 3.0
    # scores for l = 1..4: 4+1, 4.5+0.5, 1+3.5, 1.5+0.5 -> layer 4
    assert O.attn_entropy_select([5.0, 4.0, 4.5, 1.0, 1.5]) == 4
    # a flat profile: every score equals AE, the first candidate wins
    assert O.attn_entropy_select([2.0, 2.0, 2.0]) == 1
    # low entropy but a jump: layer 2 scores 0.5 + 3.5 = 4, layer 1 scores 4 + 0 = 4, tie -> 1
    assert O.attn_entropy_select([4.0, 4.0, 0.5]) == 1
    assert O.attn_entropy_select([3.0, 2.0]) == 1


ENTROPY_PINS = [pin_entropy_uniform_is_log_count, pin_entropy_two_slots_closed_form, pin_entropy_one_slot_is_zero,
                pin_entropy_bruteforce_and_bounds, pin_entropy_nonancestor_invariance, pin_entropy_layer_choice]


# ---------------------------------------------------------------------------------- visual-token selection
def pin_visual_bruteforce(orc):
    """Column means of the dense masked softmax (closure-built mask, scipy logsumexp) over every head and row
    agree to 1e-13 for any visual range, including one that runs past a sequence's prefix (those are 0)."""
    rng = np.random.default_rng(51)
    for trial in range(4):
        B, Hq, Hkv, T, D = 2, 6, 3, int(rng.integers(1, 20)), 8
        Ls = [int(rng.integers(5, 40)), int(rng.integers(5, 40))]
        S = max(Ls) + T
        q = rng.standard_normal((B, Hq, T, D)).astype(np.float32)
        k = rng.standard_normal((B, Hkv, S, D)).astype(np.float32)
        parent = np.stack([random_parent(rng, T) for _ in range(B)])
        kv = np.array(Ls, np.int32)
        v0 = int(rng.integers(0, 5))
        nv = int(rng.integers(1, S - v0))
        imp = orc.visual_importance(q, k, kv, parent, 0.6, Hkv, v0, nv)
        for b in range(B):
            L = Ls[b]
            C = ancestor_closure(parent[b])
            vis = np.concatenate([np.ones((T, L), dtype=bool), C], axis=1)
            colsum = np.zeros(L + T)
            for h in range(Hq):
                sc = 0.6 * (q[b, h].astype(np.float64) @ k[b, h // (Hq // Hkv), :L + T].astype(np.float64).T)
                sc[~vis] = -np.inf
                colsum += np.exp(sc - logsumexp(sc, axis=1)[:, None]).sum(axis=0)
            ref = np.zeros(nv)
            for j in range(nv):
                if v0 + j < L:
                    ref[j] = colsum[v0 + j] / (Hq * T)
            assert np.max(np.abs(imp[b] - ref)) <= 1e-13, (trial, b)


def pin_visual_uniform_closed_form(orc):
    """Equal keys: row i of every head spreads 1/n_i over its n_i visible slots, so a prefix token's
    importance is the mean of 1/n_i over the rows (and 0 past the prefix)."""
    rng = np.random.default_rng(52)
    L, T = 30, 11
    parent = W.random_tree(rng, T, 4, 3)[None]
    q, k, _ = random_inputs(rng, 1, 4, 2, T, 8, L)
    kc = np.broadcast_to(k[:, :, :1], k.shape).copy()
    imp = orc.visual_importance(q, kc, np.array([L], np.int32), parent, 0.3, 2, 0, L + 5)
    n = L + ancestor_closure(parent[0]).sum(axis=1)
    assert np.max(np.abs(imp[0, :L] - np.mean(1.0 / n))) <= 1e-15
    assert np.all(imp[0, L:] == 0.0)


def pin_visual_mass_balance(orc):
    """Over the whole prefix, the importances sum to one minus the mean attention mass on tree slots; that mass
    is the attention output for values that are 1 on tree slots and 0 on prefix slots (the attention oracle,
    an independent route)."""
    rng = np.random.default_rng(53)
    B, Hq, Hkv, T, D, L = 2, 4, 2, 13, 8, 17
    q, k, _ = random_inputs(rng, B, Hq, Hkv, T, D, L)
    q *= 2.0
    parent = np.stack([W.random_tree(rng, T, 5, 3) for _ in range(B)])
    kv = np.array([L, L], np.int32)
    imp = orc.visual_importance(q, k, kv, parent, 0.5, Hkv, 0, L)
    ind = np.zeros((B, Hkv, L + T, D), np.float32)
    ind[:, :, L:] = 1.0
    tree_mass, _ = orc.tree_attn(q, k, ind, kv, parent, 0.5, Hkv)
    for b in range(B):
        assert abs(imp[b].sum() - (1.0 - tree_mass[b, :, :, 0].mean())) <= 1e-13


def pin_visual_topk_and_gather(orc):
    """Top-r against a lexicographic sort (value descending, index ascending) on values with many exact ties,
    r from 1 to all; the gather against numpy fancy indexing, bit for bit."""
    rng = np.random.default_rng(54)
    for trial in range(20):
        B, n = 3, int(rng.integers(1, 60))
        vals = (rng.integers(0, 6, size=(B, n)) / 4.0).astype(np.float32)
        for r in sorted({1, n, int(rng.integers(1, n + 1))}):
            keep = orc.visual_topk(vals, r)
            for b in range(B):
                order = np.lexsort((np.arange(n), -vals[b].astype(np.float64)))
                assert np.array_equal(keep[b], np.sort(order[:r])), (trial, b, r)
    B, Hkv, S, D, v0 = 2, 3, 40, 16, 4
    kc = rng.integers(0, 65536, size=(B, Hkv, S, D), dtype=np.uint16)
    vc = rng.integers(0, 65536, size=(B, Hkv, S, D), dtype=np.uint16)
    keep = np.sort(np.stack([rng.choice(S - v0, 9, replace=False) for _ in range(B)]), axis=1).astype(np.int32)
    ko, vo = orc.visual_gather(kc, vc, v0, keep)
    for b in range(B):
        assert np.array_equal(ko[b], kc[b][:, v0 + keep[b]]) and np.array_equal(vo[b], vc[b][:, v0 + keep[b]])


VISUAL_PINS = [pin_visual_bruteforce, pin_visual_uniform_closed_form, pin_visual_mass_balance,
               pin_visual_topk_and_gather]


# ----------------------------------------------------------------------------- prefill statistics (causal)
def _prefill_inputs(rng, B, Hq, Hkv, N, D, S_cap):
    q = rng.standard_normal((B, Hq, N, D)).astype(np.float32)
    k = rng.standard_normal((B, Hkv, S_cap, D)).astype(np.float32)
    return q, k


def pin_prefill_uniform_closed_form(orc):
    """Equal keys: prompt row i spreads 1/(i+1) over slots 0..i, so lse_i = s_i + ln(i+1) (s_i = scale q_i.k),
    its entropy is ln(i+1), and slot j's importance is (1/n) sum_{i=j}^{n-1} 1/(i+1) = (H_n - H_j)/n with
    harmonic numbers H (0 at or past n); rows at or past n are not queries.  Ragged prompts, an offset window
    and grouped heads."""
    rng = np.random.default_rng(61)
    B, Hq, Hkv, N, D, S = 3, 4, 2, 23, 8, 29
    q, k = _prefill_inputs(rng, B, Hq, Hkv, N, D, S)
    kc = np.broadcast_to(k[:, :, :1], k.shape).copy()
    lens = np.array([23, 9, 1], np.int32)
    scale = 0.4
    lse, ent = orc.prefill_attn_stats(q, kc, lens, scale, Hkv)
    for b in range(B):
        n = int(lens[b])
        for h in range(Hq):
            s = scale * (q[b, h, :n].astype(np.float64) @ kc[b, h // 2, 0].astype(np.float64))
            i = np.arange(n)
            assert np.max(np.abs(lse[b, h, :n] - (s + np.log(i + 1.0)))) <= 1e-12, (b, h)
            assert np.max(np.abs(ent[b, h, :n] - np.log(i + 1.0))) <= 1e-12, (b, h)
            assert np.all(lse[b, h, n:] == -np.inf) and np.all(ent[b, h, n:] == 0.0)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, S + 1))])   # H[m] = 1 + 1/2 + ... + 1/m
    for v0, nv in ((0, S), (5, 11)):
        imp = orc.prefill_visual_importance(q, kc, lens, scale, Hkv, v0, nv)
        for b in range(B):
            n = int(lens[b])
            j = v0 + np.arange(nv)
            ref = np.where(j < n, (H[n] - H[np.minimum(j, n)]) / n, 0.0)
            assert np.max(np.abs(imp[b] - ref)) <= 1e-14, (b, v0)


def pin_prefill_mass_balance(orc):
    """Every prompt row's attention sums to one, so over a window covering the whole prompt the importances of a
    sequence sum to one (the mean over its Hq*n rows), whatever the scores; an empty prompt has none."""
    rng = np.random.default_rng(62)
    B, Hq, Hkv, N, D, S = 4, 6, 3, 31, 8, 32
    q, k = _prefill_inputs(rng, B, Hq, Hkv, N, D, S)
    q *= 3.0
    lens = np.array([31, 17, 0, 2], np.int32)
    imp = orc.prefill_visual_importance(q, k, lens, 0.5, Hkv, 0, S)
    for b in range(B):
        expect = 1.0 if lens[b] > 0 else 0.0
        assert abs(imp[b].sum() - expect) <= 1e-13, b
        assert np.all(imp[b, lens[b]:] == 0.0) and np.all(imp[b] >= 0.0)


def pin_prefill_chain_tree_agrees(orc):
    """A prompt's rows L0..n-1 are the rows of a chain-shaped tree of n - L0 nodes over a committed prefix of L0
    slots (node t at slot L0 + t sees the prefix and nodes 0..t): their lse and entropy equal the tree oracle's
    (itself pinned to brute force and to library causal attention).  Telescoping the importance over prompt
    lengths L0 and n leaves exactly the tree rows, so for a prefix slot j < L0,
    n I_j(n) - L0 I_j(L0) = T I_j(tree)."""
    rng = np.random.default_rng(63)
    for B, Hq, Hkv, N, D, L0 in ((2, 4, 2, 40, 16, 25), (1, 3, 1, 12, 8, 0), (1, 2, 2, 70, 8, 5)):
        S = N + 3
        q, k = _prefill_inputs(rng, B, Hq, Hkv, N, D, S)
        T = N - L0
        lens = np.full(B, N, np.int32)
        lse, ent = orc.prefill_attn_stats(q, k, lens, 0.35, Hkv)
        chain = np.tile(W.chain_tree(T)[None], (B, 1))
        kv = np.full(B, L0, np.int32)
        qt = np.ascontiguousarray(q[:, :, L0:N])
        vv = np.zeros_like(k)
        _, lse_t = orc.tree_attn(qt, k, vv, kv, chain, 0.35, Hkv)
        ent_t = orc.tree_attn_entropy(qt, k, kv, chain, 0.35, Hkv)
        assert np.max(np.abs(lse[:, :, L0:N] - lse_t)) <= 1e-12
        assert np.max(np.abs(ent[:, :, L0:N] - ent_t)) <= 1e-12
        if L0 > 0:
            imp_n = orc.prefill_visual_importance(q, k, lens, 0.35, Hkv, 0, L0)
            imp_0 = orc.prefill_visual_importance(q, k, np.full(B, L0, np.int32), 0.35, Hkv, 0, L0)
            imp_t = orc.visual_importance(qt, k, kv, chain, 0.35, Hkv, 0, L0)
            assert np.max(np.abs(N * imp_n - L0 * imp_0 - T * imp_t)) <= 1e-12


def pin_prefill_single_and_two_slots(orc):
    """Row 0 sees only slot 0: lse = s_00, entropy 0; with a one-token prompt slot 0 has importance 1.  Row 1
    sees two slots with score gap d: the binary entropy ln(1 + e^-d) + d e^-d / (1 + e^-d), d >= 0."""
    rng = np.random.default_rng(64)
    B, Hq, Hkv, N, D, S = 2, 2, 1, 6, 8, 6
    for trial in range(10):
        q, k = _prefill_inputs(rng, B, Hq, Hkv, N, D, S)
        q *= rng.uniform(0.2, 3.0)
        lse, ent = orc.prefill_attn_stats(q, k, np.array([6, 2], np.int32), 0.5, Hkv)
        for b in range(B):
            for h in range(Hq):
                qd, kd = q[b, h].astype(np.float64), k[b, 0].astype(np.float64)
                assert abs(lse[b, h, 0] - 0.5 * (qd[0] @ kd[0])) <= 1e-13
                assert ent[b, h, 0] == 0.0
                d = abs(0.5 * (qd[1] @ kd[1] - qd[1] @ kd[0]))
                Hb = np.log1p(np.exp(-d)) + d * np.exp(-d) / (1.0 + np.exp(-d))
                assert abs(ent[b, h, 1] - Hb) <= 1e-12, (trial, b, h)
        imp = orc.prefill_visual_importance(q, k, np.array([1, 1], np.int32), 0.5, Hkv, 0, 3)
        assert np.array_equal(imp, np.array([[1.0, 0.0, 0.0]] * B))


def pin_prefill_layer_entropy_mean(orc):
    """AE over prompts with equal keys: row i has entropy ln(i+1), so the mean over the sum(n_b) rows of every
    head is sum_b ln(n_b!) / sum_b n_b (log-gamma); each row counts once whatever the padding N."""
    from math import lgamma
    import oracle as oracle_mod
    rng = np.random.default_rng(65)
    B, Hq, Hkv, N, D, S = 3, 4, 4, 40, 8, 40
    q, k = _prefill_inputs(rng, B, Hq, Hkv, N, D, S)
    kc = np.broadcast_to(k[:, :, :1], k.shape).copy()
    lens = np.array([40, 7, 19], np.int32)
    _, ent = orc.prefill_attn_stats(q, kc, lens, 0.3, Hkv)
    ae = oracle_mod.prefill_attn_entropy_mean(ent, lens)
    ref = sum(lgamma(int(n) + 1) for n in lens) / float(lens.sum())
    assert abs(ae - ref) <= 1e-12


PREFILL_PINS = [pin_prefill_uniform_closed_form, pin_prefill_mass_balance, pin_prefill_chain_tree_agrees,
                pin_prefill_single_and_two_slots, pin_prefill_layer_entropy_mean]


# ------------------------------------------------------------------------------------ sampled acceptance
def _softmax(logits, tau):
    z = np.asarray(logits, dtype=np.float64) / tau
    z -= z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def _sample(rng, probs):
    """One index per row of `probs` (fp64 rows summing to 1), by inverse CDF of numpy uniforms."""
    c = np.cumsum(probs, axis=-1)
    u = rng.random(probs.shape[:-1])[..., None] * c[..., -1:]
    return np.minimum((c <= u).sum(axis=-1), probs.shape[-1] - 1)


def _emitted(tokens, path, alen, nxt, b):
    return [int(tokens[b, path[b, d]]) for d in range(1, alen[b] + 1)] + [int(nxt[b])]


def _chi2_ok(counts, expected, floor=1e-6):
    from scipy.stats import chi2
    keep = expected > 0
    assert np.all(counts[~keep] == 0), "a token of probability zero was emitted"
    stat = float((((counts - expected) ** 2)[keep] / expected[keep]).sum())
    dof = int(keep.sum()) - 1
    return chi2.sf(stat, dof) > floor, stat, dof


def pin_sampled_single_child_closed_form(orc):
    """One child of token x: accepted iff u < p(x)/q(x); on rejection the emitted token is the inverse CDF of
    max(p - q, 0) / sum(max(p - q, 0)) at u0 (values written out by hand from the two distributions)."""
    tau = 0.8
    tl = np.log(np.array([0.10, 0.45, 0.05, 0.40])) * tau          # p = [0.10, 0.45, 0.05, 0.40]
    dl = np.log(np.array([0.40, 0.20, 0.30, 0.10])) * tau          # q = [0.40, 0.20, 0.30, 0.10]
    p, q = _softmax(tl, tau), _softmax(dl, tau)
    np.testing.assert_allclose(p, [0.10, 0.45, 0.05, 0.40], rtol=1e-6)
    # max(p - q, 0) = [0, .25, 0, .30]: token 1 for u0 < .25/.55, token 3 above (u0 = 0 must give 1, not 0)
    parent = np.array([[-1, 0]], np.int32)
    cases = []
    for x in range(4):
        ratio = p[x] / q[x]
        for u1 in (0.999 * ratio, 1.001 * ratio, 0.0, 0.99999):
            if not u1 < 1.0:
                continue
            for u0 in (0.0, 0.2, 0.5, 0.9):
                cases.append((x, u1, u0))
    for x, u1, u0 in cases:
        tok = np.array([[0, x]], np.int32)
        uni = np.array([[u0, u1]], np.float32)
        alen, path, nxt = orc.tree_accept_sampled(tl[None, None].repeat(2, 1).astype(np.float32),
                                                  dl[None, None].repeat(2, 1).astype(np.float32), tok, parent,
                                                  uni, tau)
        if float(np.float32(u1)) < p[x] / q[x]:
            assert alen[0] == 1 and list(path[0]) == [0, 1], (x, u1)
            # the child is a leaf: its token follows the target's distribution at the child (row 1 = p)
            assert nxt[0] == int(np.searchsorted(np.cumsum(p), np.float32(u0), side="right")), (x, u1, u0)
        else:
            assert alen[0] == 0 and list(path[0]) == [0, -1], (x, u1)
            want = 1 if np.float32(u0) < 0.25 / 0.55 else 3   # the residual's support is {1, 3}
            assert nxt[0] == want, (x, u1, u0, nxt[0], want)


def pin_sampled_repeated_token_never_accepted_twice(orc):
    """Siblings carrying the same token x: once x is rejected its residual mass is zero, so every later copy is
    rejected too, whatever its uniform."""
    rng = np.random.default_rng(41)
    B, V, tau = 2000, 6, 1.0
    tl = rng.standard_normal((B, 4, V)).astype(np.float32)
    dl = rng.standard_normal((B, 4, V)).astype(np.float32)
    x = rng.integers(0, V, size=B)
    tok = np.stack([np.zeros(B, int), x, x, x], axis=1).astype(np.int32)
    parent = np.tile(np.array([-1, 0, 0, 0], np.int32), (B, 1))
    uni = rng.random((B, 4)).astype(np.float32)
    alen, path, nxt = orc.tree_accept_sampled(tl, dl, tok, parent, uni, tau)
    assert np.all(path[alen == 1, 1] == 1)              # only the first copy can be accepted
    assert np.all(nxt[alen == 0] != x[alen == 0])       # and the rejected token is never emitted instead
    assert 0 < (alen == 1).sum() < B


def pin_sampled_low_temperature_is_greedy(orc):
    """As tau -> 0 both distributions become one-hot at their argmax; with integer logits spaced >= 1 and
    tau = 1e-3 every other probability underflows to exactly zero, and with distinct sibling tokens the
    sampled walk accepts exactly the greedy rule's path and bonus token, for any uniforms."""
    rng = np.random.default_rng(42)
    B, T, V = 300, 20, 12
    parent = np.stack([W.random_tree(rng, T, int(rng.integers(2, 8)), 4) for _ in range(B)])
    tl = np.stack([rng.permutation(V) for _ in range(B * T)]).reshape(B, T, V).astype(np.float32)
    dl = np.stack([rng.permutation(V) for _ in range(B * T)]).reshape(B, T, V).astype(np.float32)
    am = tl.argmax(axis=2)
    tok = np.zeros((B, T), np.int32)
    for b in range(B):
        used = {}
        for i in range(1, T):
            sib = used.setdefault(int(parent[b, i]), set())
            # agree with the parent's target token half of the time, never repeat a sibling's token
            choice = int(am[b, parent[b, i]]) if rng.random() < 0.6 else int(rng.integers(0, V))
            while choice in sib:
                choice = int(rng.integers(0, V))
            sib.add(choice)
            tok[b, i] = choice
    uni = rng.random((B, T)).astype(np.float32)
    alen, path, nxt = orc.tree_accept_sampled(tl, dl, tok, parent, uni, 1e-3)
    galen, gpath, gnxt, _ = orc.tree_accept(tl, tok, parent)
    np.testing.assert_array_equal(alen, galen)
    np.testing.assert_array_equal(path, gpath)
    np.testing.assert_array_equal(nxt, gnxt)


def pin_sampled_identical_models(orc):
    """Draft == target: every tested child is accepted (u q(x) < q(x) for u < 1), so the walk follows
    first children to a leaf and emits a token drawn from the leaf's distribution at u0."""
    rng = np.random.default_rng(43)
    B, T, V, tau = 200, 15, 9, 0.7
    parent = np.stack([random_parent(rng, T, max_branch=3) for _ in range(B)])
    tl = rng.standard_normal((B, T, V)).astype(np.float32)
    tok = rng.integers(0, V, size=(B, T)).astype(np.int32)
    uni = rng.random((B, T)).astype(np.float32)
    alen, path, nxt = orc.tree_accept_sampled(tl, tl, tok, parent, uni, tau)
    for b in range(B):
        node, walk = 0, [0]
        while True:
            kids = [c for c in range(T) if parent[b, c] == node]
            if not kids:
                break
            node = kids[0]
            walk.append(node)
        assert alen[b] == len(walk) - 1 and list(path[b, :len(walk)]) == walk
        cdf = np.cumsum(_softmax(tl[b, node], tau))
        assert nxt[b] == int(np.searchsorted(cdf, float(uni[b, 0]) * cdf[-1], side="right"))


def _markov_tree_step(orc, rng, P_tab, Q_tab, roots, width, depth2, tau):
    """One verification step per root token: a tree whose root has `width` children drawn i.i.d. from the
    draft's distribution after the root, each with `depth2` children drawn i.i.d. from the draft's distribution
    after it.  Target and draft logits depend only on a node's own token (a Markov model)."""
    B = len(roots)
    T = 1 + width + width * depth2
    parent = np.full(T, -1, np.int32)
    for c in range(width):
        parent[1 + c] = 0
        for g in range(depth2):
            parent[1 + width + c * depth2 + g] = 1 + c
    tok = np.zeros((B, T), np.int32)
    tok[:, 0] = roots
    V = P_tab.shape[0]
    qprob = _softmax(Q_tab, tau)
    for c in range(width):
        tok[:, 1 + c] = _sample(rng, qprob[tok[:, 0]])
        for g in range(depth2):
            tok[:, 1 + width + c * depth2 + g] = _sample(rng, qprob[tok[:, 1 + c]])
    tl = P_tab[tok].astype(np.float32)
    dl = Q_tab[tok].astype(np.float32)
    uni = rng.random((B, T)).astype(np.float32)
    alen, path, nxt = orc.tree_accept_sampled(tl, dl, tok, np.tile(parent, (B, 1)), uni, tau)
    assert tl.shape == (B, T, V)
    return tok, alen, path, nxt


def pin_sampled_output_distribution(orc):
    """The defining property of speculative sampling: whatever the draft, the emitted tokens follow the
    target's own distribution.  With a Markov target P(. | previous token) the first two emitted tokens after a
    root r0 have the joint law P(x1 | r0) P(x2 | x1); a step that emits one token is followed by a fresh step
    rooted at it.  Chi-square test over all V^2 cells, at two temperatures; also the acceptance rate of the
    first child equals sum_x min(p(x), q(x)) within 5 standard errors."""
    rng = np.random.default_rng(44)
    V, N = 4, 30000
    P_tab = rng.standard_normal((V, V)) * 1.5
    Q_tab = rng.standard_normal((V, V)) * 1.5
    for tau in (1.0, 0.6):
        P = _softmax(P_tab, tau)
        Q = _softmax(Q_tab, tau)
        r0 = 2
        roots = np.full(N, r0, np.int32)
        tok, alen, path, nxt = _markov_tree_step(orc, rng, P_tab, Q_tab, roots, 3, 2, tau)
        pairs = np.full((N, 2), -1)
        short = []
        for b in range(N):
            e = _emitted(tok, path, alen, nxt, b)
            if len(e) >= 2:
                pairs[b] = e[:2]
            else:
                pairs[b, 0] = e[0]
                short.append(b)
        if short:
            tok2, alen2, path2, nxt2 = _markov_tree_step(orc, rng, P_tab, Q_tab, pairs[short, 0].astype(np.int32),
                                                         2, 1, tau)
            for k, b in enumerate(short):
                pairs[b, 1] = _emitted(tok2, path2, alen2, nxt2, k)[0]
        counts = np.zeros((V, V))
        np.add.at(counts, (pairs[:, 0], pairs[:, 1]), 1)
        expected = N * P[r0][:, None] * P
        ok, stat, dof = _chi2_ok(counts.ravel(), expected.ravel())
        assert ok, (tau, stat, dof)
        # acceptance rate of the first child, drawn from q: sum_x min(p(x), q(x))
        first_acc = (alen >= 1) & (path[:, 1] == 1)
        rate = np.minimum(P[r0], Q[r0]).sum()
        se = np.sqrt(rate * (1 - rate) / N)
        assert abs(first_acc.mean() - rate) <= 5 * se, (tau, first_acc.mean(), rate)


# --------------------------------------------------------------------------------------- LM head + argmax
def _bf16_bits(x):
    b = np.asarray(x, dtype=np.float32).view(np.uint32)
    assert np.all((b & 0xFFFF) == 0), "test values must be exactly representable in bf16"
    return (b >> 16).astype(np.uint16)


def pin_lm_head_one_hot_weights(orc):
    """Weight rows that are scaled unit vectors pick single hidden entries: logit[m, v] = c_v * h[m, k_v]
    exactly (V != H, so a transposed operand fails by shape or by value)."""
    import oracle as O
    rng = np.random.default_rng(51)
    M, H, V = 7, 24, 40
    h = rng.choice(np.array([-2.0, -0.5, 0.25, 1.0, 3.0], np.float32), size=(M, H))
    k = rng.integers(0, H, size=V)
    c = rng.choice(np.array([-1.0, 0.5, 2.0], np.float32), size=V)
    w = np.zeros((V, H), np.float32)
    w[np.arange(V), k] = c
    got = O.lm_head_logits(_bf16_bits(h), _bf16_bits(w))
    assert got.shape == (M, V)
    np.testing.assert_array_equal(got, h[:, k].astype(np.float64) * c.astype(np.float64))


def pin_lm_head_constant_closed_form(orc):
    """Constant operands: every logit is H * a * b exactly; and bf16 bit patterns decode exactly (1.0 is
    0x3F80, -2.5 is 0xC020)."""
    import oracle as O
    M, H, V = 3, 256, 5
    h = np.full((M, H), 0x3F80, np.uint16)          # 1.0
    w = np.full((V, H), 0xC020, np.uint16)          # -2.5
    np.testing.assert_array_equal(O.lm_head_logits(h, w), np.full((M, V), -2.5 * H))


def pin_lm_head_greedy_composition(orc):
    """With an identity LM head (V = H) and one-hot hidden states at planted tokens, the logits' argmax is the
    planted token of each node, and acceptance from the LM head equals the (separately pinned) greedy rule on
    those logits, row order [B, T] included."""
    import oracle as O
    rng = np.random.default_rng(52)
    B, T, H = 6, 12, 32
    parent = np.stack([W.random_tree(rng, T, 4, 3) for _ in range(B)])
    tgt = rng.integers(0, H, size=(B, T))
    hid = np.zeros((B, T, H), np.float32)
    np.put_along_axis(hid, tgt[:, :, None], 1.0, axis=2)
    logits = O.lm_head_logits(_bf16_bits(hid), _bf16_bits(np.eye(H, dtype=np.float32)))
    am = logits.argmax(axis=2)
    np.testing.assert_array_equal(am, tgt)
    tokens = np.where(rng.random((B, T)) < 0.7, tgt[np.arange(B)[:, None], np.maximum(parent, 0)],
                      rng.integers(0, H, (B, T))).astype(np.int32)
    got = O.tree_accept_from_argmax(am, tokens, parent)
    want = orc.tree_accept(logits.astype(np.float32), tokens, parent)[:3]
    for x, y in zip(got, want):
        np.testing.assert_array_equal(x, y)


LM_HEAD_PINS = [pin_lm_head_one_hot_weights, pin_lm_head_constant_closed_form, pin_lm_head_greedy_composition]

SAMPLED_PINS = [pin_sampled_single_child_closed_form, pin_sampled_repeated_token_never_accepted_twice,
                pin_sampled_low_temperature_is_greedy, pin_sampled_identical_models,
                pin_sampled_output_distribution]
ALL_PINS = (ATTN_PINS + ACCEPT_PINS + COMMIT_PINS + ENTROPY_PINS + VISUAL_PINS + PREFILL_PINS + SAMPLED_PINS
            + LM_HEAD_PINS)
