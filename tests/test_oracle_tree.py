"""Pins for the oracle's tree verification (draft trees of Sec. 3.1 checked
in the single parallel pass of Sec. 3.2; EAGLE-3 tree shape of App. A).

Masked attention is pinned to torch fp64 scaled_dot_product_attention with
an explicit boolean mask, to the block-causal oracle on chain-shaped trees,
and to single-token decoding along each node's root path (a cache rebuilt
from the ancestors' rows).  Tree acceptance is pinned to a brute-force walk
of every node's root path, to the chain acceptance rule, and to trees built
with a known accepted path.  Path compaction is pinned through attention: a
query over the compacted cache sees exactly what the tree mask showed it.
"""
import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle
import workloads as W


def _rand(shape, rng, std=1.0):
    return rng.standard_normal(shape) * std


def _random_parents(gamma, rng):
    par = np.full(gamma, -1, np.int32)
    for j in range(1, gamma):
        par[j] = rng.integers(0, j)
    return par


def _root_path(parents, i):
    path = [i]
    while path[-1] != 0:
        path.append(int(parents[path[-1]]))
    return path[::-1]


def _sdpa_masked(q, k, v, ctx_len, visible):
    """torch fp64 SDPA; visible [gamma][gamma] bool over the block keys."""
    gamma, hq, dh = q.shape
    hkv = k.shape[0]
    n = ctx_len + gamma
    group = hq // hkv
    kt = torch.from_numpy(k[:, :n]).repeat_interleave(group, dim=0)
    vt = torch.from_numpy(v[:, :n]).repeat_interleave(group, dim=0)
    qt = torch.from_numpy(q).transpose(0, 1).contiguous()
    mask = torch.ones((gamma, n), dtype=torch.bool)
    mask[:, ctx_len:] = torch.from_numpy(visible)
    out = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt,
                                                           attn_mask=mask)
    return out.transpose(0, 1).numpy()


TREES = [
    # gamma, ctx_len, n_q_heads, n_kv_heads, head_dim, seed
    (1, 9, 4, 2, 8, 1),
    (6, 0, 4, 2, 8, 2),
    (13, 21, 8, 2, 16, 3),
    (33, 40, 8, 4, 8, 4),
    (64, 17, 4, 1, 8, 5),
]


@pytest.mark.parametrize("gamma,ctx,hq,hkv,dh,seed", TREES)
def test_tree_attention_matches_torch_sdpa(gamma, ctx, hq, hkv, dh, seed):
    rng = np.random.default_rng(seed)
    par = _random_parents(gamma, rng)
    masks = W.ancestor_masks(par)
    visible = np.array([[(int(masks[i]) >> j) & 1 for j in range(gamma)]
                        for i in range(gamma)], bool)
    cap = ctx + gamma + 2
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    got = oracle.verify_attn_mask(q, k, v, ctx, masks)
    ref = _sdpa_masked(q, k, v, ctx, visible)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("gamma,ctx", [(1, 5), (8, 30), (16, 3), (64, 12)])
def test_chain_tree_is_block_causal(gamma, ctx):
    rng = np.random.default_rng(gamma + ctx)
    hq, hkv, dh = 8, 2, 16
    par = np.arange(-1, gamma - 1, dtype=np.int32)
    cap = ctx + gamma
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    got = oracle.verify_attn_mask(q, k, v, ctx, W.ancestor_masks(par))
    ref = oracle.verify_attn(q, k, v, ctx)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_each_node_equals_decode_along_its_root_path():
    """Row i of the tree equals a gamma = 1 decode whose cache is the cached
    prefix followed by the rows of i's ancestors and i, in depth order."""
    rng = np.random.default_rng(11)
    gamma, ctx, hq, hkv, dh = 24, 15, 8, 2, 16
    par = _random_parents(gamma, rng)
    cap = ctx + gamma
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    tree = oracle.verify_attn_mask(q, k, v, ctx, W.ancestor_masks(par))
    for i in range(gamma):
        path = _root_path(par, i)
        rows = list(range(ctx)) + [ctx + j for j in path]
        kp = np.ascontiguousarray(k[:, rows])
        vp = np.ascontiguousarray(v[:, rows])
        dec = oracle.verify_attn(np.ascontiguousarray(q[i:i + 1]), kp, vp,
                                 ctx + len(path) - 1)
        np.testing.assert_allclose(tree[i], dec[0], rtol=1e-12, atol=1e-12)


def test_invisible_rows_are_never_read_and_self_is_implicit():
    rng = np.random.default_rng(12)
    gamma, ctx, hq, hkv, dh = 10, 7, 4, 2, 8
    par = np.array([-1, 0, 0, 1, 1, 2, 5, 5, 3, 8], np.int32)
    masks = W.ancestor_masks(par)
    cap = ctx + gamma + 4
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    a = oracle.verify_attn_mask(q, k, v, ctx, masks)
    no_self = np.array([int(m) & ~(1 << i) for i, m in enumerate(masks)],
                       np.uint64)
    np.testing.assert_array_equal(
        a, oracle.verify_attn_mask(q, k, v, ctx, no_self))
    # node 9 sees nodes 0, 1, 3, 8, 9 only: poison every other block row
    vis = [0, 1, 3, 8, 9]
    k2, v2 = k.copy(), v.copy()
    for j in range(gamma):
        if j not in vis:
            k2[:, ctx + j] = 1e6
            v2[:, ctx + j] = np.nan
    k2[:, ctx + gamma:] = 1e6
    v2[:, ctx + gamma:] = np.nan
    b = oracle.verify_attn_mask(q, k2, v2, ctx, masks)
    np.testing.assert_array_equal(a[9], b[9])


# ---- acceptance ------------------------------------------------------------

def _brute_force_accept(argmax, entropy, tokens, parents, tau):
    """Every node's full root path is checked on its own."""
    gamma = len(argmax)
    best, best_depth = 0, 0
    for j in range(1, gamma):
        ok, v, depth = True, j, 0
        while v != 0:
            p = int(parents[v])
            if p < 0 or p >= v or tokens[v] != argmax[p]:
                ok = False
                break
            v, depth = p, depth + 1
        if ok and depth > best_depth:
            best, best_depth = j, depth
    path = [-1] * gamma
    for t, node in enumerate(_root_path(parents, best)):
        path[t] = node
    return (best_depth, int(argmax[best]), int(entropy[best] > tau), best,
            path)


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 64), st.integers(0, 2 ** 32 - 1), st.integers(2, 4))
def test_accept_tree_matches_brute_force(gamma, seed, vocab):
    rng = np.random.default_rng(seed)
    par = _random_parents(gamma, rng)
    am = rng.integers(0, vocab, gamma).astype(np.int32)
    tok = rng.integers(0, vocab, gamma).astype(np.int32)
    ent = rng.random(gamma) * 3.0
    n, bonus, route, b, ht, path = oracle.accept_tree(am, ent, tok, par, 1.5)
    ref = _brute_force_accept(am, ent, tok, par, 1.5)
    assert (n, bonus, route, b) == ref[:4]
    assert path.tolist() == ref[4]
    assert ht == ent[b]


@settings(max_examples=200, deadline=None)
@given(st.integers(1, 64), st.integers(0, 2 ** 32 - 1))
def test_chain_tree_accept_equals_prefix_accept(gamma, seed):
    rng = np.random.default_rng(seed)
    am = rng.integers(0, 3, gamma).astype(np.int32)
    draft = rng.integers(0, 3, gamma - 1).astype(np.int32)
    ent = rng.random(gamma) * 3.0
    par = np.arange(-1, gamma - 1, dtype=np.int32)
    tok = np.concatenate([[0], draft]).astype(np.int32)
    n, bonus, route, b, ht, path = oracle.accept_tree(am, ent, tok, par, 1.0)
    n2, bonus2, route2, ht2 = oracle.accept(am, ent, draft, 1.0)
    assert (n, bonus, route, ht) == (n2, bonus2, route2, ht2)
    assert b == n and path.tolist() == list(range(n + 1)) + [-1] * (gamma - 1 - n)


@pytest.mark.parametrize("k", [0, 1, 3, 8, 20])
def test_constructed_tree_accepts_the_designated_path(k):
    par = W.draft_tree(seed=W.stream_seed(6000, "tree"))
    gamma = len(par)
    rng = np.random.default_rng(k)
    am = rng.integers(0, 151936, gamma).astype(np.int32)
    tok = W.tree_tokens(am, par, k, 151936, seed=k)
    ent = rng.random(gamma)
    n, bonus, route, b, ht, path = oracle.accept_tree(am, ent, tok, par, 0.5)
    designated = [0]
    while True:
        kids = [j for j in range(1, gamma) if par[j] == designated[-1]]
        if not kids:
            break
        designated.append(min(kids))
    assert n == min(k, len(designated) - 1)
    assert path[:n + 1].tolist() == designated[:n + 1]
    assert bonus == am[designated[n]]


def test_invalid_parent_is_never_accepted():
    am = np.array([7, 7, 7, 7], np.int32)
    tok = np.array([0, 7, 7, 7], np.int32)
    ent = np.zeros(4)
    for bad in (3, 5, -2):      # not a smaller index
        par = np.array([-1, 0, 1, bad], np.int32)
        n, _, _, b, _, _ = oracle.accept_tree(am, ent, tok, par, 0.0)
        assert (n, b) == (2, 2)


def test_route_threshold_is_strict():
    par = np.array([-1, 0, 1], np.int32)
    am = np.array([4, 5, 6], np.int32)
    tok = np.array([0, 4, 5], np.int32)
    ent = np.array([0.1, 0.2, 0.75])
    assert oracle.accept_tree(am, ent, tok, par, 0.75)[2] == 0
    assert oracle.accept_tree(am, ent, tok, par, np.nextafter(0.75, 0))[2] == 1


# ---- path compaction ---------------------------------------------------------

def test_compacted_cache_shows_the_accepted_path():
    """After compaction, a decode of the deepest accepted node over the first
    ctx + n + 1 cache rows equals that node's tree-attention output."""
    rng = np.random.default_rng(21)
    gamma, ctx, hq, hkv, dh = 30, 12, 8, 2, 16
    par = W.draft_tree(levels=(4, 8, 9, 8), top_k=4, seed=3)
    assert len(par) == gamma
    cap = ctx + gamma
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    tree = oracle.verify_attn_mask(q, k, v, ctx, W.ancestor_masks(par))
    am = rng.integers(0, 50, gamma).astype(np.int32)
    tok = W.tree_tokens(am, par, 3, 50, seed=2)
    n, _, _, b, _, path = oracle.accept_tree(am, np.zeros(gamma), tok, par, 0.0)
    assert n == 3
    kc, vc = oracle.kv_compact_path(k, v, ctx, path, n)
    dec = oracle.verify_attn(np.ascontiguousarray(q[b:b + 1]), kc, vc, ctx + n)
    np.testing.assert_allclose(dec[0], tree[b], rtol=1e-12, atol=1e-12)
    # rows outside [ctx, ctx + n] are untouched
    np.testing.assert_array_equal(kc[:, :ctx], k[:, :ctx])
    np.testing.assert_array_equal(kc[:, ctx + n + 1:], k[:, ctx + n + 1:])
