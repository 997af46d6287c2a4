"""GPU parity of tree verification against the fp64 oracle: ancestor-mask
attention (draft trees of Sec. 3.1 verified in one pass, Sec. 3.2), tree
acceptance with the entropy route (Sec. 3.3.1), and path compaction of the
KV cache.  Includes the EAGLE-3-shaped workload (App. A: depth 8, top-k 10,
60 draft tokens) at its full size on the 8B shapes.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import (TOL, check_argmax, check_tree_accept, entropy_rel_err, host64,
                    max_vec_rel_err)

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _random_parents(gamma, seed):
    rng = np.random.default_rng(seed)
    par = np.full(gamma, -1, np.int32)
    for j in range(1, gamma):
        par[j] = rng.integers(max(0, j - 6), j)   # bushy, a few levels deep
    return par


def _mask_dev(par):
    m = W.ancestor_masks(par).view(np.int64)
    return torch.from_numpy(m.copy()).to(DEV)


def _inputs(dt, gamma, ctx, hq, hkv, dh, seed, cap_extra=3):
    cap = ctx + gamma + cap_extra
    dtype = DT[dt]
    q = W.normal((gamma, hq, dh), 1.0, W.stream_seed(seed, "q"), dtype, DEV)
    k = W.normal((hkv, cap, dh), 1.0, W.stream_seed(seed, "k_cache"), dtype, DEV)
    v = W.normal((hkv, cap, dh), 1.0, W.stream_seed(seed, "v_cache"), dtype, DEV)
    k[:, ctx + gamma:] = float("nan")      # past the block: never read
    v[:, ctx + gamma:] = float("nan")
    return q, k, v


CASES = [
    # dt, gamma, ctx, n_q_heads, n_kv_heads, head_dim
    ("bf16", 1, 40, 8, 2, 128),
    ("bf16", 7, 0, 8, 2, 128),
    ("bf16", 13, 31, 8, 8, 64),
    ("bf16", 33, 1000, 32, 8, 128),
    ("bf16", 61, 2049, 32, 8, 128),
    ("bf16", 64, 300, 16, 2, 128),
    ("bf16", 20, 517, 32, 8, 128),             # 80 rows per KV head: 128-row workgroups
    ("bf16", 40, 700, 16, 4, 64),              # 160 rows, head_dim 64: three row groups
    ("f32", 9, 100, 8, 2, 64),
    ("f32", 61, 257, 8, 2, 64),
]


@pytest.mark.parametrize("dt,gamma,ctx,hq,hkv,dh", CASES)
def test_tree_attention_matches_oracle(dt, gamma, ctx, hq, hkv, dh):
    print(f"tree attention {dt} gamma={gamma} ctx={ctx} {hq}/{hkv}x{dh}", flush=True)
    seed = 7000 + gamma * 31 + ctx
    q, k, v = _inputs(dt, gamma, ctx, hq, hkv, dh, seed)
    par = _random_parents(gamma, seed)
    out = torch.empty_like(q)
    wf.wf_verify_attn_tree(q, k, v, out, ctx, _mask_dev(par))
    torch.cuda.synchronize()
    n = ctx + gamma
    ref = oracle.verify_attn_mask(W.to_oracle(q), W.to_oracle(k[:, :n].contiguous()),
                                  W.to_oracle(v[:, :n].contiguous()), ctx,
                                  W.ancestor_masks(par))
    assert max_vec_rel_err(host64(out), ref) <= TOL[dt]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_chain_mask_is_bit_identical_to_block_causal(dt):
    print(f"tree chain == block-causal {dt}", flush=True)
    gamma, ctx = 16, 777
    q, k, v = _inputs(dt, gamma, ctx, 32, 8, 128 if dt == "bf16" else 64, 91)
    par = np.arange(-1, gamma - 1, dtype=np.int32)
    a = torch.empty_like(q)
    b = torch.empty_like(q)
    wf.wf_verify_attn(q, k, v, a, ctx)
    wf.wf_verify_attn_tree(q, k, v, b, ctx, _mask_dev(par))
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_mask_bits_above_gamma_and_self_bit_are_ignored():
    print("tree mask: stray bits and implicit self", flush=True)
    gamma, ctx = 20, 300
    q, k, v = _inputs("bf16", gamma, ctx, 8, 2, 128, 92)
    par = _random_parents(gamma, 92)
    m = W.ancestor_masks(par)
    noisy = np.array([(int(x) & ~(1 << i)) | (0xFFF << gamma) for i, x in enumerate(m)],
                     np.uint64).view(np.int64)
    a = torch.empty_like(q)
    b = torch.empty_like(q)
    wf.wf_verify_attn_tree(q, k, v, a, ctx, _mask_dev(par))
    wf.wf_verify_attn_tree(q, k, v, b, ctx, torch.from_numpy(noisy.copy()).to(DEV))
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("splits", [1, 3, 16, 0])
def test_tree_attention_any_split_count(splits):
    print(f"tree attention splits={splits}", flush=True)
    gamma, ctx = 61, 1500
    q, k, v = _inputs("bf16", gamma, ctx, 32, 8, 128, 93)
    par = W.draft_tree(seed=93)
    out = torch.empty_like(q)
    wf.wf_verify_attn_tree(q, k, v, out, ctx, _mask_dev(par), num_splits=splits)
    torch.cuda.synchronize()
    n = ctx + gamma
    ref = oracle.verify_attn_mask(W.to_oracle(q), W.to_oracle(k[:, :n].contiguous()),
                                  W.to_oracle(v[:, :n].contiguous()), ctx,
                                  W.ancestor_masks(par))
    assert max_vec_rel_err(host64(out), ref) <= TOL["bf16"]


# ---- acceptance ------------------------------------------------------------

def _lm_tree(h, w, logits, tok, par, tau):
    gamma = (logits if logits is not None else h).shape[0]
    am = torch.empty(gamma, dtype=torch.int32, device=DEV)
    ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
    acc = torch.empty(4, dtype=torch.int32, device=DEV)
    path = torch.empty(gamma, dtype=torch.int32, device=DEV)
    wf.wf_lmhead_accept_tree(h, w, logits, torch.from_numpy(tok).to(DEV),
                             torch.from_numpy(par).to(DEV), tau, am, ent, acc,
                             path)
    torch.cuda.synchronize()
    return am.cpu().numpy(), ent.cpu().numpy(), acc.cpu().numpy(), path.cpu().numpy()


@pytest.mark.parametrize("k", [0, 2, 5, 8])
def test_tree_accept_head_mode(k):
    """EAGLE-shaped tree, bf16 LM head; tokens put the accepted path at
    depth min(k, designated depth) using the oracle's argmax."""
    print(f"tree accept head mode k={k}", flush=True)
    gamma, d, vocab = 61, 512, 7001
    seed = 500 + k
    h = W.normal((gamma, d), 1.0, W.stream_seed(seed, "h"), torch.bfloat16, DEV)
    w = W.normal((vocab, d), 0.05, W.stream_seed(seed, "w_lm"), torch.bfloat16, DEV)
    am_ref, ent_ref, margin, z = oracle.lmhead_rows(W.to_oracle(h), W.to_oracle(w),
                                                    want_logits=True)
    par = W.draft_tree(seed=seed)
    tok = W.tree_tokens(am_ref, par, k, vocab, seed)
    tau = float(np.float32(np.median(ent_ref) + 1e-3))
    am, ent, acc, path = _lm_tree(h, w, None, tok, par, tau)
    check_argmax(am, am_ref, margin, z, "bf16")
    assert entropy_rel_err(ent, ent_ref) <= TOL["bf16"]
    check_tree_accept(am, ent, acc, path, am_ref, ent_ref, margin, tok, par,
                      tau, 1e-2)


@pytest.mark.parametrize("seed", range(6))
def test_tree_accept_logits_mode_random_trees(seed):
    """fp32 logits with a planted maximum per row; node tokens copy the
    parent's argmax with probability 1/2, so accepted subtrees branch."""
    print(f"tree accept logits mode seed={seed}", flush=True)
    rng = np.random.default_rng(seed)
    gamma = int(rng.integers(1, 65))
    vocab = 3000
    z = rng.standard_normal((gamma, vocab)).astype(np.float32)
    top = rng.integers(0, vocab, gamma)
    z[np.arange(gamma), top] = 10.0
    par = _random_parents(gamma, seed)
    am_ref, ent_ref, _ = oracle.lmhead_rows(logits=z)
    tok = rng.integers(0, vocab, gamma).astype(np.int32)
    for j in range(1, gamma):
        if rng.random() < 0.5:
            tok[j] = am_ref[par[j]]
    am, ent, acc, path = _lm_tree(None, None, torch.from_numpy(z).to(DEV), tok,
                                  par, 1.0)
    assert am.tolist() == am_ref.tolist()
    assert entropy_rel_err(ent, ent_ref) <= TOL["f32"]
    ref = oracle.accept_tree(am_ref, ent_ref, tok, par, 1.0)
    assert acc.tolist() == [ref[0], ref[1], ref[2], ref[3]]
    assert path.tolist() == ref[5].tolist()


def test_tree_accept_invalid_parents_never_accepted():
    print("tree accept invalid parents", flush=True)
    gamma, vocab = 6, 100
    z = np.zeros((gamma, vocab), np.float32)
    z[:, 7] = 5.0                          # every argmax is 7
    tok = np.full(gamma, 7, np.int32)
    par = np.array([-1, 0, 1, 9, -3, 2], np.int32)   # nodes 3, 4 invalid
    am, ent, acc, path = _lm_tree(None, None, torch.from_numpy(z).to(DEV), tok,
                                  par, 0.0)
    assert acc.tolist()[0] == 3 and acc[3] == 5
    assert path.tolist() == [0, 1, 2, 5, -1, -1]


# ---- compaction --------------------------------------------------------------

@pytest.mark.parametrize("dt,dh,layers", [("bf16", 128, 1), ("bf16", 64, 1),
                                          ("f32", 128, 1), ("bf16", 128, 5)])
def test_compaction_matches_oracle(dt, dh, layers):
    print(f"compaction {dt} D={dh} layers={layers}", flush=True)
    gamma, ctx, hkv = 61, 500, 8
    cap = ctx + gamma + 7
    shape = (hkv, cap, dh) if layers == 1 else (layers, hkv, cap, dh)
    k = W.normal(shape, 1.0, W.stream_seed(3, "k_cache"), DT[dt], DEV)
    v = W.normal(shape, 1.0, W.stream_seed(3, "v_cache"), DT[dt], DEV)
    par = W.draft_tree(seed=4)
    rng = np.random.default_rng(5)
    am = rng.integers(0, 1000, gamma).astype(np.int32)
    tok = W.tree_tokens(am, par, 6, 1000, seed=6)
    n, _, _, b, _, path = oracle.accept_tree(am, np.zeros(gamma), tok, par, 0.0)
    assert n == 6
    k0, v0 = W.to_oracle(k), W.to_oracle(v)
    acc = torch.tensor([n, 0, 0, b], dtype=torch.int32, device=DEV)
    wf.wf_kv_compact_path(k, v, acc, torch.from_numpy(path).to(DEV), ctx)
    torch.cuda.synchronize()
    k1, v1 = W.to_oracle(k), W.to_oracle(v)
    for l in range(layers):
        sl = (slice(None),) if layers == 1 else (l,)
        kref, vref = oracle.kv_compact_path(k0[sl], v0[sl], ctx, path, n)
        assert np.array_equal(k1[sl], kref)
        assert np.array_equal(v1[sl], vref)


# ---- the EAGLE-3-shaped workload at full size ----------------------------------

def test_eagle_tree_round_full_size():
    """Workload 6 (8B shapes, ctx 8192, root + 60 nodes): one layer of tree
    attention against the oracle (all rows and heads), then the LM head with
    acceptance on the tree and compaction of that layer's cache."""
    w = W.CONFIGS[6]
    print(f"eagle tree round {w.name}", flush=True)
    lay = W.generate_layer(w, 0, device=DEV)
    head = W.generate_head(w, device=DEV)
    par = W.draft_tree(seed=W.stream_seed(W.master_seed(6), "tree"))
    q, kc, vc = lay["q"], lay["k_cache"], lay["v_cache"]
    out = torch.empty_like(q)
    wf.wf_verify_attn_tree(q, kc, vc, out, w.ctx_len, _mask_dev(par))
    torch.cuda.synchronize()
    n_keys = w.ctx_len + w.gamma
    ref = oracle.verify_attn_mask(W.to_oracle(q),
                                  W.to_oracle(kc[:, :n_keys].contiguous()),
                                  W.to_oracle(vc[:, :n_keys].contiguous()),
                                  w.ctx_len, W.ancestor_masks(par))
    assert max_vec_rel_err(host64(out), ref) <= TOL["bf16"]

    am_ref, ent_ref, margin = oracle.lmhead_rows(W.to_oracle(head["h"]),
                                                 W.to_oracle(head["w_lm"]))
    k = W.prefix_len(w, 1)
    tok = W.tree_tokens(am_ref, par, k, w.vocab, 1)
    tau = 1.0
    am, ent, acc, path = _lm_tree(head["h"], head["w_lm"], None, tok, par, tau)
    assert entropy_rel_err(ent, ent_ref) <= TOL["bf16"]
    check_argmax(am, am_ref, margin, None, "bf16")
    check_tree_accept(am, ent, acc, path, am_ref, ent_ref, margin, tok, par,
                      tau, 1e-2)

    kbefore, vbefore = W.to_oracle(kc), W.to_oracle(vc)
    wf.wf_kv_compact_path(kc, vc, torch.from_numpy(acc).to(DEV),
                          torch.from_numpy(path).to(DEV), w.ctx_len)
    torch.cuda.synchronize()
    kref, vref = oracle.kv_compact_path(kbefore, vbefore, w.ctx_len, path, int(acc[0]))
    assert np.array_equal(W.to_oracle(kc), kref)
    assert np.array_equal(W.to_oracle(vc), vref)
