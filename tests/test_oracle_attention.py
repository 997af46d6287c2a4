"""Pins for the oracle's verification attention (Sec. 3.2 parallel verify).

Each check fixes the oracle against something other than its own formula:
a library routine (torch scaled_dot_product_attention in fp64 with an
explicit block-causal mask), closed forms, and invariants of causal decoding.
"""
import numpy as np
import pytest
import torch

import oracle

SHAPES = [
    # gamma, ctx_len, n_q_heads, n_kv_heads, head_dim
    (1, 0, 4, 2, 8),
    (1, 37, 8, 2, 16),
    (4, 19, 8, 2, 16),
    (7, 50, 8, 8, 8),
    (8, 33, 12, 3, 32),
    (16, 64, 8, 1, 16),
]


def _rand(shape, rng, std=1.0):
    return rng.standard_normal(shape) * std


def _sdpa_reference(q, k, v, ctx_len):
    """torch fp64 SDPA with an explicit mask; GQA by repeating kv heads."""
    gamma, hq, dh = q.shape
    hkv = k.shape[0]
    n = ctx_len + gamma
    group = hq // hkv
    kt = torch.from_numpy(k[:, :n]).repeat_interleave(group, dim=0)
    vt = torch.from_numpy(v[:, :n]).repeat_interleave(group, dim=0)
    qt = torch.from_numpy(q).transpose(0, 1).contiguous()  # [hq][gamma][dh]
    rows = torch.arange(gamma)[:, None]
    cols = torch.arange(n)[None, :]
    mask = cols <= ctx_len + rows                              # block-causal
    out = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=mask)
    return out.transpose(0, 1).numpy()


@pytest.mark.parametrize("gamma,ctx,hq,hkv,dh", SHAPES)
def test_matches_torch_sdpa(gamma, ctx, hq, hkv, dh):
    rng = np.random.default_rng(gamma * 1000 + ctx)
    cap = ctx + gamma + 3
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    got = oracle.verify_attn(q, k, v, ctx)
    ref = _sdpa_reference(q, k, v, ctx)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_rows_beyond_the_block_are_never_read():
    rng = np.random.default_rng(3)
    gamma, ctx, hq, hkv, dh = 5, 20, 4, 2, 8
    cap = ctx + gamma + 10
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    a = oracle.verify_attn(q, k, v, ctx)
    k[:, ctx + gamma:] = 1e6
    v[:, ctx + gamma:] = np.nan
    b = oracle.verify_attn(q, k, v, ctx)
    np.testing.assert_array_equal(a, b)


def test_equal_keys_give_mean_of_visible_values():
    rng = np.random.default_rng(4)
    gamma, ctx, hq, hkv, dh = 6, 11, 4, 2, 8
    cap = ctx + gamma
    q = _rand((gamma, hq, dh), rng)
    k = np.tile(_rand((hkv, 1, dh), rng), (1, cap, 1))
    v = _rand((hkv, cap, dh), rng)
    out = oracle.verify_attn(q, k, v, ctx)
    for i in range(gamma):
        for h in range(hq):
            g = h // (hq // hkv)
            np.testing.assert_allclose(out[i, h], v[g, :ctx + i + 1].mean(0),
                                       rtol=1e-12, atol=1e-12)


def test_dominant_key_selects_its_value():
    rng = np.random.default_rng(5)
    gamma, ctx, hq, hkv, dh = 4, 9, 2, 1, 8
    cap = ctx + gamma
    q = np.abs(_rand((gamma, hq, dh), rng)) + 0.5
    k = _rand((hkv, cap, dh), rng) * 1e-3
    jstar = 3
    k[0, jstar] = 1e4              # score ~ +1e4 * sum(q) / sqrt(dh)
    v = _rand((hkv, cap, dh), rng)
    out = oracle.verify_attn(q, k, v, ctx)
    np.testing.assert_allclose(out, np.broadcast_to(v[0, jstar], out.shape),
                               rtol=0, atol=1e-12)


def test_gamma1_row_i_equals_decode_on_prefix_i():
    """Row i of a block-causal block == a single-token decode at ctx+i."""
    rng = np.random.default_rng(6)
    gamma, ctx, hq, hkv, dh = 9, 40, 8, 2, 16
    cap = ctx + gamma
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    blk = oracle.verify_attn(q, k, v, ctx)
    for i in range(gamma):
        dec = oracle.verify_attn(q[i:i + 1], k, v, ctx + i)
        np.testing.assert_allclose(blk[i], dec[0], rtol=1e-13, atol=1e-14)


def test_cached_key_permutation_invariance():
    rng = np.random.default_rng(7)
    gamma, ctx, hq, hkv, dh = 3, 30, 4, 2, 8
    cap = ctx + gamma
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    a = oracle.verify_attn(q, k, v, ctx)
    perm = rng.permutation(ctx)
    k2, v2 = k.copy(), v.copy()
    k2[:, :ctx] = k[:, perm]
    v2[:, :ctx] = v[:, perm]
    b = oracle.verify_attn(q, k2, v2, ctx)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)


def test_rows_subset_matches_full():
    rng = np.random.default_rng(8)
    gamma, ctx, hq, hkv, dh = 5, 17, 8, 4, 16
    cap = ctx + gamma
    q = _rand((gamma, hq, dh), rng)
    k = _rand((hkv, cap, dh), rng)
    v = _rand((hkv, cap, dh), rng)
    full = oracle.verify_attn(q, k, v, ctx)
    pairs = [(0, 0), (4, 7), (2, 3), (1, 6)]
    sub = oracle.verify_attn_rows(q, k, v, ctx, pairs)
    for n, (i, h) in enumerate(pairs):
        np.testing.assert_array_equal(sub[n], full[i, h])


def test_bf16_storage_is_read_exactly():
    """bf16 bit patterns decode to the same values torch's bf16 -> fp32
    conversion gives (the oracle on both representations agrees exactly)."""
    g = torch.Generator().manual_seed(9)
    gamma, ctx, hq, hkv, dh = 4, 21, 4, 2, 16
    cap = ctx + gamma
    qb = torch.randn((gamma, hq, dh), generator=g).to(torch.bfloat16)
    kb = torch.randn((hkv, cap, dh), generator=g).to(torch.bfloat16)
    vb = torch.randn((hkv, cap, dh), generator=g).to(torch.bfloat16)
    bits = [t.view(torch.int16).numpy().view(np.uint16) for t in (qb, kb, vb)]
    f32 = [t.float().numpy() for t in (qb, kb, vb)]
    a = oracle.verify_attn(*bits, ctx)
    b = oracle.verify_attn(*f32, ctx)
    np.testing.assert_array_equal(a, b)


def test_rejects_bad_shapes():
    q = np.zeros((2, 3, 8))
    k = np.zeros((2, 10, 8))
    with pytest.raises(ValueError):
        oracle.verify_attn(q, k, k, 0)         # 3 q heads over 2 kv heads
    q = np.zeros((4, 4, 8))
    with pytest.raises(ValueError):
        oracle.verify_attn(q, k, k, 7)         # ctx + gamma > cap
