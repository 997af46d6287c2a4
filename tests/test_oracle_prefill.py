"""Pins for the oracle's RoPE and KV-only prefill (Sec. 3.4).

KV-only prefill must produce exactly the keys and values a full forward of
the layer would cache (catch-up only needs the KV cache), and a batched
catch-up must equal token-by-token appends (lazy catch-up leaves the result
unchanged).  RoPE is pinned by its textbook complex-rotation form and its
invariants.
"""
import numpy as np
import pytest
import torch

import oracle


def _complex_rope(v, pos, base):
    """Rotate-half RoPE as complex multiplication (textbook form): the pair
    (v_i, v_{i+D/2}) is the complex number v_i + 1j*v_{i+D/2}, multiplied by
    exp(1j * pos * base**(-2i/D))."""
    d = v.shape[-1]
    half = d // 2
    z = v[..., :half] + 1j * v[..., half:]
    freqs = base ** (-np.arange(0, d, 2) / d)
    z = z * np.exp(1j * pos * freqs)
    return np.concatenate([z.real, z.imag], axis=-1)


def test_rope_position_zero_is_identity():
    v = np.random.default_rng(0).standard_normal(64)
    np.testing.assert_array_equal(oracle.rope(v, 0, 1e4), v)


@pytest.mark.parametrize("pos,base,dh", [(1, 1e4, 64), (252, 1e4, 64),
                                         (32800, 1e6, 128),
                                         (65583, 1e6, 128)])
def test_rope_matches_complex_rotation(pos, base, dh):
    v = np.random.default_rng(pos).standard_normal(dh)
    # one ulp of theta moves the angle by ~pos * 2^-53 rad
    tol = 1e-12 + 8 * pos * 2.0 ** -53 * np.abs(v).max()
    np.testing.assert_allclose(oracle.rope(v, pos, base),
                               _complex_rope(v, pos, base), rtol=0, atol=tol)


def test_rope_frequency_at_quarter_dim():
    """For head_dim 64 and base 1e4, pair 16 turns at base^(-1/2) = 0.01 rad
    per position, so position 100 rotates it by exactly 1 rad."""
    v = np.zeros(64)
    v[16] = 1.0
    r = oracle.rope(v, 100, 1e4)
    np.testing.assert_allclose([r[16], r[48]], [np.cos(1.0), np.sin(1.0)],
                               rtol=0, atol=1e-12)
    v = np.zeros(64)
    v[0] = 1.0
    r = oracle.rope(v, 3, 1e4)       # pair 0 turns 1 rad per position
    np.testing.assert_allclose([r[0], r[32]], [np.cos(3.0), np.sin(3.0)],
                               rtol=0, atol=1e-12)


def test_rope_preserves_pair_norms_and_relative_position():
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    rq = oracle.rope(q, 1234, 1e6)
    half = 64
    np.testing.assert_allclose(np.hypot(rq[:half], rq[half:]),
                               np.hypot(q[:half], q[half:]), rtol=1e-13)
    a = oracle.rope(q, 50, 1e6) @ oracle.rope(k, 20, 1e6)
    b = oracle.rope(q, 1050, 1e6) @ oracle.rope(k, 1020, 1e6)
    np.testing.assert_allclose(a, b, rtol=1e-10)


def test_prefill_matches_matmul_and_complex_rope():
    rng = np.random.default_rng(2)
    n, d_in, hkv, dh, start = 5, 48, 2, 16, 77
    x = rng.standard_normal((n, d_in))
    wk = rng.standard_normal((hkv * dh, d_in))
    wv = rng.standard_normal((hkv * dh, d_in))
    k, v = oracle.kv_only_prefill(x, wk, wv, start, hkv, dh, 1e4)
    kp = (x @ wk.T).reshape(n, hkv, dh).transpose(1, 0, 2)
    vp = (x @ wv.T).reshape(n, hkv, dh).transpose(1, 0, 2)
    for t in range(n):
        kp[:, t] = _complex_rope(kp[:, t], start + t, 1e4)
    np.testing.assert_allclose(k, kp, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(v, vp, rtol=1e-12, atol=1e-12)


def test_batched_catch_up_equals_single_token_appends():
    rng = np.random.default_rng(3)
    n, d_in, hkv, dh, start = 6, 32, 2, 8, 100
    x = rng.standard_normal((n, d_in))
    wk = rng.standard_normal((hkv * dh, d_in))
    wv = rng.standard_normal((hkv * dh, d_in))
    kb, vb = oracle.kv_only_prefill(x, wk, wv, start, hkv, dh, 1e6)
    for t in range(n):
        k1, v1 = oracle.kv_only_prefill(x[t:t + 1], wk, wv, start + t, hkv,
                                        dh, 1e6)
        np.testing.assert_array_equal(kb[:, t], k1[:, 0])
        np.testing.assert_array_equal(vb[:, t], v1[:, 0])


def test_kv_only_prefill_equals_full_layer_cache():
    """The cache written by KV-only prefill of the normalised inputs equals
    the K/V recorded by a full forward of the same layer."""
    rng = np.random.default_rng(4)
    T, d, hq, hkv, dh, pos0 = 7, 64, 8, 2, 16, 250
    x = rng.standard_normal((T, d))
    gain = 1.0 + 0.1 * rng.standard_normal(d)
    wq = rng.standard_normal((hq * dh, d)) * 0.1
    wk = rng.standard_normal((hkv * dh, d)) * 0.1
    wv = rng.standard_normal((hkv * dh, d)) * 0.1
    fwd = oracle.layer_forward(x, gain, wq, wk, wv, pos0, hq, hkv, dh, 1e-6,
                               1e4)
    k, v = oracle.kv_only_prefill(fwd["xn"], wk, wv, pos0, hkv, dh, 1e4)
    np.testing.assert_array_equal(k, fwd["k"])
    np.testing.assert_array_equal(v, fwd["v"])


def test_layer_forward_matches_torch():
    """The full-forward pin itself is checked against torch: rms_norm and
    causal grouped-query SDPA in fp64, with the complex RoPE above."""
    rng = np.random.default_rng(5)
    T, d, hq, hkv, dh, pos0 = 6, 32, 4, 2, 8, 10
    x = rng.standard_normal((T, d))
    gain = 1.0 + 0.1 * rng.standard_normal(d)
    wq = rng.standard_normal((hq * dh, d)) * 0.2
    wk = rng.standard_normal((hkv * dh, d)) * 0.2
    wv = rng.standard_normal((hkv * dh, d)) * 0.2
    fwd = oracle.layer_forward(x, gain, wq, wk, wv, pos0, hq, hkv, dh, 1e-6,
                               1e4)
    xt = torch.from_numpy(x)
    xn = torch.nn.functional.rms_norm(xt, (d,), torch.from_numpy(gain),
                                      eps=1e-6).numpy()
    np.testing.assert_allclose(fwd["xn"], xn, rtol=1e-12, atol=1e-12)
    q = (xn @ wq.T).reshape(T, hq, dh)
    k = (xn @ wk.T).reshape(T, hkv, dh)
    v = (xn @ wv.T).reshape(T, hkv, dh)
    for t in range(T):
        q[t] = _complex_rope(q[t], pos0 + t, 1e4)
        k[t] = _complex_rope(k[t], pos0 + t, 1e4)
    qt = torch.from_numpy(q).transpose(0, 1)
    kt = torch.from_numpy(k).transpose(0, 1).repeat_interleave(hq // hkv, 0)
    vt = torch.from_numpy(v).transpose(0, 1).repeat_interleave(hq // hkv, 0)
    out = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, is_causal=True).transpose(0, 1).numpy()
    np.testing.assert_allclose(fwd["out"], out, rtol=1e-11, atol=1e-12)


def test_verify_block_equals_full_forward_rows():
    """Verifying the last gamma tokens against the cache of the first ones
    reproduces the full causal forward at those positions."""
    rng = np.random.default_rng(6)
    T, gamma, d, hq, hkv, dh = 12, 5, 32, 8, 2, 8
    x = rng.standard_normal((T, d))
    gain = np.ones(d)
    wq = rng.standard_normal((hq * dh, d)) * 0.3
    wk = rng.standard_normal((hkv * dh, d)) * 0.3
    wv = rng.standard_normal((hkv * dh, d)) * 0.3
    fwd = oracle.layer_forward(x, gain, wq, wk, wv, 0, hq, hkv, dh, 1e-6, 1e4)
    ctx = T - gamma
    out = oracle.verify_attn(fwd["q"][ctx:], fwd["k"], fwd["v"], ctx)
    np.testing.assert_allclose(out, fwd["out"][ctx:], rtol=1e-12, atol=1e-13)
