"""Pins for the oracle's drafter layer and lazy catch-up (Sec. 3.4: lazy
catch-up with KV-only prefill; only the last backlog token runs the full
layer).  The full layer is pinned to a torch fp64 implementation (rms_norm,
linear, complex-form RoPE, scaled_dot_product_attention, silu); catch-up is
pinned to the full forward over the whole backlog (lazy and eager catch-up
give the same cache and the same final hidden state, Sec. 6), and the
layer's K/V to the KV-only prefill."""
import numpy as np
import pytest
import torch

import oracle

EPS, BASE = 1e-6, 1e4


def _layer(rng, d, hq, hkv, dh, inter, std=0.05):
    return {
        "attn_norm": 1.0 + 0.1 * rng.standard_normal(d),
        "w_q": rng.standard_normal((hq * dh, d)) * std,
        "w_k": rng.standard_normal((hkv * dh, d)) * std,
        "w_v": rng.standard_normal((hkv * dh, d)) * std,
        "w_o": rng.standard_normal((d, hq * dh)) * std,
        "mlp_norm": 1.0 + 0.1 * rng.standard_normal(d),
        "w_gate": rng.standard_normal((inter, d)) * std,
        "w_up": rng.standard_normal((inter, d)) * std,
        "w_down": rng.standard_normal((d, inter)) * std,
    }


def _rope_t(x, pos, base):
    """x [..., D] rotate-half RoPE at positions pos [...], as complex numbers."""
    dh = x.shape[-1]
    half = dh // 2
    theta = base ** (-2.0 * torch.arange(half, dtype=torch.float64) / dh)
    ang = pos[..., None].double() * theta
    z = torch.complex(x[..., :half], x[..., half:]) * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([z.real, z.imag], dim=-1)


def _torch_forward(r, pos, L, kc, vc, hq, hkv):
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    r, kc, vc = T(r), T(kc).clone(), T(vc).clone()
    M, d = r.shape
    dh = kc.shape[-1]
    p = torch.arange(pos, pos + M)
    xn = torch.nn.functional.rms_norm(r, (d,), T(L["attn_norm"]), EPS)
    q = (xn @ T(L["w_q"]).T).view(M, hq, dh)
    k = (xn @ T(L["w_k"]).T).view(M, hkv, dh)
    v = (xn @ T(L["w_v"]).T).view(M, hkv, dh)
    q = _rope_t(q, p[:, None].expand(M, hq), BASE)
    k = _rope_t(k, p[:, None].expand(M, hkv), BASE)
    kc[:, pos:pos + M] = k.transpose(0, 1)
    vc[:, pos:pos + M] = v.transpose(0, 1)
    n = pos + M
    g = hq // hkv
    mask = torch.arange(n)[None, :] <= p[:, None]
    a = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(0, 1), kc[:, :n].repeat_interleave(g, 0),
        vc[:, :n].repeat_interleave(g, 0), attn_mask=mask)
    a = a.transpose(0, 1).reshape(M, hq * dh)
    h1 = r + a @ T(L["w_o"]).T
    xn2 = torch.nn.functional.rms_norm(h1, (d,), T(L["mlp_norm"]), EPS)
    act = torch.nn.functional.silu(xn2 @ T(L["w_gate"]).T) * (xn2 @ T(L["w_up"]).T)
    return (h1 + act @ T(L["w_down"]).T).numpy(), kc.numpy(), vc.numpy()


@pytest.mark.parametrize("M,pos", [(1, 0), (1, 9), (4, 13), (7, 0)])
def test_decoder_matches_torch(M, pos):
    rng = np.random.default_rng(M * 100 + pos)
    d, hq, hkv, dh, inter = 32, 4, 2, 8, 48
    L = _layer(rng, d, hq, hkv, dh, inter)
    cap = pos + M + 3
    kc = rng.standard_normal((hkv, cap, dh))
    vc = rng.standard_normal((hkv, cap, dh))
    r = rng.standard_normal((M, d))
    out, k2, v2 = oracle.decoder_forward(r, pos, L, kc, vc, hq, hkv, EPS, BASE)
    ref, kr, vr = _torch_forward(r, pos, L, kc, vc, hq, hkv)
    np.testing.assert_allclose(out, ref, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(k2[:, :pos + M], kr[:, :pos + M], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(v2[:, :pos + M], vr[:, :pos + M], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("n,pos", [(1, 5), (2, 0), (9, 17)])
def test_lazy_catchup_equals_full_forward(n, pos):
    """KV-only prefill of the backlog but its last token, then the full layer
    for that token, gives the cache and final hidden state of running the
    full layer over the whole backlog."""
    rng = np.random.default_rng(n * 7 + pos)
    d, hq, hkv, dh, inter = 32, 4, 1, 16, 64
    L = _layer(rng, d, hq, hkv, dh, inter)
    cap = pos + n + 2
    kc = rng.standard_normal((hkv, cap, dh))
    vc = rng.standard_normal((hkv, cap, dh))
    r = rng.standard_normal((n, d))
    last, k1, v1 = oracle.catchup(r, pos, L, kc, vc, hq, hkv, EPS, BASE)
    full, k2, v2 = oracle.decoder_forward(r, pos, L, kc, vc, hq, hkv, EPS, BASE)
    np.testing.assert_allclose(last, full[n - 1], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(k1, k2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(v1, v2, rtol=1e-12, atol=1e-12)


def test_single_key_attention_is_its_value():
    """At position 0 the token attends to itself alone, so the layer is
    h1 = r + Wo v (per query head, the v of its KV head) and the MLP."""
    rng = np.random.default_rng(5)
    d, hq, hkv, dh, inter = 16, 2, 1, 8, 24
    L = _layer(rng, d, hq, hkv, dh, inter)
    r = rng.standard_normal((1, d))
    kc = np.zeros((hkv, 4, dh))
    vc = np.zeros((hkv, 4, dh))
    out, _, vnew = oracle.decoder_forward(r, 0, L, kc, vc, hq, hkv, EPS, BASE)
    a = np.concatenate([vnew[0, 0]] * hq)
    h1 = r[0] + L["w_o"] @ a
    xn2 = h1 / np.sqrt(np.mean(h1 ** 2) + EPS) * L["mlp_norm"]
    zg, zu = L["w_gate"] @ xn2, L["w_up"] @ xn2
    ref = h1 + L["w_down"] @ (zg / (1 + np.exp(-zg)) * zu)
    np.testing.assert_allclose(out[0], ref, rtol=1e-12, atol=1e-12)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(8)
    x, g = rng.standard_normal((5, 40)), rng.standard_normal(40)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (40,), torch.from_numpy(g),
                                       1e-5).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-13)
