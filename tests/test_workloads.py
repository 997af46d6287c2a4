"""Host-side checks of the seeded workload generator (no GPU needed)."""
import numpy as np
import torch

import workloads as W


def test_configs_have_the_stated_shapes():
    c3 = W.CONFIGS[3]
    assert (c3.n_layers, c3.hidden, c3.n_q_heads, c3.n_kv_heads,
            c3.head_dim) == (36, 4096, 32, 8, 128)
    assert (c3.ctx_len, c3.gamma, c3.n_prefill, c3.vocab) == (32768, 16, 16,
                                                              151936)
    assert c3.cap == 32768 + 16 + 16
    b = c3.algorithmic_bytes()
    assert b["total"] == 6_699_483_136
    assert W.CONFIGS[2].algorithmic_bytes()["total"] == 2_458_583_040
    assert W.CONFIGS[5].algorithmic_bytes()["total"] == 20_145_143_808
    c1 = W.CONFIGS[1]
    assert c1.dtype == "f32" and c1.prefill_start + c1.n_prefill == 256


def test_generation_is_seeded_and_reproducible():
    w = W.CONFIGS[1]
    a = W.generate_layer(w, 0)
    b = W.generate_layer(w, 0)
    for k in a:
        assert torch.equal(a[k], b[k])
    c = W.generate_layer(w, 0, seed=12345)
    assert not torch.equal(a["q"], c["q"])
    assert abs(float(a["k_cache"].std()) - 0.02) < 0.002


def test_geometric_prefix_distribution():
    ks = [W.geometric_prefix(0.3, 1000, s) for s in range(4000)]
    assert min(ks) == 0
    assert abs(np.mean(ks) - 0.7 / 0.3) < 0.15     # mean (1-p)/p
    assert all(W.geometric_prefix(0.01, 8, s) <= 7 for s in range(100))


def test_make_drafts_forces_the_prefix():
    ref = np.array([5, 9, 9, 2, 7, 1, 0, 3], np.int32)
    for k in range(8):
        d = W.make_drafts(ref, k, vocab=10, seed=k)
        assert d.shape == (7,)
        assert np.array_equal(d[:k], ref[:k])
        if k < 7:
            assert d[k] != ref[k]
        assert d.min() >= 0 and d.max() < 10


def test_router_logits_mixture():
    z, peaked = W.router_logits(16, 5000, seed=7)
    assert z.shape == (16, 5000) and len(peaked) == 8
    for i in range(16):
        row = z[i]
        top2 = torch.topk(row, 2).values
        if i in peaked:
            assert float(top2[0] - top2[1]) >= 16.0 - 1e-3
        else:
            assert float(row.std()) < 0.6


def test_to_oracle_keeps_bf16_bits():
    t = torch.randn(5, 7).to(torch.bfloat16)
    a = W.to_oracle(t)
    assert a.dtype == np.uint16
    back = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    assert torch.equal(back, t)
