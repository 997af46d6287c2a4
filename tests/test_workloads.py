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


def test_draft_tree_shape():
    """EAGLE-3 shape (App. A): 60 drafts below the root, depth 8, at most 10
    children per node, breadth-first order (every parent precedes its
    children, depths never decrease)."""
    par = W.draft_tree(seed=W.stream_seed(6000, "tree"))
    assert par.shape == (61,) and par[0] == -1
    depth = np.zeros(61, np.int64)
    for j in range(1, 61):
        assert 0 <= par[j] < j
        depth[j] = depth[par[j]] + 1
    assert np.all(np.diff(depth) >= 0)
    assert [int((depth == d).sum()) for d in range(1, 9)] == list(W.EAGLE_LEVELS)
    counts = np.bincount(par[1:], minlength=61)
    assert counts.max() <= W.EAGLE_TOP_K


def test_ancestor_masks_mark_root_paths():
    par = np.array([-1, 0, 0, 1, 3, 2], np.int32)
    m = W.ancestor_masks(par)
    assert [bin(int(x))[2:][::-1] for x in m] == [
        "1", "11", "101", "1101", "11011", "101001"]


def test_tree_tokens_accept_exactly_k():
    par = W.draft_tree(seed=5)
    ref = np.arange(61, dtype=np.int32) * 7 % 1000
    for k in (0, 2, 5, 9):
        tok = W.tree_tokens(ref, par, k, 1000, seed=k)
        accepted = {0}
        for j in range(1, 61):
            if par[j] in accepted and tok[j] == ref[par[j]]:
                accepted.add(j)
        depth = {0: 0}
        for j in range(1, 61):
            depth[j] = depth[int(par[j])] + 1
        assert max(depth[j] for j in accepted) == min(k, 8)


def test_switch_workload_and_drafter_generator():
    """Workload 7: one drafter layer with the 8B attention shapes, a 4096-row
    cache and an 80-token backlog; the generator gives every projection its
    nn.Linear shape, gains near 1, a cache whose rows past the base are
    zero, and the same bytes for the same seed."""
    import dataclasses
    w = W.CONFIGS[7]
    assert (w.hidden, w.n_q_heads, w.n_kv_heads, w.head_dim, w.inter) == (4096, 32, 8, 128, 12288)
    assert (w.ctx_len, w.n_prefill, w.n_layers) == (4096, 80, 1)
    small = dataclasses.replace(w, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                                inter=512, ctx_len=10, n_prefill=3)
    t = W.generate_drafter(small)
    shapes = {"attn_norm": (256,), "w_q": (256, 256), "w_k": (128, 256), "w_v": (128, 256),
              "w_o": (256, 256), "mlp_norm": (256,), "w_gate": (512, 256),
              "w_up": (512, 256), "w_down": (256, 512)}
    for name, shp in shapes.items():
        assert tuple(t[name].shape) == shp, name
    assert tuple(t["k_cache"].shape) == (2, 13, 64) and tuple(t["r"].shape) == (3, 256)
    assert not t["k_cache"][:, 10:].any() and t["k_cache"][:, :10].abs().sum() > 0
    g = t["attn_norm"].float()
    assert (g - 1).abs().max() < 1.0 and (g - 1).abs().mean() > 0.01
    t2 = W.generate_drafter(small)
    for name in shapes:
        assert torch.equal(t[name], t2[name])
    assert w.drafter_weight_bytes() == (2 * 4096 * 4096 + 2 * 1024 * 4096
                                        + 3 * 12288 * 4096 + 2 * 4096) * 2
    assert w.catchup_bytes(80, 4096) == 403_988_480
