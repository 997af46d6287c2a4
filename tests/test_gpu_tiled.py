"""The tiled bf16 weight layout: wf_tile_weights against the layout's
definition written out with torch indexing, and the calls that stream
weights (KV-only prefill, the LM head) giving bit-for-bit the results of
the row-major weights."""
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
BF = torch.bfloat16


def _expected_tiles(w):
    """The layout by its definition: tile (rb, c) of 16 rows x 32 columns at
    element (rb * cols/32 + c) * 512; inside it element (16 q + r) * 8 + e
    is W[16 rb + r][32 c + 8 q + e]; rows past the end are zero."""
    rows, cols = w.shape
    rp = (rows + 15) // 16 * 16
    wp = torch.zeros((rp, cols), dtype=w.dtype, device=w.device)
    wp[:rows] = w
    t = wp.view(rp // 16, 16, cols // 32, 4, 8)        # rb, r, c, q, e
    return t.permute(0, 2, 3, 1, 4).reshape(-1)        # rb, c, q, r, e


@pytest.mark.parametrize("rows,cols", [(16, 32), (37, 96), (1024, 4096), (151936 // 8, 512)])
def test_tiling_matches_definition(rows, cols):
    print(f"tile {rows}x{cols}", flush=True)
    w = W.normal((rows, cols), 1.0, W.stream_seed(rows, "w_lm"), BF, DEV)
    t = wf.tile_weights(w)
    torch.cuda.synchronize()
    assert t.data.numel() * 2 == wf.wf_tiled_weight_bytes(rows, cols)
    assert torch.equal(t.data.view(torch.int16), _expected_tiles(w).view(torch.int16))


@pytest.mark.parametrize("n,d_in,hkv,dh,start", [(16, 4096, 8, 128, 32784), (5, 512, 2, 64, 3),
                                                 (70, 1024, 4, 128, 100)])
def test_prefill_tiled_is_bit_exact(n, d_in, hkv, dh, start):
    print(f"prefill tiled n={n} d_in={d_in}", flush=True)
    cap = start + n + 1
    x = W.normal((n, d_in), 1.0, 1, BF, DEV)
    wk = W.normal((hkv * dh, d_in), 0.02, 2, BF, DEV)
    wv = W.normal((hkv * dh, d_in), 0.02, 3, BF, DEV)
    kc = torch.zeros((hkv, cap, dh), dtype=BF, device=DEV)
    vc = torch.zeros_like(kc)
    k2, v2 = kc.clone(), vc.clone()
    wf.wf_kv_only_prefill(x, wk, wv, kc, vc, start, 1e6)
    wf.wf_kv_only_prefill(x, wf.tile_weights(wk), wf.tile_weights(wv), k2, v2, start, 1e6)
    torch.cuda.synchronize()
    assert torch.equal(kc.view(torch.int16), k2.view(torch.int16))
    assert torch.equal(vc.view(torch.int16), v2.view(torch.int16))


@pytest.mark.parametrize("L", [2, 36])
def test_prefill_layers_tiled_is_bit_exact(L):
    print(f"prefill layers tiled L={L}", flush=True)
    n, d_in, hkv, dh, start = 16, 4096, 8, 128, 1000
    cap = start + n
    x = W.normal((L, n, d_in), 1.0, 4, BF, DEV)
    wk = W.normal((L, hkv * dh, d_in), 0.02, 5, BF, DEV)
    wv = W.normal((L, hkv * dh, d_in), 0.02, 6, BF, DEV)
    kc = torch.zeros((L, hkv, cap, dh), dtype=BF, device=DEV)
    vc = torch.zeros_like(kc)
    k2, v2 = kc.clone(), vc.clone()
    wf.wf_kv_only_prefill_layers(x, wk, wv, kc, vc, start, 1e6)
    wf.wf_kv_only_prefill_layers(x, wf.tile_weights(wk), wf.tile_weights(wv), k2, v2, start, 1e6)
    torch.cuda.synchronize()
    assert torch.equal(kc.view(torch.int16), k2.view(torch.int16))
    assert torch.equal(vc.view(torch.int16), v2.view(torch.int16))


@pytest.mark.parametrize("gamma,d,vocab", [(16, 4096, 151936), (16, 4096, 50001), (8, 5120, 3001),
                                           (61, 4096, 151936), (33, 512, 70001), (16, 1024, 2000)])
def test_lmhead_tiled_is_bit_exact(gamma, d, vocab):
    print(f"LM head tiled gamma={gamma} d={d} vocab={vocab}", flush=True)
    h = W.normal((gamma, d), 1.0, W.stream_seed(gamma + d, "h"), BF, DEV)
    w = W.normal((vocab, d), 0.05, W.stream_seed(vocab, "w_lm"), BF, DEV)
    draft = torch.zeros(max(gamma - 1, 1), dtype=torch.int32, device=DEV)
    outs = []
    for wl in (w, wf.tile_weights(w)):
        am = torch.empty(gamma, dtype=torch.int32, device=DEV)
        ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
        acc = torch.empty(3, dtype=torch.int32, device=DEV)
        wf.wf_lmhead_accept_entropy(h, wl, None, draft, 1.0, am, ent, acc)
        outs.append((am, ent, acc))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("M,backlog", [(16, 0), (1, 0), (0, 80)])
def test_drafter_tiled_is_bit_exact(M, backlog):
    """The drafter layer (forward of M tokens, or catch-up over a backlog)
    with its seven projections tiled gives the row-major call's bits."""
    import dataclasses
    print(f"drafter tiled M={M} backlog={backlog}", flush=True)
    n = M or backlog
    w = dataclasses.replace(W.CONFIGS[7], cfg=77, ctx_len=1000, n_prefill=n,
                            prefill_start=1000, prefill_cap=1000 + n)
    t = W.generate_drafter(w, device=DEV)
    names = W.DECODER_WEIGHTS
    row = wf.decoder_layer({k: t[k] for k in names}, w.n_q_heads, w.n_kv_heads,
                           w.rms_eps, w.rope_base)
    tiled = wf.decoder_layer({k: (t[k] if k.endswith("norm") else wf.tile_weights(t[k]))
                              for k in names}, w.n_q_heads, w.n_kv_heads, w.rms_eps,
                             w.rope_base)
    assert tiled.tiled and not row.tiled
    res = []
    for layer in (row, tiled):
        kc, vc = t["k_cache"].clone(), t["v_cache"].clone()
        if M:
            out = torch.empty((M, w.hidden), dtype=BF, device=DEV)
            wf.wf_drafter_forward(layer, t["r"], 1000, kc, vc, out)
        else:
            out = torch.empty(w.hidden, dtype=BF, device=DEV)
            wf.wf_drafter_catchup(layer, t["r"], 1000, kc, vc, out)
        res.append((out, kc, vc))
    torch.cuda.synchronize()
    for a, b in zip(*res):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
