"""The verification calls captured in a HIP graph: a step (attention, KV-only
prefill with tiled weights, LM head with acceptance, the neural router at
the accepted row) is recorded once and replayed several times, with eager
work and synchronisations between the replays; every replay must give the
bits of the eager step.  The calls allocate nothing, memset nothing and
leave their workspace counters at zero, so one capture serves any number of
replays."""
import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
BF = torch.bfloat16


def test_step_replays_match_eager():
    print("graph replay of a small verification step", flush=True)
    g, ctx, hq, hkv, dh, d, vocab, n_pre = 16, 3000, 16, 4, 128, 1024, 20000, 8
    cap = ctx + g + n_pre
    q = W.normal((g, hq, dh), 1.0, 1, BF, DEV)
    kc = W.normal((hkv, cap, dh), 1.0, 2, BF, DEV)
    vc = W.normal((hkv, cap, dh), 1.0, 3, BF, DEV)
    x = W.normal((n_pre, d), 1.0, 4, BF, DEV)
    wk = wf.tile_weights(W.normal((hkv * dh, d), 0.02, 5, BF, DEV))
    wv = wf.tile_weights(W.normal((hkv * dh, d), 0.02, 6, BF, DEV))
    h = W.normal((g, d), 1.0, 7, BF, DEV)
    wl = wf.tile_weights(W.normal((vocab, d), 0.05, 8, BF, DEV))
    m = d // 8
    w1 = W.normal((m, d), 0.02, 9, BF, DEV)
    b1 = W.normal((m,), 0.02, 10, BF, DEV)
    w2 = W.normal((m,), 0.05, 11, BF, DEV)
    b2 = W.normal((1,), 0.05, 12, BF, DEV)
    draft = torch.zeros(g - 1, dtype=torch.int32, device=DEV)

    ws_a = wf.alloc_workspace(wf.wf_verify_attn_workspace_bytes(1, g, ctx, hq, hkv, dh), DEV)
    ws_p = wf.alloc_workspace(wf.wf_kv_only_prefill_workspace_bytes(2, n_pre, d, hkv, dh), DEV)
    ws_l = wf.alloc_workspace(wf.wf_lmhead_workspace_bytes(g, vocab), DEV)
    ws_r = wf.alloc_workspace(int(wf.lib.wf_router_workspace_bytes(1, g, d, m)), DEV)
    out = torch.empty_like(q)
    am = torch.empty(g, dtype=torch.int32, device=DEV)
    ent = torch.empty(g, dtype=torch.float32, device=DEV)
    acc = torch.empty(3, dtype=torch.int32, device=DEV)
    delta = torch.empty(g, dtype=torch.float32, device=DEV)
    route = torch.empty(1, dtype=torch.int32, device=DEV)

    def step(stream=None):
        wf.wf_verify_attn(q, kc, vc, out, ctx, workspace=ws_a, stream=stream)
        wf.wf_kv_only_prefill(x, wk, wv, kc, vc, ctx + g, 1e6, workspace=ws_p, stream=stream)
        wf.wf_lmhead_accept_entropy(h, wl, None, draft, 1.0, am, ent, acc, workspace=ws_l,
                                    stream=stream)
        wf.wf_router_neural(h, w1, b1, w2, b2, acc[:1], 0.0, delta, route, workspace=ws_r,
                            stream=stream)

    def snapshot():
        torch.cuda.synchronize()
        return [t.clone() for t in (out, kc, vc, am, ent, acc, delta, route)]

    step()
    ref = snapshot()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(side)                      # warm the side stream before capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step(torch.cuda.current_stream())
    for rep in range(3):
        for t in (out, am, ent, acc, delta, route):
            t.zero_()
        graph.replay()
        got = snapshot()
        for a, b in zip(ref, got):
            assert torch.equal(a.view(torch.uint8) if a.dtype == BF else a,
                               b.view(torch.uint8) if b.dtype == BF else b), rep
        # eager work between replays, on the same workspaces
        step()
        torch.cuda.synchronize()
    assert not bool(ws_a[:4 << 20].any().item()) and not bool(ws_l[:4 << 20].any().item())
    assert int(route[0]) in (0, 1) and np.isfinite(delta.cpu().numpy()).all()


def test_tree_step_and_catchup_replay_match_eager():
    """Tree verification (masked attention, tree acceptance, path
    compaction of the caches) and a drafter catch-up, captured together."""
    import dataclasses
    print("graph replay of a tree step and a catch-up", flush=True)
    g, ctx, hq, hkv, dh, d, vocab = 61, 2000, 16, 4, 128, 1024, 5000
    cap = ctx + g
    par = W.draft_tree(seed=3)
    mask = torch.from_numpy(W.ancestor_masks(par).view(np.int64).copy()).to(DEV)
    parents = torch.from_numpy(par).to(DEV)
    q = W.normal((g, hq, dh), 1.0, 21, BF, DEV)
    kc0 = W.normal((hkv, cap, dh), 1.0, 22, BF, DEV)
    vc0 = W.normal((hkv, cap, dh), 1.0, 23, BF, DEV)
    h = W.normal((g, d), 1.0, 24, BF, DEV)
    wl = wf.tile_weights(W.normal((vocab, d), 0.05, 25, BF, DEV))
    tokens = torch.randint(0, vocab, (g,), generator=torch.Generator().manual_seed(5)).to(
        torch.int32).to(DEV)
    kc, vc = kc0.clone(), vc0.clone()
    out = torch.empty_like(q)
    am = torch.empty(g, dtype=torch.int32, device=DEV)
    ent = torch.empty(g, dtype=torch.float32, device=DEV)
    acc = torch.empty(4, dtype=torch.int32, device=DEV)
    path = torch.empty(g, dtype=torch.int32, device=DEV)
    ws_a = wf.alloc_workspace(wf.wf_verify_attn_workspace_bytes(1, g, ctx, hq, hkv, dh), DEV)
    ws_l = wf.alloc_workspace(wf.wf_lmhead_workspace_bytes(g, vocab), DEV)
    wd = dataclasses.replace(W.CONFIGS[7], cfg=91, hidden=512, n_q_heads=4, n_kv_heads=2,
                             head_dim=128, inter=1024, ctx_len=300, n_prefill=20,
                             prefill_start=300, prefill_cap=320)
    t = W.generate_drafter(wd, device=DEV)
    layer = wf.decoder_layer({k: (t[k] if k.endswith("norm") else wf.tile_weights(t[k]))
                              for k in W.DECODER_WEIGHTS}, 4, 2, wd.rms_eps, wd.rope_base)
    dout = torch.empty(512, dtype=BF, device=DEV)
    ws_d = wf.alloc_workspace(wf.wf_drafter_catchup_workspace_bytes(layer, 20, 300), DEV)
    lib = wf.lib

    def step(stream=None):
        s = wf._stream(stream)
        kc.copy_(kc0)
        vc.copy_(vc0)
        wf.wf_verify_attn_tree(q, kc, vc, out, ctx, mask, workspace=ws_a, stream=stream)
        wf.wf_lmhead_accept_tree(h, wl, None, tokens, parents, 1.0, am, ent, acc, path,
                                 workspace=ws_l, stream=stream)
        assert lib.wf_kv_compact_path(1, wf._dev(kc, "k"), wf._dev(vc, "v"),
                                      wf._dev(acc, "a"), wf._dev(path, "p"), g, ctx, cap,
                                      hkv, dh, 1, 0, s) == 0
        wf.wf_drafter_catchup(layer, t["r"], 300, t["k_cache"], t["v_cache"], dout,
                              workspace=ws_d, stream=stream)

    def snapshot():
        torch.cuda.synchronize()
        return [x.clone() for x in (out, am, ent, acc, path, kc, vc, dout, t["k_cache"])]

    step()
    ref = snapshot()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(torch.cuda.current_stream())
    for rep in range(3):
        for x in (out, am, ent, acc, path, dout):
            x.zero_()
        graph.replay()
        got = snapshot()
        for a, b in zip(ref, got):
            assert torch.equal(a.view(torch.uint8) if a.dtype == BF else a,
                               b.view(torch.uint8) if b.dtype == BF else b), rep
        step()
        torch.cuda.synchronize()
