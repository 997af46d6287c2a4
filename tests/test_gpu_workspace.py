"""GPU checks of the workspace contract: a workspace zero-filled once serves
any sequence of calls of the three kinds and of different sizes, every call
leaves the leading counter block at zero, and results do not depend on what
earlier calls left in the partial-result area.  Also covers the LM head at
a vocabulary of 2^28 entries."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import TOL, entropy_rel_err

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
COUNTER_BLOCK = 4 << 20


def _lm(h, w, logits, draft, ws):
    gamma = (logits if logits is not None else h).shape[0]
    am = torch.empty(gamma, dtype=torch.int32, device=DEV)
    ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
    acc = torch.empty(3, dtype=torch.int32, device=DEV)
    wf.wf_lmhead_accept_entropy(h, w, logits, draft, 1.0, am, ent, acc,
                                workspace=ws)
    return am, ent, acc


def _counters_zero(ws):
    torch.cuda.synchronize()
    return not bool(ws[:COUNTER_BLOCK].any().item())


def test_one_workspace_across_kinds_and_sizes():
    print("workspace reuse across kinds and sizes", flush=True)
    bf = torch.bfloat16
    # LM head, two sizes
    h1 = W.normal((16, 1024), 1.0, W.stream_seed(5, "h"), bf, DEV)
    w1 = W.normal((20000, 1024), 0.05, W.stream_seed(5, "w_lm"), bf, DEV)
    h2 = W.normal((5, 512), 1.0, W.stream_seed(6, "h"), bf, DEV)
    w2 = W.normal((3001, 512), 0.05, W.stream_seed(6, "w_lm"), bf, DEV)
    d1 = torch.zeros(15, dtype=torch.int32, device=DEV)
    d2 = torch.zeros(4, dtype=torch.int32, device=DEV)
    # prefill
    x = W.normal((70, 1024), 1.0, W.stream_seed(7, "x"), bf, DEV)
    wk = W.normal((4 * 128, 1024), 0.02, W.stream_seed(7, "w_k"), bf, DEV)
    wv = W.normal((4 * 128, 1024), 0.02, W.stream_seed(7, "w_v"), bf, DEV)
    # attention
    q = W.normal((16, 16, 128), 1.0, W.stream_seed(8, "q"), bf, DEV)
    kc = W.normal((4, 4000, 128), 1.0, W.stream_seed(8, "k_cache"), bf, DEV)
    vc = W.normal((4, 4000, 128), 1.0, W.stream_seed(8, "v_cache"), bf, DEV)

    need = max(wf.wf_lmhead_workspace_bytes(16, 20000),
               wf.wf_kv_only_prefill_workspace_bytes(1, 70, 1024, 4, 128),
               wf.wf_verify_attn_workspace_bytes(1, 16, 3054, 16, 4, 128))
    shared = wf.alloc_workspace(need, DEV)

    def fresh_lm(h, w, d):
        gamma, vocab = h.shape[0], w.shape[0]
        return _lm(h, w, None, d,
                   wf.alloc_workspace(wf.wf_lmhead_workspace_bytes(gamma, vocab), DEV))

    ref1, ref2 = fresh_lm(h1, w1, d1), fresh_lm(h2, w2, d2)
    kref, vref = kc.clone(), vc.clone()
    wf.wf_kv_only_prefill(x, wk, wv, kref, vref, 3000, 1e6)
    out_ref = torch.empty_like(q)
    wf.wf_verify_attn(q, kref, vref, out_ref, 3054)

    # the same calls, interleaved, through one workspace
    for _ in range(2):
        got1 = _lm(h1, w1, None, d1, shared)
        assert _counters_zero(shared)
        got2 = _lm(h2, w2, None, d2, shared)
        assert _counters_zero(shared)
        k2, v2 = kc.clone(), vc.clone()
        wf.wf_kv_only_prefill(x, wk, wv, k2, v2, 3000, 1e6, workspace=shared)
        assert _counters_zero(shared)
        out = torch.empty_like(q)
        wf.wf_verify_attn(q, k2, v2, out, 3054, workspace=shared)
        assert _counters_zero(shared)
        torch.cuda.synchronize()
        for a, b in zip(got1 + got2, ref1 + ref2):
            assert torch.equal(a, b)
        assert torch.equal(k2, kref) and torch.equal(v2, vref)
        assert torch.equal(out, out_ref)


def test_lmhead_reused_workspace_many_calls():
    """Back-to-back calls on one workspace without a host synchronisation in
    between: every call must see its counters at zero."""
    print("lmhead back-to-back calls on one workspace", flush=True)
    gamma, d, vocab = 16, 4096, 151936
    h = W.normal((gamma, d), 1.0, W.stream_seed(9, "h"), torch.bfloat16, DEV)
    w = W.normal((vocab, d), 0.02, W.stream_seed(9, "w_lm"), torch.bfloat16, DEV)
    dr = torch.zeros(gamma - 1, dtype=torch.int32, device=DEV)
    ws = wf.alloc_workspace(wf.wf_lmhead_workspace_bytes(gamma, vocab), DEV)
    first = _lm(h, w, None, dr, ws)
    outs = [_lm(h, w, None, dr, ws) for _ in range(20)]
    torch.cuda.synchronize()
    for o in outs:
        for a, b in zip(o, first):
            assert torch.equal(a, b)
    assert _counters_zero(ws)


def test_lmhead_logits_mode_huge_vocab():
    """2^28 logits in one row: 2^20 tile states for one finishing
    workgroup."""
    print("lmhead logits mode vocab 2^28", flush=True)
    vocab = 1 << 28
    g = torch.Generator(device=DEV)
    g.manual_seed(1234)
    z = torch.randn((1, vocab), generator=g, device=DEV, dtype=torch.float32)
    z[0, 987654321 % vocab] = 12.0          # a clear maximum (the rest stay below 7)
    ws = wf.alloc_workspace(wf.wf_lmhead_workspace_bytes(1, vocab), DEV)
    am, ent, acc = _lm(None, None, z, None, ws)
    torch.cuda.synchronize()
    am_ref, ent_ref, _ = oracle.lmhead_rows(logits=z.cpu().numpy())
    assert int(am[0]) == int(am_ref[0]) == 987654321 % vocab
    assert entropy_rel_err(ent.cpu().numpy(), ent_ref) <= 1e-4
    assert int(acc[0]) == 0 and int(acc[1]) == int(am_ref[0])
    assert _counters_zero(ws)
