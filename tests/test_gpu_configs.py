"""The five workload configurations at full size, in the launch configuration
the benchmark times (automatic split plan, same shapes), against the oracle.

Attention: the first and last layer, every (block row, q head) pair.
KV-only prefill: the same layers, all written rows.  LM head: every row,
argmax/entropy/accept, over 16 draft seeds per configuration, and the route
bit against the oracle's wherever the oracle's entropy at the accepted row
is farther from the threshold than the entropy bar (thresholds on both
sides of it); the router-heavy case also runs the logits-only mode.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import (TOL, accept_is_consistent, check_argmax, entropy_rel_err,
                    host64, max_vec_rel_err)

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_layers(cfg):
    w = W.CONFIGS[cfg]
    tol = TOL[w.dtype]
    for layer in sorted({0, w.n_layers - 1}):
        print(f"config {cfg} layer {layer}: generate", flush=True)
        t = W.generate_layer(w, layer, device=DEV)
        if w.n_prefill:
            kc = t["drafter_k_cache"] if w.separate_drafter_cache else t["k_cache"]
            vc = t["drafter_v_cache"] if w.separate_drafter_cache else t["v_cache"]
            # as the benchmark runs it: bf16 weights in the tiled layout
            tiled = w.dtype == "bf16"
            wk = wf.tile_weights(t["w_k"]) if tiled else t["w_k"]
            wv = wf.tile_weights(t["w_v"]) if tiled else t["w_v"]
            wf.wf_kv_only_prefill(t["x"], wk, wv, kc, vc, w.prefill_start, w.rope_base)
            torch.cuda.synchronize()
            kr, vr = oracle.kv_only_prefill(
                W.to_oracle(t["x"]), W.to_oracle(t["w_k"]),
                W.to_oracle(t["w_v"]), w.prefill_start, w.n_kv_heads,
                w.head_dim, w.rope_base)
            s0, s1 = w.prefill_start, w.prefill_start + w.n_prefill
            assert max_vec_rel_err(host64(kc[:, s0:s1]), kr) <= tol
            assert max_vec_rel_err(host64(vc[:, s0:s1]), vr) <= tol
            print(f"config {cfg} layer {layer}: prefill ok", flush=True)
        out = torch.empty_like(t["q"])
        wf.wf_verify_attn(t["q"], t["k_cache"], t["v_cache"], out, w.ctx_len)
        torch.cuda.synchronize()
        n = w.ctx_len + w.gamma
        ref = oracle.verify_attn(
            W.to_oracle(t["q"]), W.to_oracle(t["k_cache"][:, :n].contiguous()),
            W.to_oracle(t["v_cache"][:, :n].contiguous()), w.ctx_len)
        got = host64(out)
        assert np.isfinite(got).all()
        err = max_vec_rel_err(got, ref)
        print(f"config {cfg} layer {layer}: attention max rel err {err:.3e}",
              flush=True)
        assert err <= tol
        del t, out


def _lm(h, w_lm, logits, draft, tau, gamma):
    am = torch.empty(gamma, dtype=torch.int32, device=DEV)
    ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
    acc = torch.empty(3, dtype=torch.int32, device=DEV)
    dr = torch.as_tensor(draft, device=DEV)
    wf.wf_lmhead_accept_entropy(h, w_lm, logits, dr, tau, am, ent, acc)
    torch.cuda.synchronize()
    return am.cpu().numpy(), ent.cpu().numpy(), acc.cpu().numpy()


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_lmhead(cfg):
    w = W.CONFIGS[cfg]
    print(f"config {cfg}: LM head generate", flush=True)
    hd = W.generate_head(w, device=DEV)
    am_ref, ent_ref, margin, z = oracle.lmhead_rows(
        W.to_oracle(hd["h"]), W.to_oracle(hd["w_lm"]), want_logits=True)
    print(f"config {cfg}: LM head oracle done", flush=True)
    tau = float(np.median(ent_ref))
    bar = 1e-2 if w.dtype == "bf16" else 1e-6
    # as the benchmark runs it: bf16 W_lm in the tiled layout
    w_lm = wf.tile_weights(hd["w_lm"]) if w.dtype == "bf16" else hd["w_lm"]
    routes_checked = 0
    for ds in range(16):
        k = W.prefix_len(w, ds)
        draft = W.make_drafts(am_ref, k, w.vocab, 100 * cfg + ds)
        # the entropy bar at row k: thresholds just outside it on both sides
        # flip the route, the median threshold is wherever it falls
        eb = TOL[w.dtype] * max(abs(ent_ref[k]), 1e-3)
        for t in (tau, ent_ref[k] + 3 * eb, ent_ref[k] - 3 * eb):
            t = float(t)
            am, ent, acc = _lm(hd["h"], w_lm, None, draft, t, w.gamma)
            if ds == 0 and t == tau:
                check_argmax(am, am_ref, margin, z, w.dtype)
                assert entropy_rel_err(ent, ent_ref) <= TOL[w.dtype]
            assert accept_is_consistent(acc[0], acc[1], acc[2], am, ent, draft, t)
            n = int(acc[0])
            if all(margin[j] > bar for j in range(k + 1)):
                assert n == k and acc[1] == am_ref[k]
                n_ref, _, route_ref, _ = oracle.accept(am_ref, ent_ref, draft, t)
                assert n_ref == n
            else:
                route_ref = int(ent_ref[n] > t)
            # the route bit against the oracle's entropy, wherever the GPU
            # entropy bar cannot put it on the other side of the threshold
            if abs(ent_ref[n] - t) > TOL[w.dtype] * max(abs(ent_ref[n]), 1e-3):
                assert int(acc[2]) == route_ref, (ds, t, ent_ref[n])
                routes_checked += 1
    assert routes_checked >= 32
    if w.router_logits:
        zl = hd["router_logits"].contiguous()
        am_r, ent_r, _ = oracle.lmhead_rows(logits=zl.cpu().numpy())
        draft = W.make_drafts(am_r, 4, w.vocab, 7)
        am, ent, acc = _lm(None, None, zl, draft, 1.0, w.gamma)
        np.testing.assert_array_equal(am, am_r)
        assert entropy_rel_err(ent, ent_r) <= 1e-4
        assert tuple(acc) == oracle.accept(am_r, ent_r, draft, 1.0)[:3]
