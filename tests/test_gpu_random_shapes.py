"""Seeded random-shape GPU parity sweep against the fp64 oracle: verify
attention (block-causal and tree masks, Sec. 3.2), KV-only prefill (Sec.
3.4; one layer, and all layers in one launch), the LM head with acceptance
and entropy (Sec. 3.3.1) or with tree acceptance (Sec. 3.1), the drafter
layer of the switch path (full layer and lazy catch-up, Sec. 3.4) and the
neural routing policy (Sec. 3.3.2), over shapes drawn from the ranges the C
ABI accepts (tests/random_cases.py: gamma 1..64, ragged context and
vocabulary, head_dim 64 and 128, fp32 and bf16, row-major and tiled
weights).  Each test runs a bounded number of cases from a fixed seed,
prints every case before it runs, and stops at the first mismatch.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
import random_cases as R
import workloads as W
from parity import (TOL, accept_is_consistent, check_argmax, check_tree_accept,
                    entropy_rel_err, host64, max_vec_rel_err)

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def test_attention_random_shapes():
    for c in R.attn_cases():
        print(f"random attn #{c['case']}: {c['dt']} gamma={c['gamma']} "
              f"ctx={c['ctx']} hq={c['hq']} hkv={c['hkv']} dh={c['dh']} "
              f"splits={c['splits']} tree={c['tree']} std={c['std']}", flush=True)
        dt, gamma, ctx, seed = c["dt"], c["gamma"], c["ctx"], c["seed"]
        hq, hkv, dh, cap, std = c["hq"], c["hkv"], c["dh"], c["cap"], c["std"]
        q = W.normal((gamma, hq, dh), std, W.stream_seed(seed, "q"), DT[dt], DEV)
        k = W.normal((hkv, cap, dh), std, W.stream_seed(seed, "k_cache"), DT[dt], DEV)
        v = W.normal((hkv, cap, dh), std, W.stream_seed(seed, "v_cache"), DT[dt], DEV)
        k[:, ctx + gamma:] = float("nan")       # past the block: never read
        v[:, ctx + gamma:] = float("nan")
        out = torch.empty_like(q)
        n = ctx + gamma
        kk = W.to_oracle(k[:, :n].contiguous())
        vv = W.to_oracle(v[:, :n].contiguous())
        if c["tree"]:
            mask = W.ancestor_masks(c["parents"])
            md = torch.from_numpy(mask.view(np.int64).copy()).to(DEV)
            wf.wf_verify_attn_tree(q, k, v, out, ctx, md, num_splits=c["splits"])
            torch.cuda.synchronize()
            ref = oracle.verify_attn_mask(W.to_oracle(q), kk, vv, ctx, mask)
        else:
            wf.wf_verify_attn(q, k, v, out, ctx, num_splits=c["splits"])
            torch.cuda.synchronize()
            ref = oracle.verify_attn(W.to_oracle(q), kk, vv, ctx)
        got = host64(out)
        assert np.isfinite(got).all(), c["case"]
        err = max_vec_rel_err(got, ref)
        assert err <= TOL[dt], (c["case"], err)


def test_prefill_random_shapes():
    for c in R.prefill_cases():
        print(f"random prefill #{c['case']}: {c['dt']} tiled={c['tiled']} "
              f"n={c['n']} d_in={c['d_in']} hkv={c['hkv']} dh={c['dh']} "
              f"start={c['start']} base={c['base']:g}", flush=True)
        dt, n, d_in, hkv, dh = c["dt"], c["n"], c["d_in"], c["hkv"], c["dh"]
        start, seed = c["start"], c["seed"]
        xs = 1.0 if dt == "bf16" else 0.5
        x = W.normal((n, d_in), xs, W.stream_seed(seed, "x"), DT[dt], DEV)
        wk = W.normal((hkv * dh, d_in), 0.02, W.stream_seed(seed, "w_k"), DT[dt], DEV)
        wv = W.normal((hkv * dh, d_in), 0.02, W.stream_seed(seed, "w_v"), DT[dt], DEV)
        kc = torch.zeros((hkv, c["cap"], dh), dtype=DT[dt], device=DEV)
        vc = torch.zeros_like(kc)
        wkp = wf.tile_weights(wk) if c["tiled"] else wk
        wvp = wf.tile_weights(wv) if c["tiled"] else wv
        wf.wf_kv_only_prefill(x, wkp, wvp, kc, vc, start, c["base"])
        torch.cuda.synchronize()
        kr, vr = oracle.kv_only_prefill(W.to_oracle(x), W.to_oracle(wk),
                                        W.to_oracle(wv), start, hkv, dh, c["base"])
        ek = max_vec_rel_err(host64(kc[:, start:start + n]), kr)
        ev = max_vec_rel_err(host64(vc[:, start:start + n]), vr)
        assert ek <= TOL[dt] and ev <= TOL[dt], (c["case"], ek, ev)
        # rows outside the catch-up stay untouched
        assert not kc[:, :start].any() and not kc[:, start + n:].any(), c["case"]
        assert not vc[:, :start].any() and not vc[:, start + n:].any(), c["case"]


def test_lmhead_random_shapes():
    for c in R.lmhead_cases():
        print(f"random lmhead #{c['case']}: {c['dt']} tiled={c['tiled']} "
              f"gamma={c['gamma']} d={c['d']} vocab={c['vocab']} "
              f"w_std={c['w_std']}", flush=True)
        dt, gamma, d, vocab, seed = c["dt"], c["gamma"], c["d"], c["vocab"], c["seed"]
        h = W.normal((gamma, d), 1.0, W.stream_seed(seed, "h"), DT[dt], DEV)
        w = W.normal((vocab, d), c["w_std"], W.stream_seed(seed, "w_lm"), DT[dt], DEV)
        am_ref, ent_ref, margin, z = oracle.lmhead_rows(W.to_oracle(h), W.to_oracle(w),
                                                        want_logits=True)
        k = W.geometric_prefix(0.3, gamma, seed)
        draft = W.make_drafts(am_ref, k, vocab, seed)
        tau = float(np.median(ent_ref))
        am = torch.empty(gamma, dtype=torch.int32, device=DEV)
        ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
        acc = torch.empty(3, dtype=torch.int32, device=DEV)
        dr = torch.as_tensor(draft, device=DEV) if gamma > 1 else None
        wl = wf.tile_weights(w) if c["tiled"] else w
        wf.wf_lmhead_accept_entropy(h, wl, None, dr, tau, am, ent, acc)
        torch.cuda.synchronize()
        am, ent, acc = am.cpu().numpy(), ent.cpu().numpy(), acc.cpu().numpy()
        check_argmax(am, am_ref, margin, z, dt)
        assert entropy_rel_err(ent, ent_ref) <= TOL[dt], c["case"]
        assert accept_is_consistent(acc[0], acc[1], acc[2], am, ent, draft, tau), c["case"]
        bar = 1e-2 if dt == "bf16" else 1e-6
        if all(margin[j] > bar for j in range(min(k, gamma - 1) + 1)):
            n_ref, bonus_ref, route_ref, _ = oracle.accept(am_ref, ent_ref, draft, tau)
            assert (acc[0], acc[1]) == (n_ref, bonus_ref), c["case"]
            if abs(ent_ref[n_ref] - tau) > TOL[dt] * max(abs(ent_ref[n_ref]), 1e-3):
                assert acc[2] == route_ref, c["case"]


def test_drafter_random_shapes():
    """The drafter layer (Sec. 3.4 switch path): full layer over a few
    tokens or lazy catch-up over a backlog, against the oracle; written
    cache rows within the bar, every other row unchanged bit for bit."""
    for c in R.drafter_cases():
        print(f"random drafter #{c['case']}: {c['kind']} hidden={c['hidden']} "
              f"heads={c['hq']}/{c['hkv']}x{c['dh']} inter={c['inter']} pos={c['pos']} "
              f"n={c['n']} tiled={c['tiled']}", flush=True)
        hidden, hq, hkv, pos, n = c["hidden"], c["hq"], c["hkv"], c["pos"], c["n"]
        w = dataclasses.replace(W.CONFIGS[7], cfg=c["cfg"], hidden=hidden, n_q_heads=hq,
                                n_kv_heads=hkv, head_dim=c["dh"], inter=c["inter"],
                                ctx_len=pos, n_prefill=n, prefill_start=pos,
                                prefill_cap=pos + n, qkv_std=0.02 * np.sqrt(hidden))
        t = W.generate_drafter(w, device=DEV)
        spare = lambda x: torch.cat([x, torch.full((x.shape[0], 2, x.shape[2]), 7.0,
                                                   dtype=x.dtype, device=DEV)], dim=1)
        kc, vc = spare(t["k_cache"]), spare(t["v_cache"])
        kc0, vc0 = kc.clone(), vc.clone()
        names = W.DECODER_WEIGHTS
        weights = {k: (t[k] if k.endswith("norm") or not c["tiled"] else wf.tile_weights(t[k]))
                   for k in names}
        layer = wf.decoder_layer(weights, hq, hkv, w.rms_eps, w.rope_base)
        host = {k: W.to_oracle(t[k]) for k in names}
        if c["kind"] == "catchup":
            out = torch.empty(hidden, dtype=torch.bfloat16, device=DEV)
            wf.wf_drafter_catchup(layer, t["r"], pos, kc, vc, out)
            torch.cuda.synchronize()
            ref, kref, vref = oracle.catchup(W.to_oracle(t["r"]), pos, host, W.to_oracle(kc0),
                                             W.to_oracle(vc0), hq, hkv, w.rms_eps, w.rope_base)
            got, ref = host64(out)[None], ref[None]
        else:
            out = torch.empty((n, hidden), dtype=torch.bfloat16, device=DEV)
            wf.wf_drafter_forward(layer, t["r"], pos, kc, vc, out)
            torch.cuda.synchronize()
            ref, kref, vref = oracle.decoder_forward(
                W.to_oracle(t["r"]), pos, host, W.to_oracle(kc0), W.to_oracle(vc0),
                hq, hkv, w.rms_eps, w.rope_base)
            got = host64(out)
        assert np.isfinite(got).all(), c["case"]
        err = max_vec_rel_err(got, ref)
        assert err <= TOL["bf16"], (c["case"], "out", err)
        for name, g, g0, r in (("k", kc, kc0, kref), ("v", vc, vc0, vref)):
            e = max_vec_rel_err(host64(g)[:, pos:pos + n], r[:, pos:pos + n])
            assert e <= TOL["bf16"], (c["case"], name, e)
            before, after = g0.view(torch.int16).cpu(), g.view(torch.int16).cpu()
            assert torch.equal(before[:, :pos], after[:, :pos]), (c["case"], name)
            assert torch.equal(before[:, pos + n:], after[:, pos + n:]), (c["case"], name)


def _router_scale(h, w1, b1, w2, b2):
    """|b2| + sum_u |w2_u GELU(z_u)| per row: the size of the terms the
    predicted gain sums, which bounds its rounding error."""
    h, w1, b1, w2, b2 = (t.double().cpu().numpy() for t in (h, w1, b1, w2, b2))
    z = h @ w1.T + b1
    g = 0.5 * z * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))
    return np.abs(b2[0]) + np.abs(g * w2).sum(axis=1)


def test_router_random_shapes():
    """The neural routing policy (Sec. 3.3.2): the predicted gain of every
    row within the router's bar (TOL x the size of the terms it sums) and
    the route at a device-named row, against the oracle."""
    for c in R.router_cases():
        print(f"random router #{c['case']}: {c['dt']} gamma={c['gamma']} d={c['d']} "
              f"m={c['m']}", flush=True)
        dt, gamma, d, m, seed = c["dt"], c["gamma"], c["d"], c["m"], c["seed"]
        h = W.normal((gamma, d), 1.0, W.stream_seed(seed, "h"), DT[dt], DEV)
        w1 = W.normal((m, d), 0.02, W.stream_seed(seed, "router_w1"), DT[dt], DEV)
        b1 = W.normal((m,), 0.02, W.stream_seed(seed, "router_b1"), DT[dt], DEV)
        w2 = W.normal((m,), 0.05, W.stream_seed(seed, "router_w2"), DT[dt], DEV)
        b2 = W.normal((1,), 0.05, W.stream_seed(seed, "router_b2"), DT[dt], DEV)
        ref = oracle.router_mlp(*(W.to_oracle(t) for t in (h, w1, b1, w2, b2)))
        scale = _router_scale(h, w1, b1, w2, b2)
        tau = float(np.float32(np.median(ref)))
        row = gamma - 1 - c["case"] % gamma
        rowt = torch.tensor([row], dtype=torch.int32, device=DEV)
        delta = torch.empty(gamma, dtype=torch.float32, device=DEV)
        route = torch.empty(1, dtype=torch.int32, device=DEV)
        wf.wf_router_neural(h, w1, b1, w2, b2, rowt, tau, delta, route)
        torch.cuda.synchronize()
        got = delta.cpu().numpy().astype(np.float64)
        assert np.isfinite(got).all(), c["case"]
        assert np.all(np.abs(got - ref) <= TOL[dt] * scale), (c["case"], np.abs(got - ref).max())
        assert int(route[0]) == int(got[row] > tau), c["case"]
        if abs(ref[row] - tau) > TOL[dt] * scale[row]:
            assert int(route[0]) == oracle.route_neural(ref, row, tau), c["case"]


def test_tree_lmhead_random_shapes():
    """Tree verification's LM head (Sec. 3.1 draft trees verified in one
    pass, Sec. 3.3.1 route): argmax and entropy of every node, then the
    accepted path, its bonus token and the route, against the oracle."""
    for c in R.tree_lmhead_cases():
        print(f"random tree lmhead #{c['case']}: gamma={c['gamma']} d={c['d']} "
              f"vocab={c['vocab']} tiled={c['tiled']} k={c['k']}", flush=True)
        gamma, d, vocab, seed, par = c["gamma"], c["d"], c["vocab"], c["seed"], c["parents"]
        h = W.normal((gamma, d), 1.0, W.stream_seed(seed, "h"), torch.bfloat16, DEV)
        w = W.normal((vocab, d), 0.05, W.stream_seed(seed, "w_lm"), torch.bfloat16, DEV)
        am_ref, ent_ref, margin, z = oracle.lmhead_rows(W.to_oracle(h), W.to_oracle(w),
                                                        want_logits=True)
        tok = W.tree_tokens(am_ref, par, c["k"], vocab, seed)
        tau = float(np.float32(np.median(ent_ref) + 1e-3))
        am = torch.empty(gamma, dtype=torch.int32, device=DEV)
        ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
        acc = torch.empty(4, dtype=torch.int32, device=DEV)
        path = torch.empty(gamma, dtype=torch.int32, device=DEV)
        wl = wf.tile_weights(w) if c["tiled"] else w
        wf.wf_lmhead_accept_tree(h, wl, None, torch.from_numpy(tok).to(DEV),
                                 torch.from_numpy(par).to(DEV), tau, am, ent, acc, path)
        torch.cuda.synchronize()
        am, ent, acc, path = (t.cpu().numpy() for t in (am, ent, acc, path))
        check_argmax(am, am_ref, margin, z, "bf16")
        assert entropy_rel_err(ent, ent_ref) <= TOL["bf16"], c["case"]
        check_tree_accept(am, ent, acc, path, am_ref, ent_ref, margin, tok, par, tau, 1e-2)


def test_layer_prefill_random_shapes():
    """All layers' KV-only prefill in one launch (Sec. 3.4): every layer's
    written rows against the oracle, the other rows unchanged."""
    for c in R.layer_prefill_cases():
        print(f"random layer prefill #{c['case']}: layers={c['layers']} n={c['n']} "
              f"d_in={c['d_in']} hkv={c['hkv']} dh={c['dh']} start={c['start']} "
              f"tiled={c['tiled']}", flush=True)
        L, n, d_in, hkv, dh, start, seed = (c[k] for k in ("layers", "n", "d_in", "hkv", "dh",
                                                            "start", "seed"))
        cap = start + n + 2
        bf = torch.bfloat16
        x = W.normal((L, n, d_in), 1.0, W.stream_seed(seed, "x"), bf, DEV)
        wk = W.normal((L, hkv * dh, d_in), 0.02, W.stream_seed(seed, "w_k"), bf, DEV)
        wv = W.normal((L, hkv * dh, d_in), 0.02, W.stream_seed(seed, "w_v"), bf, DEV)
        kc = W.normal((L, hkv, cap, dh), 1.0, W.stream_seed(seed, "k_cache"), bf, DEV)
        vc = W.normal((L, hkv, cap, dh), 1.0, W.stream_seed(seed, "v_cache"), bf, DEV)
        k0, v0 = kc.clone(), vc.clone()
        wkt, wvt = (wf.tile_weights(wk), wf.tile_weights(wv)) if c["tiled"] else (wk, wv)
        wf.wf_kv_only_prefill_layers(x, wkt, wvt, kc, vc, start, 1e6)
        torch.cuda.synchronize()
        rows = slice(start, start + n)
        for l in range(L):
            kr, vr = oracle.kv_only_prefill(W.to_oracle(x[l]), W.to_oracle(wk[l]),
                                            W.to_oracle(wv[l]), start, hkv, dh, 1e6)
            assert max_vec_rel_err(host64(kc[l][:, rows]), kr) <= TOL["bf16"], (c["case"], l)
            assert max_vec_rel_err(host64(vc[l][:, rows]), vr) <= TOL["bf16"], (c["case"], l)
        for a, b in ((kc, k0), (vc, v0)):
            assert torch.equal(a[:, :, :start], b[:, :, :start]), c["case"]
            assert torch.equal(a[:, :, start + n:], b[:, :, start + n:]), c["case"]
