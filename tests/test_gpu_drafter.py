"""GPU parity of the drafter side of a switch (Sec. 3.4): one full decoder
layer (RMSNorm, GQA attention with RoPE, SwiGLU MLP, both residuals) over M
new tokens, and lazy catch-up -- KV-only prefill for every backlog token but
the last, the full layer for the last -- against the fp64 oracle.

The GPU rounds each activation to bf16 between steps, as a bf16 model
stores them; the bar is the bf16 one (max-norm relative error per output
vector), for the layer output and for every K/V cache row written.  Rows
the call must not write are checked unchanged, bit for bit."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import TOL, host64, max_vec_rel_err

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
COUNTER_BLOCK = 4 << 20


def _workload(hidden, nqh, nkvh, hd, inter, pos, n_rows, seed_cfg):
    base = W.CONFIGS[7]
    return dataclasses.replace(
        base, cfg=seed_cfg, hidden=hidden, n_q_heads=nqh, n_kv_heads=nkvh,
        head_dim=hd, inter=inter, ctx_len=pos, n_prefill=n_rows,
        prefill_start=pos, prefill_cap=pos + n_rows,
        qkv_std=0.02 * np.sqrt(hidden))


def _setup(w, extra_cap=3):
    t = W.generate_drafter(w, device=DEV)
    if extra_cap:
        # spare rows past the written ones: must stay untouched
        pad = lambda c: torch.cat([c, torch.full((c.shape[0], extra_cap, c.shape[2]), 7.0,
                                                 dtype=c.dtype, device=DEV)], dim=1)
        t["k_cache"], t["v_cache"] = pad(t["k_cache"]), pad(t["v_cache"])
    layer_w = {n: t[n] for n in W.DECODER_WEIGHTS}
    layer = wf.decoder_layer(layer_w, w.n_q_heads, w.n_kv_heads, w.rms_eps, w.rope_base)
    host = {n: W.to_oracle(t[n]) for n in W.DECODER_WEIGHTS}
    return t, layer, host


def _check_cache(kc_gpu, kc0, ref, lo, hi):
    """Rows [lo, hi) within the bar against the oracle; the rest unchanged."""
    got = host64(kc_gpu)
    assert max_vec_rel_err(got[:, lo:hi], ref[:, lo:hi]) <= TOL["bf16"]
    before = kc0.view(torch.int16).cpu()
    after = kc_gpu.view(torch.int16).cpu()
    assert torch.equal(before[:, :lo], after[:, :lo])
    assert torch.equal(before[:, hi:], after[:, hi:])


FORWARD_CASES = [
    # hidden, n_q_heads, n_kv_heads, head_dim, inter, pos, M
    (512, 4, 2, 128, 1024, 300, 1),
    (512, 4, 2, 128, 1024, 300, 16),
    (512, 8, 2, 64, 1536, 0, 5),
    (1024, 8, 8, 128, 2048, 1000, 33),
    (768, 6, 3, 128, 2048, 77, 64),
    (4096, 32, 8, 128, 12288, 1024, 1),
    (4096, 32, 8, 128, 12288, 700, 16),
    (4096, 32, 8, 128, 12288, 2000, 64),
    # 34 feature blocks in W_o and W_down: two blocks per workgroup, with
    # one and with two 16-row blocks; four blocks per workgroup elsewhere
    (544, 4, 2, 64, 1056, 50, 14),
    (544, 4, 2, 64, 1056, 50, 27),
    # 1032 feature blocks in [W_gate; W_up]: six blocks per workgroup, with
    # two and with three 16-row blocks
    (256, 2, 1, 128, 8256, 30, 20),
    (256, 2, 1, 128, 8256, 30, 40),
]


@pytest.mark.parametrize("hidden,nqh,nkvh,hd,inter,pos,M", FORWARD_CASES)
def test_forward_matches_oracle(hidden, nqh, nkvh, hd, inter, pos, M):
    print(f"drafter forward hidden={hidden} heads={nqh}/{nkvh}x{hd} inter={inter} "
          f"pos={pos} M={M}", flush=True)
    w = _workload(hidden, nqh, nkvh, hd, inter, pos, M, seed_cfg=70 + M + pos)
    t, layer, host = _setup(w)
    kc0, vc0 = t["k_cache"].clone(), t["v_cache"].clone()
    out = torch.empty((M, hidden), dtype=torch.bfloat16, device=DEV)
    wf.wf_drafter_forward(layer, t["r"], pos, t["k_cache"], t["v_cache"], out)
    torch.cuda.synchronize()
    ref, kref, vref = oracle.decoder_forward(
        W.to_oracle(t["r"]), pos, host, W.to_oracle(kc0), W.to_oracle(vc0),
        nqh, nkvh, w.rms_eps, w.rope_base)
    assert np.isfinite(host64(out)).all()
    assert max_vec_rel_err(host64(out), ref) <= TOL["bf16"]
    _check_cache(t["k_cache"], kc0, kref, pos, pos + M)
    _check_cache(t["v_cache"], vc0, vref, pos, pos + M)


CATCHUP_CASES = [
    # hidden, n_q_heads, n_kv_heads, head_dim, inter, pos, backlog
    (512, 4, 2, 128, 1024, 200, 1),
    (512, 4, 2, 128, 1024, 200, 2),
    (512, 4, 2, 64, 1024, 0, 37),
    (1024, 8, 4, 128, 2048, 513, 80),
    (4096, 32, 8, 128, 12288, 4096, 80),
    (1024, 8, 4, 128, 2048, 100, 500),         # two-pair units beside q in one launch
    (256, 4, 2, 64, 512, 10, 4096),            # the largest single prefill batch
    (256, 4, 2, 64, 512, 3, 9000),             # three batches: 4096 + 4096 + 808
]


@pytest.mark.parametrize("hidden,nqh,nkvh,hd,inter,pos,n", CATCHUP_CASES)
def test_catchup_matches_oracle(hidden, nqh, nkvh, hd, inter, pos, n):
    print(f"drafter catch-up hidden={hidden} heads={nqh}/{nkvh}x{hd} inter={inter} "
          f"pos={pos} backlog={n}", flush=True)
    w = _workload(hidden, nqh, nkvh, hd, inter, pos, n, seed_cfg=170 + n + pos)
    t, layer, host = _setup(w)
    kc0, vc0 = t["k_cache"].clone(), t["v_cache"].clone()
    out = torch.empty(hidden, dtype=torch.bfloat16, device=DEV)
    wf.wf_drafter_catchup(layer, t["r"], pos, t["k_cache"], t["v_cache"], out)
    torch.cuda.synchronize()
    ref, kref, vref = oracle.catchup(
        W.to_oracle(t["r"]), pos, host, W.to_oracle(kc0), W.to_oracle(vc0),
        nqh, nkvh, w.rms_eps, w.rope_base)
    assert max_vec_rel_err(host64(out)[None], ref[None]) <= TOL["bf16"]
    _check_cache(t["k_cache"], kc0, kref, pos, pos + n)
    _check_cache(t["v_cache"], vc0, vref, pos, pos + n)


def test_catchup_agrees_with_full_forward():
    """Catch-up's output is the last row of the full layer run over the
    whole backlog at once (the backlog tokens' own outputs are what
    catch-up skips), and both leave the same K/V rows."""
    print("drafter catch-up vs full forward", flush=True)
    w = _workload(1024, 8, 2, 128, 2048, 400, 24, seed_cfg=4242)
    t, layer, _ = _setup(w, extra_cap=0)
    kf, vf = t["k_cache"].clone(), t["v_cache"].clone()
    full = torch.empty((24, 1024), dtype=torch.bfloat16, device=DEV)
    wf.wf_drafter_forward(layer, t["r"], 400, kf, vf, full)
    out = torch.empty(1024, dtype=torch.bfloat16, device=DEV)
    wf.wf_drafter_catchup(layer, t["r"], 400, t["k_cache"], t["v_cache"], out)
    torch.cuda.synchronize()
    assert max_vec_rel_err(host64(out)[None], host64(full[-1])[None]) <= TOL["bf16"]
    assert max_vec_rel_err(host64(kf), host64(t["k_cache"])) <= TOL["bf16"]
    assert max_vec_rel_err(host64(vf), host64(t["v_cache"])) <= TOL["bf16"]


def test_shared_workspace_and_repeat():
    """One workspace, zero-filled once, serves calls of both kinds and
    sizes; each call leaves its counter block at zero and gives the same
    bits when repeated."""
    print("drafter workspace reuse", flush=True)
    w1 = _workload(512, 4, 2, 128, 1024, 900, 16, seed_cfg=501)
    w2 = _workload(512, 4, 2, 128, 1024, 100, 40, seed_cfg=502)
    t1, l1, _ = _setup(w1, extra_cap=0)
    t2, l2, _ = _setup(w2, extra_cap=0)
    need = max(wf.wf_drafter_forward_workspace_bytes(l1, 16, 900),
               wf.wf_drafter_catchup_workspace_bytes(l2, 40, 100))
    ws = wf.alloc_workspace(need, DEV)
    outs = []
    for _ in range(2):
        k1, v1 = t1["k_cache"].clone(), t1["v_cache"].clone()
        k2, v2 = t2["k_cache"].clone(), t2["v_cache"].clone()
        o1 = torch.empty((16, 512), dtype=torch.bfloat16, device=DEV)
        o2 = torch.empty(512, dtype=torch.bfloat16, device=DEV)
        wf.wf_drafter_forward(l1, t1["r"], 900, k1, v1, o1, workspace=ws)
        torch.cuda.synchronize()
        assert not bool(ws[:COUNTER_BLOCK].any().item())
        wf.wf_drafter_catchup(l2, t2["r"], 100, k2, v2, o2, workspace=ws)
        torch.cuda.synchronize()
        assert not bool(ws[:COUNTER_BLOCK].any().item())
        outs.append((o1, o2, k1, k2))
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
