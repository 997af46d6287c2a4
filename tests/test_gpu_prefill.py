"""GPU parity of wf_kv_only_prefill against the fp64 oracle (Sec. 3.4 KV-only
prefill): projected and rotated K, projected V, written only to rows
[start_pos, start_pos + n_tok); batched catch-up equals single-token
appends."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import TOL, host64, max_vec_rel_err

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _setup(dt, n, d_in, hkv, dh, start, seed, cap=None):
    cap = cap or start + n + 3
    dtype = DT[dt]
    xs = 0.02 if dt == "f32" else 1.0
    x = W.normal((n, d_in), xs, W.stream_seed(seed, "x"), dtype, DEV)
    wk = W.normal((hkv * dh, d_in), 0.02, W.stream_seed(seed, "w_k"), dtype, DEV)
    wv = W.normal((hkv * dh, d_in), 0.02, W.stream_seed(seed, "w_v"), dtype, DEV)
    kc = W.normal((hkv, cap, dh), 1.0, W.stream_seed(seed, "k_cache"), dtype, DEV)
    vc = W.normal((hkv, cap, dh), 1.0, W.stream_seed(seed, "v_cache"), dtype, DEV)
    return x, wk, wv, kc, vc


CASES = [
    # dt, n_tok, d_in, n_kv_heads, head_dim, start_pos, rope_base
    ("bf16", 1, 512, 1, 128, 0, 1e6),
    ("bf16", 4, 512, 2, 64, 252, 1e4),
    ("bf16", 16, 4096, 8, 128, 32784, 1e6),
    ("bf16", 17, 1024, 8, 128, 1000, 1e6),
    ("bf16", 32, 5120, 8, 128, 65552, 1e6),
    ("bf16", 70, 256, 2, 64, 5, 1e4),
    ("bf16", 80, 4096, 8, 128, 4096, 1e6),     # two-pair units, 48 + 32 tokens
    ("bf16", 200, 2048, 4, 128, 777, 1e6),     # two-pair units, four 16-token blocks each
    ("bf16", 100, 1024, 2, 64, 3, 1e4),        # two-pair units at head_dim 64
    ("bf16", 4096, 512, 2, 64, 100, 1e4),      # the largest catch-up a call takes
    ("f32", 4, 512, 2, 64, 252, 1e4),
    ("f32", 9, 100, 3, 128, 65000, 1e6),
]


@pytest.mark.parametrize("dt,n,d_in,hkv,dh,start,base", CASES)
def test_matches_oracle(dt, n, d_in, hkv, dh, start, base):
    print(f"prefill parity {dt} n={n} d_in={d_in} hkv={hkv} dh={dh} "
          f"start={start}", flush=True)
    x, wk, wv, kc, vc = _setup(dt, n, d_in, hkv, dh, start, seed=n * 17 + d_in)
    k0, v0 = kc.clone(), vc.clone()
    wf.wf_kv_only_prefill(x, wk, wv, kc, vc, start, base)
    torch.cuda.synchronize()
    kr, vr = oracle.kv_only_prefill(W.to_oracle(x), W.to_oracle(wk),
                                    W.to_oracle(wv), start, hkv, dh, base)
    kg = host64(kc[:, start:start + n])
    vg = host64(vc[:, start:start + n])
    assert max_vec_rel_err(kg, kr) <= TOL[dt]
    assert max_vec_rel_err(vg, vr) <= TOL[dt]
    # nothing outside the catch-up rows changes
    assert torch.equal(kc[:, :start], k0[:, :start])
    assert torch.equal(kc[:, start + n:], k0[:, start + n:])
    assert torch.equal(vc[:, :start], v0[:, :start])
    assert torch.equal(vc[:, start + n:], v0[:, start + n:])


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_batched_equals_single_token_appends(dt):
    n, d_in, hkv, dh, start = 12, 512, 2, 128, 40000
    x, wk, wv, kc, vc = _setup(dt, n, d_in, hkv, dh, start, seed=3)
    kb, vb = kc.clone(), vc.clone()
    wf.wf_kv_only_prefill(x, wk, wv, kb, vb, start, 1e6)
    for t in range(n):
        wf.wf_kv_only_prefill(x[t:t + 1].contiguous(), wk, wv, kc, vc,
                              start + t, 1e6)
    torch.cuda.synchronize()
    assert torch.equal(kb, kc) and torch.equal(vb, vc)


def test_zero_tokens_is_a_noop():
    x, wk, wv, kc, vc = _setup("bf16", 1, 512, 2, 128, 10, seed=4)
    k0 = kc.clone()
    wf.wf_kv_only_prefill(x[:0], wk, wv, kc, vc, 10, 1e6)
    torch.cuda.synchronize()
    assert torch.equal(kc, k0)


LAYER_CASES = [
    # n_layers, n_tok, d_in, n_kv_heads, head_dim, start_pos, checked layers
    (3, 16, 1024, 2, 128, 100, (0, 1, 2)),
    (5, 70, 512, 2, 64, 7, (0, 4)),
    (36, 16, 4096, 8, 128, 32784, (0, 17, 35)),
]


@pytest.mark.parametrize("L,n,d_in,hkv,dh,start,check", LAYER_CASES)
def test_layers_match_oracle_and_single_layer_calls(L, n, d_in, hkv, dh, start, check):
    """All layers' catch-up in one launch: each layer's rows within the bar
    of the oracle (the layers listed) and of a single-layer call (all), the
    other rows untouched."""
    print(f"prefill layers L={L} n={n} d_in={d_in} hkv={hkv} dh={dh} start={start}",
          flush=True)
    cap = start + n + 2
    bf = torch.bfloat16
    x = W.normal((L, n, d_in), 1.0, W.stream_seed(L, "x"), bf, DEV)
    wk = W.normal((L, hkv * dh, d_in), 0.02, W.stream_seed(L, "w_k"), bf, DEV)
    wv = W.normal((L, hkv * dh, d_in), 0.02, W.stream_seed(L, "w_v"), bf, DEV)
    kc = W.normal((L, hkv, cap, dh), 1.0, W.stream_seed(L, "k_cache"), bf, DEV)
    vc = W.normal((L, hkv, cap, dh), 1.0, W.stream_seed(L, "v_cache"), bf, DEV)
    k0, v0 = kc.clone(), vc.clone()
    k1, v1 = kc.clone(), vc.clone()
    wf.wf_kv_only_prefill_layers(x, wk, wv, kc, vc, start, 1e6)
    for l in range(L):
        wf.wf_kv_only_prefill(x[l], wk[l], wv[l], k1[l], v1[l], start, 1e6)
    torch.cuda.synchronize()
    rows = slice(start, start + n)
    for l in range(L):
        assert max_vec_rel_err(host64(kc[l][:, rows]), host64(k1[l][:, rows])) <= TOL["bf16"]
        assert max_vec_rel_err(host64(vc[l][:, rows]), host64(v1[l][:, rows])) <= TOL["bf16"]
    for l in check:
        kr, vr = oracle.kv_only_prefill(W.to_oracle(x[l]), W.to_oracle(wk[l]),
                                        W.to_oracle(wv[l]), start, hkv, dh, 1e6)
        assert max_vec_rel_err(host64(kc[l][:, rows]), kr) <= TOL["bf16"]
        assert max_vec_rel_err(host64(vc[l][:, rows]), vr) <= TOL["bf16"]
    for a, b in ((kc, k0), (vc, v0)):
        assert torch.equal(a[:, :, :start], b[:, :, :start])
        assert torch.equal(a[:, :, start + n:], b[:, :, start + n:])


def test_layers_f32_equals_single_layer_calls():
    L, n, d_in, hkv, dh, start = 3, 5, 100, 3, 64, 20
    f = torch.float32
    x = W.normal((L, n, d_in), 0.02, 1, f, DEV)
    wk = W.normal((L, hkv * dh, d_in), 0.02, 2, f, DEV)
    wv = W.normal((L, hkv * dh, d_in), 0.02, 3, f, DEV)
    kc = W.normal((L, hkv, start + n, dh), 1.0, 4, f, DEV)
    vc = W.normal((L, hkv, start + n, dh), 1.0, 5, f, DEV)
    k1, v1 = kc.clone(), vc.clone()
    wf.wf_kv_only_prefill_layers(x, wk, wv, kc, vc, start, 1e4)
    for l in range(L):
        wf.wf_kv_only_prefill(x[l], wk[l], wv[l], k1[l], v1[l], start, 1e4)
    torch.cuda.synchronize()
    assert torch.equal(kc, k1) and torch.equal(vc, v1)
