"""GPU parity of wf_lmhead_accept_route_neural -- the LM head, greedy
acceptance and the neural routing policy (Sec. 3.3.2; architecture in the
appendix on the neural router) in one pass -- against the fp64 oracle:
argmax and entropy per row, the accept length and bonus token, the
predicted gain delta of every row, and the route taken on the final
accepted row.  Covers the fused shapes (gamma <= 16, d 4096/5120, tiled and
row-major weights) and the fallback schedule for other shapes."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import TOL, check_argmax, entropy_rel_err

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _scale(h, w1, b1, w2, b2):
    """|b2| + sum_u |w2_u GELU(z_u)| per row: the size of the terms delta
    sums, which bounds its rounding error."""
    h, w1, b1, w2, b2 = (t.double().cpu().numpy() for t in (h, w1, b1, w2, b2))
    z = h @ w1.T + b1
    g = 0.5 * z * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))
    return np.abs(b2[0]) + np.abs(g * w2).sum(axis=1)


CASES = [
    # dt, tiled, gamma, d, vocab, m
    ("bf16", True, 16, 4096, 151936, 512),      # the 8B head, as the benchmark runs it
    ("bf16", False, 16, 4096, 151936, 512),
    ("bf16", True, 8, 4096, 20011, 512),
    ("bf16", True, 1, 5120, 3001, 640),
    ("bf16", False, 5, 5120, 70000, 640),
    ("bf16", False, 24, 512, 5000, 64),         # fallback: LM head, then the router kernels
    ("f32", False, 3, 100, 1001, 7),             # fallback, fp32
]


@pytest.mark.parametrize("dt,tiled,gamma,d,vocab,m", CASES)
def test_matches_oracle(dt, tiled, gamma, d, vocab, m):
    print(f"lmhead+router {dt} tiled={tiled} gamma={gamma} d={d} vocab={vocab} m={m}",
          flush=True)
    seed = 7000 + gamma + d + m
    dtype = DT[dt]
    ws_std = 0.02 if dt == "bf16" else 0.1
    h = W.normal((gamma, d), 1.0, W.stream_seed(seed, "h"), dtype, DEV)
    w_lm = W.normal((vocab, d), ws_std, W.stream_seed(seed, "w_lm"), dtype, DEV)
    w1 = W.normal((m, d), 0.02, W.stream_seed(seed, "router_w1"), dtype, DEV)
    b1 = W.normal((m,), 0.02, W.stream_seed(seed, "router_b1"), dtype, DEV)
    w2 = W.normal((m,), 0.05, W.stream_seed(seed, "router_w2"), dtype, DEV)
    b2 = W.normal((1,), 0.05, W.stream_seed(seed, "router_b2"), dtype, DEV)
    am_ref, ent_ref, margin, z = oracle.lmhead_rows(W.to_oracle(h), W.to_oracle(w_lm),
                                                    want_logits=True)
    d_ref = oracle.router_mlp(*(W.to_oracle(t) for t in (h, w1, b1, w2, b2)))
    scale = _scale(h, w1, b1, w2, b2)
    wl = wf.tile_weights(w_lm) if tiled else w_lm
    w1p = wf.tile_weights(w1) if tiled else w1
    bar = 1e-2 if dt == "bf16" else 1e-6
    am = torch.empty(gamma, dtype=torch.int32, device=DEV)
    ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
    acc = torch.empty(3, dtype=torch.int32, device=DEV)
    delta = torch.empty(gamma, dtype=torch.float32, device=DEV)
    checked = 0
    for ds in range(4):
        k = W.geometric_prefix(0.3, gamma, seed + ds)
        draft = W.make_drafts(am_ref, k, vocab, seed + ds)
        dr = torch.as_tensor(draft, device=DEV) if gamma > 1 else None
        kk = min(k, gamma - 1)
        db = TOL[dt] * scale[kk]
        for tau in (float(np.median(d_ref)), float(d_ref[kk] + 3 * db),
                    float(d_ref[kk] - 3 * db)):
            wf.wf_lmhead_accept_route_neural(h, wl, dr, w1p, b1, w2, b2, tau, am, ent, acc,
                                             delta)
            torch.cuda.synchronize()
            a, e, c, dg = (am.cpu().numpy(), ent.cpu().numpy(), acc.cpu().numpy(),
                           delta.cpu().numpy().astype(np.float64))
            check_argmax(a, am_ref, margin, z, dt)
            assert entropy_rel_err(e, ent_ref) <= TOL[dt]
            assert np.all(np.abs(dg - d_ref) <= TOL[dt] * scale)
            n = int(c[0])
            # the GPU's own triple is consistent with its argmax and gain
            j = 0
            while j < gamma - 1 and draft[j] == a[j]:
                j += 1
            assert n == j and c[1] == a[n] and c[2] == int(dg[n] > tau)
            if all(margin[i] > bar for i in range(kk + 1)):
                assert n == kk and c[1] == am_ref[kk]
            if abs(d_ref[n] - tau) > TOL[dt] * scale[n]:
                assert int(c[2]) == oracle.route_neural(d_ref, n, tau)
                checked += 1
    assert checked >= 4
