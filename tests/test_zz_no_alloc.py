"""wf_verify_attn_noalloc (the verify attention of Sec. 3.2 on the library's
static device scratch, for callers that cannot allocate) against
wf_verify_attn on the same inputs and against the fp64 oracle: two calls in
a row, the second smaller than the first, then an fp32 call; and a call too
large for the scratch is rejected before anything is launched."""
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


def _inputs(dt, gamma, ctx, hq, hkv, dh, seed):
    cap = ctx + gamma + 2
    q = W.normal((gamma, hq, dh), 1.28, W.stream_seed(seed, "q"), DT[dt], DEV)
    k = W.normal((hkv, cap, dh), 1.28, W.stream_seed(seed, "k_cache"), DT[dt], DEV)
    v = W.normal((hkv, cap, dh), 1.28, W.stream_seed(seed, "v_cache"), DT[dt], DEV)
    return q, k, v


CALLS = [
    # dt, gamma, ctx, n_q_heads, n_kv_heads, head_dim, num_splits
    ("bf16", 16, 20000, 32, 8, 128, 0),
    ("bf16", 5, 700, 8, 2, 64, 0),
    ("f32", 8, 256, 8, 2, 64, 3),
]


def test_noalloc_matches_workspace_call():
    for dt, gamma, ctx, hq, hkv, dh, splits in CALLS:
        print(f"noalloc attn {dt} gamma={gamma} ctx={ctx} hq={hq} hkv={hkv} "
              f"dh={dh} splits={splits}", flush=True)
        q, k, v = _inputs(dt, gamma, ctx, hq, hkv, dh, seed=gamma * 13 + ctx)
        ref_out = torch.empty_like(q)
        wf.wf_verify_attn(q, k, v, ref_out, ctx, num_splits=splits)
        out = torch.full_like(q, float("nan"))
        wf.wf_verify_attn_noalloc(q, k, v, out, ctx, num_splits=splits)
        torch.cuda.synchronize()
        # the same kernels on the same plan: bit-identical
        assert torch.equal(out, ref_out)
        n = ctx + gamma
        ref = oracle.verify_attn(W.to_oracle(q), W.to_oracle(k[:, :n].contiguous()),
                                 W.to_oracle(v[:, :n].contiguous()), ctx)
        err = max_vec_rel_err(host64(out), ref)
        assert err <= TOL[dt], err


def test_noalloc_rejects_what_does_not_fit():
    q = torch.zeros((64, 256, 128), dtype=torch.bfloat16, device=DEV)
    k = torch.zeros((8, 4096 + 64, 128), dtype=torch.bfloat16, device=DEV)
    out = torch.zeros_like(q)
    need = wf.wf_verify_attn_workspace_bytes(torch.bfloat16, 64, 4096, 256, 8, 128, 64)
    assert need > wf.NOALLOC_SCRATCH_BYTES
    with pytest.raises(wf.WfError) as e:
        wf.wf_verify_attn_noalloc(q, k, k, out, 4096, num_splits=64)
    assert e.value.status == wf.WF_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert not out.any()                 # nothing was launched
