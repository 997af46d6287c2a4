"""GPU parity of wf_verify_attn against the fp64 oracle (Sec. 3.2 parallel
verification), plus the invariants of causal verification: gamma == 1 is
decoding, row i of a block equals a decode on prefix i, the split count does
not change the result beyond rounding, and repeated calls are bit-identical.
"""
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


def _inputs(dt, gamma, ctx, hq, hkv, dh, seed, std=1.0, cap_extra=5,
            poison=True):
    cap = ctx + gamma + cap_extra
    dtype = DT[dt]
    q = W.normal((gamma, hq, dh), std, W.stream_seed(seed, "q"), dtype, DEV)
    k = W.normal((hkv, cap, dh), std, W.stream_seed(seed, "k_cache"), dtype, DEV)
    v = W.normal((hkv, cap, dh), std, W.stream_seed(seed, "v_cache"), dtype, DEV)
    if poison and cap_extra:
        # rows past ctx + gamma must never be read
        k[:, ctx + gamma:] = float("nan")
        v[:, ctx + gamma:] = float("nan")
    return q, k, v


# Two runs of the same math under different split plans.  bf16: each side
# rounds its output once (at most half an ulp, 2^-8 of the vector's max
# norm) and its probabilities to bf16 against a different running maximum,
# so the two may differ by two half-ulps plus that rounding noise: 2^-6.
SAME_MATH_TOL = {"bf16": 2.0 ** -6, "f32": 1e-5}


def _run(q, k, v, ctx, splits=0):
    out = torch.empty_like(q)
    wf.wf_verify_attn(q, k, v, out, ctx, num_splits=splits)
    torch.cuda.synchronize()
    return out


CASES = [
    # dt, gamma, ctx, n_q_heads, n_kv_heads, head_dim
    ("bf16", 1, 0, 8, 2, 128),
    ("bf16", 1, 1000, 32, 8, 128),
    ("bf16", 2, 77, 8, 8, 64),
    ("bf16", 7, 1000, 32, 8, 128),
    ("bf16", 8, 2049, 32, 8, 128),
    ("bf16", 16, 3001, 32, 8, 128),
    ("bf16", 16, 31, 32, 8, 128),
    ("bf16", 17, 500, 16, 2, 128),
    ("bf16", 64, 300, 8, 8, 64),
    ("bf16", 16, 4000, 64, 8, 128),
    ("bf16", 3, 129, 12, 4, 64),
    ("bf16", 12, 700, 32, 4, 64),        # 96 rows per KV head: 128-row groups
    ("bf16", 30, 900, 16, 4, 128),       # 120 rows per KV head
    ("f32", 8, 256, 8, 2, 64),
    ("f32", 3, 1000, 4, 4, 128),
    ("f32", 1, 0, 2, 1, 64),
    ("f32", 16, 77, 16, 4, 128),
]


@pytest.mark.parametrize("dt,gamma,ctx,hq,hkv,dh", CASES)
def test_matches_oracle(dt, gamma, ctx, hq, hkv, dh):
    print(f"attn parity {dt} gamma={gamma} ctx={ctx} hq={hq} hkv={hkv} "
          f"dh={dh}", flush=True)
    std = 1.28 if dt == "bf16" else 1.0
    q, k, v = _inputs(dt, gamma, ctx, hq, hkv, dh, seed=gamma * 7919 + ctx,
                      std=std)
    out = _run(q, k, v, ctx)
    n = ctx + gamma
    ref = oracle.verify_attn(W.to_oracle(q), W.to_oracle(k[:, :n].contiguous()),
                             W.to_oracle(v[:, :n].contiguous()), ctx)
    got = host64(out)
    assert np.isfinite(got).all()
    err = max_vec_rel_err(got, ref)
    assert err <= TOL[dt], err


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_tiny_values_and_peaked_scores(dt):
    """Near-uniform attention (std 0.02) and sharply peaked attention
    (std 4 -> scores of order 180)."""
    for std in (0.02, 4.0):
        q, k, v = _inputs(dt, 8, 700, 32, 8, 128, seed=11, std=std)
        out = _run(q, k, v, 700)
        ref = oracle.verify_attn(W.to_oracle(q), W.to_oracle(k[:, :708].contiguous()),
                                 W.to_oracle(v[:, :708].contiguous()), 700)
        assert max_vec_rel_err(host64(out), ref) <= TOL[dt]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_row_i_equals_decode_on_prefix_i(dt):
    gamma, ctx, hq, hkv, dh = 16, 1500, 32, 8, 128
    q, k, v = _inputs(dt, gamma, ctx, hq, hkv, dh, seed=21, std=1.28)
    blk = _run(q, k, v, ctx)
    for i in (0, 1, 7, 15):
        dec = _run(q[i:i + 1].contiguous(), k, v, ctx + i)
        a, b = host64(blk[i]), host64(dec[0])
        assert max_vec_rel_err(a, b) <= SAME_MATH_TOL[dt], i


# split counts on both sides of the one-round-trip merge's limit (32
# splits at head_dim 128, 64 at head_dim 64; more go to the general merge)
@pytest.mark.parametrize("dt,dh,splits", [
    ("bf16", 128, (2, 5, 11, 17, 32, 33, 48, 0)), ("f32", 128, (2, 5, 11, 17, 32, 33, 0)),
    ("bf16", 64, (2, 17, 64, 65, 0))])
def test_split_count_invariance_and_determinism(dt, dh, splits):
    gamma, ctx, hq, hkv = 16, 3000, 32, 8
    q, k, v = _inputs(dt, gamma, ctx, hq, hkv, dh, seed=31, std=1.28)
    ref = oracle.verify_attn(W.to_oracle(q), W.to_oracle(k[:, :ctx + gamma].contiguous()),
                             W.to_oracle(v[:, :ctx + gamma].contiguous()), ctx)
    base = _run(q, k, v, ctx, splits=1)
    for s in splits:
        o = _run(q, k, v, ctx, splits=s)
        assert max_vec_rel_err(host64(o), ref) <= TOL[dt], s
        assert max_vec_rel_err(host64(o), host64(base)) <= SAME_MATH_TOL[dt], s
        o2 = _run(q, k, v, ctx, splits=s)
        assert torch.equal(o, o2), s


def test_cached_key_permutation_invariance():
    gamma, ctx, hq, hkv, dh = 8, 2000, 32, 8, 128
    q, k, v = _inputs("bf16", gamma, ctx, hq, hkv, dh, seed=41, std=1.28,
                      poison=False)
    a = _run(q, k, v, ctx)
    perm = torch.randperm(ctx, generator=torch.Generator().manual_seed(1)).to(DEV)
    k2, v2 = k.clone(), v.clone()
    k2[:, :ctx] = k[:, perm]
    v2[:, :ctx] = v[:, perm]
    b = _run(q, k2, v2, ctx)
    assert max_vec_rel_err(host64(b), host64(a)) <= SAME_MATH_TOL["bf16"]


def test_equal_keys_give_mean_of_visible_values():
    gamma, ctx, hq, hkv, dh = 5, 300, 8, 2, 128
    q, k, v = _inputs("bf16", gamma, ctx, hq, hkv, dh, seed=51, std=1.0,
                      poison=False)
    k.copy_(k[:, :1].expand_as(k).clone())
    out = host64(_run(q, k, v, ctx))
    vh = host64(v)
    for i in range(gamma):
        for h in range(hq):
            ref = vh[h // 4, :ctx + i + 1].mean(0)
            assert max_vec_rel_err(out[i, h], ref) <= 2e-2
