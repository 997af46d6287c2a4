"""GPU parity of verification attention (Sec. 3.2) when one key dominates a
row's scores: the closed form (the output is that key's value row) and the
bf16 kernel's rescaling path.

The bf16 partial kernel fixes each row's reference maximum at the first tile
of a key stream that has a visible key, and reruns its split with per-tile
rescaling when a later tile of the same stream outgrows that reference by
more than 64 log2 units.  Scores drawn like the workloads' never come near
that margin, so these cases plant one key per chosen row whose scaled score
is 100 nats above everything else, in the last tile of a split (a split of
at least five tiles, more than any stream count of a workgroup, so that tile
is never a stream's first): every such split must take the rerun.  The
split plan is fixed through num_splits; the bf16 kernel deals whole 32-key
tiles evenly, split s owning tiles [s*T/S, (s+1)*T/S), and the split count
in use is read back from the workspace query.
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
TILE = 32
COUNTER_BYTES = 4 << 20
NATS = 100.0


def _splits_in_use(dt, gamma, ctx, hq, hkv, dh, num_splits):
    """Split count of the bf16 plan, from the workspace size: the counter
    block, then per split and (row, head) pair 2 fp32 and head_dim bf16."""
    ws = wf.wf_verify_attn_workspace_bytes(DT[dt], gamma, ctx, hq, hkv, dh,
                                           num_splits)
    per = gamma * hq * (8 + 2 * dh)
    assert (ws - COUNTER_BYTES) % per == 0
    return (ws - COUNTER_BYTES) // per


def _plant(q, k, scale, row, head, key, group):
    """Key `key` of q head `head`'s KV head scores NATS (scaled) for the
    query (row, head): k = a * q with a = NATS / (scale * |q|^2)."""
    qv = q[row, head].double()
    a = NATS / (scale * float((qv * qv).sum()))
    k[head // group, key] = (a * qv).to(k.dtype)


def _planted_case(dt, gamma, ctx, hq, hkv, dh, num_splits, seed, tree_mask=None,
                  in_block=True):
    cap = ctx + gamma + 3
    dtype = DT[dt]
    q = W.normal((gamma, hq, dh), 1.28, W.stream_seed(seed, "q"), dtype, DEV)
    k = W.normal((hkv, cap, dh), 1.28, W.stream_seed(seed, "k_cache"), dtype, DEV)
    v = W.normal((hkv, cap, dh), 1.28, W.stream_seed(seed, "v_cache"), dtype, DEV)
    k[:, ctx + gamma:] = float("nan")          # past the block: never read
    v[:, ctx + gamma:] = float("nan")
    group = hq // hkv
    scale = dh ** -0.5
    n_keys = ctx + gamma
    tiles = (n_keys + TILE - 1) // TILE
    S = _splits_in_use("bf16", gamma, ctx, hq, hkv, dh, num_splits)
    assert S == min(num_splits, tiles)
    planted = {}                               # (row, head) -> key
    rows_per_head = group * gamma
    for g in range(hkv):
        for s in range(S):
            t_first, t_last = s * tiles // S, (s + 1) * tiles // S
            assert t_last - t_first >= 5, "split too short to reach a later tile"
            # the last cached key of the split's last tile
            key = min(t_last * TILE, ctx) - 1
            if key < (t_last - 1) * TILE:
                continue                       # that tile holds block keys only
            r = (7 * s + 3 * g) % rows_per_head
            i, h = r // group, g * group + r % group
            if (i, h) in planted:
                continue
            _plant(q, k, scale, i, h, key, group)
            planted[(i, h)] = key
    if in_block:
        # the last row's own key (block region, masked for every other row)
        h = hq - 1
        if (gamma - 1, h) not in planted:
            _plant(q, k, scale, gamma - 1, h, ctx + gamma - 1, group)
            planted[(gamma - 1, h)] = ctx + gamma - 1
    return q, k, v, planted


def _check(dt, q, k, v, ctx, out, planted, mask=None):
    n = ctx + q.shape[0]
    kk = W.to_oracle(k[:, :n].contiguous())
    vv = W.to_oracle(v[:, :n].contiguous())
    if mask is None:
        ref = oracle.verify_attn(W.to_oracle(q), kk, vv, ctx)
    else:
        ref = oracle.verify_attn_mask(W.to_oracle(q), kk, vv, ctx, mask)
    got = host64(out)
    assert np.isfinite(got).all()
    err = max_vec_rel_err(got, ref)
    assert err <= TOL[dt], err
    # closed form: a key 100 nats above the rest carries all the weight, so
    # the row's output is that key's value row (to the output's rounding)
    group = q.shape[1] // k.shape[0]
    vh = host64(v)
    cf = 2.0 ** -8 if dt == "bf16" else 1e-6
    for (i, h), key in planted.items():
        e = max_vec_rel_err(got[i, h], vh[h // group, key])
        assert e <= cf, ((i, h), key, e)
    return err


BLOCK_CASES = [
    # dt, gamma, ctx, n_q_heads, n_kv_heads, head_dim, num_splits
    ("bf16", 16, 4000, 32, 8, 128, 8),       # 64 rows per KV head (4 row groups x 2 streams)
    ("bf16", 8, 3000, 8, 2, 64, 4),          # 32 rows (2 row groups x 4 streams)
    ("bf16", 2, 2500, 8, 8, 128, 6),         # 2 rows (1 row group x 4 streams)
    ("bf16", 16, 3000, 64, 8, 128, 5),       # 128 rows (two 16-row blocks per wave)
    ("bf16", 30, 2200, 16, 4, 64, 3),        # 120 rows, head_dim 64
    ("bf16", 16, 5000, 32, 8, 128, 1),       # one split: the whole range reruns
    ("f32", 16, 3000, 32, 8, 128, 4),
    ("f32", 4, 2000, 8, 2, 64, 3),
]


@pytest.mark.parametrize("dt,gamma,ctx,hq,hkv,dh,splits", BLOCK_CASES)
def test_dominant_key_block_causal(dt, gamma, ctx, hq, hkv, dh, splits):
    print(f"attn dominant-key {dt} gamma={gamma} ctx={ctx} hq={hq} hkv={hkv} "
          f"dh={dh} splits={splits}", flush=True)
    q, k, v, planted = _planted_case(dt, gamma, ctx, hq, hkv, dh, splits,
                                     seed=gamma * 101 + ctx)
    out = torch.empty_like(q)
    wf.wf_verify_attn(q, k, v, out, ctx, num_splits=splits)
    torch.cuda.synchronize()
    _check(dt, q, k, v, ctx, out, planted)
    # the rerun is deterministic too
    out2 = torch.empty_like(q)
    wf.wf_verify_attn(q, k, v, out2, ctx, num_splits=splits)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)


TREE_CASES = [
    # dt, ctx, n_q_heads, n_kv_heads, head_dim, num_splits
    ("bf16", 3000, 32, 8, 128, 4),           # 244 rows per KV head
    ("bf16", 2600, 16, 4, 64, 3),            # head_dim 64
    ("f32", 2000, 8, 2, 64, 3),
]


@pytest.mark.parametrize("dt,ctx,hq,hkv,dh,splits", TREE_CASES)
def test_dominant_key_tree(dt, ctx, hq, hkv, dh, splits):
    parents = W.draft_tree(seed=5)               # root + 60 nodes, depth 8
    gamma = parents.shape[0]
    print(f"tree attn dominant-key {dt} gamma={gamma} ctx={ctx} hq={hq} "
          f"hkv={hkv} dh={dh} splits={splits}", flush=True)
    mask = W.ancestor_masks(parents)
    q, k, v, planted = _planted_case(dt, gamma, ctx, hq, hkv, dh, splits,
                                     seed=ctx + dh, in_block=False)
    # a tree node's own key is visible to it alone among its siblings
    leaf = gamma - 1
    h = hq - 1
    if (leaf, h) not in planted:
        _plant(q, k, dh ** -0.5, leaf, h, ctx + leaf, hq // hkv)
        planted[(leaf, h)] = ctx + leaf
    md = torch.from_numpy(mask.view(np.int64).copy()).to(DEV)
    out = torch.empty_like(q)
    wf.wf_verify_attn_tree(q, k, v, out, ctx, md, num_splits=splits)
    torch.cuda.synchronize()
    _check(dt, q, k, v, ctx, out, planted, mask=mask)


@pytest.mark.parametrize("ctx,splits", [(0, 1), (0, 2), (16, 1), (16, 3)])
def test_first_visible_tile_after_a_masked_one(ctx, splits):
    """Tree masks under which rows 32..63 see none of block rows 0..31: with
    ctx 0 their first tile (and at two splits their whole first split) is
    fully masked, and their first visible key lies in a later tile."""
    gamma, hq, hkv, dh = 64, 8, 2, 128
    print(f"tree attn masked-first-tile ctx={ctx} splits={splits}", flush=True)
    masks = np.zeros(gamma, np.uint64)
    for i in range(gamma):
        lo = 0 if i < 32 else 32
        m = 0
        for j in range(lo, i + 1):
            m |= 1 << j
        masks[i] = np.uint64(m)
    cap = ctx + gamma + 3
    q = W.normal((gamma, hq, dh), 1.28, W.stream_seed(ctx + 9, "q"), torch.bfloat16, DEV)
    k = W.normal((hkv, cap, dh), 1.28, W.stream_seed(ctx + 9, "k_cache"), torch.bfloat16, DEV)
    v = W.normal((hkv, cap, dh), 1.28, W.stream_seed(ctx + 9, "v_cache"), torch.bfloat16, DEV)
    # a dominant key late in the visible range of row 63 (its own key)
    _plant(q, k, dh ** -0.5, gamma - 1, 0, ctx + gamma - 1, hq // hkv)
    md = torch.from_numpy(masks.view(np.int64).copy()).to(DEV)
    out = torch.empty_like(q)
    wf.wf_verify_attn_tree(q, k, v, out, ctx, md, num_splits=splits)
    torch.cuda.synchronize()
    _check("bf16", q, k, v, ctx, out, {(gamma - 1, 0): ctx + gamma - 1}, mask=masks)
