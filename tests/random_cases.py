"""Seeded random shapes for the GPU parity sweep (tests/test_gpu_random_shapes.py),
drawn from the ranges the C ABI accepts.  Pure case generation: no GPU, no
arithmetic of the method; a host-side test checks that the library accepts
every case drawn here."""
import numpy as np

HEADS = [(1, 1), (2, 1), (4, 4), (8, 2), (12, 4), (16, 2), (32, 8), (64, 8)]


def attn_cases(n=40, seed=20260602):
    rng = np.random.default_rng(seed)
    out = []
    for case in range(n):
        dt = "bf16" if rng.random() < 0.8 else "f32"
        gamma = int(rng.integers(1, 65))
        ctx = int(rng.choice([rng.integers(0, 64), rng.integers(64, 1500),
                              rng.integers(1500, 6000)]))
        hq, hkv = HEADS[int(rng.integers(len(HEADS)))]
        dh = int(rng.choice([64, 128]))
        splits = int(rng.choice([0, 0, 1, int(rng.integers(2, 40))]))
        tree = bool(rng.random() < 0.3)
        std = float(rng.choice([0.5, 1.28, 2.5]))
        cap = ctx + gamma + int(rng.integers(0, 4))
        parents = None
        if tree:
            parents = np.full(gamma, -1, np.int32)
            for j in range(1, gamma):
                parents[j] = rng.integers(max(0, j - 8), j)
        out.append(dict(case=case, dt=dt, gamma=gamma, ctx=ctx, hq=hq, hkv=hkv,
                        dh=dh, splits=splits, tree=tree, std=std, cap=cap,
                        parents=parents, seed=1000 + case))
    return out


def prefill_cases(n=30, seed=20260603):
    rng = np.random.default_rng(seed)
    out = []
    for case in range(n):
        dt = "bf16" if rng.random() < 0.8 else "f32"
        tiled = bool(dt == "bf16" and rng.random() < 0.5)
        n_tok = int(rng.choice([rng.integers(1, 17), rng.integers(17, 80),
                                rng.integers(80, 300)]))
        d_in = 32 * int(rng.integers(1, 80))
        if dt == "f32":
            d_in = int(rng.integers(1, 1200))
        hkv = int(rng.choice([1, 2, 3, 4, 8]))
        dh = int(rng.choice([64, 128]))
        start = int(rng.integers(0, 70000))
        base = float(rng.choice([1e4, 1e6]))
        cap = start + n_tok + int(rng.integers(0, 3))
        out.append(dict(case=case, dt=dt, tiled=tiled, n=n_tok, d_in=d_in, hkv=hkv,
                        dh=dh, start=start, base=base, cap=cap, seed=2000 + case))
    return out


def lmhead_cases(n=30, seed=20260604):
    rng = np.random.default_rng(seed)
    out = []
    for case in range(n):
        dt = "bf16" if rng.random() < 0.75 else "f32"
        gamma = int(rng.choice([rng.integers(1, 17), rng.integers(17, 65)]))
        vocab = int(rng.choice([rng.integers(1, 300), rng.integers(300, 40000),
                                rng.integers(40000, 160000)]))
        if dt == "bf16":
            d = int(rng.choice([512 * int(rng.integers(1, 5)),
                                32 * int(rng.integers(1, 40)), 4096]))
        else:
            d = int(rng.integers(1, 700))
        tileable = dt == "bf16" and (d % 512 == 0 or (gamma <= 16 and d in (4096, 5120)))
        tiled = bool(tileable and rng.random() < 0.6)
        ws = float(rng.choice([0.02, 0.05, 0.2]))
        out.append(dict(case=case, dt=dt, tiled=tiled, gamma=gamma, d=d, vocab=vocab,
                        w_std=ws, seed=3000 + case))
    return out


DRAFTER_HEADS = [(1, 1), (2, 1), (4, 2), (4, 4), (6, 3), (8, 2), (12, 4)]


def drafter_cases(n=16, seed=20260605):
    """One drafter decoder layer: the full layer over 1..64 tokens
    (`forward`) or a lazy catch-up over a backlog of 1..400 (`catchup`);
    hidden and SwiGLU widths multiples of 32, head_dim 64 or 128, row-major
    or tiled projections."""
    rng = np.random.default_rng(seed)
    out = []
    for case in range(n):
        kind = "catchup" if rng.random() < 0.6 else "forward"
        hq, hkv = DRAFTER_HEADS[int(rng.integers(len(DRAFTER_HEADS)))]
        dh = int(rng.choice([64, 128]))
        hidden = 32 * int(rng.integers(4, 49))
        inter = 32 * int(rng.integers(4, 97))
        pos = int(rng.choice([rng.integers(0, 40), rng.integers(40, 2500)]))
        if kind == "catchup":
            n_tok = int(rng.choice([rng.integers(1, 17), rng.integers(17, 101),
                                    rng.integers(101, 401)]))
        else:
            n_tok = int(rng.integers(1, 65))
        tiled = bool(rng.random() < 0.5)
        out.append(dict(case=case, kind=kind, hq=hq, hkv=hkv, dh=dh, hidden=hidden,
                        inter=inter, pos=pos, n=n_tok, tiled=tiled, cfg=5000 + case))
    return out


def router_cases(n=24, seed=20260606):
    """The neural routing policy's MLP (d -> m -> GELU -> 1) over gamma
    rows: bf16 with d % 32 == 0 and m % 16 == 0, or fp32 of any size."""
    rng = np.random.default_rng(seed)
    out = []
    for case in range(n):
        dt = "bf16" if rng.random() < 0.75 else "f32"
        gamma = int(rng.integers(1, 65))
        if dt == "bf16":
            d = 32 * int(rng.integers(1, 161))
            m = 16 * int(rng.integers(1, 65))
        else:
            d = int(rng.integers(1, 700))
            m = int(rng.integers(1, 300))
        out.append(dict(case=case, dt=dt, gamma=gamma, d=d, m=m, seed=6000 + case))
    return out


def tree_lmhead_cases(n=20, seed=20260607):
    """The LM head with tree acceptance: gamma 1..64 tree nodes (bushy random
    parents), ragged vocabularies, bf16 weights row-major or tiled (the
    tiled layout where the ABI takes it: d % 512 == 0, or gamma <= 16 with
    d in {4096, 5120}), and the depth k of the accepted path the node
    tokens plant."""
    rng = np.random.default_rng(seed)
    out = []
    for case in range(n):
        gamma = int(rng.choice([rng.integers(1, 17), rng.integers(17, 65)]))
        vocab = int(rng.choice([rng.integers(2, 500), rng.integers(500, 40000)]))
        if gamma <= 16 and rng.random() < 0.4:
            d = int(rng.choice([4096, 5120]))        # the persistent stream kernel's shapes
        else:
            d = int(rng.choice([512 * int(rng.integers(1, 5)), 32 * int(rng.integers(1, 40))]))
        tileable = d % 512 == 0 or (gamma <= 16 and d in (4096, 5120))
        tiled = bool(tileable and rng.random() < 0.6)
        parents = np.full(gamma, -1, np.int32)
        for j in range(1, gamma):
            parents[j] = rng.integers(max(0, j - 6), j)
        k = int(rng.integers(0, 9))
        out.append(dict(case=case, gamma=gamma, vocab=vocab, d=d, tiled=tiled,
                        parents=parents, k=k, seed=8000 + case))
    return out


def layer_prefill_cases(n=12, seed=20260608):
    """All layers' KV-only prefill in one launch: 2..12 layers, 1..200
    tokens, bf16 row-major or tiled weights."""
    rng = np.random.default_rng(seed)
    out = []
    for case in range(n):
        n_layers = int(rng.integers(2, 13))
        n_tok = int(rng.choice([rng.integers(1, 17), rng.integers(17, 80),
                                rng.integers(80, 201)]))
        d_in = 32 * int(rng.integers(1, 48))
        hkv = int(rng.choice([1, 2, 4, 8]))
        dh = int(rng.choice([64, 128]))
        start = int(rng.integers(0, 5000))
        tiled = bool(rng.random() < 0.5)
        out.append(dict(case=case, layers=n_layers, n=n_tok, d_in=d_in, hkv=hkv, dh=dh,
                        start=start, tiled=tiled, seed=9000 + case))
    return out
