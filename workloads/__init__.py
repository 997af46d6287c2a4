"""Seeded synthetic workloads for the verification step.

This module holds the five workload shapes and the seeded generators that
fill their inputs.  It contains none of the verification arithmetic: it
draws random tensors, builds draft-token sequences from a given reference
argmax, and converts tensors into the plain arrays the CPU oracle reads.
Both the GPU tests / benchmark and the CPU oracle take their inputs from
here, so the two sides always see identical bytes.

Inputs are synthetic because the paper's models, drafters and datasets are
not available; the shapes follow the paper's targets (Qwen3-8B attention
geometry and vocabulary, Sec. 4 "Models"; a verify block of 16 for the
diffusion drafter and chains for the autoregressive one, App. A drafter
hyper-parameters; tens of catch-up tokens per switch, Sec. 6).

Distributions (std = standard deviation):
  * tiny fp32 case: every tensor N(0, 0.02).
  * 8B / 32B shapes: layer inputs x and final hidden states h ~ N(0, 1)
    (post-RMSNorm activations); projection and LM-head weights ~ N(0, 0.02);
    queries and cached K/V ~ N(0, 0.02 * sqrt(hidden)), the distribution of
    a projection of those activations.
  * router-heavy logits: half of the rows (chosen by a seeded permutation)
    N(0, 8) with one uniformly chosen id raised to the row max + 16; the
    other half N(0, 0.5).
  * drafts: draft[j] (the token at block row j+1) equals the reference
    argmax of row j for j < k, draft[k] is a uniform id different from the
    reference argmax of row k, later drafts are uniform ids.  k follows
    Geometric(p) on {0, 1, ...} clipped to gamma-1, or is fixed.
"""
from __future__ import annotations

import hashlib
import math
from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    dtype: str               # "f32" or "bf16"
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ctx_len: int
    gamma: int
    vocab: int
    rope_base: float
    n_prefill: int           # catch-up tokens per layer (0: none)
    prefill_start: int       # cache row of the first catch-up token
    prefill_cap: int         # capacity of the cache the prefill writes
    separate_drafter_cache: bool
    act_std: float           # x, h
    w_std: float             # W_k, W_v, W_lm
    qkv_std: float           # q, cached K/V
    accept_p: float | None   # Geometric(p) prefix; None -> fixed_prefix
    fixed_prefix: int | None
    router_logits: bool      # config with logits-only router rows
    description: str = field(default="", compare=False)
    # draft-tree verification: nodes per depth below the root (empty: the
    # block is a chain or a diffusion block, verified block-causally)
    tree_levels: tuple = ()
    # drafter layer of the switch path: MLP width (0: none)
    inter: int = 0
    rms_eps: float = 1e-6

    @property
    def is_tree(self) -> bool:
        return len(self.tree_levels) > 0

    @property
    def cap(self) -> int:
        """Capacity of the verify cache (block rows plus in-cache prefill)."""
        extra = 0 if self.separate_drafter_cache else self.n_prefill
        return self.ctx_len + self.gamma + extra

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def algorithmic_bytes(self) -> dict:
        """Bytes each step must move at least once (inputs read, outputs
        written); split partials and scratch are excluded."""
        b = self.elem_bytes
        hkv, hq, dh, g = self.n_kv_heads, self.n_q_heads, self.head_dim, self.gamma
        attn = 2 * hkv * (self.ctx_len + g) * dh * b + 2 * g * hq * dh * b
        if self.n_prefill:
            n, d = self.n_prefill, self.hidden
            pre = 2 * hkv * dh * d * b + n * d * b + 2 * n * hkv * dh * b
        else:
            pre = 0
        lm = self.vocab * self.hidden * b + g * self.hidden * b
        logits = g * self.vocab * 4 if self.router_logits else 0
        return {"attn_per_layer": attn, "prefill_per_layer": pre,
                "lmhead": lm, "router_logits": logits,
                "total": self.n_layers * (attn + pre) + lm + logits}

    def drafter_weight_bytes(self) -> int:
        """Bytes of one drafter layer's weights (projections and norms)."""
        d, qd, kd, i = (self.hidden, self.n_q_heads * self.head_dim,
                        self.n_kv_heads * self.head_dim, self.inter)
        return (2 * qd * d + 2 * kd * d + 3 * i * d + 2 * d) * self.elem_bytes

    def catchup_bytes(self, n: int, pos: int) -> int:
        """Bytes a lazy catch-up over n backlog tokens from cache row pos must
        move at least once: the layer's weights, the backlog inputs, the K/V
        rows written, the cache rows the last token attends over, its
        output."""
        b, d, kd = self.elem_bytes, self.hidden, self.n_kv_heads * self.head_dim
        return (self.drafter_weight_bytes() + n * d * b + 2 * n * kd * b
                + 2 * (pos + n) * kd * b + d * b)

    def flops(self) -> dict:
        hq, dh, g, L = self.n_q_heads, self.head_dim, self.gamma, self.ctx_len
        attn = 4 * hq * dh * (g * L + g * (g + 1) // 2)
        pre = 4 * self.n_prefill * self.hidden * self.n_kv_heads * dh
        lm = 2 * g * self.hidden * self.vocab
        return {"attn_per_layer": attn, "prefill_per_layer": pre, "lmhead": lm}


def _qwen_like(cfg, name, n_layers, hidden, hq, ctx, gamma, n_pre, p, desc,
               router=False, tree_levels=()):
    return Workload(cfg=cfg, name=name, dtype="bf16", n_layers=n_layers,
                    hidden=hidden, n_q_heads=hq, n_kv_heads=8, head_dim=128,
                    ctx_len=ctx, gamma=gamma, vocab=151936, rope_base=1e6,
                    n_prefill=n_pre, prefill_start=ctx + gamma,
                    prefill_cap=ctx + gamma + n_pre,
                    separate_drafter_cache=False, act_std=1.0, w_std=0.02,
                    qkv_std=0.02 * math.sqrt(hidden), accept_p=p,
                    fixed_prefix=None, router_logits=router, description=desc,
                    tree_levels=tuple(tree_levels))


# Nodes per depth of the synthetic EAGLE-3-shaped draft tree: depth 8 and
# 60 draft tokens (App. A drafter settings), at most 10 children per node
# (top-k 10), thinning with depth as a top-scored expansion does.
EAGLE_LEVELS = (10, 10, 10, 8, 8, 6, 4, 4)
EAGLE_TOP_K = 10


CONFIGS = {
    1: Workload(cfg=1, name="tiny-f32", dtype="f32", n_layers=1, hidden=512,
                n_q_heads=8, n_kv_heads=2, head_dim=64, ctx_len=256, gamma=8,
                vocab=4096, rope_base=1e4, n_prefill=4, prefill_start=252,
                prefill_cap=256, separate_drafter_cache=True, act_std=0.02,
                w_std=0.02, qkv_std=0.02, accept_p=None, fixed_prefix=5,
                router_logits=False,
                description="tiny fp32 verify step: 1 layer, hidden 512, 8/2 "
                            "heads, head_dim 64, ctx 256, gamma 8, 4 catch-up "
                            "tokens, vocab 4096"),
    2: _qwen_like(2, "8b-chain-ctx8k", 36, 4096, 32, 8192, 8, 0, 0.3,
                  "8B shapes, 36 layers, ctx 8192, gamma 8 chain, vocab "
                  "151936"),
    3: _qwen_like(3, "8b-block16-ctx32k", 36, 4096, 32, 32768, 16, 16, 0.15,
                  "8B shapes, 36 layers, ctx 32768, gamma 16 block-causal, "
                  "16 catch-up tokens per layer, vocab 151936"),
    4: _qwen_like(4, "8b-router-ctx16k", 36, 4096, 32, 16384, 16, 0, 0.3,
                  "8B shapes, 36 layers, ctx 16384, gamma 16, router logits "
                  "16 x 151936 fp32 plus target LM head", router=True),
    5: _qwen_like(5, "32b-block16-ctx64k", 64, 5120, 64, 65536, 16, 32, 0.3,
                  "32B shapes, 64 layers, ctx 65536, gamma 16 block-causal, "
                  "32 catch-up tokens per layer, vocab 151936"),
    7: Workload(cfg=7, name="8b-switch-catchup", dtype="bf16", n_layers=1,
                hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                ctx_len=4096, gamma=1, vocab=151936, rope_base=1e6,
                n_prefill=80, prefill_start=4096, prefill_cap=4096 + 80,
                separate_drafter_cache=True, act_std=1.0, w_std=0.02,
                qkv_std=0.02 * math.sqrt(4096), accept_p=None,
                fixed_prefix=0, router_logits=False,
                description="switch to a one-layer drafter with the 8B "
                            "attention shapes and a 12288-wide SwiGLU MLP: "
                            "lazy catch-up of its cache (4096 rows) over a "
                            "backlog of 80 tokens -- KV-only prefill of 79, "
                            "the full layer for the last",
                inter=12288),
    6: _qwen_like(6, "8b-tree61-ctx8k", 36, 4096, 32, 8192,
                  1 + sum(EAGLE_LEVELS), 0, 0.3,
                  "8B shapes, 36 layers, ctx 8192, EAGLE-3-shaped draft tree "
                  "(root + 60 nodes, depth 8, top-k 10) verified with an "
                  "ancestor mask, vocab 151936", tree_levels=EAGLE_LEVELS),
}

# Fixed tensor identifiers: each named tensor (and layer) gets its own stream.
TENSOR_IDS = {"q": 1, "k_cache": 2, "v_cache": 3, "x": 4, "w_k": 5, "w_v": 6,
              "h": 7, "w_lm": 8, "router_logits": 9, "router_rows": 10,
              "router_boost": 11, "drafts": 12, "prefix": 13,
              "drafter_k_cache": 14, "drafter_v_cache": 15, "tree": 16,
              "tree_tokens": 17, "router_w1": 18, "router_b1": 19,
              "router_w2": 20, "router_b2": 21, "drafter": 22, "backlog": 23}


def stream_seed(master: int, tensor: str | int, layer: int = 0) -> int:
    """64-bit seed for one named tensor of one layer (SHA-256 of the triple)."""
    tid = TENSOR_IDS[tensor] if isinstance(tensor, str) else int(tensor)
    h = hashlib.sha256(f"{master}:{tid}:{layer}".encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def master_seed(cfg: int) -> int:
    return 1000 * cfg


def normal(shape, std, seed, dtype, device="cpu"):
    """N(0, std^2) tensor from torch's generator on `device`, seeded."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = torch.empty(shape, dtype=dtype, device=device)
    if dtype == torch.float32:
        t.normal_(0.0, std, generator=g)
    else:
        tmp = torch.empty(shape, dtype=torch.float32, device=device)
        tmp.normal_(0.0, std, generator=g)
        t.copy_(tmp)
        del tmp
    return t


def normal_into(t, std, seed):
    """Fill an existing tensor in place with N(0, std^2), seeded."""
    g = torch.Generator(device=t.device)
    g.manual_seed(seed)
    if t.dtype == torch.float32:
        t.normal_(0.0, std, generator=g)
    else:
        # chunked through fp32 so large bf16 caches need little extra memory
        flat = t.view(-1)
        step = 1 << 26
        for s in range(0, flat.numel(), step):
            e = min(flat.numel(), s + step)
            tmp = torch.empty(e - s, dtype=torch.float32, device=t.device)
            tmp.normal_(0.0, std, generator=g)
            flat[s:e].copy_(tmp)
    return t


def to_oracle(t) -> np.ndarray:
    """Host copy of a tensor in the storage the oracle reads: fp32 stays fp32,
    bf16 becomes its raw uint16 bit patterns, fp64 stays fp64."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype in (torch.float32, torch.float64):
        return t.numpy()
    raise TypeError(f"unsupported dtype {t.dtype}")


def geometric_prefix(p: float, gamma: int, seed: int) -> int:
    """k ~ Geometric(p) on {0, 1, ...}: P(k) = (1-p)^k p, clipped to gamma-1."""
    rng = np.random.default_rng(seed)
    k = int(rng.geometric(p)) - 1      # numpy's geometric counts trials >= 1
    return min(k, gamma - 1)


def make_drafts(ref_argmax, k: int, vocab: int, seed: int) -> np.ndarray:
    """Drafts [gamma-1] agreeing with ref_argmax on rows < k, forced to
    disagree at row k (if k < gamma-1), uniform afterwards."""
    ref = np.asarray(ref_argmax, np.int64)
    gamma = ref.shape[0]
    rng = np.random.default_rng(seed)
    d = rng.integers(0, vocab, size=max(gamma - 1, 0), dtype=np.int64)
    for j in range(min(k, gamma - 1)):
        d[j] = ref[j]
    if k < gamma - 1:
        r = int(rng.integers(0, vocab - 1))
        d[k] = r if r < ref[k] else r + 1   # uniform over ids != ref[k]
    return d.astype(np.int32)


def draft_tree(levels=EAGLE_LEVELS, top_k=EAGLE_TOP_K, seed=0) -> np.ndarray:
    """Parents [1 + sum(levels)] int32 of a draft tree in breadth-first
    order: node 0 is the root (parent -1) and depth d holds levels[d-1]
    nodes, each the child of a depth d-1 node with at most top_k children
    per node.  A node's children are numbered consecutively, in the order of
    their parents, so every parent precedes its children.  Parents are drawn
    with weights 1/(rank+1) over the previous depth, favouring its earlier
    (higher-ranked) nodes."""
    rng = np.random.default_rng(seed)
    parents = [-1]
    prev = [0]
    for count in levels:
        if count > top_k * len(prev):
            raise ValueError("level larger than top_k children per node allow")
        load = np.zeros(len(prev), np.int64)
        picks = []
        for _ in range(count):
            wts = np.array([0.0 if load[r] >= top_k else 1.0 / (r + 1)
                            for r in range(len(prev))])
            r = int(rng.choice(len(prev), p=wts / wts.sum()))
            load[r] += 1
            picks.append(r)
        picks.sort()
        first = len(parents)
        parents.extend(prev[r] for r in picks)
        prev = list(range(first, len(parents)))
    return np.asarray(parents, np.int32)


def ancestor_masks(parents) -> np.ndarray:
    """mask[i] (uint64): bit j set iff node j is node i or one of its
    ancestors -- the rows of the block that node i's query may see."""
    parents = np.asarray(parents, np.int64)
    gamma = parents.shape[0]
    if gamma > 64:
        raise ValueError("at most 64 nodes")
    masks = np.zeros(gamma, np.uint64)
    for i in range(gamma):
        m, v = 0, i
        while v >= 0:
            m |= 1 << v
            v = int(parents[v]) if v > 0 else -1
        masks[i] = np.uint64(m)
    return masks


def tree_tokens(ref_argmax, parents, k: int, vocab: int, seed: int) -> np.ndarray:
    """Node tokens [gamma] int32 for a tree whose accepted path has exactly
    min(k, depth of the designated path) drafts.  The designated path starts
    at the root and follows the lowest-index child down to a leaf.  Its
    first k nodes carry the reference argmax of their parent; every other
    child of the root and of those k nodes carries an id different from its
    parent's reference argmax; all remaining nodes carry uniform ids.
    tokens[0] (the root) is 0."""
    ref = np.asarray(ref_argmax, np.int64)
    parents = np.asarray(parents, np.int64)
    gamma = parents.shape[0]
    rng = np.random.default_rng(seed)
    tok = rng.integers(0, vocab, size=gamma, dtype=np.int64)
    tok[0] = 0
    children = [[] for _ in range(gamma)]
    for j in range(1, gamma):
        children[int(parents[j])].append(j)
    path = [0]
    while children[path[-1]]:
        path.append(min(children[path[-1]]))
    k = min(k, len(path) - 1)
    for t in range(k + 1):
        node = path[t]
        for c in children[node]:
            if t < k and c == path[t + 1]:
                tok[c] = ref[node]
            else:
                r = int(rng.integers(0, vocab - 1))
                tok[c] = r if r < ref[node] else r + 1
    return tok.astype(np.int32)


def prefix_len(w: Workload, draft_seed: int) -> int:
    if w.accept_p is None:
        return int(w.fixed_prefix)
    return geometric_prefix(w.accept_p, w.gamma, draft_seed)


def router_logits(gamma, vocab, seed, device="cpu"):
    """Router-heavy logits: half the rows peaked, half flat (fp32)."""
    rng = np.random.default_rng(seed)
    perm = rng.permutation(gamma)
    peaked = set(int(r) for r in perm[: gamma // 2])
    rows = []
    for i in range(gamma):
        s = stream_seed(seed, "router_logits", i)
        if i in peaked:
            z = normal((vocab,), 8.0, s, torch.float32, device)
            boost = int(rng.integers(0, vocab))
            z[boost] = z.max() + 16.0
        else:
            z = normal((vocab,), 0.5, s, torch.float32, device)
        rows.append(z)
    return torch.stack(rows), sorted(peaked)


def generate_layer(w: Workload, layer: int, device="cpu", seed=None):
    """Per-layer tensors: q, k_cache, v_cache and (if any) x, w_k, w_v."""
    m = master_seed(w.cfg) if seed is None else seed
    dt = w.torch_dtype
    out = {
        "q": normal((w.gamma, w.n_q_heads, w.head_dim), w.qkv_std,
                    stream_seed(m, "q", layer), dt, device),
        "k_cache": normal_into(torch.empty((w.n_kv_heads, w.cap, w.head_dim),
                                           dtype=dt, device=device),
                               w.qkv_std, stream_seed(m, "k_cache", layer)),
        "v_cache": normal_into(torch.empty((w.n_kv_heads, w.cap, w.head_dim),
                                           dtype=dt, device=device),
                               w.qkv_std, stream_seed(m, "v_cache", layer)),
    }
    if w.n_prefill:
        out["x"] = normal((w.n_prefill, w.hidden), w.act_std,
                          stream_seed(m, "x", layer), dt, device)
        feat = w.n_kv_heads * w.head_dim
        out["w_k"] = normal((feat, w.hidden), w.w_std,
                            stream_seed(m, "w_k", layer), dt, device)
        out["w_v"] = normal((feat, w.hidden), w.w_std,
                            stream_seed(m, "w_v", layer), dt, device)
        if w.separate_drafter_cache:
            out["drafter_k_cache"] = normal(
                (w.n_kv_heads, w.prefill_cap, w.head_dim), w.qkv_std,
                stream_seed(m, "drafter_k_cache", layer), dt, device)
            out["drafter_v_cache"] = normal(
                (w.n_kv_heads, w.prefill_cap, w.head_dim), w.qkv_std,
                stream_seed(m, "drafter_v_cache", layer), dt, device)
    return out


def router_hidden(hidden: int) -> int:
    """Width of the neural router's hidden layer: d/8 (appendix on the
    neural router)."""
    return hidden // 8


def generate_router(w: Workload, device="cpu", seed=None):
    """Neural-router weights with random values (the trained router is not
    available): W1 [d/8][d] and b1 [d/8] ~ N(0, w_std), w2 [d/8] and b2 [1]
    ~ N(0, 0.05), which spreads the predicted gain over about +-1 token for
    post-norm activations, the range of the paper's thresholds."""
    m_seed = master_seed(w.cfg) if seed is None else seed
    dt = w.torch_dtype
    m = router_hidden(w.hidden)
    return {
        "w1": normal((m, w.hidden), w.w_std, stream_seed(m_seed, "router_w1"), dt, device),
        "b1": normal((m,), w.w_std, stream_seed(m_seed, "router_b1"), dt, device),
        "w2": normal((m,), 0.05, stream_seed(m_seed, "router_w2"), dt, device),
        "b2": normal((1,), 0.05, stream_seed(m_seed, "router_b2"), dt, device),
    }


DECODER_WEIGHTS = ("attn_norm", "w_q", "w_k", "w_v", "w_o", "mlp_norm",
                   "w_gate", "w_up", "w_down")


def generate_drafter(w: Workload, device="cpu", seed=None, cache_rows=None):
    """One drafter layer with random weights (the trained drafters are not
    available): projections N(0, w_std), RMSNorm gains 1 + N(0, 0.1); its KV
    cache [Hkv][cap][D] with the first `cache_rows` rows (default ctx_len)
    N(0, qkv_std) and the rest zero; the backlog's layer inputs r
    [n_prefill][hidden] N(0, act_std)."""
    m = master_seed(w.cfg) if seed is None else seed
    dt = w.torch_dtype
    d, qd, kd = w.hidden, w.n_q_heads * w.head_dim, w.n_kv_heads * w.head_dim
    shapes = {"attn_norm": (d,), "w_q": (qd, d), "w_k": (kd, d), "w_v": (kd, d),
              "w_o": (d, qd), "mlp_norm": (d,), "w_gate": (w.inter, d),
              "w_up": (w.inter, d), "w_down": (d, w.inter)}
    out = {}
    for i, name in enumerate(DECODER_WEIGHTS):
        s = stream_seed(m, "drafter", i)
        if name.endswith("norm"):
            t = normal(shapes[name], 0.1, s, torch.float32, device) + 1.0
            out[name] = t.to(dt)
        else:
            out[name] = normal(shapes[name], w.w_std, s, dt, device)
    rows = w.ctx_len if cache_rows is None else cache_rows
    cap = rows + w.n_prefill
    for name, tid in (("k_cache", 100), ("v_cache", 101)):
        c = torch.zeros((w.n_kv_heads, cap, w.head_dim), dtype=dt, device=device)
        if rows:
            c[:, :rows] = normal((w.n_kv_heads, rows, w.head_dim), w.qkv_std,
                                 stream_seed(m, "drafter", tid), dt, device)
        out[name] = c
    out["r"] = normal((w.n_prefill, d), w.act_std, stream_seed(m, "backlog"), dt, device)
    return out


def generate_head(w: Workload, device="cpu", seed=None):
    """LM-head inputs: h [gamma][hidden], w_lm [vocab][hidden] (+ logits)."""
    m = master_seed(w.cfg) if seed is None else seed
    dt = w.torch_dtype
    out = {
        "h": normal((w.gamma, w.hidden), w.act_std, stream_seed(m, "h"), dt,
                    device),
        "w_lm": normal_into(torch.empty((w.vocab, w.hidden), dtype=dt,
                                        device=device),
                            w.w_std, stream_seed(m, "w_lm")),
    }
    if w.router_logits:
        z, peaked = router_logits(w.gamma, w.vocab,
                                  stream_seed(m, "router_rows"), device)
        out["router_logits"] = z
        out["router_peaked_rows"] = peaked
    return out
