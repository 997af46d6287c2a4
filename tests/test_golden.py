"""Values the paper prints, kept as small text fixtures under tests/golden/
(each file names its source): the neural router's parameter counts pin the
router's shape reading (m = d/8 hidden units, biases on both layers), and
the drafter settings pin the verify shapes of the workloads (the EAGLE-3
draft tree, the DFlash block)."""
import os

import numpy as np

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_router_parameter_counts():
    for model, hidden, params_m in _rows("router_parameter_counts.txt"):
        d = int(hidden)
        m = W.router_hidden(d)
        count = m * d + m + m + 1                # W1, b1, w2, b2
        assert round(count / 1e6, 2) == float(params_m), model
        # the oracle's router runs on exactly those shapes
        rng = np.random.default_rng(d)
        h = rng.standard_normal((2, d)).astype(np.float32)
        w1 = rng.standard_normal((m, d)).astype(np.float32) * 0.02
        b1 = np.zeros(m, np.float32)
        w2 = rng.standard_normal(m).astype(np.float32) * 0.05
        b2 = np.zeros(1, np.float32)
        assert oracle.router_mlp(h, w1, b1, w2, b2).shape == (2,)


def test_drafter_settings_shape_the_workloads():
    g = {k: int(v) for k, v in _rows("drafter_settings.txt")}
    tree = W.CONFIGS[6]
    assert len(tree.tree_levels) == g["eagle3_tree_depth"]
    assert sum(tree.tree_levels) == g["eagle3_draft_tokens"]
    assert tree.gamma == g["eagle3_draft_tokens"] + 1        # root + drafts
    par = W.draft_tree(seed=1)
    children = np.bincount(par[1:], minlength=len(par))
    assert children.max() <= g["eagle3_top_k"]
    for cfg in (3, 4, 5):                                     # diffusion blocks
        assert W.CONFIGS[cfg].gamma == g["dflash_block_qwen3"]
