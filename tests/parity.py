"""Comparison helpers for the GPU-vs-oracle parity tests.

Tolerances (per output vector, max-norm relative): 2e-2 for bf16 storage,
1e-4 for fp32, the bar the verification step is held to.  Entropy: absolute
difference over max(|H_ref|, 1e-3 nats).  Argmax and acceptance: exact
wherever the oracle's top-2 logit margin exceeds 1e-2 (fp32 cases: 1e-6).
"""
import numpy as np
import torch

TOL = {"f32": 1e-4, "bf16": 2e-2}
ARGMAX_MARGIN = {"f32": 1e-6, "bf16": 1e-2}


def dtype_name(t) -> str:
    return "f32" if t.dtype == torch.float32 else "bf16"


def host64(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def max_vec_rel_err(got, ref, axis=-1) -> float:
    """max over vectors of ||got - ref||_inf / ||ref||_inf (vectors along
    `axis`)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.abs(got - ref).max(axis=axis)
    den = np.maximum(np.abs(ref).max(axis=axis), 1e-30)
    return float((num / den).max())


def entropy_rel_err(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float((np.abs(got - ref) / np.maximum(np.abs(ref), 1e-3)).max())


def check_argmax(got, ref, margin, logits_ref, dt):
    """Exact where the oracle margin exceeds the bar; elsewhere the GPU's
    choice must be (within the bar) a maximiser of the oracle logits."""
    bar = ARGMAX_MARGIN[dt]
    got = np.asarray(got)
    for i in range(len(ref)):
        if margin[i] > bar:
            assert got[i] == ref[i], (i, got[i], ref[i], margin[i])
        elif logits_ref is not None:
            zmax = logits_ref[i].max()
            assert logits_ref[i][got[i]] >= zmax - bar, (i, got[i], ref[i])


def accept_is_consistent(n, bonus, route, argmax, entropy, draft, tau):
    """The GPU accept triple agrees with its own argmax/entropy outputs."""
    gamma = len(argmax)
    k = 0
    while k < gamma - 1 and draft[k] == argmax[k]:
        k += 1
    return n == k and bonus == argmax[k] and route == int(entropy[k] > tau)


def check_tree_accept(am, ent, acc, path, am_ref, ent_ref, margin, tok, par, tau, bar):
    """Tree acceptance (Sec. 3.1 draft trees, Sec. 3.3.1 route): the GPU's
    accept outputs follow exactly from its own argmax and entropy; and
    wherever the oracle's margins on its accepted path exceed the bar (so
    both sides agree on those argmaxes), they equal the oracle's.  Returns
    the oracle's acceptance."""
    import oracle
    own = oracle.accept_tree(am, ent.astype(np.float64), tok, par, tau)
    assert acc.tolist() == [own[0], own[1], own[2], own[3]]
    assert path.tolist() == own[5].tolist()
    ref = oracle.accept_tree(am_ref, ent_ref, tok, par, tau)
    on_path = ref[5][:ref[0] + 1]
    if np.all(margin[on_path] > bar):
        assert [acc[0], acc[1], acc[3]] == [ref[0], ref[1], ref[3]]
        assert path.tolist() == ref[5].tolist()
        if abs(ent_ref[ref[3]] - tau) > 1e-3 * max(1.0, abs(tau)):
            assert acc[2] == ref[2]
    return ref
