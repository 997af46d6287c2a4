"""GPU parity of wf_lmhead_accept_entropy against the fp64 oracle (Sec. 3.3.1
entropy and routing rule; greedy acceptance), including the logits-only
mode, ragged vocabulary tiles, closed-form entropies and the accept
construction used by the workloads."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import (TOL, accept_is_consistent, check_argmax, entropy_rel_err)

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _run(h=None, w=None, logits=None, draft=None, tau=1.0):
    gamma = (logits if logits is not None else h).shape[0]
    am = torch.empty(gamma, dtype=torch.int32, device=DEV)
    ent = torch.empty(gamma, dtype=torch.float32, device=DEV)
    acc = torch.empty(3, dtype=torch.int32, device=DEV)
    dr = None
    if gamma > 1:
        dr = torch.as_tensor(np.asarray(draft, np.int32), device=DEV)
    wf.wf_lmhead_accept_entropy(h, w, logits, dr, tau, am, ent, acc)
    torch.cuda.synchronize()
    return am.cpu().numpy(), ent.cpu().numpy(), acc.cpu().numpy()


CASES = [
    # dt, gamma, d, vocab, h std, w std
    ("bf16", 1, 256, 1000, 1.0, 0.05),
    ("bf16", 5, 512, 4096 + 13, 1.0, 0.05),
    ("bf16", 16, 4096, 20000, 1.0, 0.02),
    ("bf16", 17, 1024, 3000, 1.0, 0.05),
    ("bf16", 64, 256, 2000, 1.0, 0.1),
    ("bf16", 8, 4096, 151936, 1.0, 0.02),
    # the wide-row kernel (hidden size a multiple of 512): every row-group
    # count, runs of one to five blocks per wave, ragged vocabularies
    ("bf16", 24, 1024, 2000, 1.0, 0.05),
    ("bf16", 40, 512, 70001, 1.0, 0.05),
    ("bf16", 61, 4096, 151936, 1.0, 0.02),
    ("bf16", 64, 512, 300000, 1.0, 0.05),
    ("bf16", 33, 512, 15, 1.0, 0.05),
    ("f32", 8, 512, 4096, 0.02, 0.02),
    ("f32", 3, 100, 1001, 1.0, 0.1),
    ("f32", 1, 64, 77, 1.0, 0.3),
]


@pytest.mark.parametrize("dt,gamma,d,vocab,hs,ws", CASES)
def test_matches_oracle(dt, gamma, d, vocab, hs, ws):
    print(f"lmhead parity {dt} gamma={gamma} d={d} vocab={vocab}", flush=True)
    seed = gamma * 131 + vocab
    h = W.normal((gamma, d), hs, W.stream_seed(seed, "h"), DT[dt], DEV)
    w = W.normal((vocab, d), ws, W.stream_seed(seed, "w_lm"), DT[dt], DEV)
    am_ref, ent_ref, margin, z = oracle.lmhead_rows(W.to_oracle(h),
                                                    W.to_oracle(w),
                                                    want_logits=True)
    k = W.geometric_prefix(0.3, gamma, seed)
    draft = W.make_drafts(am_ref, k, vocab, seed)
    tau = float(np.median(ent_ref))
    am, ent, acc = _run(h, w, draft=draft, tau=tau)
    check_argmax(am, am_ref, margin, z, dt)
    assert entropy_rel_err(ent, ent_ref) <= TOL[dt]
    assert accept_is_consistent(acc[0], acc[1], acc[2], am, ent, draft, tau)
    bar = 1e-2 if dt == "bf16" else 1e-6
    if all(margin[j] > bar for j in range(min(k, gamma - 1) + 1)):
        n_ref, bonus_ref, _, _ = oracle.accept(am_ref, ent_ref, draft, tau)
        assert (acc[0], acc[1]) == (n_ref, bonus_ref) and n_ref == k


def test_logits_mode_router_mixture():
    gamma, vocab = 16, 151936
    z, peaked = W.router_logits(gamma, vocab, seed=77, device=DEV)
    am_ref, ent_ref, margin = oracle.lmhead_rows(logits=z.cpu().numpy())
    draft = W.make_drafts(am_ref, 3, vocab, 5)
    am, ent, acc = _run(logits=z.contiguous(), draft=draft, tau=2.0)
    np.testing.assert_array_equal(am, am_ref)
    assert entropy_rel_err(ent, ent_ref) <= 1e-4
    assert tuple(acc) == oracle.accept(am_ref, ent_ref, draft, 2.0)[:3]
    for r in peaked:                  # boosted rows: entropy ~ 0
        assert ent[r] < 1e-3


@pytest.mark.parametrize("vocab", [4096, 151936, 1000, 257])
def test_uniform_logits_give_log_vocab(vocab):
    z = torch.full((3, vocab), 0.75, dtype=torch.float32, device=DEV)
    am, ent, acc = _run(logits=z, draft=[0, 0], tau=0.0)
    np.testing.assert_allclose(ent, math.log(vocab), rtol=1e-5)
    assert list(am) == [0, 0, 0]
    assert tuple(acc) == (2, 0, 1)


def test_one_hot_logits_give_zero_entropy():
    vocab = 5000
    z = torch.full((4, vocab), float("-inf"), dtype=torch.float32, device=DEV)
    hot = [17, 4999, 0, 2048]
    for r, v in enumerate(hot):
        z[r, v] = 3.0 - r
    am, ent, acc = _run(logits=z, draft=[17, 4999, 1], tau=0.5)
    assert list(am) == hot
    np.testing.assert_array_equal(ent, 0.0)
    assert tuple(acc) == (2, 0, 0)
    z = torch.zeros((2, vocab), dtype=torch.float32, device=DEV)
    z[:, 123] = 1e4
    am, ent, _ = _run(logits=z, draft=[123], tau=0.0)
    assert list(am) == [123, 123] and float(ent.max()) == 0.0


def test_ties_resolve_to_lowest_index():
    vocab = 3000
    z = torch.zeros((2, vocab), dtype=torch.float32, device=DEV)
    z[0, [2999, 1500, 700]] = 5.0
    z[1, [64, 63]] = 2.0
    am, _, _ = _run(logits=z, draft=[700], tau=0.0)
    assert list(am) == [700, 63]


def test_gamma_one_and_full_accept():
    vocab, d = 4096, 512
    h = W.normal((1, d), 1.0, 5, torch.bfloat16, DEV)
    w = W.normal((vocab, d), 0.05, 6, torch.bfloat16, DEV)
    am, ent, acc = _run(h, w, tau=1e9)
    assert tuple(acc) == (0, am[0], 0)
    h = W.normal((8, d), 1.0, 7, torch.bfloat16, DEV)
    am_ref, ent_ref, margin = oracle.lmhead_rows(W.to_oracle(h), W.to_oracle(w))
    am, ent, acc = _run(h, w, draft=am_ref[:7], tau=-1.0)
    if (margin > 1e-2).all():
        assert tuple(acc) == (7, am_ref[7], 1)


def test_repeated_calls_are_bit_identical():
    vocab, d = 20000, 4096
    h = W.normal((16, d), 1.0, 8, torch.bfloat16, DEV)
    w = W.normal((vocab, d), 0.02, 9, torch.bfloat16, DEV)
    a = _run(h, w, draft=list(range(15)), tau=1.0)
    b = _run(h, w, draft=list(range(15)), tau=1.0)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
