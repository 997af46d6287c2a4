"""The switch path end to end (Sec. 3.4): verify rounds commit tokens, the
router picks the next drafter, the lazy catch-up bookkeeping hands out the
due backlog and wf_drafter_catchup brings the autoregressive drafter's
cache up to date.  Every catch-up output and the final cache are checked
against the fp64 oracle run over the same schedule, and the naive scheme
(catch-up every round) must leave the same cache rows."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity import TOL, host64, max_vec_rel_err

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
AR, DIFF = 0, 1


def _schedule(seed, n_rounds, p_ar):
    rng = np.random.default_rng(seed)
    rounds = [(int(rng.integers(1, 10)), AR if rng.random() < p_ar else DIFF)
              for _ in range(n_rounds)]
    return rounds + [(2, AR)]


@pytest.mark.parametrize("seed,prompt,first", [(1, 50, DIFF), (2, 7, AR), (3, 200, DIFF)])
def test_rounds_with_lazy_catchup(seed, prompt, first):
    print(f"switch path seed={seed} prompt={prompt}", flush=True)
    rounds = _schedule(seed, 30, 0.35)
    total = prompt + sum(n for n, _ in rounds)
    base = W.CONFIGS[7]
    w = dataclasses.replace(base, cfg=600 + seed, hidden=512, n_q_heads=4, n_kv_heads=2,
                            head_dim=128, inter=1024, ctx_len=prompt,
                            n_prefill=total - prompt, prefill_start=prompt,
                            prefill_cap=total, qkv_std=0.02 * np.sqrt(512))
    t = W.generate_drafter(w, device=DEV)
    r_all = torch.cat([W.normal((prompt, 512), 1.0, 17, torch.bfloat16, DEV), t["r"]])
    layer_w = {n: t[n] for n in W.DECODER_WEIGHTS}
    layer = wf.decoder_layer(layer_w, 4, 2, w.rms_eps, w.rope_base)
    host = {n: W.to_oracle(t[n]) for n in W.DECODER_WEIGHTS}
    r_host = W.to_oracle(r_all)

    caches = {}
    for lazy in (1, 0):
        kc, vc = t["k_cache"].clone(), t["v_cache"].clone()
        kref, vref = W.to_oracle(kc), W.to_oracle(vc)
        s = wf.wf_switch_init(first, lazy, prompt)
        out = torch.empty(512, dtype=torch.bfloat16, device=DEV)
        calls = 0
        for n_new, nxt in rounds:
            start, count = wf.wf_switch_commit(s, n_new, nxt)
            if count == 0:
                continue
            wf.wf_drafter_catchup(layer, r_all[start:start + count], start, kc, vc, out)
            ref, kref, vref = oracle.catchup(r_host[start:start + count], start, host,
                                             kref, vref, 4, 2, w.rms_eps, w.rope_base)
            torch.cuda.synchronize()
            assert max_vec_rel_err(host64(out)[None], ref[None]) <= TOL["bf16"], (lazy, start)
            calls += 1
        assert s.ar_cache_len == s.committed == total
        assert calls == s.catchups
        got_k, got_v = host64(kc), host64(vc)
        assert max_vec_rel_err(got_k[:, prompt:], kref[:, prompt:]) <= TOL["bf16"]
        assert max_vec_rel_err(got_v[:, prompt:], vref[:, prompt:]) <= TOL["bf16"]
        # the prompt rows were never touched
        assert torch.equal(kc[:, :prompt].view(torch.int16),
                           t["k_cache"][:, :prompt].view(torch.int16))
        caches[lazy] = (got_k, got_v, s.catchups)
    # lazy and naive leave the same rows; lazy in fewer calls
    assert max_vec_rel_err(caches[1][0], caches[0][0]) <= TOL["bf16"]
    assert max_vec_rel_err(caches[1][1], caches[0][1]) <= TOL["bf16"]
    assert caches[1][2] < caches[0][2]
