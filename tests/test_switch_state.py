"""Host-side lazy catch-up bookkeeping (Sec. 3.4; the lazy vs naive study
of Sec. 4): which backlog of the autoregressive drafter's KV cache is due
after each verify round.  Checked against the scheme written out round by
round, on random round sequences, with no GPU."""
import ctypes
import random

import pytest

wf = pytest.importorskip("paper_2606_07710_amd")
AR, DIFF = wf.WF_DRAFTER_AR, wf.WF_DRAFTER_DIFFUSION


def _rounds(seed, n_rounds, p_ar=0.5):
    rng = random.Random(seed)
    return [(rng.randint(1, 17), AR if rng.random() < p_ar else DIFF)
            for _ in range(n_rounds)]


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("first", [AR, DIFF])
def test_lazy_hands_out_the_whole_backlog_on_a_switch(seed, first):
    prompt = 37 + seed
    s = wf.wf_switch_init(first, 1, prompt)
    committed, cache, due_calls = prompt, prompt, []
    for n_new, nxt in _rounds(seed, 200):
        start, count = wf.wf_switch_commit(s, n_new, nxt)
        committed += n_new
        if nxt == AR:
            # the AR drafter drafts next: every token since its cache last
            # caught up, in one batch starting at its cache length
            assert (start, count) == (cache, committed - cache)
            cache = committed
            due_calls.append(count)
        else:
            assert count == 0                  # no work for the inactive drafter
            assert start == cache
        assert s.committed == committed and s.ar_cache_len == cache
        assert s.active == nxt
        assert s.ar_cache_len <= s.committed
        if s.active == AR:
            assert s.ar_cache_len == s.committed
    assert s.caught_up == sum(due_calls) == cache - prompt
    assert s.catchups == len(due_calls)
    assert s.max_backlog == max(due_calls, default=0)


def test_switch_count_and_backlog_sizes():
    s = wf.wf_switch_init(AR, 1, 100)
    seq = [(5, AR), (3, DIFF), (4, DIFF), (7, DIFF), (2, AR), (6, DIFF), (1, AR)]
    got = [wf.wf_switch_commit(s, n, d) for n, d in seq]
    assert got == [(100, 5), (105, 0), (105, 0), (105, 0), (105, 16), (121, 0),
                   (121, 7)]
    assert s.switches == 2                     # DIFF -> AR twice
    assert (s.committed, s.ar_cache_len, s.max_backlog) == (128, 128, 16)


@pytest.mark.parametrize("seed", range(4))
def test_naive_updates_every_round_and_matches_lazy_rows(seed):
    """The naive scheme hands out each round's tokens every round; both
    schemes end with the same cache rows once the AR drafter is active,
    lazy in fewer, larger batches."""
    prompt = 64
    lazy = wf.wf_switch_init(DIFF, 1, prompt)
    naive = wf.wf_switch_init(DIFF, 0, prompt)
    committed = prompt
    rows_lazy, rows_naive = [], []
    for n_new, nxt in _rounds(100 + seed, 150, p_ar=0.3) + [(3, AR)]:
        a, n = wf.wf_switch_commit(naive, n_new, nxt)
        assert (a, n) == (committed, n_new)
        committed += n_new
        rows_naive += range(a, a + n)
        a, n = wf.wf_switch_commit(lazy, n_new, nxt)
        rows_lazy += range(a, a + n)
    # every row exactly once, in order, under both schemes
    assert rows_lazy == rows_naive == list(range(prompt, committed))
    assert lazy.catchups <= naive.catchups == 151
    assert lazy.max_backlog >= naive.max_backlog


def test_rejects():
    with pytest.raises(wf.WfError):
        wf.wf_switch_init(2, 1, 0)
    with pytest.raises(wf.WfError):
        wf.wf_switch_init(AR, 2, 0)
    with pytest.raises(wf.WfError):
        wf.wf_switch_init(AR, 1, -1)
    s = wf.wf_switch_init(DIFF, 1, 10)
    before = bytes(s)
    for n_new, nxt in ((0, AR), (-3, AR), (1, 2), (1, -1)):
        with pytest.raises(wf.WfError):
            wf.wf_switch_commit(s, n_new, nxt)
        assert bytes(s) == before              # state unchanged on error
    s = wf.wf_switch_init(DIFF, 1, 2**31 - 10)
    with pytest.raises(wf.WfError):
        wf.wf_switch_commit(s, 10, AR)         # sequence length past INT32_MAX
    assert wf.wf_switch_commit(s, 9, AR) == (2**31 - 10, 9)
    assert wf.lib.wf_switch_commit(None, 1, AR, None, None) == wf.WF_ERR_INVALID_ARG


def _fake_layer(hidden=4096, hq=32, hkv=8, hd=128, inter=12288):
    fake = 1 << 20                        # 16-byte aligned, never dereferenced
    return wf.DecoderLayer(*([fake] * len(wf.DECODER_WEIGHTS)), hidden, hq, hkv, hd, inter,
                           1e-6, 1e6)


def test_a_long_lazy_backlog_is_accepted_by_the_catchup():
    """Rounds on the diffusion drafter pile up a backlog far beyond one
    KV-only prefill batch (4096 tokens); the switch back hands it out in one
    piece, and the catch-up takes it (in 4096-token prefill batches)."""
    s = wf.wf_switch_init(AR, 1, 100)
    for _ in range(700):
        assert wf.wf_switch_commit(s, 16, DIFF) == (100, 0)
    start, count = wf.wf_switch_commit(s, 16, AR)
    assert (start, count) == (100, 701 * 16) and count > 4096
    layer = _fake_layer()
    for code in (wf.WF_BF16, wf.WF_BF16_TILED):
        need = int(wf.lib.wf_drafter_catchup_workspace_bytes(code, ctypes.byref(layer),
                                                             count, start))
        assert need >= count * 4096 * 2     # the normalised backlog is staged
    assert int(wf.lib.wf_drafter_catchup_workspace_bytes(
        wf.WF_BF16, ctypes.byref(layer), (1 << 20) + 1, 0)) == 0
