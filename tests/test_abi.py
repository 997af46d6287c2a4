"""CPU checks of the C ABI: the library loads, exports every function the
header declares, and rejects invalid arguments on the host before anything
would touch the GPU (no compute call is made here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wf.h")

wf = pytest.importorskip("paper_2606_07710_amd")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wf_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_three_calls():
    names = _declared_functions()
    for n in ("wf_verify_attn", "wf_kv_only_prefill",
              "wf_lmhead_accept_entropy"):
        assert n in names


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(wf.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert set(_declared_functions()) == set(wf.EXPORTED_SYMBOLS)


def test_status_strings_and_version():
    assert wf.abi_version() == 9
    assert wf.status_string(wf.WF_OK) == "ok"
    assert "workspace" in wf.status_string(wf.WF_ERR_WORKSPACE)
    assert wf.status_string(99) == "unknown status"


FAKE = ctypes.c_void_p(1 << 20)      # 16-byte aligned, never dereferenced
ODD = ctypes.c_void_p((1 << 20) + 8)


def _attn(**kw):
    a = dict(dt=1, q=FAKE, k=FAKE, v=FAKE, out=FAKE, gamma=16, ctx=100,
             cap=116, hq=32, hkv=8, dh=128, scale=0.088, splits=0, ws=FAKE,
             ws_bytes=1 << 30)
    a.update(kw)
    return wf.lib.wf_verify_attn(a["dt"], a["q"], a["k"], a["v"], a["out"],
                                 a["gamma"], a["ctx"], a["cap"], a["hq"],
                                 a["hkv"], a["dh"], a["scale"], a["splits"],
                                 a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), 1), (dict(out=None), 1), (dict(gamma=0), 1),
    (dict(gamma=65), 1), (dict(ctx=-1), 1), (dict(cap=115), 1),
    (dict(hq=30), 1), (dict(dh=96), 2), (dict(dh=256), 2),
    (dict(q=ODD), 1), (dict(scale=0.0), 1), (dict(scale=float("nan")), 1),
    (dict(splits=-1), 1), (dict(splits=5000), 1), (dict(dt=7), 1),
    (dict(ws=None), 3), (dict(ws_bytes=16), 3), (dict(ws=ODD), 3),
])
def test_verify_attn_rejects(kw, status):
    assert _attn(**kw) == status


def _attn_noalloc(**kw):
    a = dict(dt=1, q=FAKE, k=FAKE, v=FAKE, out=FAKE, gamma=16, ctx=100,
             cap=116, hq=32, hkv=8, dh=128, scale=0.088, splits=0)
    a.update(kw)
    return wf.lib.wf_verify_attn_noalloc(a["dt"], a["q"], a["k"], a["v"], a["out"],
                                         a["gamma"], a["ctx"], a["cap"], a["hq"],
                                         a["hkv"], a["dh"], a["scale"], a["splits"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), 1), (dict(gamma=65), 1), (dict(cap=115), 1), (dict(hq=30), 1),
    (dict(dh=96), 2), (dict(q=ODD), 1), (dict(scale=0.0), 1), (dict(splits=5000), 1),
    # partials beyond the static scratch: 64 rows x 256 heads x 64 splits
    (dict(gamma=64, hq=256, ctx=4096, cap=4160, splits=64), 3),
])
def test_verify_attn_noalloc_rejects(kw, status):
    assert _attn_noalloc(**kw) == status


@pytest.mark.parametrize("args,status", [
    ((None, 1 << 20, FAKE, 1 << 20, 16), 1), ((FAKE, 1 << 20, None, 1 << 20, 16), 1),
    ((ODD, 1 << 20, FAKE, 1 << 20, 16), 1), ((FAKE, 1000, FAKE, 1 << 20, 16), 1),
    ((FAKE, 0, FAKE, 1 << 20, 16), 1), ((FAKE, 1 << 20, FAKE, 1 << 20, 0), 1),
    ((FAKE, 1 << 20, FAKE, 1 << 20, 70000), 1), ((FAKE, 1 << 20, FAKE, 4095, 1), 3),
])
def test_read_probe_rejects(args, status):
    assert wf.lib.wf_read_probe(*args, None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(base=None), 1), (dict(sink=None), 1), (dict(base=ODD), 1), (dict(nbytes=1000), 1),
    (dict(nbytes=0), 1), (dict(stride=1 << 19), 1), (dict(stride=(1 << 20) + 8), 1),
    (dict(n_bufs=0), 1), (dict(reps=0), 1), (dict(wgs=0), 1), (dict(wgs=70000), 1),
    (dict(depth=16), 1), (dict(depth=0), 1), (dict(sink_bytes=4095), 3),
])
def test_read_probe_series_rejects(kw, status):
    a = dict(base=FAKE, nbytes=1 << 20, stride=1 << 20, n_bufs=4, reps=2, sink=FAKE,
             sink_bytes=1 << 20, wgs=16, depth=4)
    a.update(kw)
    assert wf.lib.wf_read_probe_series(a["base"], a["nbytes"], a["stride"], a["n_bufs"],
                                       a["reps"], a["sink"], a["sink_bytes"], a["wgs"],
                                       a["depth"], None) == status


def _route(**kw):
    a = dict(dt=1, h=FAKE, w=FAKE, draft=FAKE, gamma=16, d=4096, vocab=151936, w1=FAKE,
             b1=FAKE, w2=FAKE, b2=FAKE, m=512, tau=0.5, am=FAKE, ent=FAKE, acc=FAKE,
             delta=FAKE, ws=FAKE, ws_bytes=1 << 34)
    a.update(kw)
    return wf.lib.wf_lmhead_accept_route_neural(
        a["dt"], a["h"], a["w"], a["draft"], a["gamma"], a["d"], a["vocab"], a["w1"], a["b1"],
        a["w2"], a["b2"], a["m"], a["tau"], a["am"], a["ent"], a["acc"], a["delta"], a["ws"],
        a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(w1=None), 1), (dict(b2=None), 1), (dict(delta=None), 1), (dict(w1=ODD), 1),
    (dict(m=0), 1), (dict(m=70000), 1), (dict(draft=None), 1), (dict(gamma=65), 1),
    (dict(tau=float("nan")), 1), (dict(m=500), 2), (dict(ws=None), 3), (dict(ws_bytes=4096), 3),
    (dict(dt=2, gamma=24, d=512), 2),      # tiled weights outside the fused shapes
])
def test_route_neural_rejects(kw, status):
    assert _route(**kw) == status


def test_route_neural_workspace_query():
    fused = wf.lib.wf_lmhead_route_neural_workspace_bytes(2, 16, 151936, 4096, 512)
    assert fused == wf.wf_lmhead_workspace_bytes(16, 151936) + 16 * 512 * 4
    assert wf.lib.wf_lmhead_route_neural_workspace_bytes(1, 24, 5000, 512, 64) > 0
    assert wf.lib.wf_lmhead_route_neural_workspace_bytes(1, 0, 5000, 512, 64) == 0


def test_noalloc_scratch_size_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define WF_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == wf.NOALLOC_SCRATCH_BYTES


# every workspace starts with the same block of arrival counters
COUNTER_BLOCK = 4 << 20


def test_workspace_query():
    need = wf.wf_verify_attn_workspace_bytes(1, 16, 32768, 32, 8, 128)
    assert need > 0 and need % 4 == 0
    assert wf.wf_verify_attn_workspace_bytes(1, 0, 32768, 32, 8, 128) == 0
    forced = wf.wf_verify_attn_workspace_bytes(1, 16, 32768, 32, 8, 128, 7)
    # bf16 partial outputs, fp32 (max, sum) per split and (row, head)
    assert forced == COUNTER_BLOCK + 7 * 16 * 32 * (128 * 2 + 8)
    # counter block, then one 16-byte row state per (row, 64-entry tile)
    assert wf.wf_lmhead_workspace_bytes(16, 151936) == COUNTER_BLOCK + 16 * 2374 * 16
    assert wf.wf_lmhead_workspace_bytes(0, 10) == 0


def _prefill(**kw):
    a = dict(dt=1, x=FAKE, wk=FAKE, wv=FAKE, kc=FAKE, vc=FAKE, n=16, start=10,
             cap=26, d_in=4096, hkv=8, dh=128, base=1e6, ws=FAKE,
             ws_bytes=1 << 30)
    a.update(kw)
    return wf.lib.wf_kv_only_prefill(a["dt"], a["x"], a["wk"], a["wv"],
                                     a["kc"], a["vc"], a["n"], a["start"],
                                     a["cap"], a["d_in"], a["hkv"], a["dh"],
                                     a["base"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), 1), (dict(vc=None), 1), (dict(n=-1), 1),
    (dict(cap=25), 1), (dict(start=-2), 1), (dict(dh=80), 2),
    (dict(d_in=100), 2), (dict(base=0.0), 1), (dict(hkv=0), 1),
    (dict(kc=ODD), 1), (dict(n=5000, cap=6000), 1), (dict(ws=None), 3),
    (dict(ws_bytes=64), 3), (dict(ws=ODD), 3),
])
def test_prefill_rejects(kw, status):
    assert _prefill(**kw) == status


def test_prefill_workspace_query():
    # the bf16 path only needs the zero block (its exchange slots live there)
    need = wf.wf_kv_only_prefill_workspace_bytes(1, 16, 4096, 8, 128)
    assert need == COUNTER_BLOCK
    assert wf.wf_kv_only_prefill_workspace_bytes(0, 16, 4096, 8, 128) == 0
    assert wf.wf_kv_only_prefill_workspace_bytes(1, 0, 4096, 8, 128) == 0
    assert wf.wf_kv_only_prefill_workspace_bytes(1, 16, 100, 8, 128) == 0


def test_prefill_zero_tokens_is_a_noop():
    assert _prefill(n=0) == 0


def _prefill_layers(**kw):
    a = dict(dt=1, x=FAKE, wk=FAKE, wv=FAKE, kc=FAKE, vc=FAKE, n=16, start=10,
             cap=26, d_in=4096, hkv=8, dh=128, base=1e6, layers=36,
             xs=16 * 4096, ws_=8 * 128 * 4096, cs=8 * 26 * 128, ws=FAKE,
             ws_bytes=1 << 30)
    a.update(kw)
    return wf.lib.wf_kv_only_prefill_layers(
        a["dt"], a["x"], a["wk"], a["wv"], a["kc"], a["vc"], a["n"], a["start"],
        a["cap"], a["d_in"], a["hkv"], a["dh"], a["base"], a["layers"], a["xs"],
        a["ws_"], a["cs"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(layers=0), 1), (dict(layers=1025), 1), (dict(xs=16 * 4096 - 8), 1),
    (dict(ws_=8 * 128 * 4096 - 8), 1), (dict(cs=8 * 26 * 128 - 8), 1),
    (dict(xs=16 * 4096 + 4), 1), (dict(cs=8 * 26 * 128 + 1), 1),
    (dict(x=None), 1), (dict(cap=25), 1), (dict(dh=80), 2), (dict(d_in=100), 2),
    (dict(ws=None), 3), (dict(ws_bytes=64), 3), (dict(kc=ODD), 1),
    (dict(dt=0, xs=16 * 4096 + 2), 1),
])
def test_prefill_layers_rejects(kw, status):
    assert _prefill_layers(**kw) == status


def test_prefill_layers_workspace_query_and_noop():
    assert wf.wf_kv_only_prefill_layers_workspace_bytes(1, 16, 4096, 8, 128, 36) == COUNTER_BLOCK
    assert wf.wf_kv_only_prefill_layers_workspace_bytes(1, 16, 4096, 8, 128, 0) == 0
    assert wf.wf_kv_only_prefill_layers_workspace_bytes(0, 16, 4096, 8, 128, 36) == 0
    assert _prefill_layers(n=0) == 0


def _lm(**kw):
    a = dict(dt=1, h=FAKE, w=FAKE, logits=None, draft=FAKE, gamma=16,
             d=4096, vocab=151936, tau=1.0, am=FAKE, ent=FAKE, acc=FAKE,
             ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return wf.lib.wf_lmhead_accept_entropy(
        a["dt"], a["h"], a["w"], a["logits"], a["draft"], a["gamma"], a["d"],
        a["vocab"], a["tau"], a["am"], a["ent"], a["acc"], a["ws"],
        a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(h=None), 1), (dict(gamma=0), 1), (dict(gamma=65), 1),
    (dict(vocab=0), 1), (dict(draft=None), 1), (dict(d=100), 2),
    (dict(logits=FAKE), 1), (dict(am=None), 1), (dict(tau=float("nan")), 1),
    (dict(ws_bytes=100), 3), (dict(ws=None), 3), (dict(w=ODD), 1),
])
def test_lmhead_rejects(kw, status):
    assert _lm(**kw) == status


def _attn_tree(**kw):
    a = dict(dt=1, q=FAKE, k=FAKE, v=FAKE, out=FAKE, mask=FAKE, gamma=61,
             ctx=100, cap=161, hq=32, hkv=8, dh=128, scale=0.088, splits=0,
             ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return wf.lib.wf_verify_attn_tree(
        a["dt"], a["q"], a["k"], a["v"], a["out"], a["mask"], a["gamma"],
        a["ctx"], a["cap"], a["hq"], a["hkv"], a["dh"], a["scale"],
        a["splits"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(mask=None), 1), (dict(mask=ODD), 1), (dict(q=None), 1),
    (dict(gamma=65), 1), (dict(cap=160), 1), (dict(dh=96), 2),
    (dict(ws_bytes=100), 3),
])
def test_verify_attn_tree_rejects(kw, status):
    assert _attn_tree(**kw) == status


def _lm_tree(**kw):
    a = dict(dt=1, h=FAKE, w=FAKE, logits=None, tok=FAKE, par=FAKE, gamma=61,
             d=4096, vocab=151936, tau=1.0, am=FAKE, ent=FAKE, acc=FAKE,
             path=FAKE, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return wf.lib.wf_lmhead_accept_tree(
        a["dt"], a["h"], a["w"], a["logits"], a["tok"], a["par"], a["gamma"],
        a["d"], a["vocab"], a["tau"], a["am"], a["ent"], a["acc"], a["path"],
        a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(tok=None), 1), (dict(par=None), 1), (dict(path=None), 1),
    (dict(gamma=65), 1), (dict(h=None), 1), (dict(d=100), 2),
    (dict(ws_bytes=100), 3), (dict(tau=float("nan")), 1),
])
def test_lmhead_tree_rejects(kw, status):
    assert _lm_tree(**kw) == status


def _compact(**kw):
    a = dict(dt=1, k=FAKE, v=FAKE, acc=FAKE, path=FAKE, gamma=61, ctx=100,
             cap=161, hkv=8, dh=128, layers=36, stride=8 * 161 * 128)
    a.update(kw)
    return wf.lib.wf_kv_compact_path(a["dt"], a["k"], a["v"], a["acc"],
                                     a["path"], a["gamma"], a["ctx"],
                                     a["cap"], a["hkv"], a["dh"], a["layers"],
                                     a["stride"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(k=None), 1), (dict(acc=None), 1), (dict(path=None), 1),
    (dict(gamma=0), 1), (dict(gamma=65), 1), (dict(cap=160), 1),
    (dict(k=ODD), 1), (dict(dh=96), 2), (dict(dt=7), 1),
    (dict(layers=0), 1), (dict(stride=8 * 161 * 128 - 1), 1),
    (dict(layers=1025), 1),
])
def test_compact_rejects(kw, status):
    assert _compact(**kw) == status


def _router(**kw):
    a = dict(dt=1, h=FAKE, w1=FAKE, b1=FAKE, w2=FAKE, b2=FAKE, row=FAKE,
             gamma=16, d=4096, m=512, tau=1.0, delta=FAKE, route=FAKE,
             ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return wf.lib.wf_router_neural(
        a["dt"], a["h"], a["w1"], a["b1"], a["w2"], a["b2"], a["row"],
        a["gamma"], a["d"], a["m"], a["tau"], a["delta"], a["route"], a["ws"],
        a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(h=None), 1), (dict(row=None), 1), (dict(delta=None), 1),
    (dict(gamma=0), 1), (dict(gamma=65), 1), (dict(m=0), 1), (dict(d=0), 1),
    (dict(d=100), 2), (dict(m=40), 2), (dict(tau=float("nan")), 1),
    (dict(w1=ODD), 1), (dict(ws_bytes=100), 3), (dict(ws=None), 3),
])
def test_router_rejects(kw, status):
    assert _router(**kw) == status


def test_router_workspace_query():
    # z in 16 slices of d (32 unit tiles x 16 slices = 512 workgroups), then
    # 32 unit-group sums, per row
    need = wf.lib.wf_router_workspace_bytes(1, 16, 4096, 512)
    assert need == COUNTER_BLOCK + (16 * 512 + 32) * 16 * 4
    assert wf.lib.wf_router_workspace_bytes(1, 16, 4096, 40) == 0
    assert wf.lib.wf_router_workspace_bytes(0, 3, 100, 40) == COUNTER_BLOCK + (40 + 3) * 3 * 4


def _layer(**kw):
    f = dict(hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128, inter=12288,
             rms_eps=1e-6, rope_base=1e6)
    f.update(kw)
    return wf.DecoderLayer(*[FAKE.value] * 9, f["hidden"], f["n_q_heads"],
                           f["n_kv_heads"], f["head_dim"], f["inter"], f["rms_eps"],
                           f["rope_base"])


def _drafter(fn, layer=None, **kw):
    a = dict(dt=1, r=FAKE, n=16, pos=4000, k=FAKE, v=FAKE, cap=4200, out=FAKE, ws=FAKE,
             ws_bytes=1 << 34)
    a.update(kw)
    lay = _layer() if layer is None else layer
    return getattr(wf.lib, fn)(a["dt"], ctypes.byref(lay), a["r"], a["n"], a["pos"],
                               a["k"], a["v"], a["cap"], a["out"], a["ws"],
                               a["ws_bytes"], None)


@pytest.mark.parametrize("fn", ["wf_drafter_forward", "wf_drafter_catchup"])
@pytest.mark.parametrize("kw,lay,status", [
    (dict(dt=0), None, 2), (dict(n=0), None, 1), (dict(cap=4015), None, 1),
    (dict(r=None), None, 1), (dict(out=ODD), None, 1), (dict(pos=-1), None, 1),
    (dict(ws_bytes=100), None, 3), (dict(ws=None), None, 3),
    ({}, dict(head_dim=96), 2), ({}, dict(hidden=4010), 2),
    ({}, dict(n_kv_heads=5), 1), ({}, dict(rms_eps=0.0), 1),
    ({}, dict(rope_base=-1.0), 1),
])
def test_drafter_rejects(fn, kw, lay, status):
    layer = _layer(**lay) if lay else None
    assert _drafter(fn, layer, **kw) == status


def test_drafter_token_limits():
    assert _drafter("wf_drafter_forward", n=65, cap=5000) == 1
    # the catch-up takes backlogs up to 2^20 tokens (KV-only prefill in
    # 4096-token batches); one more is rejected before anything is launched
    assert _drafter("wf_drafter_catchup", n=(1 << 20) + 1, pos=0, cap=(1 << 20) + 8) == 1
    lay = _layer()
    assert wf.lib.wf_drafter_catchup_workspace_bytes(1, ctypes.byref(lay), 4097, 4096) > 0
    lay = _layer()
    assert wf.lib.wf_drafter_forward_workspace_bytes(1, ctypes.byref(lay), 1, 4096) > COUNTER_BLOCK
    assert wf.lib.wf_drafter_catchup_workspace_bytes(1, ctypes.byref(lay), 80, 4096) > COUNTER_BLOCK
    assert wf.lib.wf_drafter_forward_workspace_bytes(0, ctypes.byref(lay), 1, 4096) == 0


def test_tiled_weight_bytes_and_rejects():
    assert wf.wf_tiled_weight_bytes(16, 32) == 16 * 32 * 2
    assert wf.wf_tiled_weight_bytes(37, 96) == 48 * 96 * 2          # rows padded to 16
    assert wf.wf_tiled_weight_bytes(151936, 4096) == 151936 * 4096 * 2
    for rows, cols in ((0, 32), (16, 16), (16, 100), (-1, 64)):
        assert wf.wf_tiled_weight_bytes(rows, cols) == 0
    t = wf.lib.wf_tile_weights
    assert t(None, 16, 32, FAKE, 1 << 20, None) == 1
    assert t(FAKE, 16, 32, None, 1 << 20, None) == 1
    assert t(ODD, 16, 32, FAKE, 1 << 20, None) == 1
    assert t(FAKE, 16, 100, 1 << 30, 1 << 20, None) == 1
    assert t(FAKE, 16, 32, 1 << 30, 64, None) == 3               # too small
    assert t(FAKE, 16, 32, (1 << 20) + 512, 1 << 20, None) == 1   # overlapping


def test_tiled_dtype_only_where_weights_are_streamed():
    # calls without weights reject it
    assert _attn(dt=2) == 1
    assert _compact(dt=2) == 1
    # LM head: the persistent kernels only
    assert _lm(dt=2, d=96, gamma=16) == 2
    assert _lm(dt=2, d=1056, gamma=16) == 2
    # prefill: accepted (validated like bf16), workspace as bf16
    assert _prefill(dt=2, d_in=100) == 2
    assert _prefill(dt=2, n=0) == 0
    assert wf.wf_kv_only_prefill_workspace_bytes(2, 16, 4096, 8, 128) == COUNTER_BLOCK
    assert wf.wf_kv_only_prefill_layers_workspace_bytes(2, 16, 4096, 8, 128, 36) == COUNTER_BLOCK
    assert _prefill_layers(dt=2, xs=16 * 4096 + 4) == 1
