"""Host-side check of the GPU random-shape sweep's cases (tests/random_cases.py):
every drawn shape lies in the ranges the C ABI accepts, so the sweep tests
the kernels rather than argument validation.  No GPU call is made."""
import ctypes

import pytest

import random_cases as R

wf = pytest.importorskip("paper_2606_07710_amd")


def test_attention_cases_are_accepted():
    cases = R.attn_cases()
    assert any(c["tree"] for c in cases) and any(not c["tree"] for c in cases)
    assert {c["dh"] for c in cases} == {64, 128}
    assert {c["dt"] for c in cases} == {"f32", "bf16"}
    for c in cases:
        code = wf.WF_F32 if c["dt"] == "f32" else wf.WF_BF16
        assert 1 <= c["gamma"] <= 64 and c["ctx"] + c["gamma"] <= c["cap"]
        assert wf.wf_verify_attn_workspace_bytes(code, c["gamma"], c["ctx"], c["hq"],
                                                 c["hkv"], c["dh"], c["splits"]) > 0, c


def test_prefill_cases_are_accepted():
    for c in R.prefill_cases():
        if c["dt"] == "f32":
            code = wf.WF_F32
        else:
            code = wf.WF_BF16_TILED if c["tiled"] else wf.WF_BF16
            assert c["d_in"] % 32 == 0
            # bf16 plans need their exchange slots to fit: the query says 0 otherwise
            assert wf.wf_kv_only_prefill_workspace_bytes(code, c["n"], c["d_in"], c["hkv"],
                                                         c["dh"]) > 0, c
        assert c["start"] + c["n"] <= c["cap"]


def test_lmhead_cases_are_accepted():
    cases = R.lmhead_cases()
    assert any(c["tiled"] for c in cases)
    for c in cases:
        assert wf.wf_lmhead_workspace_bytes(c["gamma"], c["vocab"]) > 0, c
        if c["dt"] == "bf16":
            assert c["d"] % 32 == 0
        if c["tiled"]:
            assert c["d"] % 512 == 0 or (c["gamma"] <= 16 and c["d"] in (4096, 5120))


def test_drafter_cases_are_accepted():
    cases = R.drafter_cases()
    assert {c["kind"] for c in cases} == {"catchup", "forward"}
    assert any(c["tiled"] for c in cases) and any(not c["tiled"] for c in cases)
    assert {c["dh"] for c in cases} == {64, 128}
    for c in cases:
        assert c["hidden"] % 32 == 0 and c["inter"] % 32 == 0
        assert c["hq"] % c["hkv"] == 0
        # the workspace queries read only the layer's shapes: stand-in
        # pointers (never dereferenced) give its shape struct
        fake = [4096] * len(wf.DECODER_WEIGHTS)
        layer = wf.DecoderLayer(*fake, c["hidden"], c["hq"], c["hkv"], c["dh"],
                                c["inter"], 1e-6, 1e6)
        code = wf.WF_BF16_TILED if c["tiled"] else wf.WF_BF16
        if c["kind"] == "catchup":
            need = wf.lib.wf_drafter_catchup_workspace_bytes(code, ctypes.byref(layer),
                                                             c["n"], c["pos"])
        else:
            assert 1 <= c["n"] <= 64
            need = wf.lib.wf_drafter_forward_workspace_bytes(code, ctypes.byref(layer),
                                                             c["n"], c["pos"])
        assert need > 0, c


def test_router_cases_are_accepted():
    cases = R.router_cases()
    assert {c["dt"] for c in cases} == {"f32", "bf16"}
    for c in cases:
        code = wf.WF_F32 if c["dt"] == "f32" else wf.WF_BF16
        assert 1 <= c["gamma"] <= 64 and c["d"] >= 1 and 1 <= c["m"] <= 65536
        if c["dt"] == "bf16":
            assert c["d"] % 32 == 0 and c["m"] % 16 == 0
        assert wf.lib.wf_router_workspace_bytes(code, c["gamma"], c["d"], c["m"]) > 0, c


def test_tree_lmhead_cases_are_accepted():
    cases = R.tree_lmhead_cases()
    assert any(c["tiled"] for c in cases) and any(not c["tiled"] for c in cases)
    for c in cases:
        assert 1 <= c["gamma"] <= 64 and c["d"] % 32 == 0
        assert wf.wf_lmhead_workspace_bytes(c["gamma"], c["vocab"]) > 0, c
        if c["tiled"]:
            assert c["d"] % 512 == 0 or (c["gamma"] <= 16 and c["d"] in (4096, 5120))
        par = c["parents"]
        assert par[0] == -1 and all(0 <= par[j] < j for j in range(1, c["gamma"]))


def test_layer_prefill_cases_are_accepted():
    cases = R.layer_prefill_cases()
    assert any(c["tiled"] for c in cases) and any(not c["tiled"] for c in cases)
    for c in cases:
        code = wf.WF_BF16_TILED if c["tiled"] else wf.WF_BF16
        assert c["d_in"] % 32 == 0 and c["layers"] >= 2
        assert wf.wf_kv_only_prefill_layers_workspace_bytes(
            code, c["n"], c["d_in"], c["hkv"], c["dh"], c["layers"]) > 0, c
