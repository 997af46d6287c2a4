#!/usr/bin/env python3
"""Benchmark of the WhiFlash verification step on one MI355X.

One step = the whole hot path over one synthetic batch, issued on one
stream in model order:
  n_layers x wf_verify_attn      (block-causal GQA attention vs the cache)
  n_layers x wf_kv_only_prefill  (catch-up K/V projection + RoPE + append;
                                  --batch-prefill-layers: one
                                  wf_kv_only_prefill_layers call for all
                                  layers, reported as an upper bound only)
  1 x wf_lmhead_accept_entropy   (LM head -> argmax, entropy, accept, route)
W_k, W_v and W_lm are streamed in the tiled layout (wf_tile_weights, done
once at setup like weight preprocessing at model load;
--row-major-weights: the untiled tensors).
(the router-heavy workload adds the logits-only LM-head call).  Inputs are
seeded synthetic tensors already resident in HBM.  The default workload is
8B shapes at 32K context with a 16-token block (36 layers).

Output: ONE JSON line.  `value` is the verify-step time in microseconds
(lower is better); the roofline object reports the dominant kernel, the
per-layer verify attention, against HBM bandwidth using the algorithmic
bytes of one call; cpu_baseline is the fp64 oracle timed on host cores on a
bounded sample of the same step, scaled to one step.
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
PEAK_BF16_FLOPS = 2.5e15       # dense bf16 MFMA


def parse():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3,
                    help="workload 1..7 (default 3: 8B shapes, ctx 32K, "
                         "gamma 16, 16 catch-up tokens; 6: draft-tree "
                         "verification; 7: drafter switch catch-up)")
    ap.add_argument("--switch-table", action="store_true",
                    help="with --config 7: also sweep base KV length x "
                         "backlog, compare KV-only catch-up with the full "
                         "layer over the backlog and with per-round updates")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step as one captured HIP graph")
    ap.add_argument("--overlap", action="store_true",
                    help="run the catch-up prefill on a second stream, "
                         "concurrent with the verification attention.  Off by "
                         "default: in a round the catch-up follows the route "
                         "decision and reads the target's features of the "
                         "accepted tokens, so it depends on the verification")
    ap.add_argument("--batch-prefill-layers", action="store_true",
                    help="one wf_kv_only_prefill_layers call for all layers "
                         "instead of one call per layer (an upper bound: a "
                         "real forward has a layer-to-layer dependency)")
    ap.add_argument("--row-major-weights", action="store_true",
                    help="stream W_k, W_v and W_lm in their row-major layout "
                         "instead of the tiled copies made once at setup")
    ap.add_argument("--router", choices=("entropy", "neural"), default="entropy",
                    help="routing policy: the entropy rule evaluated with the "
                         "LM head (default), or the neural policy (a two-layer "
                         "MLP on the final accepted row's hidden state) as "
                         "one more call per step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=20.0,
                    help="approximate seconds of oracle work for cpu_baseline")
    ap.add_argument("--cpu-sample-layers", type=int, default=None,
                    help="cap on the layers the cpu baseline runs")
    ap.add_argument("--copy-probe-mib", type=int, default=1024,
                    help="size of the plain device copy run after timing "
                         "(the known-size reference that scales the HBM "
                         "traffic counters of a profiling run; not timed "
                         "for the roofline); 0 = off")
    ap.add_argument("--read-probe-mib", type=int, default=1024,
                    help="buffer the streaming-read ceiling is measured on "
                         "(larger than the 256 MB last-level cache); 0 = off")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Step:
    """Pre-marshalled C-ABI calls of one verification step."""

    def __init__(self, w, layers, head, outs, lmouts, draft, tau, ws_attn,
                 ws_pre, ws_lm, wf, tree=None, router=None, pre_stack=None,
                 w_lm_tiled=None):
        self.w, self.layers, self.head = w, layers, head
        self.outs, self.lmouts, self.draft, self.tau = outs, lmouts, draft, tau
        self.ws_attn, self.ws_pre, self.ws_lm, self.wf = ws_attn, ws_pre, ws_lm, wf
        # draft-tree workloads: {"mask", "parents", "path", "k_all", "v_all"}
        # (draft then holds the node tokens)
        self.tree = tree
        # neural routing policy: {"w1", "b1", "w2", "b2", "delta", "route", "ws"}
        self.router = router
        # all layers' catch-up inputs and caches as [L][...] stacks: one
        # multi-layer prefill call ({"x", "w_k", "w_v", "k", "v"})
        self.pre_stack = pre_stack
        # the LM head's weight in the tiled layout (None: row-major)
        self.w_lm_tiled = w_lm_tiled

    def build(self, stream, catchup=None):
        """Marshal every call for `stream`; with `catchup` (a second stream),
        the KV-only prefill calls go there and run concurrently with the
        verification attention: they write disjoint cache rows and read
        nothing the attention writes."""
        import torch
        w, wf = self.w, self.wf
        P = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
        code = wf.WF_BF16 if w.dtype == "bf16" else wf.WF_F32
        s = ctypes.c_void_p(stream.cuda_stream)
        s2 = ctypes.c_void_p((catchup or stream).cuda_stream)
        self.stream, self.catchup = stream, catchup
        self.fork = torch.cuda.Event()
        self.join = torch.cuda.Event()
        self.attn = []
        self.pre = []
        self.compact = []
        tr = self.tree
        self.attn_fn = wf.lib.wf_verify_attn_tree if tr else wf.lib.wf_verify_attn
        for l, t in enumerate(self.layers):
            mask = (P(tr["mask"]),) if tr else ()
            self.attn.append((code, P(t["q"]), P(t["k_cache"]), P(t["v_cache"]),
                              P(self.outs[l])) + mask +
                             (w.gamma, w.ctx_len, w.cap,
                              w.n_q_heads, w.n_kv_heads, w.head_dim,
                              w.softmax_scale, 0, P(self.ws_attn),
                              self.ws_attn.numel(), s))
            if w.n_prefill and self.pre_stack is None:
                kc = t["drafter_k_cache"] if w.separate_drafter_cache else t["k_cache"]
                vc = t["drafter_v_cache"] if w.separate_drafter_cache else t["v_cache"]
                wk, wv = t.get("w_k_tiled", t["w_k"]), t.get("w_v_tiled", t["w_v"])
                pc = wf.WF_BF16_TILED if isinstance(wk, wf.TiledWeight) else code
                self.pre.append((pc, P(t["x"]), P(wk), P(wv), P(kc),
                                 P(vc), w.n_prefill, w.prefill_start,
                                 kc.shape[1], w.hidden, w.n_kv_heads,
                                 w.head_dim, w.rope_base, P(self.ws_pre),
                                 self.ws_pre.numel(), s2))
        self.pre_fn = wf.lib.wf_kv_only_prefill
        ps = self.pre_stack
        if ps is not None:
            self.pre_fn = wf.lib.wf_kv_only_prefill_layers
            pcode = wf.WF_BF16_TILED if isinstance(ps["w_k"], wf.TiledWeight) else code
            self.pre = [(pcode, P(ps["x"]), P(ps["w_k"]), P(ps["w_v"]), P(ps["k"]),
                         P(ps["v"]), w.n_prefill, w.prefill_start, ps["k"].shape[2],
                         w.hidden, w.n_kv_heads, w.head_dim, w.rope_base,
                         ps["x"].shape[0], ps["x"].stride(0), ps["w_k"].stride(0),
                         ps["k"].stride(0), P(self.ws_pre), self.ws_pre.numel(), s2)]
        am, ent, acc = self.lmouts[0]
        w_lm = self.head["w_lm"] if self.w_lm_tiled is None else self.w_lm_tiled
        lcode = code if self.w_lm_tiled is None else wf.WF_BF16_TILED
        self.route = []
        rt = self.router
        if rt:
            m = rt["w1"].shape[0]
            row = ctypes.c_void_p(acc.data_ptr() + (12 if tr else 0))
            self.route = [(code, P(self.head["h"]), P(rt["w1"]), P(rt["b1"]),
                           P(rt["w2"]), P(rt["b2"]), row, w.gamma, w.hidden, m,
                           1.0, P(rt["delta"]), P(rt["route"]), P(rt["ws"]),
                           rt["ws"].numel(), s)]
        if tr:
            self.lm_fn = wf.lib.wf_lmhead_accept_tree
            self.lm = [(lcode, P(self.head["h"]), P(w_lm), None,
                        P(self.draft), P(tr["parents"]), w.gamma, w.hidden,
                        w.vocab, self.tau, P(am), P(ent), P(acc), P(tr["path"]),
                        P(self.ws_lm), self.ws_lm.numel(), s)]
            ka, va = tr["k_all"], tr["v_all"]
            self.compact = [(code, P(ka), P(va), P(acc), P(tr["path"]), w.gamma,
                             w.ctx_len, w.cap, w.n_kv_heads, w.head_dim,
                             ka.shape[0], ka[0].numel(), s)]
            return
        # (each LM-head entry is (C function, arguments...))
        self.lm_fn = lambda fn, *a: fn(*a)
        if rt:
            # the neural policy in the LM-head pass: one call forms the
            # logits' row states and the router's hidden layer from h
            m = rt["w1"].shape[0]
            w1 = rt.get("w1_tiled", rt["w1"])
            self.lm = [(wf.lib.wf_lmhead_accept_route_neural, lcode, P(self.head["h"]),
                        P(w_lm), P(self.draft), w.gamma, w.hidden, w.vocab, P(w1),
                        P(rt["b1"]), P(rt["w2"]), P(rt["b2"]), m, 1.0, P(am), P(ent),
                        P(acc), P(rt["delta"]), P(self.ws_lm), self.ws_lm.numel(), s)]
            self.route = []
        else:
            self.lm = [(wf.lib.wf_lmhead_accept_entropy, lcode, P(self.head["h"]),
                        P(w_lm), None, P(self.draft), w.gamma, w.hidden, w.vocab,
                        self.tau, P(am), P(ent), P(acc), P(self.ws_lm),
                        self.ws_lm.numel(), s)]
        if w.router_logits:
            am2, ent2, acc2 = self.lmouts[1]
            self.lm.append((wf.lib.wf_lmhead_accept_entropy, code, None, None,
                            P(self.head["router_logits"]), P(self.draft), w.gamma, 0,
                            w.vocab, self.tau, P(am2), P(ent2), P(acc2), P(self.ws_lm),
                            self.ws_lm.numel(), s))

    def run(self, check=False):
        lib = self.wf.lib

        def prefill():
            for a in self.pre:
                rc = self.pre_fn(*a)
                if check and rc:
                    raise RuntimeError(f"KV-only prefill: {self.wf.status_string(rc)}")
        if self.catchup is not None:
            self.fork.record(self.stream)
            self.catchup.wait_event(self.fork)
            prefill()                       # marshalled for the catch-up stream
        for a in self.attn:
            rc = self.attn_fn(*a)
            if check and rc:
                raise RuntimeError(f"verify attention: {self.wf.status_string(rc)}")
        if self.catchup is None:
            prefill()
        else:
            self.join.record(self.catchup)
            self.stream.wait_event(self.join)
        for a in self.lm:
            rc = self.lm_fn(*a)
            if check and rc:
                raise RuntimeError(f"LM head: {self.wf.status_string(rc)}")
        for a in self.compact:
            rc = lib.wf_kv_compact_path(*a)
            if check and rc:
                raise RuntimeError(f"wf_kv_compact_path: {self.wf.status_string(rc)}")
        for a in self.route:
            rc = lib.wf_router_neural(*a)
            if check and rc:
                raise RuntimeError(f"wf_router_neural: {self.wf.status_string(rc)}")

    def phases(self):
        """(name, C function, argument tuples, stream) of the step's three
        phases."""
        lib = self.wf.lib
        ph = [("attention", self.attn_fn, self.attn, self.stream),
              ("prefill", self.pre_fn, self.pre,
               self.catchup or self.stream),
              ("lmhead", self.lm_fn, self.lm, self.stream)]
        if self.compact:
            ph.append(("compaction", lib.wf_kv_compact_path, self.compact,
                       self.stream))
        if self.route:
            ph.append(("router", lib.wf_router_neural, self.route, self.stream))
        return ph


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "verify_attn_8b_ctx32k_hbm_traffic.md")


MFMA_PROFILE = os.path.join(ROOT, "profiles", "verify_step_8b_ctx32k_sq_counters.md")


def profile_field(path, key, prefix):
    """A value recorded in a committed counter summary (`prefix`_`key`: ...),
    or None when the summary is missing or the kernel sources it names have
    changed since the counters were taken (their SHA-256 is recorded)."""
    import hashlib
    try:
        text = open(path).read()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines()
                  if line.startswith(prefix + "_"))
    try:
        h = hashlib.sha256()
        for src in fields[prefix + "_sources"].split():
            h.update(open(os.path.join(ROOT, src), "rb").read())
        if h.hexdigest() != fields[prefix + "_sources_sha256"].strip():
            return None
        return fields[prefix + "_" + key].strip()
    except (KeyError, OSError, ValueError):
        return None


def measured_traffic():
    """HBM bytes per wf_verify_attn call from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy), or None when the
    summary is missing or the kernel sources changed since it was taken."""
    v = profile_field(TRAFFIC_PROFILE, "bytes_per_call", "traffic")
    return int(v) if v is not None else None


def measured_mfma_busy():
    """MFMA busy fraction of attn_partial_bf16 (SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE x SIMDs) from the committed counter summary, or None."""
    v = profile_field(MFMA_PROFILE, "attn_partial_mfma_busy", "sq")
    return float(v) if v is not None else None


def read_ceiling(wf, dev, mib, reps=3):
    """Best rate (GB/s) of the library's plain streaming-read probe over a
    `mib` MiB buffer, at a few grid sizes; each launch reads the whole
    buffer, which the 256 MB last-level cache cannot hold."""
    import torch
    buf = torch.ones(mib << 20, dtype=torch.uint8, device=dev)
    rates = {}
    for wgs in (256, 512, 1024, 2048):
        sink = torch.empty(wgs * 4096, dtype=torch.uint8, device=dev)
        wf.wf_read_probe(buf, sink, wgs)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            wf.wf_read_probe(buf, sink, wgs)
        e1.record()
        torch.cuda.synchronize()
        rates[wgs] = reps * buf.numel() / (e0.elapsed_time(e1) * 1e-3) / 1e9
        del sink
    del buf
    return max(rates.values()), rates


def size_matched_read_us(wf, dev, nbytes, total_mib=640, reps=5):
    """Per-call time (us) of the library's plain streaming read of `nbytes`,
    the reads launched back to back over consecutive pieces of a buffer that
    together exceed the 256 MB last-level cache: the best over a few grid
    sizes and load depths.  It is the time any kernel needs just to move
    that many bytes in one launch on this part (launch, first-byte latency
    and drain included)."""
    import torch
    n_bufs = max(1, -(-(total_mib << 20) // nbytes))
    buf = torch.ones(n_bufs * nbytes, dtype=torch.uint8, device=dev)
    best = None
    for wgs in (256, 512, 1024, 2048):
        sink = torch.empty(wgs * 4096, dtype=torch.uint8, device=dev)
        for depth in (4, 8):
            wf.wf_read_probe_series(buf, nbytes, n_bufs, 1, sink, wgs, depth)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            wf.wf_read_probe_series(buf, nbytes, n_bufs, reps, sink, wgs, depth)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / (reps * n_bufs)
            best = us if best is None else min(best, us)
        del sink
    del buf
    return best


def _vec_rel_err(got, ref):
    """max over output vectors (last axis) of ||got - ref||_inf / ||ref||_inf"""
    import numpy as np
    num = np.abs(got - ref).max(axis=-1)
    return float((num / np.maximum(np.abs(ref).max(axis=-1), 1e-30)).max())


def cpu_baseline(w, layers, head, budget_s, max_layers=None, tree_mask=None,
                 outs=None, lmouts=None, draft=None, tau=None):
    """The oracle as it stands, on host cores, over a bounded sample of the
    step: the LM head, then as many layers of attention and prefill as fit
    in about `budget_s` seconds (all of them if they fit); scaled to one
    full step.  With the step's GPU outputs (outs: attention per layer,
    lmouts: argmax / entropy / accept, the caches in `layers` holding the
    prefill's rows) it also compares them with the oracle's results of the
    same inputs -> (check, baseline)."""
    import numpy as np

    import oracle
    import workloads as W
    n = w.ctx_len + w.gamma
    h, wl = W.to_oracle(head["h"]), W.to_oracle(head["w_lm"])
    t0 = time.perf_counter()
    am_ref, ent_ref, margin = oracle.lmhead_rows(h, wl)
    t_lm = time.perf_counter() - t0
    del h, wl
    check = {}
    bar = 2e-2 if w.dtype == "bf16" else 1e-4
    amar = 1e-2 if w.dtype == "bf16" else 1e-6

    def lm_check(key, outs3, a_ref, e_ref, mg):
        am, ent, acc = (t.cpu().numpy() for t in outs3)
        sure = mg > amar
        check[key + "_argmax_mismatches"] = int((am[sure] != a_ref[sure]).sum())
        check[key + "_entropy_rel_err"] = float(
            (np.abs(ent - e_ref) / np.maximum(np.abs(e_ref), 1e-3)).max())
        if tree_mask is None and draft is not None and bool(sure.all()):
            n_ref, bonus_ref, route_ref, _ = oracle.accept(a_ref, e_ref, draft, tau)
            check[key + "_accept_matches"] = bool(
                (int(acc[0]), int(acc[1]), int(acc[2])) == (n_ref, bonus_ref, route_ref))

    if lmouts is not None:
        lm_check("lmhead", lmouts[0], am_ref, ent_ref, margin)
    if w.router_logits:
        z = head["router_logits"].cpu().numpy()
        t0 = time.perf_counter()
        a2, e2, m2 = oracle.lmhead_rows(logits=z)
        t_lm += time.perf_counter() - t0
        if lmouts is not None:
            lm_check("logits_only", lmouts[1], a2, e2, m2)
    log(f"cpu baseline: LM head {t_lm:.2f}s")
    t_attn = t_pre = 0.0
    done = 0
    limit = w.n_layers if max_layers is None else min(max_layers, w.n_layers)
    while done < limit:
        t = layers[done]
        q = W.to_oracle(t["q"])
        k = W.to_oracle(t["k_cache"][:, :n].contiguous())
        v = W.to_oracle(t["v_cache"][:, :n].contiguous())
        t0 = time.perf_counter()
        if tree_mask is None:
            o_ref = oracle.verify_attn(q, k, v, w.ctx_len)
        else:
            o_ref = oracle.verify_attn_mask(q, k, v, w.ctx_len, tree_mask)
        t_attn += time.perf_counter() - t0
        del q, k, v
        if outs is not None:
            e = _vec_rel_err(outs[done].float().cpu().numpy().astype(np.float64), o_ref)
            check["attention_max_rel_err"] = max(check.get("attention_max_rel_err", 0.0), e)
        if w.n_prefill:
            x, wk, wv = (W.to_oracle(t[k_]) for k_ in ("x", "w_k", "w_v"))
            t0 = time.perf_counter()
            k_ref, v_ref = oracle.kv_only_prefill(x, wk, wv, w.prefill_start, w.n_kv_heads,
                                                  w.head_dim, w.rope_base)
            t_pre += time.perf_counter() - t0
            if outs is not None:
                kc = t["drafter_k_cache"] if w.separate_drafter_cache else t["k_cache"]
                vc = t["drafter_v_cache"] if w.separate_drafter_cache else t["v_cache"]
                rows = slice(w.prefill_start, w.prefill_start + w.n_prefill)
                e = max(_vec_rel_err(kc[:, rows].float().cpu().numpy().astype(np.float64), k_ref),
                        _vec_rel_err(vc[:, rows].float().cpu().numpy().astype(np.float64), v_ref))
                check["prefill_max_rel_err"] = max(check.get("prefill_max_rel_err", 0.0), e)
        done += 1
        spent = t_lm + t_attn + t_pre
        log(f"cpu baseline: layer {done - 1} done ({spent:.1f}s)")
        if spent + (t_attn + t_pre) / done > budget_s:
            break
    per_step_s = (t_attn + t_pre) / done * w.n_layers + t_lm
    whole = done == w.n_layers
    if check:
        check["layers_checked"] = done
        check["tolerance"] = bar
        check["ok"] = bool(
            check.get("attention_max_rel_err", 0.0) <= bar
            and check.get("prefill_max_rel_err", 0.0) <= bar
            and all(v == 0 for k_, v in check.items() if k_.endswith("_mismatches"))
            and all(v for k_, v in check.items() if k_.endswith("_accept_matches"))
            and all(v <= bar for k_, v in check.items() if k_.endswith("_entropy_rel_err")))
        log("oracle check of the step's outputs: " + json.dumps(check))
    return check or None, {
        "value": round(per_step_s * 1e6, 1),
        "unit": "us",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": ("the whole step: " if whole else
                   f"{done} of {w.n_layers} layers, scaled to one step: ")
                  + f"{'tree ' if tree_mask is not None else ''}attention over all "
                    f"{w.gamma * w.n_q_heads} rows x heads"
                  + (", KV-only prefill" if w.n_prefill else "")
                  + ", full LM head",
        "measured_s": round(t_attn + t_pre + t_lm, 2),
    }


def _time_calls(torch, fn, steps, warmup):
    """Average ms of fn() over `steps` back-to-back calls on the current
    stream, after `warmup` untimed ones."""
    for _ in range(warmup):
        fn()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def bench_switch(args, w):
    """The drafter side of a switch: lazy catch-up of a one-layer drafter's
    cache over the backlog (KV-only prefill of all backlog tokens but the
    last, the full layer for the last).  One step = one catch-up."""
    import dataclasses

    import numpy as np
    import torch

    import paper_2606_07710_amd as wf
    import workloads as W

    dev = "cuda:0"
    bases = (512, 1024, 2048, 4096, 8192, 16384) if args.switch_table else ()
    backlogs = (1, 64, 128, 512, 1024) if args.switch_table else ()
    max_rows = max((w.ctx_len,) + bases) + max((w.n_prefill,) + backlogs)
    t0 = time.perf_counter()
    big = dataclasses.replace(w, n_prefill=max(w.n_prefill, *backlogs) if backlogs
                              else w.n_prefill)
    t = W.generate_drafter(big, device=dev, cache_rows=max_rows - big.n_prefill)
    tiled = not args.row_major_weights
    # static weights: the projections tiled once at setup, as at model load
    lw = {n: (t[n] if n.endswith("norm") or not tiled else wf.tile_weights(t[n]))
          for n in W.DECODER_WEIGHTS}
    layer = wf.decoder_layer(lw, w.n_q_heads, w.n_kv_heads, w.rms_eps, w.rope_base)
    kc, vc, r_all = t["k_cache"], t["v_cache"], t["r"]
    torch.cuda.synchronize()
    log(f"inputs generated in {time.perf_counter() - t0:.1f}s "
        f"(drafter weights {w.drafter_weight_bytes() / 2**20:.0f} MiB)")
    ws = wf.alloc_workspace(max(
        wf.wf_drafter_catchup_workspace_bytes(layer, n, b)
        for n in (w.n_prefill,) + backlogs for b in (w.ctx_len,) + bases), dev)
    fws = wf.alloc_workspace(max(
        [wf.wf_drafter_forward_workspace_bytes(layer, n, b)
         for n in (1, 64) for b in (w.ctx_len,) + bases]), dev)
    pws = wf.alloc_workspace(wf.wf_kv_only_prefill_workspace_bytes(
        1, 64, w.hidden, w.n_kv_heads, w.head_dim), dev)
    out = torch.empty(w.hidden, dtype=torch.bfloat16, device=dev)
    fout = torch.empty((64, w.hidden), dtype=torch.bfloat16, device=dev)

    def catchup(n, pos):
        return lambda: wf.wf_drafter_catchup(layer, r_all[:n], pos, kc, vc, out,
                                             workspace=ws)

    n, pos = w.n_prefill, w.ctx_len
    catchup(n, pos)()
    torch.cuda.synchronize()
    ms = _time_calls(torch, catchup(n, pos), args.steps, args.warmup)
    by = w.catchup_bytes(n, pos)
    gbps = by / (ms * 1e-3) / 1e9
    log(f"catch-up of {n} tokens at base KV {pos}: {ms * 1e3:.1f} us "
        f"({gbps:.0f} GB/s of algorithmic bytes)")

    table = None
    if args.switch_table:
        table = {"base_kv": list(bases), "backlog": list(backlogs),
                 "lazy_catchup_us": [], "kv_only_vs_full_layer": [],
                 "lazy_vs_per_round": []}
        for b in bases:
            row = []
            for nb in backlogs:
                row.append(round(_time_calls(torch, catchup(nb, b), args.steps,
                                             args.warmup) * 1e3, 1))
            table["lazy_catchup_us"].append(row)
            log(f"base KV {b}: " + ", ".join(f"{nb}: {u} us" for nb, u in
                                             zip(backlogs, row)))
        # KV-only catch-up vs the full layer on every backlog token (one
        # forward call; the forward takes at most 64 tokens)
        for nb in (1, 16, 32, 64):
            lazy = _time_calls(torch, catchup(nb, pos), args.steps, args.warmup)
            full = _time_calls(torch, lambda: wf.wf_drafter_forward(
                layer, r_all[:nb], pos, kc, vc, fout[:nb], workspace=fws),
                args.steps, args.warmup)
            table["kv_only_vs_full_layer"].append(
                {"backlog": nb, "base_kv": pos, "kv_only_us": round(lazy * 1e3, 1),
                 "full_layer_us": round(full * 1e3, 1),
                 "saving": round(1.0 - lazy / full, 3)})
            log(f"backlog {nb}: KV-only {lazy * 1e3:.1f} us, full layer "
                f"{full * 1e3:.1f} us")
        # one batched catch-up vs keeping the cache current every round
        # (KV-only prefill of each round's tokens, the last token in full at
        # the switch), same tokens
        for per_round, rounds in ((4, 20), (8, 10), (2, 40)):
            nb = per_round * rounds

            def naive(per_round=per_round, rounds=rounds, nb=nb):
                for k in range(rounds - 1):
                    wf.wf_kv_only_prefill(r_all[k * per_round:(k + 1) * per_round],
                                          lw["w_k"], lw["w_v"], kc, vc,
                                          pos + k * per_round, w.rope_base,
                                          workspace=pws)
                wf.wf_drafter_catchup(layer, r_all[nb - per_round:nb],
                                      pos + nb - per_round, kc, vc, out, workspace=ws)
            lazy = _time_calls(torch, catchup(nb, pos), args.steps, args.warmup)
            per = _time_calls(torch, naive, args.steps, args.warmup)
            table["lazy_vs_per_round"].append(
                {"tokens": nb, "rounds": rounds, "lazy_us": round(lazy * 1e3, 1),
                 "per_round_us": round(per * 1e3, 1)})
            log(f"{nb} tokens: lazy {lazy * 1e3:.1f} us, per round over {rounds} "
                f"rounds {per * 1e3:.1f} us")

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        host = {k: W.to_oracle(t[k]) for k in W.DECODER_WEIGHTS}
        rh = W.to_oracle(r_all[:n])
        kh = W.to_oracle(kc[:, :pos + n].contiguous())
        vh = W.to_oracle(vc[:, :pos + n].contiguous())
        t0 = time.perf_counter()
        oracle.catchup(rh, pos, host, kh, vh, w.n_q_heads, w.n_kv_heads,
                       w.rms_eps, w.rope_base)
        cs = time.perf_counter() - t0
        cpu = {"value": round(cs * 1e6, 1), "unit": "us",
               "cores": oracle.num_threads(), "kind": "oracle",
               "sample": f"one whole catch-up ({n} backlog tokens, base KV {pos})",
               "measured_s": round(cs, 2)}

    line = {
        "metric": f"drafter switch catch-up us (8B-shape drafter layer, base KV "
                  f"{pos}, backlog {n}, 1 GPU)",
        "value": round(ms * 1e3, 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded; one drafter layer with the 8B attention "
                "shapes and a 12288-wide SwiGLU MLP, random weights)",
        "config": {"workload": w.name, "hidden": w.hidden, "q_heads": w.n_q_heads,
                   "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "inter": w.inter, "base_kv": pos, "backlog": n,
                   "weights": "tiled (16x32 tiles, made once at setup)" if tiled
                              else "row-major"},
        "roofline": {
            "kernel": "wf_drafter_catchup, whole call (rmsnorm, KV-only "
                      "prefill, then the full layer for the last token)",
            "bound": "hbm",
            "achieved": round(gbps, 1),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(gbps / PEAK_HBM_GBPS, 4),
            "traffic": None,
            "bytes_per_launch": by,
            "avg_launch_us": round(ms * 1e3, 2),
        },
        "cpu_baseline": cpu,
    } | ({"switch_table": table} if table else {})
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the verification step is built "
              "and timed on a single MI355X (no multi-GPU path exists); run "
              "with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_07710_amd as wf
    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    w = W.CONFIGS[args.config]
    log(f"workload {w.name}: {w.description}")
    if w.inter:
        return bench_switch(args, w)

    t0 = time.perf_counter()
    layers = [W.generate_layer(w, l, device=dev) for l in range(w.n_layers)]
    head = W.generate_head(w, device=dev)
    tree = None
    if w.is_tree:
        # one [layers][heads][cap][D] cache per K and V, so the path
        # compaction covers every layer in one call
        tree = {"k_all": torch.stack([t.pop("k_cache") for t in layers]),
                "v_all": torch.stack([t.pop("v_cache") for t in layers])}
        for l, t in enumerate(layers):
            t["k_cache"], t["v_cache"] = tree["k_all"][l], tree["v_all"][l]
        par = W.draft_tree(seed=W.stream_seed(W.master_seed(w.cfg), "tree"))
        tree["parents_np"] = par
        tree["parents"] = torch.from_numpy(par).to(dev)
        tree["mask"] = torch.from_numpy(
            W.ancestor_masks(par).view(np.int64).copy()).to(dev)
        tree["path"] = torch.empty(w.gamma, dtype=torch.int32, device=dev)
    pre_stack = None
    if w.n_prefill and w.n_layers > 1 and args.batch_prefill_layers:
        # the layers' catch-up inputs, weights and caches as dense [L][...]
        # stacks (per-layer views into them), so one call covers all layers
        ck, cv = (("drafter_k_cache", "drafter_v_cache") if w.separate_drafter_cache
                  else ("k_cache", "v_cache"))
        pre_stack = {}
        for key, name in (("x", "x"), ("w_k", "w_k"), ("w_v", "w_v"), ("k", ck), ("v", cv)):
            st = torch.stack([t.pop(name) for t in layers])
            for l, t in enumerate(layers):
                t[name] = st[l]
            pre_stack[key] = st
            torch.cuda.empty_cache()
    tiled = w.dtype == "bf16" and not args.row_major_weights
    if pre_stack is not None and tiled:
        # static weights: tiled once at setup, as at model load
        pre_stack["w_k"] = wf.tile_weights(pre_stack["w_k"])
        pre_stack["w_v"] = wf.tile_weights(pre_stack["w_v"])
    elif w.n_prefill and tiled:
        for t in layers:
            t["w_k_tiled"] = wf.tile_weights(t["w_k"])
            t["w_v_tiled"] = wf.tile_weights(t["w_v"])
    w_lm_tiled = wf.tile_weights(head["w_lm"]) if tiled else None
    torch.cuda.synchronize()
    log(f"inputs generated in {time.perf_counter() - t0:.1f}s")

    outs = [torch.empty_like(t["q"]) for t in layers]
    ws_attn = wf.alloc_workspace(
        wf.wf_verify_attn_workspace_bytes(1 if w.dtype == "bf16" else 0,
                                          w.gamma, w.ctx_len, w.n_q_heads,
                                          w.n_kv_heads, w.head_dim), dev)
    ws_pre = wf.alloc_workspace(
        wf.wf_kv_only_prefill_layers_workspace_bytes(
            1 if w.dtype == "bf16" else 0, w.n_prefill, w.hidden, w.n_kv_heads,
            w.head_dim, w.n_layers if pre_stack else 1), dev)
    ws_lm = wf.alloc_workspace(wf.wf_lmhead_workspace_bytes(w.gamma, w.vocab), dev)
    lmouts = [(torch.empty(w.gamma, dtype=torch.int32, device=dev),
               torch.empty(w.gamma, dtype=torch.float32, device=dev),
               torch.empty(4 if tree else 3, dtype=torch.int32, device=dev))
              for _ in range(2)]

    # drafts: the workload's accept prefix, built from this GPU's own argmax
    # (the timed work does not depend on draft content)
    am, ent, acc = lmouts[0]
    wf.wf_lmhead_accept_entropy(head["h"], head["w_lm"], None,
                                torch.zeros(max(w.gamma - 1, 1), dtype=torch.int32,
                                            device=dev),
                                0.0, am, ent, acc, workspace=ws_lm)
    torch.cuda.synchronize()
    k = W.prefix_len(w, 0)
    if tree:
        # node tokens: the accepted root path has min(k, its depth) drafts
        draft = torch.as_tensor(W.tree_tokens(am.cpu().numpy(), tree["parents_np"],
                                              k, w.vocab, 1), device=dev)
    else:
        draft = torch.as_tensor(W.make_drafts(am.cpu().numpy(), k, w.vocab, 1),
                                device=dev)
    tau = float(np.median(ent.cpu().numpy()))

    router = None
    if args.router == "neural":
        router = W.generate_router(w, device=dev)
        m = router["w1"].shape[0]
        router["delta"] = torch.empty(w.gamma, dtype=torch.float32, device=dev)
        router["route"] = torch.empty(1, dtype=torch.int32, device=dev)
        router["ws"] = wf.alloc_workspace(int(wf.lib.wf_router_workspace_bytes(
            1 if w.dtype == "bf16" else 0, w.gamma, w.hidden, m)), dev)
        if not tree:
            # chain/block rounds: the router rides in the LM-head call, its
            # W1 in the LM head's layout
            if w_lm_tiled is not None:
                router["w1_tiled"] = wf.tile_weights(router["w1"])
            code = (wf.WF_BF16_TILED if w_lm_tiled is not None else
                    wf.WF_BF16 if w.dtype == "bf16" else wf.WF_F32)
            ws_lm = wf.alloc_workspace(int(wf.lib.wf_lmhead_route_neural_workspace_bytes(
                code, w.gamma, w.vocab, w.hidden, m)), dev)
    step = Step(w, layers, head, outs, lmouts, draft, tau, ws_attn, ws_pre,
                ws_lm, wf, tree, router, pre_stack, w_lm_tiled)
    stream = torch.cuda.current_stream()
    catchup = torch.cuda.Stream() if args.overlap else None
    step.build(stream, catchup)
    step.run(check=True)
    torch.cuda.synchronize()
    log(f"step ok: accept {tuple(acc.tolist())} (expected n = {k})")

    graph = None
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        with torch.cuda.stream(side):
            step.build(side, catchup)
            step.run(check=True)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            step.build(torch.cuda.current_stream(), catchup)
            step.run(check=True)
        step.build(stream, catchup)
        torch.cuda.synchronize()

    def one_step():
        if graph is not None:
            graph.replay()
        else:
            step.run()

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    log("warmup done")

    # ---- timed region 1: the step ------------------------------------------
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        one_step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = e0.elapsed_time(e1) / args.steps
    log(f"timed {args.steps} steps: {ms_per_step * 1e3:.1f} us/step "
        f"(host wall {wall / args.steps * 1e6:.1f} us/step)")

    # the spread of single steps (a second run of K steps, an event between
    # consecutive steps; not part of `value`)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    for i in range(args.steps):
        one_step()
        evs[i + 1].record()
    torch.cuda.synchronize()
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    spread = {q: round(float(np.percentile(per_step, p)) * 1e3, 1)
              for q, p in (("p10", 10), ("median", 50), ("p90", 90))}
    log(f"single steps (us): {spread}")

    # ---- timed region 2: each phase alone, calls back to back --------------
    # Events bracket only whole runs of one kind of call, so a per-call
    # average includes no event overhead and matches what a kernel trace
    # reports for the kernels of that call.
    # (on the stream each phase's calls are marshalled for)
    per_call_ms = {}
    for name, fn, calls, st in step.phases():
        if not calls:
            per_call_ms[name] = 0.0
            continue
        for a in calls:                       # warm this phase alone
            fn(*a)
        a_ev = torch.cuda.Event(enable_timing=True)
        b_ev = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a_ev.record(st)
        for _ in range(args.steps):
            for a in calls:
                fn(*a)
        b_ev.record(st)
        torch.cuda.synchronize()
        per_call_ms[name] = a_ev.elapsed_time(b_ev) / (args.steps * len(calls))
    attn_avg_ms = per_call_ms["attention"]
    breakdown = {name: round(per_call_ms[name] * len(calls) * 1e3, 1)
                 for name, _, calls, _ in step.phases()}
    log(f"per call (us): " + ", ".join(f"{k} {v * 1e3:.2f}"
                                       for k, v in per_call_ms.items()))

    by = w.algorithmic_bytes()
    if router is not None:
        # the router reads its weights and the verify rows' hidden states
        m = router["w1"].shape[0]
        by["router"] = (m * w.hidden + 2 * m + 1 + w.gamma * w.hidden) * w.elem_bytes
        by["total"] += by["router"]
    achieved = by["attn_per_layer"] / (attn_avg_ms * 1e-3) / 1e9
    step_gbps = by["total"] / (ms_per_step * 1e-3) / 1e9

    # ---- plain copy for the HBM traffic counters (not timed) ---------------
    copy_gbps = None
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        # the same copy timed: a plain-streaming reference for the roofline
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(4):
            dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        copy_gbps = 4 * 2 * n / (c0.elapsed_time(c1) * 1e-3) / 1e9
        log(f"device copy: {copy_gbps:.0f} GB/s (read + write; counter reference only)")
        del src, dst

    # ---- streaming-read ceiling (not timed with the step) -------------------
    ceiling = None
    if args.read_probe_mib:
        ceiling, rates = read_ceiling(wf, dev, args.read_probe_mib)
        log("read ceiling: " + ", ".join(f"{k} WGs {v:.0f}" for k, v in rates.items())
            + f" GB/s -> {ceiling:.0f}")

    # ---- size-matched read floors (not timed with the step) -----------------
    # a plain read of each kernel's bytes, one launch per call: what the
    # step would take if every launch only streamed its bytes
    floors = None
    if args.read_probe_mib and by["attn_per_layer"] >= (16 << 20):
        floors = {"attention": size_matched_read_us(wf, dev, by["attn_per_layer"]),
                  "lmhead": size_matched_read_us(wf, dev, by["lmhead"])}
        if by["prefill_per_layer"]:
            floors["prefill"] = size_matched_read_us(wf, dev, by["prefill_per_layer"])
        floors["step"] = (w.n_layers * (floors["attention"] + floors.get("prefill", 0.0))
                          + floors["lmhead"])
        floors = {k: round(v, 2) for k, v in floors.items()}
        log("size-matched plain reads (us per launch): "
            + ", ".join(f"{k} {v:.2f}" for k, v in floors.items()))

    cpu = check = None
    if not args.no_cpu_baseline:
        log(f"cpu baseline: about {args.cpu_budget_s:.0f}s of oracle work ...")
        check, cpu = cpu_baseline(w, layers, head, args.cpu_budget_s,
                                  args.cpu_sample_layers,
                                  W.ancestor_masks(tree["parents_np"]) if tree else None,
                                  outs=outs, lmouts=lmouts, draft=draft.cpu().numpy(),
                                  tau=tau)

    line = {
        "metric": "verify-step us and achieved HBM GB/s (gamma=16, 32K ctx, "
                  "8B shapes, 1 GPU)" if w.cfg == 3 else
                  f"verify-step us and achieved HBM GB/s ({w.name}, 1 GPU)",
        "value": round(ms_per_step * 1e3, 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded; shapes of the paper's Qwen3-8B-class "
                "targets, random inputs)",
        "config": {"workload": w.name, "layers": w.n_layers,
                   "hidden": w.hidden, "q_heads": w.n_q_heads,
                   "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "ctx_len": w.ctx_len, "gamma": w.gamma,
                   "catch_up_tokens": w.n_prefill, "vocab": w.vocab,
                   "graph": bool(graph is not None),
                   "schedule": "one stream, model order" if catchup is None else
                               "catch-up prefill on a second stream",
                   "prefill": "one call for all layers (upper bound)"
                              if step.pre_stack is not None else "one call per layer",
                   "weights": "tiled (16x32 tiles, made once at setup)"
                              if w_lm_tiled is not None else "row-major"}
                  | {"router": args.router}
                  | ({"draft_tree": {"nodes": w.gamma - 1,
                                     "depth": len(w.tree_levels),
                                     "nodes_per_depth": list(w.tree_levels)}}
                     if tree else {}),
        "step_hbm_gbps": round(step_gbps, 1),
        "step_us_spread": spread,
        # catch-up prefill / step: the analog of the paper's switching cost
        "prefill_share": round(breakdown.get("prefill", 0.0) / (ms_per_step * 1e3), 4),
        "step_algorithmic_bytes": by["total"],
        "breakdown_us": breakdown,   # each phase run alone, back to back
        # a plain read of each launch's algorithmic bytes, one launch per
        # call, back to back (the step row: all of the step's launches)
        "size_matched_read_us": floors,
        "step_frac_of_size_matched": round(floors["step"] / (ms_per_step * 1e3), 4)
                                     if floors else None,
        "roofline": {
            "kernel": ("wf_verify_attn_tree" if tree else "wf_verify_attn")
                      + ", one layer (attn_partial_bf16 + attn_merge)",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": measured_traffic() if w.cfg == 3 else None,
            "bytes_per_launch": by["attn_per_layer"],
            "avg_launch_us": round(attn_avg_ms * 1e3, 2),
            # the best rate of a plain streaming read over a buffer larger
            # than the last-level cache, measured in this run
            "read_ceiling_gbps": round(ceiling, 1) if ceiling else None,
            "frac_of_read_ceiling": round(achieved / ceiling, 4) if ceiling else None,
            # a plain read of the launch's bytes on its own over the call time
            "frac_of_size_matched_read": round(floors["attention"] / (attn_avg_ms * 1e3), 4)
                                         if floors else None,
            # secondary, derived (not a counter): the call's flops over its
            # time, against the dense bf16 MFMA peak
            "mfma_util_from_flops": round(w.flops()["attn_per_layer"] / (attn_avg_ms * 1e-3)
                                          / PEAK_BF16_FLOPS, 4),
            # counter-based: MFMA busy cycles of attn_partial_bf16 over its
            # active cycles x SIMDs (committed rocprofv3 summary; None when
            # the kernel sources changed since it was taken)
            "mfma_busy_counter": measured_mfma_busy() if w.cfg == 3 else None,
        },
        "cpu_baseline": cpu,
        # the timed step's own outputs against the oracle's for the same
        # inputs (the layers the baseline's time budget covered)
        "oracle_check": check,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
