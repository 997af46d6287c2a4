"""CPU oracle for the WhiFlash target-verification step (fp64, plain loops).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the GPU library (paper_2606_07710_amd).

The arithmetic lives in wfref.c; this module only marshals numpy arrays.
Storage codes: float32 arrays -> fp32, uint16 arrays -> bf16 bit patterns,
float64 arrays -> fp64.  Every result is fp64.

Paper: arXiv 2606.07710 (WhiFlash).  What each call computes:
  verify_attn      -- Sec. 3.2 parallel verification of the drafted block:
                      block-causal grouped-query softmax attention against
                      the KV cache.
  kv_only_prefill  -- Sec. 3.4 "KV-only Prefill": K/V projection, RoPE on K.
  lmhead_rows      -- Sec. 3.3.1: next-token logits, argmax and the entropy
                      H = -sum p log p of the softmax distribution.
  accept           -- greedy acceptance of the longest matching draft prefix
                      plus the Sec. 3.3.1 entropy routing rule (H > tau -> AR).
  verify_attn_mask -- tree verification (Sec. 3.1 draft trees, Sec. 3.2
                      parallel verification): row i sees the cache, itself
                      and the block rows its mask bits name.
  accept_tree      -- greedy acceptance of the deepest accepted tree node
                      and its root path, plus the same entropy route.
  kv_compact_path  -- after tree acceptance, the accepted path's K/V rows
                      move to consecutive cache rows after the prefix.
  router_mlp       -- the neural routing policy (Sec. 3.3.2 and its
                      appendix): delta = w2 . GELU(W1 h + b1) + b2 per row;
                      route = delta > tau_neural.
  decoder_forward  -- one full drafter layer (attention + SwiGLU MLP) for
                      tokens against a cache: what lazy catch-up (Sec. 3.4)
                      still runs for the last backlog token.
  catchup          -- lazy catch-up of a drafter's cache: KV-only prefill of
                      the backlog but its last token, which runs the full
                      layer.
  layer_forward    -- a full single attention layer, used to pin that KV-only
                      prefill yields the cache a full forward would.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# WFREF_LIB names another build of wfref.c (the sanitizer run of the tests)
_LIB_PATH = os.environ.get("WFREF_LIB") or os.path.join(_HERE, "libwfref.so")
_lib = None

_CODES = {np.dtype(np.float32): 0, np.dtype(np.uint16): 1,
          np.dtype(np.float64): 2}

_p = ctypes.c_void_p
_i = ctypes.c_int
_d = ctypes.c_double


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.wfref_num_threads.restype = _i
    lib.wfref_verify_attn.argtypes = [_i, _p, _p, _p, _p, _i, _i, _i, _i, _i,
                                      _i, _d]
    lib.wfref_verify_attn_rows.argtypes = [_i, _p, _p, _p, _p, _i, _i, _i, _i,
                                           _i, _i, _d, _i, _p]
    lib.wfref_kv_only_prefill.argtypes = [_i, _p, _p, _p, _p, _p, _i, _i, _i,
                                          _i, _i, _d]
    lib.wfref_lmhead_rows.argtypes = [_i, _p, _p, _p, _i, _i, _i, _p, _p, _p,
                                      _p]
    lib.wfref_accept.argtypes = [_p, _p, _p, _i, _d, _p, _p]
    lib.wfref_verify_attn_mask.argtypes = [_i, _p, _p, _p, _p, _p, _i, _i, _i,
                                           _i, _i, _i, _d]
    lib.wfref_accept_tree.argtypes = [_p, _p, _p, _p, _i, _d, _p, _p, _p]
    lib.wfref_router_mlp.argtypes = [_i, _p, _p, _p, _p, _p, _i, _i, _i, _p]
    lib.wfref_rmsnorm.argtypes = [_i, _p, _p, _i, _i, _d, _p]
    lib.wfref_decoder_forward.argtypes = [_i, _p, _i, _i] + [_p] * 9 + [_i] * 5 + \
        [_d, _d, _p, _p, _i, _p]
    lib.wfref_rope_inplace.argtypes = [_p, _i, _d, _d]
    lib.wfref_rope_inplace.restype = None
    lib.wfref_layer_forward.argtypes = [_i, _p, _p, _p, _p, _p, _i, _i, _i, _i,
                                        _i, _i, _d, _d, _p, _p, _p, _p, _p]
    for name in ("wfref_verify_attn", "wfref_verify_attn_rows",
                 "wfref_kv_only_prefill", "wfref_lmhead_rows", "wfref_accept",
                 "wfref_verify_attn_mask", "wfref_accept_tree",
                 "wfref_router_mlp", "wfref_rmsnorm", "wfref_decoder_forward",
                 "wfref_layer_forward"):
        getattr(lib, name).restype = _i
    _lib = lib
    return lib


def _arr(a):
    a = np.ascontiguousarray(a)
    if a.dtype not in _CODES:
        raise TypeError(f"oracle input dtype {a.dtype} not supported")
    return a, _CODES[a.dtype]


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


def num_threads() -> int:
    return int(_load().wfref_num_threads())


def verify_attn(q, k_cache, v_cache, ctx_len, scale=None):
    """q [gamma][Hq][D]; caches [Hkv][cap][D] (same storage); -> fp64 out."""
    lib = _load()
    q, code = _arr(q)
    k_cache, c2 = _arr(k_cache)
    v_cache, c3 = _arr(v_cache)
    if not (code == c2 == c3):
        raise TypeError("q and caches must share a storage type")
    gamma, hq, dh = q.shape
    hkv, cap, dh2 = k_cache.shape
    if dh2 != dh or v_cache.shape != k_cache.shape:
        raise ValueError("shape mismatch")
    if scale is None:
        scale = 1.0 / np.sqrt(dh)
    out = np.empty((gamma, hq, dh), np.float64)
    rc = lib.wfref_verify_attn(code, _ptr(q), _ptr(k_cache), _ptr(v_cache),
                               _ptr(out), gamma, int(ctx_len), cap, hq, hkv,
                               dh, float(scale))
    _check(rc, "verify_attn")
    return out


def verify_attn_rows(q, k_cache, v_cache, ctx_len, rows_heads, scale=None):
    """Attention output at the listed (block row, q head) pairs only."""
    lib = _load()
    q, code = _arr(q)
    k_cache, _ = _arr(k_cache)
    v_cache, _ = _arr(v_cache)
    gamma, hq, dh = q.shape
    hkv, cap, _ = k_cache.shape
    rh = np.ascontiguousarray(np.asarray(rows_heads, np.int32).reshape(-1, 2))
    if scale is None:
        scale = 1.0 / np.sqrt(dh)
    out = np.empty((rh.shape[0], dh), np.float64)
    rc = lib.wfref_verify_attn_rows(code, _ptr(q), _ptr(k_cache),
                                    _ptr(v_cache), _ptr(out), gamma,
                                    int(ctx_len), cap, hq, hkv, dh,
                                    float(scale), rh.shape[0], _ptr(rh))
    _check(rc, "verify_attn_rows")
    return out


def kv_only_prefill(x, w_k, w_v, start_pos, n_kv_heads, head_dim, rope_base):
    """x [n][d_in]; w_k, w_v [Hkv*D][d_in] -> (K, V) each [Hkv][n][D] fp64."""
    lib = _load()
    x, code = _arr(x)
    w_k, _ = _arr(w_k)
    w_v, _ = _arr(w_v)
    n_tok, d_in = x.shape
    k = np.empty((n_kv_heads, n_tok, head_dim), np.float64)
    v = np.empty_like(k)
    rc = lib.wfref_kv_only_prefill(code, _ptr(x), _ptr(w_k), _ptr(w_v),
                                   _ptr(k), _ptr(v), n_tok, int(start_pos),
                                   d_in, n_kv_heads, head_dim,
                                   float(rope_base))
    _check(rc, "kv_only_prefill")
    return k, v


def lmhead_rows(h=None, w=None, logits=None, want_logits=False):
    """Per-row argmax (int32), entropy (nats), top-2 margin, optional logits.

    Either (h [gamma][d], w [vocab][d]) or logits [gamma][vocab] float32.
    """
    lib = _load()
    if logits is not None:
        logits = np.ascontiguousarray(logits, np.float32)
        gamma, vocab = logits.shape
        d, code = 0, 0
        hp = wp = None
    else:
        h, code = _arr(h)
        w, c2 = _arr(w)
        if code != c2:
            raise TypeError("h and w must share a storage type")
        gamma, d = h.shape
        vocab = w.shape[0]
        hp, wp = h, w
    am = np.empty(gamma, np.int32)
    ent = np.empty(gamma, np.float64)
    margin = np.empty(gamma, np.float64)
    z = np.empty((gamma, vocab), np.float64) if want_logits else None
    rc = lib.wfref_lmhead_rows(code, _ptr(hp), _ptr(wp), _ptr(logits), gamma,
                               d, vocab, _ptr(am), _ptr(ent), _ptr(margin),
                               _ptr(z))
    _check(rc, "lmhead_rows")
    if want_logits:
        return am, ent, margin, z
    return am, ent, margin


def accept(argmax, entropy, draft, tau):
    """-> (n_accepted, bonus, route, H_t)."""
    lib = _load()
    argmax = np.ascontiguousarray(argmax, np.int32)
    entropy = np.ascontiguousarray(entropy, np.float64)
    gamma = argmax.shape[0]
    dr = np.ascontiguousarray(draft, np.int32) if gamma > 1 else None
    if dr is not None and dr.shape[0] != gamma - 1:
        raise ValueError("draft must hold gamma-1 tokens")
    out3 = np.empty(3, np.int32)
    ht = ctypes.c_double()
    rc = lib.wfref_accept(_ptr(argmax), _ptr(entropy), _ptr(dr), gamma,
                          float(tau), _ptr(out3), ctypes.byref(ht))
    _check(rc, "accept")
    return int(out3[0]), int(out3[1]), int(out3[2]), float(ht.value)


def verify_attn_mask(q, k_cache, v_cache, ctx_len, mask, scale=None):
    """Tree verification attention: mask [gamma] uint64, bit j of mask[i]
    lets row i see block row j (it always sees itself) -> fp64 out."""
    lib = _load()
    q, code = _arr(q)
    k_cache, c2 = _arr(k_cache)
    v_cache, c3 = _arr(v_cache)
    if not (code == c2 == c3):
        raise TypeError("q and caches must share a storage type")
    gamma, hq, dh = q.shape
    hkv, cap, dh2 = k_cache.shape
    if dh2 != dh or v_cache.shape != k_cache.shape:
        raise ValueError("shape mismatch")
    m = np.ascontiguousarray(np.asarray(mask, np.uint64))
    if m.shape != (gamma,):
        raise ValueError("mask must hold gamma words")
    if scale is None:
        scale = 1.0 / np.sqrt(dh)
    out = np.empty((gamma, hq, dh), np.float64)
    rc = lib.wfref_verify_attn_mask(code, _ptr(q), _ptr(k_cache),
                                    _ptr(v_cache), _ptr(out), _ptr(m), gamma,
                                    int(ctx_len), cap, hq, hkv, dh,
                                    float(scale))
    _check(rc, "verify_attn_mask")
    return out


def accept_tree(argmax, entropy, tokens, parents, tau):
    """-> (n, bonus, route, deepest node, H_t, path [gamma] int32)."""
    lib = _load()
    argmax = np.ascontiguousarray(argmax, np.int32)
    entropy = np.ascontiguousarray(entropy, np.float64)
    gamma = argmax.shape[0]
    tok = np.ascontiguousarray(tokens, np.int32)
    par = np.ascontiguousarray(parents, np.int32)
    if tok.shape != (gamma,) or par.shape != (gamma,):
        raise ValueError("tokens and parents must hold gamma entries")
    out4 = np.empty(4, np.int32)
    path = np.empty(gamma, np.int32)
    ht = ctypes.c_double()
    rc = lib.wfref_accept_tree(_ptr(argmax), _ptr(entropy), _ptr(tok),
                               _ptr(par), gamma, float(tau), _ptr(out4),
                               _ptr(path), ctypes.byref(ht))
    _check(rc, "accept_tree")
    return (int(out4[0]), int(out4[1]), int(out4[2]), int(out4[3]),
            float(ht.value), path)


def kv_compact_path(k_cache, v_cache, ctx_len, path, n):
    """Caches [Hkv][cap][D]: block row path[t] (cache row ctx_len + path[t])
    moves to block row t for t = 0..n; every other row is unchanged.
    Returns new arrays."""
    k = np.array(k_cache, copy=True)
    v = np.array(v_cache, copy=True)
    src = [ctx_len + int(path[t]) for t in range(n + 1)]
    dst = [ctx_len + t for t in range(n + 1)]
    k[:, dst] = np.asarray(k_cache)[:, src]
    v[:, dst] = np.asarray(v_cache)[:, src]
    return k, v


def router_mlp(h, w1, b1, w2, b2):
    """h [gamma][d]; w1 [m][d]; b1, w2 [m]; b2 [1] (one storage type)
    -> delta [gamma] fp64."""
    lib = _load()
    h, code = _arr(h)
    arrs = []
    for a in (w1, b1, w2, b2):
        a, c = _arr(a)
        if c != code:
            raise TypeError("router inputs must share a storage type")
        arrs.append(a)
    w1, b1, w2, b2 = arrs
    gamma, d = h.shape
    m = w1.shape[0]
    if w1.shape != (m, d) or b1.shape != (m,) or w2.shape != (m,) or b2.shape != (1,):
        raise ValueError("router shapes")
    out = np.empty(gamma, np.float64)
    rc = lib.wfref_router_mlp(code, _ptr(h), _ptr(w1), _ptr(b1), _ptr(w2),
                              _ptr(b2), gamma, d, m, _ptr(out))
    _check(rc, "router_mlp")
    return out


def route_neural(delta, row, tau):
    """Sec. 3.3.2 decision: 1 (autoregressive) iff delta[row] > tau."""
    return int(float(delta[row]) > float(tau))


DECODER_WEIGHTS = ("attn_norm", "w_q", "w_k", "w_v", "w_o", "mlp_norm",
                   "w_gate", "w_up", "w_down")


def rmsnorm(x, gain, eps):
    """x [M][d], gain [d] (one storage type) -> fp64 [M][d]."""
    lib = _load()
    x, code = _arr(x)
    gain, c2 = _arr(gain)
    if code != c2:
        raise TypeError("x and gain must share a storage type")
    M, d = x.shape
    y = np.empty((M, d), np.float64)
    _check(lib.wfref_rmsnorm(code, _ptr(x), _ptr(gain), M, d, float(eps), _ptr(y)),
           "rmsnorm")
    return y


def decoder_forward(r, pos, layer, k_cache, v_cache, n_q_heads, n_kv_heads,
                    rms_eps, rope_base):
    """r [M][d]; layer: dict of DECODER_WEIGHTS arrays (storage as r);
    k_cache, v_cache [Hkv][cap][D] (any storage; rows [0, pos) used).
    Returns (out [M][d], k_cache, v_cache) in fp64, the caches with rows
    pos .. pos+M-1 written."""
    lib = _load()
    r, code = _arr(r)
    ws = []
    for name in DECODER_WEIGHTS:
        a, c = _arr(layer[name])
        if c != code:
            raise TypeError(f"{name} must share r's storage type")
        ws.append(a)
    M, d = r.shape
    hkv, cap, dh = np.asarray(k_cache).shape
    inter = ws[6].shape[0]
    kc = _decode64(k_cache)
    vc = _decode64(v_cache)
    out = np.empty((M, d), np.float64)
    rc = lib.wfref_decoder_forward(code, _ptr(r), M, int(pos), *[_ptr(a) for a in ws],
                                   d, n_q_heads, n_kv_heads, dh, inter,
                                   float(rms_eps), float(rope_base), _ptr(kc),
                                   _ptr(vc), cap, _ptr(out))
    _check(rc, "decoder_forward")
    return out, kc, vc


def catchup(r, pos, layer, k_cache, v_cache, n_q_heads, n_kv_heads, rms_eps,
            rope_base):
    """Lazy catch-up over a backlog r [n][d] starting at cache row pos: the
    first n-1 tokens get K/V only (KV-only prefill of RMSNorm(r) * g1), the
    last runs the full layer.  Returns (out [d], k_cache, v_cache) fp64."""
    r = np.asarray(r)
    n = r.shape[0]
    kc = _decode64(k_cache)
    vc = _decode64(v_cache)
    hkv, cap, dh = kc.shape
    if n > 1:
        xn = rmsnorm(r[:n - 1], layer["attn_norm"], rms_eps)
        k, v = kv_only_prefill(xn, _decode64(layer["w_k"]), _decode64(layer["w_v"]),
                               pos, hkv, dh, rope_base)
        kc[:, pos:pos + n - 1] = k
        vc[:, pos:pos + n - 1] = v
    out, kc, vc = decoder_forward(r[n - 1:], pos + n - 1, layer, kc, vc, n_q_heads,
                                  n_kv_heads, rms_eps, rope_base)
    return out[0], kc, vc


def _decode64(a):
    """fp64 copy of an oracle array (bf16 bit patterns decoded exactly)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.ascontiguousarray(a, np.float64).copy()


def rope(v, pos, base):
    """RoPE (rotate-half) of a fp64 vector at position pos."""
    lib = _load()
    v = np.array(v, np.float64, copy=True)
    lib.wfref_rope_inplace(_ptr(v), v.shape[0], float(pos), float(base))
    return v


def layer_forward(x, gain, w_q, w_k, w_v, pos0, n_q_heads, n_kv_heads,
                  head_dim, rms_eps, rope_base):
    """Full single-layer forward; returns dict of fp64 arrays."""
    lib = _load()
    x, code = _arr(x)
    gain, _ = _arr(gain)
    w_q, _ = _arr(w_q)
    w_k, _ = _arr(w_k)
    w_v, _ = _arr(w_v)
    T, d = x.shape
    xn = np.empty((T, d), np.float64)
    q = np.empty((T, n_q_heads, head_dim), np.float64)
    k = np.empty((n_kv_heads, T, head_dim), np.float64)
    v = np.empty_like(k)
    out = np.empty_like(q)
    rc = lib.wfref_layer_forward(code, _ptr(x), _ptr(gain), _ptr(w_q),
                                 _ptr(w_k), _ptr(w_v), T, int(pos0), d,
                                 n_q_heads, n_kv_heads, head_dim,
                                 float(rms_eps), float(rope_base), _ptr(xn),
                                 _ptr(q), _ptr(k), _ptr(v), _ptr(out))
    _check(rc, "layer_forward")
    return {"xn": xn, "q": q, "k": k, "v": v, "out": out}
