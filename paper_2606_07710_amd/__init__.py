"""Python binding of libwf, the MI355X verification-step library for WhiFlash
cross-paradigm speculative decoding (arXiv 2606.07710).

Argument marshalling only: every function passes torch tensors' device
pointers and the current HIP stream to the C ABI declared in include/wf.h,
and raises WfError on a non-OK status.  All computation runs in the HIP
kernels of libwf.so; there is no fallback path.  If the library has not been
built, importing this package raises ImportError.
"""
import ctypes
import os

import torch  # loaded first so libwf binds to the same HIP runtime as torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# WF_LIB names another build of the library (the host-sanitizer CPU run)
LIB_PATH = os.environ.get("WF_LIB") or os.path.join(_HERE, "libwf.so")

WF_OK, WF_ERR_INVALID_ARG, WF_ERR_UNSUPPORTED, WF_ERR_WORKSPACE, WF_ERR_HIP = range(5)
WF_F32, WF_BF16, WF_BF16_TILED = 0, 1, 2

EXPORTED_SYMBOLS = (
    "wf_abi_version", "wf_status_string", "wf_verify_attn",
    "wf_verify_attn_workspace_bytes", "wf_kv_only_prefill",
    "wf_lmhead_accept_entropy", "wf_lmhead_workspace_bytes",
    "wf_kv_only_prefill_workspace_bytes", "wf_verify_attn_tree",
    "wf_lmhead_accept_tree", "wf_kv_compact_path", "wf_router_neural",
    "wf_router_workspace_bytes", "wf_drafter_forward",
    "wf_drafter_forward_workspace_bytes", "wf_drafter_catchup",
    "wf_drafter_catchup_workspace_bytes", "wf_switch_init", "wf_switch_commit",
    "wf_kv_only_prefill_layers", "wf_kv_only_prefill_layers_workspace_bytes",
    "wf_tiled_weight_bytes", "wf_tile_weights", "wf_verify_attn_noalloc",
    "wf_read_probe", "wf_read_probe_series", "wf_lmhead_accept_route_neural",
    "wf_lmhead_route_neural_workspace_bytes",
)
NOALLOC_SCRATCH_BYTES = 32 << 20     # WF_NOALLOC_SCRATCH_BYTES
WF_DRAFTER_AR, WF_DRAFTER_DIFFUSION = 0, 1

DECODER_WEIGHTS = ("attn_norm", "w_q", "w_k", "w_v", "w_o", "mlp_norm",
                   "w_gate", "w_up", "w_down")


class DecoderLayer(ctypes.Structure):
    """wf_decoder_layer_t: device pointers of a drafter layer's weights and
    its shape."""
    _fields_ = [(n, ctypes.c_void_p) for n in DECODER_WEIGHTS] + [
        ("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("inter", ctypes.c_int32), ("rms_eps", ctypes.c_float),
        ("rope_base", ctypes.c_double)]


class SwitchState(ctypes.Structure):
    """wf_switch_state_t: host-side lazy catch-up bookkeeping."""
    _fields_ = [("active", ctypes.c_int32), ("lazy", ctypes.c_int32),
                ("committed", ctypes.c_int32), ("ar_cache_len", ctypes.c_int32),
                ("switches", ctypes.c_int32), ("max_backlog", ctypes.c_int32),
                ("caught_up", ctypes.c_int64), ("catchups", ctypes.c_int64)]


class WfError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with "
            "`python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(LIB_PATH)
    p, i32, sz, f32, f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t,
                            ctypes.c_float, ctypes.c_double)
    lib.wf_abi_version.restype = i32
    lib.wf_status_string.argtypes = [i32]
    lib.wf_status_string.restype = ctypes.c_char_p
    lib.wf_verify_attn.argtypes = [i32, p, p, p, p, i32, i32, i32, i32, i32,
                                   i32, f32, i32, p, sz, p]
    lib.wf_verify_attn.restype = i32
    lib.wf_verify_attn_noalloc.argtypes = [i32, p, p, p, p, i32, i32, i32, i32, i32,
                                           i32, f32, i32, p]
    lib.wf_verify_attn_noalloc.restype = i32
    lib.wf_verify_attn_workspace_bytes.argtypes = [i32, i32, i32, i32, i32,
                                                   i32, i32]
    lib.wf_verify_attn_workspace_bytes.restype = sz
    lib.wf_kv_only_prefill.argtypes = [i32, p, p, p, p, p, i32, i32, i32, i32,
                                       i32, i32, f64, p, sz, p]
    lib.wf_kv_only_prefill.restype = i32
    lib.wf_kv_only_prefill_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
    lib.wf_kv_only_prefill_workspace_bytes.restype = sz
    lib.wf_lmhead_accept_entropy.argtypes = [i32, p, p, p, p, i32, i32, i32,
                                             f32, p, p, p, p, sz, p]
    lib.wf_lmhead_accept_entropy.restype = i32
    lib.wf_lmhead_workspace_bytes.argtypes = [i32, i32]
    lib.wf_lmhead_workspace_bytes.restype = sz
    lib.wf_verify_attn_tree.argtypes = [i32, p, p, p, p, p, i32, i32, i32,
                                        i32, i32, i32, f32, i32, p, sz, p]
    lib.wf_verify_attn_tree.restype = i32
    lib.wf_lmhead_accept_tree.argtypes = [i32, p, p, p, p, p, i32, i32, i32,
                                          f32, p, p, p, p, p, sz, p]
    lib.wf_lmhead_accept_tree.restype = i32
    lib.wf_kv_compact_path.argtypes = [i32, p, p, p, p, i32, i32, i32, i32,
                                       i32, i32, sz, p]
    lib.wf_kv_compact_path.restype = i32
    lib.wf_router_neural.argtypes = [i32, p, p, p, p, p, p, i32, i32, i32, f32,
                                     p, p, p, sz, p]
    lib.wf_router_neural.restype = i32
    lib.wf_router_workspace_bytes.argtypes = [i32, i32, i32, i32]
    lib.wf_router_workspace_bytes.restype = sz
    for name in ("wf_drafter_forward", "wf_drafter_catchup"):
        fn = getattr(lib, name)
        fn.argtypes = [i32, p, p, i32, i32, p, p, i32, p, p, sz, p]
        fn.restype = i32
        q = getattr(lib, name + "_workspace_bytes")
        q.argtypes = [i32, p, i32, i32]
        q.restype = sz
    lib.wf_kv_only_prefill_layers.argtypes = [i32, p, p, p, p, p, i32, i32, i32, i32,
                                              i32, i32, f64, i32, sz, sz, sz, p, sz, p]
    lib.wf_kv_only_prefill_layers.restype = i32
    lib.wf_kv_only_prefill_layers_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
    lib.wf_kv_only_prefill_layers_workspace_bytes.restype = sz
    lib.wf_tiled_weight_bytes.argtypes = [i32, i32]
    lib.wf_tiled_weight_bytes.restype = sz
    lib.wf_tile_weights.argtypes = [p, i32, i32, p, sz, p]
    lib.wf_tile_weights.restype = i32
    lib.wf_lmhead_accept_route_neural.argtypes = [i32, p, p, p, i32, i32, i32, p, p, p, p,
                                                  i32, f32, p, p, p, p, p, sz, p]
    lib.wf_lmhead_accept_route_neural.restype = i32
    lib.wf_lmhead_route_neural_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
    lib.wf_lmhead_route_neural_workspace_bytes.restype = sz
    lib.wf_read_probe.argtypes = [p, sz, p, sz, i32, p]
    lib.wf_read_probe.restype = i32
    lib.wf_read_probe_series.argtypes = [p, sz, sz, i32, i32, p, sz, i32, i32, p]
    lib.wf_read_probe_series.restype = i32
    lib.wf_switch_init.argtypes = [p, i32, i32, i32]
    lib.wf_switch_init.restype = i32
    lib.wf_switch_commit.argtypes = [p, i32, i32, p, p]
    lib.wf_switch_commit.restype = i32
    return lib


lib = _load()


def status_string(status: int) -> str:
    return lib.wf_status_string(int(status)).decode()


def abi_version() -> int:
    return int(lib.wf_abi_version())


class TiledWeight:
    """A bf16 weight (or a [L] stack of them) in the tiled layout that
    wf_tile_weights writes: `data` [L?][n] holds the tiles, `shape` is the
    logical [L?][rows][cols].  Passed wherever a weight is, it selects
    WF_BF16_TILED."""

    def __init__(self, data, shape):
        self.data, self.shape = data, tuple(shape)
        self.dtype, self.device, self.is_cuda = data.dtype, data.device, data.is_cuda

    def data_ptr(self):
        return self.data.data_ptr()

    def is_contiguous(self):
        return self.data.is_contiguous()

    def stride(self, dim):
        if dim != 0 or len(self.shape) != 3:
            raise ValueError("layer stride of a tiled stack only")
        return self.data.stride(0)


def wf_tiled_weight_bytes(rows, cols) -> int:
    return int(lib.wf_tiled_weight_bytes(int(rows), int(cols)))


def tile_weights(w, stream=None) -> TiledWeight:
    """Tiled copy of a bf16 weight [rows][cols] or stack [L][rows][cols]."""
    if w.dtype != torch.bfloat16:
        raise TypeError("tiled weights are bf16")
    rows, cols = w.shape[-2:]
    n = wf_tiled_weight_bytes(rows, cols) // 2
    if n == 0:
        raise ValueError(f"cannot tile a [{rows}][{cols}] weight (cols % 32 != 0)")
    layers = w.shape[0] if w.dim() == 3 else None
    out = torch.empty((layers, n) if layers else (n,), dtype=torch.bfloat16, device=w.device)
    for l in range(layers or 1):
        src, dst = (w[l], out[l]) if layers else (w, out)
        _check(lib.wf_tile_weights(_dev(src, "w"), rows, cols, _dev(dst, "tiled"), 2 * n,
                                   _stream(stream)), "wf_tile_weights")
    return TiledWeight(out, w.shape)


def _weight_code(x, *ws) -> int:
    """dtype code of a call whose activations are x and weights ws."""
    tiled = [isinstance(w, TiledWeight) for w in ws if w is not None]
    if any(tiled):
        if not all(tiled) or x.dtype != torch.bfloat16:
            raise TypeError("tiled weights: all weights tiled, bf16 activations")
        return WF_BF16_TILED
    return _dtype_code(x)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return WF_F32
    if t.dtype == torch.bfloat16:
        return WF_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _dev(t, name):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(status, what):
    if status != WF_OK:
        raise WfError(status, what)


def wf_verify_attn_workspace_bytes(dtype, gamma, ctx_len, n_q_heads,
                                   n_kv_heads, head_dim, num_splits=0) -> int:
    code = dtype if isinstance(dtype, int) else (
        WF_F32 if dtype == torch.float32 else WF_BF16)
    return int(lib.wf_verify_attn_workspace_bytes(
        code, gamma, ctx_len, n_q_heads, n_kv_heads, head_dim, num_splits))


def wf_lmhead_workspace_bytes(gamma, vocab) -> int:
    return int(lib.wf_lmhead_workspace_bytes(gamma, vocab))


def alloc_workspace(nbytes: int, device) -> torch.Tensor:
    """Caller-owned scratch for the workspace arguments: 16-byte aligned and
    zero-filled, as the calls require before a workspace's first use (each
    call leaves its arrival counters at zero again, so one workspace serves
    any number of calls that do not overlap in time)."""
    return torch.zeros(max(16, (nbytes + 15) // 16 * 16), dtype=torch.uint8,
                       device=device)


def wf_verify_attn(q, k_cache, v_cache, out, ctx_len, softmax_scale=None,
                   num_splits=0, workspace=None, stream=None):
    """q [gamma][Hq][D]; k_cache, v_cache [Hkv][cap][D]; out like q."""
    gamma, hq, dh = q.shape
    hkv, cap, dh2 = k_cache.shape
    if dh2 != dh or tuple(v_cache.shape) != tuple(k_cache.shape):
        raise ValueError("cache shapes do not match q")
    if tuple(out.shape) != tuple(q.shape) or out.dtype != q.dtype:
        raise ValueError("out must match q in shape and dtype")
    code = _dtype_code(q)
    if softmax_scale is None:
        softmax_scale = dh ** -0.5
    need = wf_verify_attn_workspace_bytes(code, gamma, ctx_len, hq, hkv, dh,
                                          num_splits)
    if workspace is None:
        workspace = alloc_workspace(need, q.device)
    st = lib.wf_verify_attn(code, _dev(q, "q"), _dev(k_cache, "k_cache"),
                            _dev(v_cache, "v_cache"), _dev(out, "out"), gamma,
                            int(ctx_len), cap, hq, hkv, dh,
                            float(softmax_scale), int(num_splits),
                            _dev(workspace, "workspace"), workspace.numel(),
                            _stream(stream))
    _check(st, "wf_verify_attn")
    return out


def wf_verify_attn_noalloc(q, k_cache, v_cache, out, ctx_len, softmax_scale=None,
                           num_splits=0, stream=None):
    """wf_verify_attn with the library's static device scratch instead of a
    workspace: nothing is allocated (for graph capture and callers that
    cannot allocate).  Calls that overlap in time on one GPU race."""
    gamma, hq, dh = q.shape
    hkv, cap, dh2 = k_cache.shape
    if dh2 != dh or tuple(v_cache.shape) != tuple(k_cache.shape):
        raise ValueError("cache shapes do not match q")
    if tuple(out.shape) != tuple(q.shape) or out.dtype != q.dtype:
        raise ValueError("out must match q in shape and dtype")
    if softmax_scale is None:
        softmax_scale = dh ** -0.5
    st = lib.wf_verify_attn_noalloc(_dtype_code(q), _dev(q, "q"), _dev(k_cache, "k_cache"),
                                    _dev(v_cache, "v_cache"), _dev(out, "out"), gamma,
                                    int(ctx_len), cap, hq, hkv, dh, float(softmax_scale),
                                    int(num_splits), _stream(stream))
    _check(st, "wf_verify_attn_noalloc")
    return out


def wf_kv_only_prefill_workspace_bytes(dtype, n_tok, d_in, n_kv_heads,
                                       head_dim) -> int:
    code = dtype if isinstance(dtype, int) else (
        WF_F32 if dtype == torch.float32 else WF_BF16)
    return int(lib.wf_kv_only_prefill_workspace_bytes(code, n_tok, d_in,
                                                      n_kv_heads, head_dim))


def wf_kv_only_prefill(x, w_k, w_v, k_cache, v_cache, start_pos, rope_base,
                       workspace=None, stream=None):
    """x [n][d_in]; w_k, w_v [Hkv*D][d_in]; caches [Hkv][cap][D]."""
    n_tok, d_in = x.shape
    hkv, cap, dh = k_cache.shape
    code = _weight_code(x, w_k, w_v)
    need = wf_kv_only_prefill_workspace_bytes(code, n_tok, d_in, hkv, dh)
    if workspace is None and need:
        workspace = alloc_workspace(need, x.device)
    st = lib.wf_kv_only_prefill(code, _dev(x, "x"), _dev(w_k, "w_k"),
                                _dev(w_v, "w_v"), _dev(k_cache, "k_cache"),
                                _dev(v_cache, "v_cache"), n_tok,
                                int(start_pos), cap, d_in, hkv, dh,
                                float(rope_base), _dev(workspace, "workspace"),
                                workspace.numel() if workspace is not None else 0,
                                _stream(stream))
    _check(st, "wf_kv_only_prefill")


def wf_kv_only_prefill_layers_workspace_bytes(dtype, n_tok, d_in, n_kv_heads, head_dim,
                                              n_layers) -> int:
    code = dtype if isinstance(dtype, int) else (
        WF_F32 if dtype == torch.float32 else WF_BF16)
    return int(lib.wf_kv_only_prefill_layers_workspace_bytes(code, n_tok, d_in, n_kv_heads,
                                                             head_dim, n_layers))


def wf_kv_only_prefill_layers(x, w_k, w_v, k_cache, v_cache, start_pos, rope_base,
                              workspace=None, stream=None):
    """x [L][n][d_in]; w_k, w_v [L][Hkv*D][d_in]; caches [L][Hkv][cap][D]
    (each a dense stack, so the layer strides are those of dim 0)."""
    n_layers, n_tok, d_in = x.shape
    _, hkv, cap, dh = k_cache.shape
    if w_k.shape[0] != n_layers or v_cache.stride(0) != k_cache.stride(0) or \
            w_v.stride(0) != w_k.stride(0) or k_cache.shape[0] != n_layers:
        raise ValueError("layer stacks must match")
    code = _weight_code(x, w_k, w_v)
    need = wf_kv_only_prefill_layers_workspace_bytes(code, n_tok, d_in, hkv, dh, n_layers)
    if workspace is None and need:
        workspace = alloc_workspace(need, x.device)
    st = lib.wf_kv_only_prefill_layers(
        code, _dev(x, "x"), _dev(w_k, "w_k"), _dev(w_v, "w_v"), _dev(k_cache, "k_cache"),
        _dev(v_cache, "v_cache"), n_tok, int(start_pos), cap, d_in, hkv, dh,
        float(rope_base), n_layers, x.stride(0), w_k.stride(0), k_cache.stride(0),
        _dev(workspace, "workspace"), workspace.numel() if workspace is not None else 0,
        _stream(stream))
    _check(st, "wf_kv_only_prefill_layers")


def wf_lmhead_accept_entropy(h, w_lm, logits, draft, tau, argmax_out,
                             entropy_out, accept_out, workspace=None,
                             stream=None, gamma=None, vocab=None):
    """Either (h [gamma][d], w_lm [vocab][d]) or logits [gamma][vocab] fp32.
    draft [gamma-1] int32 (None when gamma == 1); outputs int32 [gamma],
    fp32 [gamma], int32 [3]."""
    if logits is not None:
        gamma, vocab = logits.shape
        d, code = 0, WF_F32
    else:
        gamma, d = h.shape
        vocab = w_lm.shape[0]
        code = _weight_code(h, w_lm)
    need = wf_lmhead_workspace_bytes(gamma, vocab)
    dev = (logits if logits is not None else h).device
    if workspace is None:
        workspace = alloc_workspace(need, dev)
    st = lib.wf_lmhead_accept_entropy(
        code, _dev(h, "h"), _dev(w_lm, "w_lm"), _dev(logits, "logits"),
        _dev(draft, "draft"), gamma, d, vocab, float(tau),
        _dev(argmax_out, "argmax_out"), _dev(entropy_out, "entropy_out"),
        _dev(accept_out, "accept_out"), _dev(workspace, "workspace"),
        workspace.numel(), _stream(stream))
    _check(st, "wf_lmhead_accept_entropy")


def wf_verify_attn_tree(q, k_cache, v_cache, out, ctx_len, tree_mask,
                        softmax_scale=None, num_splits=0, workspace=None,
                        stream=None):
    """Tree verification attention: tree_mask [gamma] int64/uint64 device
    tensor (bit j of row i: row i sees block row j); else as wf_verify_attn."""
    gamma, hq, dh = q.shape
    hkv, cap, dh2 = k_cache.shape
    if dh2 != dh or tuple(v_cache.shape) != tuple(k_cache.shape):
        raise ValueError("cache shapes do not match q")
    if tuple(out.shape) != tuple(q.shape) or out.dtype != q.dtype:
        raise ValueError("out must match q in shape and dtype")
    if tree_mask.numel() != gamma or tree_mask.element_size() != 8:
        raise ValueError("tree_mask must hold gamma 64-bit words")
    code = _dtype_code(q)
    if softmax_scale is None:
        softmax_scale = dh ** -0.5
    need = wf_verify_attn_workspace_bytes(code, gamma, ctx_len, hq, hkv, dh,
                                          num_splits)
    if workspace is None:
        workspace = alloc_workspace(need, q.device)
    st = lib.wf_verify_attn_tree(code, _dev(q, "q"), _dev(k_cache, "k_cache"),
                                 _dev(v_cache, "v_cache"), _dev(out, "out"),
                                 _dev(tree_mask, "tree_mask"), gamma,
                                 int(ctx_len), cap, hq, hkv, dh,
                                 float(softmax_scale), int(num_splits),
                                 _dev(workspace, "workspace"),
                                 workspace.numel(), _stream(stream))
    _check(st, "wf_verify_attn_tree")
    return out


def wf_lmhead_accept_route_neural(h, w_lm, draft, w1, b1, w2, b2, tau_neural, argmax_out,
                                  entropy_out, accept_out, delta_out, workspace=None,
                                  stream=None):
    """h [gamma][d]; w_lm [vocab][d] and w1 [m][d] (both tiled or both
    row-major); b1, w2 [m], b2 [1]; draft [gamma-1] int32 (None when gamma
    == 1); outputs int32 [gamma], fp32 [gamma], int32 [3] (route: the neural
    policy), fp32 [gamma] (predicted gain per row)."""
    gamma, d = h.shape
    vocab = w_lm.shape[0]
    m = w1.shape[0]
    code = _weight_code(h, w_lm, w1)
    need = int(lib.wf_lmhead_route_neural_workspace_bytes(code, gamma, vocab, d, m))
    if workspace is None:
        workspace = alloc_workspace(need, h.device)
    st = lib.wf_lmhead_accept_route_neural(
        code, _dev(h, "h"), _dev(w_lm, "w_lm"), _dev(draft, "draft"), gamma, d, vocab,
        _dev(w1, "w1"), _dev(b1, "b1"), _dev(w2, "w2"), _dev(b2, "b2"), m, float(tau_neural),
        _dev(argmax_out, "argmax_out"), _dev(entropy_out, "entropy_out"),
        _dev(accept_out, "accept_out"), _dev(delta_out, "delta_out"),
        _dev(workspace, "workspace"), workspace.numel(), _stream(stream))
    _check(st, "wf_lmhead_accept_route_neural")


def wf_lmhead_accept_tree(h, w_lm, logits, tokens, parents, tau, argmax_out,
                          entropy_out, accept_out, path_out, workspace=None,
                          stream=None):
    """Either (h [gamma][d], w_lm [vocab][d]) or logits [gamma][vocab] fp32;
    tokens, parents [gamma] int32; outputs int32 [gamma], fp32 [gamma],
    int32 [4], int32 [gamma]."""
    if logits is not None:
        gamma, vocab = logits.shape
        d, code = 0, WF_F32
    else:
        gamma, d = h.shape
        vocab = w_lm.shape[0]
        code = _weight_code(h, w_lm)
    need = wf_lmhead_workspace_bytes(gamma, vocab)
    dev = (logits if logits is not None else h).device
    if workspace is None:
        workspace = alloc_workspace(need, dev)
    st = lib.wf_lmhead_accept_tree(
        code, _dev(h, "h"), _dev(w_lm, "w_lm"), _dev(logits, "logits"),
        _dev(tokens, "tokens"), _dev(parents, "parents"), gamma, d, vocab,
        float(tau), _dev(argmax_out, "argmax_out"),
        _dev(entropy_out, "entropy_out"), _dev(accept_out, "accept_out"),
        _dev(path_out, "path_out"), _dev(workspace, "workspace"),
        workspace.numel(), _stream(stream))
    _check(st, "wf_lmhead_accept_tree")


def wf_kv_compact_path(k_cache, v_cache, accept, path, ctx_len, stream=None):
    """Caches [Hkv][cap][D] (one layer) or [L][Hkv][cap][D] (all layers);
    accept (n at [0]) and path [gamma] int32 device tensors, as written by
    wf_lmhead_accept_tree."""
    if tuple(v_cache.shape) != tuple(k_cache.shape) or v_cache.dtype != k_cache.dtype:
        raise ValueError("k_cache and v_cache must match")
    if k_cache.dim() == 4:
        n_layers, hkv, cap, dh = k_cache.shape
        stride = hkv * cap * dh
    else:
        (hkv, cap, dh), n_layers, stride = k_cache.shape, 1, 0
    gamma = path.numel()
    st = lib.wf_kv_compact_path(_dtype_code(k_cache), _dev(k_cache, "k_cache"),
                                _dev(v_cache, "v_cache"), _dev(accept, "accept"),
                                _dev(path, "path"), gamma, int(ctx_len), cap,
                                hkv, dh, n_layers, stride, _stream(stream))
    _check(st, "wf_kv_compact_path")


def wf_router_neural(h, w1, b1, w2, b2, row, tau, delta_out, route_out,
                     workspace=None, stream=None):
    """h [gamma][d]; w1 [m][d]; b1, w2 [m]; b2 [1] (one dtype); row: int32
    device tensor holding the row to route on; outputs fp32 [gamma] and
    int32 [1]."""
    gamma, d = h.shape
    m = w1.shape[0]
    code = _dtype_code(h)
    need = int(lib.wf_router_workspace_bytes(code, gamma, d, m))
    if workspace is None:
        workspace = alloc_workspace(need, h.device)
    st = lib.wf_router_neural(code, _dev(h, "h"), _dev(w1, "w1"), _dev(b1, "b1"),
                              _dev(w2, "w2"), _dev(b2, "b2"), _dev(row, "row"),
                              gamma, d, m, float(tau), _dev(delta_out, "delta_out"),
                              _dev(route_out, "route_out"),
                              _dev(workspace, "workspace"), workspace.numel(),
                              _stream(stream))
    _check(st, "wf_router_neural")


def decoder_layer(weights, n_q_heads, n_kv_heads, rms_eps, rope_base):
    """DecoderLayer from a dict of DECODER_WEIGHTS device tensors (bf16)."""
    w_q, w_k, w_gate = weights["w_q"], weights["w_k"], weights["w_gate"]
    head_dim = w_q.shape[0] // n_q_heads
    if w_k.shape[0] != n_kv_heads * head_dim:
        raise ValueError("w_k rows must be n_kv_heads * head_dim")
    layer = DecoderLayer(*[_dev(weights[n], n).value for n in DECODER_WEIGHTS],
                         w_q.shape[1], n_q_heads, n_kv_heads, head_dim,
                         w_gate.shape[0], float(rms_eps), float(rope_base))
    # the struct holds raw device pointers: keep the tensors alive with it
    layer.keepalive = dict(weights)
    # projections tiled (wf_tile_weights) -> the calls pass WF_BF16_TILED
    mats = [weights[n] for n in DECODER_WEIGHTS if not n.endswith("norm")]
    layer.tiled = all(isinstance(m, TiledWeight) for m in mats)
    if not layer.tiled and any(isinstance(m, TiledWeight) for m in mats):
        raise TypeError("tile all seven projections or none")
    return layer


def wf_drafter_forward_workspace_bytes(layer, n_tok, pos) -> int:
    """Workspace of a bf16 wf_drafter_forward call (0: shapes rejected)."""
    code = WF_BF16_TILED if getattr(layer, "tiled", False) else WF_BF16
    return int(lib.wf_drafter_forward_workspace_bytes(code, ctypes.byref(layer),
                                                      int(n_tok), int(pos)))


def wf_drafter_catchup_workspace_bytes(layer, n_backlog, pos) -> int:
    """Workspace of a bf16 wf_drafter_catchup call (0: shapes rejected)."""
    code = WF_BF16_TILED if getattr(layer, "tiled", False) else WF_BF16
    return int(lib.wf_drafter_catchup_workspace_bytes(code, ctypes.byref(layer),
                                                      int(n_backlog), int(pos)))


def wf_drafter_forward(layer, r, pos, k_cache, v_cache, out, workspace=None,
                       stream=None):
    """layer: DecoderLayer; r, out [n_tok][hidden]; caches [Hkv][cap][D]."""
    n_tok = r.shape[0]
    code = WF_BF16_TILED if getattr(layer, "tiled", False) else _dtype_code(r)
    need = int(lib.wf_drafter_forward_workspace_bytes(code, ctypes.byref(layer), n_tok,
                                                      int(pos)))
    if workspace is None:
        workspace = alloc_workspace(need, r.device)
    st = lib.wf_drafter_forward(code, ctypes.byref(layer), _dev(r, "r"), n_tok, int(pos),
                                _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
                                k_cache.shape[1], _dev(out, "out"),
                                _dev(workspace, "workspace"), workspace.numel(),
                                _stream(stream))
    _check(st, "wf_drafter_forward")
    return out


def wf_drafter_catchup(layer, r, pos, k_cache, v_cache, out, workspace=None,
                       stream=None):
    """layer: DecoderLayer; r [n_backlog][hidden]; out [hidden]."""
    n = r.shape[0]
    code = WF_BF16_TILED if getattr(layer, "tiled", False) else _dtype_code(r)
    need = int(lib.wf_drafter_catchup_workspace_bytes(code, ctypes.byref(layer), n,
                                                      int(pos)))
    if workspace is None:
        workspace = alloc_workspace(need, r.device)
    st = lib.wf_drafter_catchup(code, ctypes.byref(layer), _dev(r, "r"), n, int(pos),
                                _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
                                k_cache.shape[1], _dev(out, "out"),
                                _dev(workspace, "workspace"), workspace.numel(),
                                _stream(stream))
    _check(st, "wf_drafter_catchup")
    return out


def wf_read_probe(src, sink, workgroups, stream=None):
    """Measurement support: one plain streaming read of the whole device
    tensor src (sink: device tensor of at least workgroups * 4 KB)."""
    _check(lib.wf_read_probe(_dev(src, "src"), src.numel() * src.element_size(),
                             _dev(sink, "sink"), sink.numel() * sink.element_size(),
                             int(workgroups), _stream(stream)), "wf_read_probe")


def wf_read_probe_series(buf, nbytes, n_bufs, reps, sink, workgroups, depth, stream=None):
    """Measurement support: reps rounds of plain reads of the n_bufs
    consecutive nbytes-long pieces of the device tensor buf, launched back
    to back by the library."""
    if n_bufs * nbytes > buf.numel() * buf.element_size():
        raise ValueError("wf_read_probe_series: buf holds fewer than n_bufs pieces")
    _check(lib.wf_read_probe_series(_dev(buf, "buf"), int(nbytes), int(nbytes), int(n_bufs),
                                    int(reps), _dev(sink, "sink"),
                                    sink.numel() * sink.element_size(), int(workgroups),
                                    int(depth), _stream(stream)), "wf_read_probe_series")


def wf_switch_init(active, lazy, prompt_len) -> SwitchState:
    s = SwitchState()
    _check(lib.wf_switch_init(ctypes.byref(s), int(active), int(lazy), int(prompt_len)),
           "wf_switch_init")
    return s


def wf_switch_commit(state, n_new, next_drafter):
    """-> (start, count) of the backlog now due (count 0: none)."""
    start, count = ctypes.c_int32(), ctypes.c_int32()
    _check(lib.wf_switch_commit(ctypes.byref(state), int(n_new), int(next_drafter),
                                ctypes.byref(start), ctypes.byref(count)),
           "wf_switch_commit")
    return start.value, count.value
