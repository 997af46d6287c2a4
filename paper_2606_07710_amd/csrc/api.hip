// api.hip -- the extern "C" boundary of libwf: argument validation on the
// host, workspace queries and dispatch to the kernel launchers.  Nothing is
// enqueued unless every check passes.  The library holds no global state.
#include <algorithm>
#include <climits>
#include <cmath>

#include "wf_api_internal.h"

namespace {

constexpr int kMaxGamma = 64;
constexpr int kMaxQHeads = 256;
constexpr int kMaxSplits = 1024;
constexpr int kMaxPrefillTokens = 4096;
constexpr int kMaxBacklog = 1 << 20;        // drafter catch-up, in 4096-token batches
constexpr int kMaxLayers = 1024;
constexpr int kMaxRouterHidden = 1 << 16;

inline bool aligned16(const void *p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

inline bool dtype_ok(wf_dtype_t dt) { return dt == WF_F32 || dt == WF_BF16; }

// bf16 storage, weights row-major or tiled (the calls that take weights)
inline bool is_bf16(wf_dtype_t dt) { return dt == WF_BF16 || dt == WF_BF16_TILED; }
inline bool weight_dtype_ok(wf_dtype_t dt) { return dtype_ok(dt) || dt == WF_BF16_TILED; }
inline wf_dtype_t storage(wf_dtype_t dt) { return is_bf16(dt) ? WF_BF16 : dt; }

inline bool head_dim_ok(int dh) { return dh == 64 || dh == 128; }

wf_status_t check_attn(wf_dtype_t dt, int gamma, int ctx_len, int n_q_heads,
                       int n_kv_heads, int head_dim, int num_splits) {
    if (!dtype_ok(dt))
        return WF_ERR_INVALID_ARG;
    if (gamma < 1 || gamma > kMaxGamma || ctx_len < 0)
        return WF_ERR_INVALID_ARG;
    if (n_kv_heads < 1 || n_q_heads < 1 || n_q_heads > kMaxQHeads ||
        n_q_heads % n_kv_heads != 0)
        return WF_ERR_INVALID_ARG;
    if (num_splits < 0 || num_splits > kMaxSplits)
        return WF_ERR_INVALID_ARG;
    if ((long long)ctx_len + gamma > (long long)INT32_MAX / 2)
        return WF_ERR_INVALID_ARG;
    if (!head_dim_ok(head_dim))
        return WF_ERR_UNSUPPORTED;
    return WF_OK;
}

}  // namespace

extern "C" {

int32_t wf_abi_version(void) { return 9; }

const char *wf_status_string(wf_status_t s) {
    switch (s) {
    case WF_OK: return "ok";
    case WF_ERR_INVALID_ARG: return "invalid argument";
    case WF_ERR_UNSUPPORTED: return "unsupported configuration";
    case WF_ERR_WORKSPACE: return "workspace missing or too small";
    case WF_ERR_HIP: return "HIP kernel launch failed";
    default: break;
    }
    return "unknown status";
}

size_t wf_verify_attn_workspace_bytes(wf_dtype_t dt, int32_t gamma,
                                      int32_t ctx_len, int32_t n_q_heads,
                                      int32_t n_kv_heads, int32_t head_dim,
                                      int32_t num_splits) {
    if (check_attn(dt, gamma, ctx_len, n_q_heads, n_kv_heads, head_dim,
                   num_splits) != WF_OK)
        return 0;
    const wf::AttnPlan p = wf::plan_attn(dt, gamma, ctx_len, n_q_heads,
                                         n_kv_heads, head_dim, num_splits);
    return wf::attn_workspace_bytes(p, gamma, n_q_heads, head_dim);
}

}  // extern "C"

namespace wf {
// Host-side checks of a verify-attention call, everything but the
// workspace; on WF_OK *plan holds the call's split plan.
wf_status_t validate_verify_attn(wf_dtype_t dt, const void *q, const void *k_cache,
                                 const void *v_cache, const void *out, int32_t gamma,
                                 int32_t ctx_len, int32_t cap, int32_t n_q_heads,
                                 int32_t n_kv_heads, int32_t head_dim, float softmax_scale,
                                 int32_t num_splits, AttnPlan *plan) {
    wf_status_t st = check_attn(dt, gamma, ctx_len, n_q_heads, n_kv_heads,
                                head_dim, num_splits);
    if (st != WF_OK)
        return st;
    if (!q || !k_cache || !v_cache || !out)
        return WF_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) ||
        !aligned16(out))
        return WF_ERR_INVALID_ARG;
    if ((long long)ctx_len + gamma > cap)
        return WF_ERR_INVALID_ARG;
    if (!std::isfinite(softmax_scale) || softmax_scale <= 0.f)
        return WF_ERR_INVALID_ARG;
    *plan = plan_attn(dt, gamma, ctx_len, n_q_heads, n_kv_heads, head_dim, num_splits);
    return WF_OK;
}
}  // namespace wf

extern "C" {

namespace {
wf_status_t verify_attn_common(wf_dtype_t dt, const void *q, const void *k_cache,
                               const void *v_cache, void *out,
                               const uint64_t *tree_mask, int32_t gamma,
                               int32_t ctx_len, int32_t cap, int32_t n_q_heads,
                               int32_t n_kv_heads, int32_t head_dim,
                               float softmax_scale, int32_t num_splits,
                               void *workspace, size_t workspace_bytes,
                               void *stream) {
    wf::AttnPlan p{};
    const wf_status_t st = wf::validate_verify_attn(dt, q, k_cache, v_cache, out, gamma,
                                                    ctx_len, cap, n_q_heads, n_kv_heads,
                                                    head_dim, softmax_scale, num_splits, &p);
    if (st != WF_OK)
        return st;
    const size_t need = wf::attn_workspace_bytes(p, gamma, n_q_heads, head_dim);
    if (!workspace || workspace_bytes < need || !aligned16(workspace))
        return WF_ERR_WORKSPACE;
    return wf::launch_attn(dt, q, k_cache, v_cache, out, gamma, ctx_len, cap,
                           n_q_heads, n_kv_heads, head_dim, softmax_scale,
                           tree_mask, p, workspace,
                           static_cast<hipStream_t>(stream));
}
}  // namespace

wf_status_t wf_verify_attn(wf_dtype_t dt, const void *q, const void *k_cache,
                           const void *v_cache, void *out, int32_t gamma,
                           int32_t ctx_len, int32_t cap, int32_t n_q_heads,
                           int32_t n_kv_heads, int32_t head_dim,
                           float softmax_scale, int32_t num_splits,
                           void *workspace, size_t workspace_bytes,
                           void *stream) {
    return verify_attn_common(dt, q, k_cache, v_cache, out, nullptr, gamma,
                              ctx_len, cap, n_q_heads, n_kv_heads, head_dim,
                              softmax_scale, num_splits, workspace,
                              workspace_bytes, stream);
}

wf_status_t wf_verify_attn_tree(wf_dtype_t dt, const void *q,
                                const void *k_cache, const void *v_cache,
                                void *out, const uint64_t *tree_mask,
                                int32_t gamma, int32_t ctx_len, int32_t cap,
                                int32_t n_q_heads, int32_t n_kv_heads,
                                int32_t head_dim, float softmax_scale,
                                int32_t num_splits, void *workspace,
                                size_t workspace_bytes, void *stream) {
    if (!tree_mask || !aligned16(tree_mask))
        return WF_ERR_INVALID_ARG;
    return verify_attn_common(dt, q, k_cache, v_cache, out, tree_mask, gamma,
                              ctx_len, cap, n_q_heads, n_kv_heads, head_dim,
                              softmax_scale, num_splits, workspace,
                              workspace_bytes, stream);
}

namespace {
wf_status_t check_prefill(wf_dtype_t dt, int n_tok, int start_pos, int cap,
                          int d_in, int n_kv_heads, int head_dim,
                          double rope_base) {
    if (!weight_dtype_ok(dt))
        return WF_ERR_INVALID_ARG;
    if (n_tok < 0 || n_tok > kMaxPrefillTokens || start_pos < 0 ||
        (long long)start_pos + n_tok > cap || d_in < 1 || n_kv_heads < 1 ||
        n_kv_heads > kMaxQHeads)
        return WF_ERR_INVALID_ARG;
    if (!std::isfinite(rope_base) || rope_base <= 0.0)
        return WF_ERR_INVALID_ARG;
    if (!head_dim_ok(head_dim))
        return WF_ERR_UNSUPPORTED;
    if (is_bf16(dt) && d_in % 32 != 0)
        return WF_ERR_UNSUPPORTED;
    if (is_bf16(dt) && n_tok > 0 && !wf::prefill_fits(n_tok, d_in, n_kv_heads, head_dim))
        return WF_ERR_UNSUPPORTED;
    return WF_OK;
}
}  // namespace

size_t wf_kv_only_prefill_workspace_bytes(wf_dtype_t dt, int32_t n_tok,
                                          int32_t d_in, int32_t n_kv_heads,
                                          int32_t head_dim) {
    if (check_prefill(dt, n_tok, 0, n_tok, d_in, n_kv_heads, head_dim, 1.0) != WF_OK)
        return 0;
    return wf::prefill_workspace_bytes(storage(dt), n_tok, d_in, n_kv_heads, head_dim);
}

wf_status_t wf_kv_only_prefill(wf_dtype_t dt, const void *x, const void *w_k,
                               const void *w_v, void *k_cache, void *v_cache,
                               int32_t n_tok, int32_t start_pos, int32_t cap,
                               int32_t d_in, int32_t n_kv_heads,
                               int32_t head_dim, double rope_base,
                               void *workspace, size_t workspace_bytes,
                               void *stream) {
    const wf_status_t st = check_prefill(dt, n_tok, start_pos, cap, d_in,
                                         n_kv_heads, head_dim, rope_base);
    if (st != WF_OK)
        return st;
    if (n_tok == 0)
        return WF_OK;
    if (!x || !w_k || !w_v || !k_cache || !v_cache)
        return WF_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(w_k) || !aligned16(w_v) ||
        !aligned16(k_cache) || !aligned16(v_cache))
        return WF_ERR_INVALID_ARG;
    const size_t need = wf::prefill_workspace_bytes(storage(dt), n_tok, d_in, n_kv_heads,
                                                    head_dim);
    if (need && (!workspace || workspace_bytes < need || !aligned16(workspace)))
        return WF_ERR_WORKSPACE;
    return wf::launch_prefill(dt, x, w_k, w_v, k_cache, v_cache, n_tok,
                              start_pos, cap, d_in, n_kv_heads, head_dim,
                              rope_base, workspace, static_cast<hipStream_t>(stream));
}

namespace {
wf_status_t check_prefill_layers(wf_dtype_t dt, int n_tok, int cap, int d_in, int n_kv_heads,
                                 int head_dim, int n_layers, size_t x_ls, size_t w_ls,
                                 size_t c_ls) {
    if (n_layers < 1 || n_layers > kMaxLayers)
        return WF_ERR_INVALID_ARG;
    if (n_layers == 1)
        return WF_OK;
    const size_t eb = is_bf16(dt) ? 2 : 4;
    if (x_ls < (size_t)n_tok * d_in || w_ls < (size_t)n_kv_heads * head_dim * d_in ||
        c_ls < (size_t)n_kv_heads * cap * head_dim)
        return WF_ERR_INVALID_ARG;
    if ((x_ls * eb) % 16 || (w_ls * eb) % 16 || (c_ls * eb) % 16)
        return WF_ERR_INVALID_ARG;
    if (is_bf16(dt) && n_tok > 0 &&
        !wf::prefill_fits(n_tok, d_in, n_kv_heads, head_dim, n_layers))
        return WF_ERR_UNSUPPORTED;
    return WF_OK;
}
}  // namespace

size_t wf_kv_only_prefill_layers_workspace_bytes(wf_dtype_t dt, int32_t n_tok, int32_t d_in,
                                                 int32_t n_kv_heads, int32_t head_dim,
                                                 int32_t n_layers) {
    if (check_prefill(dt, n_tok, 0, n_tok, d_in, n_kv_heads, head_dim, 1.0) != WF_OK ||
        n_layers < 1 || n_layers > kMaxLayers ||
        (is_bf16(dt) && n_tok > 0 &&
         !wf::prefill_fits(n_tok, d_in, n_kv_heads, head_dim, n_layers)))
        return 0;
    return wf::prefill_workspace_bytes(storage(dt), n_tok, d_in, n_kv_heads, head_dim);
}

wf_status_t wf_kv_only_prefill_layers(wf_dtype_t dt, const void *x, const void *w_k,
                                      const void *w_v, void *k_cache, void *v_cache,
                                      int32_t n_tok, int32_t start_pos, int32_t cap,
                                      int32_t d_in, int32_t n_kv_heads, int32_t head_dim,
                                      double rope_base, int32_t n_layers,
                                      size_t x_layer_stride, size_t w_layer_stride,
                                      size_t cache_layer_stride, void *workspace,
                                      size_t workspace_bytes, void *stream) {
    wf_status_t st = check_prefill(dt, n_tok, start_pos, cap, d_in, n_kv_heads, head_dim,
                                   rope_base);
    if (st != WF_OK)
        return st;
    st = check_prefill_layers(dt, n_tok, cap, d_in, n_kv_heads, head_dim, n_layers,
                              x_layer_stride, w_layer_stride, cache_layer_stride);
    if (st != WF_OK)
        return st;
    if (n_tok == 0)
        return WF_OK;
    if (!x || !w_k || !w_v || !k_cache || !v_cache)
        return WF_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(w_k) || !aligned16(w_v) ||
        !aligned16(k_cache) || !aligned16(v_cache))
        return WF_ERR_INVALID_ARG;
    const size_t need = wf::prefill_workspace_bytes(storage(dt), n_tok, d_in, n_kv_heads,
                                                    head_dim);
    if (need && (!workspace || workspace_bytes < need || !aligned16(workspace)))
        return WF_ERR_WORKSPACE;
    const bool one = n_layers == 1;
    return wf::launch_prefill(dt, x, w_k, w_v, k_cache, v_cache, n_tok, start_pos, cap, d_in,
                              n_kv_heads, head_dim, rope_base, workspace,
                              static_cast<hipStream_t>(stream), n_layers,
                              one ? 0 : (long long)x_layer_stride,
                              one ? 0 : (long long)w_layer_stride,
                              one ? 0 : (long long)cache_layer_stride);
}

size_t wf_lmhead_workspace_bytes(int32_t gamma, int32_t vocab) {
    if (gamma < 1 || gamma > kMaxGamma || vocab < 1 || vocab > (1 << 30))
        return 0;
    return wf::lmhead_workspace_bytes(gamma, vocab);
}

namespace {
// Shared checks of the two LM-head entry points (the head/logits inputs,
// outputs and workspace); the caller checks its own draft arguments.
wf_status_t check_lmhead(wf_dtype_t dt, const void *h, const void *w_lm,
                         const float *logits, int32_t gamma, int32_t d,
                         int32_t vocab, float tau_entropy,
                         const int32_t *argmax_out, const float *entropy_out,
                         const int32_t *accept_out, const void *workspace,
                         size_t workspace_bytes) {
    if (gamma < 1 || gamma > kMaxGamma || vocab < 1 || vocab > (1 << 30))
        return WF_ERR_INVALID_ARG;
    if (std::isnan(tau_entropy))
        return WF_ERR_INVALID_ARG;
    if (logits) {
        if (h || w_lm || !aligned16(logits))
            return WF_ERR_INVALID_ARG;
    } else {
        if (!weight_dtype_ok(dt) || !h || !w_lm || d < 1)
            return WF_ERR_INVALID_ARG;
        if (!aligned16(h) || !aligned16(w_lm))
            return WF_ERR_INVALID_ARG;
        if (is_bf16(dt) && d % 32 != 0)
            return WF_ERR_UNSUPPORTED;
        // tiled weights: only the persistent kernels read them
        if (dt == WF_BF16_TILED &&
            !((gamma <= 16 && (d == 4096 || d == 5120)) || d % 512 == 0))
            return WF_ERR_UNSUPPORTED;
    }
    if (!argmax_out || !entropy_out || !accept_out)
        return WF_ERR_INVALID_ARG;
    const size_t need = wf::lmhead_workspace_bytes(gamma, vocab);
    if (!workspace || workspace_bytes < need || !aligned16(workspace))
        return WF_ERR_WORKSPACE;
    return WF_OK;
}
}  // namespace

wf_status_t wf_lmhead_accept_entropy(wf_dtype_t dt, const void *h,
                                     const void *w_lm, const float *logits,
                                     const int32_t *draft, int32_t gamma,
                                     int32_t d, int32_t vocab,
                                     float tau_entropy, int32_t *argmax_out,
                                     float *entropy_out, int32_t *accept_out,
                                     void *workspace, size_t workspace_bytes,
                                     void *stream) {
    const wf_status_t st = check_lmhead(dt, h, w_lm, logits, gamma, d, vocab,
                                        tau_entropy, argmax_out, entropy_out,
                                        accept_out, workspace, workspace_bytes);
    if (st != WF_OK)
        return st;
    if (gamma > 1 && !draft)
        return WF_ERR_INVALID_ARG;
    return wf::launch_lmhead(dt, h, w_lm, logits, draft, nullptr, gamma, d,
                             vocab, tau_entropy, argmax_out, entropy_out,
                             accept_out, nullptr, workspace,
                             static_cast<hipStream_t>(stream));
}

wf_status_t wf_lmhead_accept_tree(wf_dtype_t dt, const void *h,
                                  const void *w_lm, const float *logits,
                                  const int32_t *tokens, const int32_t *parents,
                                  int32_t gamma, int32_t d, int32_t vocab,
                                  float tau_entropy, int32_t *argmax_out,
                                  float *entropy_out, int32_t *accept_out,
                                  int32_t *path_out, void *workspace,
                                  size_t workspace_bytes, void *stream) {
    const wf_status_t st = check_lmhead(dt, h, w_lm, logits, gamma, d, vocab,
                                        tau_entropy, argmax_out, entropy_out,
                                        accept_out, workspace, workspace_bytes);
    if (st != WF_OK)
        return st;
    if (!tokens || !parents || !path_out)
        return WF_ERR_INVALID_ARG;
    return wf::launch_lmhead(dt, h, w_lm, logits, tokens, parents, gamma, d,
                             vocab, tau_entropy, argmax_out, entropy_out,
                             accept_out, path_out, workspace,
                             static_cast<hipStream_t>(stream));
}

namespace {
size_t route_neural_ws(wf_dtype_t dt, int gamma, int vocab, int d, int m) {
    if (wf::lmhead_router_fusable(dt, gamma, d, m))
        return wf::lmhead_router_workspace_bytes(gamma, vocab, m);
    return std::max(wf::lmhead_workspace_bytes(gamma, vocab),
                    wf::router_workspace_bytes(storage(dt), gamma, d, m));
}
}  // namespace

size_t wf_lmhead_route_neural_workspace_bytes(wf_dtype_t dt, int32_t gamma, int32_t vocab,
                                              int32_t d, int32_t m) {
    if (!weight_dtype_ok(dt) || gamma < 1 || gamma > kMaxGamma || vocab < 1 ||
        vocab > (1 << 30) || d < 1 || m < 1 || m > kMaxRouterHidden)
        return 0;
    return route_neural_ws(dt, gamma, vocab, d, m);
}

wf_status_t wf_lmhead_accept_route_neural(wf_dtype_t dt, const void *h, const void *w_lm,
                                          const int32_t *draft, int32_t gamma, int32_t d,
                                          int32_t vocab, const void *w1, const void *b1,
                                          const void *w2, const void *b2, int32_t m,
                                          float tau_neural, int32_t *argmax_out,
                                          float *entropy_out, int32_t *accept_out,
                                          float *delta_out, void *workspace,
                                          size_t workspace_bytes, void *stream) {
    if (m < 1 || m > kMaxRouterHidden || !w1 || !b1 || !w2 || !b2 || !delta_out ||
        !aligned16(w1))
        return WF_ERR_INVALID_ARG;
    // the LM-head checks, with a workspace large enough for either schedule
    // (they are repeated below with the size this call needs)
    wf_status_t st = check_lmhead(dt, h, w_lm, nullptr, gamma, d, vocab, tau_neural,
                                  argmax_out, entropy_out, accept_out, workspace,
                                  ~(size_t)0);
    if (st != WF_OK)
        return st;
    if (gamma > 1 && !draft)
        return WF_ERR_INVALID_ARG;
    if (is_bf16(dt) && m % 16 != 0)
        return WF_ERR_UNSUPPORTED;
    if (!workspace || workspace_bytes < route_neural_ws(dt, gamma, vocab, d, m) ||
        !aligned16(workspace))
        return WF_ERR_WORKSPACE;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (wf::lmhead_router_fusable(dt, gamma, d, m)) {
        const wf::LmRouter r{w1, b1, w2, b2, m, tau_neural, delta_out};
        return wf::launch_lmhead(dt, h, w_lm, nullptr, draft, nullptr, gamma, d, vocab, 0.f,
                                 argmax_out, entropy_out, accept_out, nullptr, workspace, s, &r);
    }
    // other shapes: the LM head, then the separate router on row n (its
    // route replaces the entropy rule's in accept_out[2])
    if (dt == WF_BF16_TILED)
        return WF_ERR_UNSUPPORTED;
    st = wf::launch_lmhead(dt, h, w_lm, nullptr, draft, nullptr, gamma, d, vocab, 0.f,
                           argmax_out, entropy_out, accept_out, nullptr, workspace, s);
    if (st != WF_OK)
        return st;
    return wf::launch_router(dt, h, w1, b1, w2, b2, accept_out, gamma, d, m, tau_neural,
                             delta_out, accept_out + 2, workspace, s);
}

namespace {
wf_status_t check_router(wf_dtype_t dt, int gamma, int d, int m) {
    if (!dtype_ok(dt) || gamma < 1 || gamma > kMaxGamma || d < 1 || m < 1 ||
        m > kMaxRouterHidden)
        return WF_ERR_INVALID_ARG;
    if (dt == WF_BF16 && (d % 32 != 0 || m % 16 != 0))
        return WF_ERR_UNSUPPORTED;
    return WF_OK;
}
}  // namespace

size_t wf_router_workspace_bytes(wf_dtype_t dt, int32_t gamma, int32_t d,
                                 int32_t m) {
    if (check_router(dt, gamma, d, m) != WF_OK)
        return 0;
    return wf::router_workspace_bytes(dt, gamma, d, m);
}

wf_status_t wf_router_neural(wf_dtype_t dt, const void *h, const void *w1,
                             const void *b1, const void *w2, const void *b2,
                             const int32_t *row, int32_t gamma, int32_t d,
                             int32_t m, float tau_neural, float *delta_out,
                             int32_t *route_out, void *workspace,
                             size_t workspace_bytes, void *stream) {
    const wf_status_t st = check_router(dt, gamma, d, m);
    if (st != WF_OK)
        return st;
    if (std::isnan(tau_neural))
        return WF_ERR_INVALID_ARG;
    if (!h || !w1 || !b1 || !w2 || !b2 || !row || !delta_out || !route_out)
        return WF_ERR_INVALID_ARG;
    if (!aligned16(h) || !aligned16(w1))
        return WF_ERR_INVALID_ARG;
    const size_t need = wf::router_workspace_bytes(dt, gamma, d, m);
    if (!workspace || workspace_bytes < need || !aligned16(workspace))
        return WF_ERR_WORKSPACE;
    return wf::launch_router(dt, h, w1, b1, w2, b2, row, gamma, d, m, tau_neural,
                             delta_out, route_out, workspace,
                             static_cast<hipStream_t>(stream));
}

namespace {
// Shapes and pointers of a drafter layer call (the backlog or token count
// is checked by the caller).
wf_status_t check_drafter(wf_dtype_t dt, const wf_decoder_layer_t *L, int pos, int last_row,
                          int cap) {
    if (!weight_dtype_ok(dt) || !L)
        return WF_ERR_INVALID_ARG;
    if (L->hidden < 1 || L->inter < 1 || L->n_kv_heads < 1 || L->n_q_heads < 1 ||
        L->n_q_heads > kMaxQHeads || L->n_q_heads % L->n_kv_heads != 0)
        return WF_ERR_INVALID_ARG;
    if (pos < 0 || (long long)last_row >= cap || cap < 1)
        return WF_ERR_INVALID_ARG;
    if (!std::isfinite(L->rope_base) || L->rope_base <= 0.0 || !std::isfinite(L->rms_eps) ||
        L->rms_eps <= 0.f)
        return WF_ERR_INVALID_ARG;
    const void *ws[] = {L->attn_norm, L->w_q, L->w_k, L->w_v, L->w_o,
                        L->mlp_norm, L->w_gate, L->w_up, L->w_down};
    for (const void *p : ws)
        if (!p || !aligned16(p))
            return WF_ERR_INVALID_ARG;
    if (!is_bf16(dt) || !head_dim_ok(L->head_dim))
        return WF_ERR_UNSUPPORTED;
    if (L->hidden % 32 != 0 || L->inter % 32 != 0 || (L->n_q_heads * L->head_dim) % 32 != 0)
        return WF_ERR_UNSUPPORTED;
    return WF_OK;
}
}  // namespace

size_t wf_drafter_forward_workspace_bytes(wf_dtype_t dt, const wf_decoder_layer_t *layer,
                                          int32_t n_tok, int32_t pos) {
    if (n_tok < 1 || n_tok > kMaxGamma ||
        check_drafter(dt, layer, pos, pos + n_tok - 1, pos + n_tok) != WF_OK ||
        !wf::prefill_fits(n_tok, layer->hidden, layer->n_kv_heads, layer->head_dim))
        return 0;
    return wf::drafter_forward_workspace_bytes(*layer, n_tok, pos);
}

wf_status_t wf_drafter_forward(wf_dtype_t dt, const wf_decoder_layer_t *layer, const void *r,
                               int32_t n_tok, int32_t pos, void *k_cache, void *v_cache,
                               int32_t cap, void *out, void *workspace,
                               size_t workspace_bytes, void *stream) {
    if (n_tok < 1 || n_tok > kMaxGamma)
        return WF_ERR_INVALID_ARG;
    const wf_status_t st = check_drafter(dt, layer, pos, pos + n_tok - 1, cap);
    if (st != WF_OK)
        return st;
    if (!r || !k_cache || !v_cache || !out || !aligned16(r) || !aligned16(k_cache) ||
        !aligned16(v_cache) || !aligned16(out))
        return WF_ERR_INVALID_ARG;
    if (!wf::prefill_fits(n_tok, layer->hidden, layer->n_kv_heads, layer->head_dim))
        return WF_ERR_UNSUPPORTED;
    const size_t need = wf::drafter_forward_workspace_bytes(*layer, n_tok, pos);
    if (!workspace || workspace_bytes < need || !aligned16(workspace))
        return WF_ERR_WORKSPACE;
    return wf::launch_drafter_forward(*layer, r, n_tok, pos, k_cache, v_cache, cap, out,
                                      workspace, static_cast<hipStream_t>(stream),
                                      dt == WF_BF16_TILED);
}

namespace {
// Every KV-only prefill batch of a catch-up (full 4096-token batches and the
// last, shorter one) fits the prefill plan.
bool catchup_fits(int n, const wf_decoder_layer_t &L) {
    const int full = std::min(n, wf::kCatchupChunk), tail = n % wf::kCatchupChunk;
    return wf::prefill_fits(full, L.hidden, L.n_kv_heads, L.head_dim) &&
           (tail == 0 || wf::prefill_fits(tail, L.hidden, L.n_kv_heads, L.head_dim));
}
}  // namespace

size_t wf_drafter_catchup_workspace_bytes(wf_dtype_t dt, const wf_decoder_layer_t *layer,
                                          int32_t n_backlog, int32_t pos) {
    if (n_backlog < 1 || n_backlog > kMaxBacklog ||
        check_drafter(dt, layer, pos, pos + n_backlog - 1, pos + n_backlog) != WF_OK)
        return 0;
    if (!catchup_fits(n_backlog, *layer))
        return 0;
    return wf::drafter_catchup_workspace_bytes(*layer, n_backlog, pos);
}

wf_status_t wf_drafter_catchup(wf_dtype_t dt, const wf_decoder_layer_t *layer, const void *r,
                               int32_t n_backlog, int32_t pos, void *k_cache, void *v_cache,
                               int32_t cap, void *out, void *workspace,
                               size_t workspace_bytes, void *stream) {
    if (n_backlog < 1 || n_backlog > kMaxBacklog)
        return WF_ERR_INVALID_ARG;
    const wf_status_t st = check_drafter(dt, layer, pos, pos + n_backlog - 1, cap);
    if (st != WF_OK)
        return st;
    if (!r || !k_cache || !v_cache || !out || !aligned16(r) || !aligned16(k_cache) ||
        !aligned16(v_cache) || !aligned16(out))
        return WF_ERR_INVALID_ARG;
    if (!catchup_fits(n_backlog, *layer))
        return WF_ERR_UNSUPPORTED;
    const size_t need = wf::drafter_catchup_workspace_bytes(*layer, n_backlog, pos);
    if (!workspace || workspace_bytes < need || !aligned16(workspace))
        return WF_ERR_WORKSPACE;
    return wf::launch_drafter_catchup(*layer, r, n_backlog, pos, k_cache, v_cache, cap, out,
                                      workspace, static_cast<hipStream_t>(stream),
                                      dt == WF_BF16_TILED);
}

wf_status_t wf_kv_compact_path(wf_dtype_t dt, void *k_cache, void *v_cache,
                               const int32_t *accept, const int32_t *path,
                               int32_t gamma, int32_t ctx_len, int32_t cap,
                               int32_t n_kv_heads, int32_t head_dim,
                               int32_t n_layers, size_t layer_stride,
                               void *stream) {
    if (!dtype_ok(dt) || gamma < 1 || gamma > kMaxGamma || ctx_len < 0 ||
        (long long)ctx_len + gamma > cap || n_kv_heads < 1 ||
        n_kv_heads > kMaxQHeads || n_layers < 1 || n_layers > kMaxLayers)
        return WF_ERR_INVALID_ARG;
    if (n_layers > 1 &&
        layer_stride < (size_t)n_kv_heads * (size_t)cap * (size_t)head_dim)
        return WF_ERR_INVALID_ARG;
    if (n_layers > 1 && (layer_stride * (dt == WF_BF16 ? 2 : 4)) % 16 != 0)
        return WF_ERR_INVALID_ARG;
    if (!k_cache || !v_cache || !accept || !path)
        return WF_ERR_INVALID_ARG;
    if (!aligned16(k_cache) || !aligned16(v_cache))
        return WF_ERR_INVALID_ARG;
    if (!head_dim_ok(head_dim))
        return WF_ERR_UNSUPPORTED;
    return wf::launch_compact(dt, k_cache, v_cache, accept, path, gamma,
                              ctx_len, cap, n_kv_heads, head_dim, n_layers,
                              n_layers > 1 ? layer_stride : 0,
                              static_cast<hipStream_t>(stream));
}

size_t wf_tiled_weight_bytes(int32_t rows, int32_t cols) {
    if (rows < 1 || cols < 32 || cols % 32 != 0)
        return 0;
    return wf::tiled_weight_bytes(rows, cols);
}

wf_status_t wf_tile_weights(const void *w, int32_t rows, int32_t cols, void *tiled,
                            size_t tiled_bytes, void *stream) {
    if (!w || !tiled || !aligned16(w) || !aligned16(tiled) || rows < 1 || cols < 32 ||
        cols % 32 != 0)
        return WF_ERR_INVALID_ARG;
    const size_t need = wf::tiled_weight_bytes(rows, cols);
    if (tiled_bytes < need)
        return WF_ERR_WORKSPACE;
    const auto a = reinterpret_cast<uintptr_t>(w), b = reinterpret_cast<uintptr_t>(tiled);
    const size_t in_bytes = (size_t)rows * cols * 2;
    if (a < b + need && b < a + in_bytes)
        return WF_ERR_INVALID_ARG;                  // overlapping copies
    return wf::launch_tile_weights(w, rows, cols, tiled, static_cast<hipStream_t>(stream));
}

wf_status_t wf_read_probe(const void *src, size_t bytes, void *sink, size_t sink_bytes,
                          int32_t workgroups, void *stream) {
    if (!src || !sink || !aligned16(src) || !aligned16(sink) || bytes < 16 || bytes % 16 != 0 ||
        workgroups < 1 || workgroups > 65536)
        return WF_ERR_INVALID_ARG;
    if (sink_bytes < (size_t)workgroups * 4096)
        return WF_ERR_WORKSPACE;
    return wf::launch_read_probe(src, bytes, sink, workgroups, static_cast<hipStream_t>(stream));
}

wf_status_t wf_read_probe_series(const void *base, size_t bytes, size_t stride,
                                 int32_t n_bufs, int32_t reps, void *sink, size_t sink_bytes,
                                 int32_t workgroups, int32_t depth, void *stream) {
    if (!base || !sink || !aligned16(base) || !aligned16(sink) || bytes < 16 ||
        bytes % 16 != 0 || stride < bytes || stride % 16 != 0 || n_bufs < 1 || reps < 1 ||
        workgroups < 1 || workgroups > 65536 || (depth != 4 && depth != 8))
        return WF_ERR_INVALID_ARG;
    if (sink_bytes < (size_t)workgroups * 4096)
        return WF_ERR_WORKSPACE;
    return wf::launch_read_probe_series(base, bytes, stride, n_bufs, reps, sink, workgroups,
                                        depth, static_cast<hipStream_t>(stream));
}

wf_status_t wf_switch_init(wf_switch_state_t *s, int32_t active, int32_t lazy,
                           int32_t prompt_len) {
    if (!s || prompt_len < 0 || (active != WF_DRAFTER_AR && active != WF_DRAFTER_DIFFUSION) ||
        (lazy != 0 && lazy != 1))
        return WF_ERR_INVALID_ARG;
    *s = wf_switch_state_t{};
    s->active = active;
    s->lazy = lazy;
    s->committed = prompt_len;
    s->ar_cache_len = prompt_len;
    return WF_OK;
}

wf_status_t wf_switch_commit(wf_switch_state_t *s, int32_t n_new, int32_t next_drafter,
                             int32_t *start, int32_t *count) {
    if (!s || !start || !count || n_new < 1 ||
        (next_drafter != WF_DRAFTER_AR && next_drafter != WF_DRAFTER_DIFFUSION))
        return WF_ERR_INVALID_ARG;
    if (s->committed < 0 || s->ar_cache_len < 0 || s->ar_cache_len > s->committed ||
        (long long)s->committed + n_new > INT32_MAX)
        return WF_ERR_INVALID_ARG;
    const int32_t committed = s->committed + n_new;
    const bool due = !s->lazy || next_drafter == WF_DRAFTER_AR;
    const int32_t from = s->ar_cache_len;
    const int32_t n = due ? committed - from : 0;
    if (next_drafter == WF_DRAFTER_AR && s->active != WF_DRAFTER_AR)
        ++s->switches;
    s->committed = committed;
    s->active = next_drafter;
    if (n > 0) {
        s->ar_cache_len = committed;
        s->caught_up += n;
        ++s->catchups;
        s->max_backlog = std::max(s->max_backlog, n);
    }
    *start = from;
    *count = n;
    return WF_OK;
}

}  // extern "C"
