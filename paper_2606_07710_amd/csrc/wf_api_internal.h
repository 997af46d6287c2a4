// wf_api_internal.h -- host-side plumbing between the C ABI (api.hip) and
// the kernel launchers.  Internal header; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstddef>
#include <cstdint>

#include "wf.h"

namespace wf {

// Every workspace starts with a fixed zero block (the same offset and size
// for the three kinds of call) holding arrival counters and exchange slots,
// followed by that call's partial results.  Calls leave the block at zero,
// so a workspace zeroed once can be reused by any later call, whatever its
// kind or sizes.
constexpr size_t kCounterBytes = (size_t)4 << 20;
constexpr int kCounterSlots = static_cast<int>(kCounterBytes / sizeof(unsigned));

struct AttnPlan {
    int rows;            // G * gamma query rows per KV head
    int nb;              // 16-row blocks per wave (bf16 path)
    int rg;              // row groups of waves per workgroup
    int ks;              // key streams per workgroup
    int nbuf;            // LDS ring depth in stages of ks tiles (bf16 path)
    int n_row_groups;    // workgroup row groups of 16*nb*rg rows
    int splits;          // key splits per KV head
    int keys_per_split;  // multiple of the 32-key tile
    int part_bytes;      // bytes per partial-output element (bf16 path: 2)
};

AttnPlan plan_attn(wf_dtype_t dt, int gamma, int ctx_len, int n_q_heads,
                   int n_kv_heads, int head_dim, int num_splits);
size_t attn_workspace_bytes(const AttnPlan &p, int gamma, int n_q_heads,
                            int head_dim);
// Host-side checks of a verify-attention call (api.hip), everything but the
// workspace; on WF_OK *plan holds the split plan of the call.
wf_status_t validate_verify_attn(wf_dtype_t dt, const void *q, const void *k_cache,
                                 const void *v_cache, const void *out, int32_t gamma,
                                 int32_t ctx_len, int32_t cap, int32_t n_q_heads,
                                 int32_t n_kv_heads, int32_t head_dim, float softmax_scale,
                                 int32_t num_splits, AttnPlan *plan);
wf_status_t launch_attn(wf_dtype_t dt, const void *q, const void *k_cache,
                        const void *v_cache, void *out, int gamma, int ctx_len,
                        int cap, int n_q_heads, int n_kv_heads, int head_dim,
                        float softmax_scale, const uint64_t *tree_mask,
                        const AttnPlan &p, void *workspace, hipStream_t stream);

size_t lmhead_workspace_bytes(int gamma, int vocab);
// The neural routing policy folded into the LM-head pass (bf16 weights in
// the LM head's layout; b1, w2, b2 bf16): route = delta[n] > tau.
struct LmRouter {
    const void *w1, *b1, *w2, *b2;
    int m;
    float tau;
    float *delta_out;
};
// Shapes whose persistent LM-head kernel carries the router's W1 blocks.
bool lmhead_router_fusable(wf_dtype_t dt, int gamma, int d, int m);
size_t lmhead_router_workspace_bytes(int gamma, int vocab, int m);
// Chain mode: draft [gamma-1], parents == path_out == nullptr, accept_out
// [3].  Tree mode: draft = node tokens [gamma], parents [gamma], accept_out
// [4], path_out [gamma].  router: chain mode on a fusable shape only.
wf_status_t launch_lmhead(wf_dtype_t dt, const void *h, const void *w_lm,
                          const float *logits, const int32_t *draft,
                          const int32_t *parents, int gamma, int d, int vocab,
                          float tau, int32_t *argmax_out, float *entropy_out,
                          int32_t *accept_out, int32_t *path_out,
                          void *workspace, hipStream_t stream,
                          const LmRouter *router = nullptr);

// Skinny linear layer (gemv.hip): zpart[k][f][r] = sum over the k-th input
// slice of W[f] . x[r] for rows <= 64, features n_a + n_b (a multiple of
// 16; [0, n_a) from w_a, the rest from w_b) and k_in a multiple of 32.
int linear_slices(int k_in, int n_out);
constexpr int kLinearMaxSlices = 16;     // linear_slices never exceeds this
wf_status_t launch_linear_partial(const uint16_t *x, const uint16_t *w_a,
                                  const uint16_t *w_b, int n_a, int n_b, int rows,
                                  int k_in, float *zpart, hipStream_t stream,
                                  bool tiled = false);
// act[r][f] = bf16(SiLU(W_gate[f] . x[r]) * (W_up[f] . x[r])) in one launch,
// for 12..64 rows where the input dimension is not split (otherwise
// WF_ERR_UNSUPPORTED, and the caller takes launch_linear_partial and a
// separate SwiGLU pass, which give the same bits).
wf_status_t launch_linear_swiglu(const uint16_t *x, const uint16_t *w_gate,
                                 const uint16_t *w_up, int inter, int rows, int k_in,
                                 uint16_t *act, hipStream_t stream, bool tiled = false);

// Single-token skinny linear layers with their epilogue in the kernel
// (gemv.hip): y = res + W x; act = SiLU(Wg x') * (Wu x') with
// x' = RMSNorm(x) * gain.  n_out, inter multiples of 16, k_in of 32.
wf_status_t launch_linear_resid(const uint16_t *x, const uint16_t *w, const uint16_t *res,
                                int k_in, int n_out, uint16_t *y, hipStream_t stream,
                                bool tiled);
wf_status_t launch_linear_norm_swiglu(const uint16_t *x, const uint16_t *gain, float eps,
                                      const uint16_t *w_gate, const uint16_t *w_up, int k_in,
                                      int inter, uint16_t *act, hipStream_t stream,
                                      bool tiled);

// Neural routing policy: delta = w2 . GELU(W1 h + b1) + b2 for every row,
// route at the row *row names.
size_t router_workspace_bytes(wf_dtype_t dt, int gamma, int d, int m);
wf_status_t launch_router(wf_dtype_t dt, const void *h, const void *w1,
                          const void *b1, const void *w2, const void *b2,
                          const int32_t *row, int gamma, int d, int m, float tau,
                          float *delta_out, int32_t *route_out, void *workspace,
                          hipStream_t stream);

// Drafter layer and lazy catch-up (drafter.hip); bf16 only, the weight
// matrices row-major or (tiled) in 16x32 tiles.
// Backlogs longer than this are caught up in several KV-only prefill
// batches of at most this many tokens (the prefill's own limit).
constexpr int kCatchupChunk = 4096;
size_t drafter_forward_workspace_bytes(const wf_decoder_layer_t &L, int M, int pos);
size_t drafter_catchup_workspace_bytes(const wf_decoder_layer_t &L, int n, int pos);
wf_status_t launch_drafter_forward(const wf_decoder_layer_t &L, const void *r, int M, int pos,
                                   void *k_cache, void *v_cache, int cap, void *out,
                                   void *workspace, hipStream_t stream, bool tiled);
wf_status_t launch_drafter_catchup(const wf_decoder_layer_t &L, const void *r, int n, int pos,
                                   void *k_cache, void *v_cache, int cap, void *out,
                                   void *workspace, hipStream_t stream, bool tiled);

// Path compaction after tree acceptance: block rows path[t] -> t, t <= n,
// in n_layers caches layer_stride elements apart.
wf_status_t launch_compact(wf_dtype_t dt, void *k_cache, void *v_cache,
                           const int32_t *accept, const int32_t *path,
                           int gamma, int ctx_len, int cap, int n_kv_heads,
                           int head_dim, int n_layers, size_t layer_stride,
                           hipStream_t stream);

struct PrefillPlan {
    int nbt;             // 16-token blocks per workgroup
    int token_blocks;    // workgroups along the tokens
    int ppu;             // RoPE block pairs per work unit
    int units;           // (kv head, K|V, group of ppu RoPE block pairs) work units
    int ksplit;          // slices of the input dimension
    int chunks_per_split;
};

// beside_q: the plan of a prefill that shares its launch with the drafter
// catch-up's q projection (prefill_pair_bf16).
PrefillPlan plan_prefill(int n_tok, int d_in, int n_kv_heads, int head_dim, int n_layers = 1,
                         int kinds = 2, bool beside_q = false);
size_t prefill_workspace_bytes(wf_dtype_t dt, int n_tok, int d_in, int n_kv_heads,
                               int head_dim);
// Whether the bf16 plan's exchange slots fit the workspace zero block (and
// its grid the launch limits).
bool prefill_fits(int n_tok, int d_in, int n_kv_heads, int head_dim, int n_layers = 1);
// n_layers independent prefills in one launch: layer l reads x + l*x_ls,
// w_k/w_v + l*w_ls and writes the caches at + l*c_ls (element strides).
wf_status_t launch_prefill(wf_dtype_t dt, const void *x, const void *w_k,
                           const void *w_v, void *k_cache, void *v_cache,
                           int n_tok, int start_pos, int cap, int d_in,
                           int n_kv_heads, int head_dim, double rope_base,
                           void *workspace, hipStream_t stream, int n_layers = 1,
                           long long x_ls = 0, long long w_ls = 0, long long c_ls = 0,
                           bool x_tiled = false);

// Streaming-read probe (probe.hip): `workgroups` workgroups of 256 threads
// read [src, src + bytes) once; sink takes workgroups * 4 KB.
wf_status_t launch_read_probe(const void *src, size_t bytes, void *sink, int workgroups,
                              hipStream_t stream);
wf_status_t launch_read_probe_series(const void *base, size_t bytes, size_t stride, int n_bufs,
                                     int reps, void *sink, int workgroups, int depth,
                                     hipStream_t stream);

// q = RoPE(W_q x) for one token at position pos, q [n_heads][head_dim],
// on the KV-only prefill kernel (its exchange slots live in the workspace's
// zero block).
wf_status_t launch_q_rope(const uint16_t *x, const uint16_t *w_q, uint16_t *q, int d_in,
                          int n_heads, int head_dim, int pos, double rope_base,
                          void *workspace, hipStream_t stream, bool tiled);

// The KV-only prefill of n_tok tiled rows and q = RoPE(W_q x_last) in one
// launch (their exchange slots in the two halves of the zero block);
// WF_ERR_UNSUPPORTED if they do not fit there.
wf_status_t launch_prefill_and_q(bool tiled, const uint16_t *x_rows, const void *w_k,
                                 const void *w_v, void *k_cache, void *v_cache, int n_tok,
                                 int start_pos, int cap, int d_in, int n_kv_heads,
                                 const uint16_t *x_last, const uint16_t *w_q, uint16_t *q,
                                 int n_q_heads, int head_dim, int q_pos, double rope_base,
                                 void *workspace, hipStream_t stream);

// Tiled bf16 weights (16x32 tiles of 1 KB, one wave operand load each).
size_t tiled_weight_bytes(int rows, int cols);
wf_status_t launch_tile_weights(const void *w, int rows, int cols, void *tiled,
                                hipStream_t stream);

}  // namespace wf
