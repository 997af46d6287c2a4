/*
 * wf.h -- C ABI of libwf, the MI355X (gfx950) verification-step library for
 * WhiFlash cross-paradigm speculative decoding (arXiv 2606.07710).
 *
 * One speculation round of the paper (Sec. 3.2) drafts a block of tokens,
 * hands it to the target model for parallel verification, accepts the
 * longest prefix the target agrees with, and routes the next round by the
 * entropy of the target's next-token distribution at the final accepted
 * position (Sec. 3.3.1).  A drafter switch first catches the incoming
 * drafter's KV cache up on the backlog tokens with a KV-only prefill
 * (Sec. 3.4).  This library implements the three data-parallel pieces of
 * that step on one GPU:
 *
 *   wf_verify_attn            block-causal grouped-query attention of the
 *                             gamma verify rows against the KV cache
 *   wf_kv_only_prefill        K/V projection + RoPE + cache append for
 *                             catch-up tokens
 *   wf_kv_only_prefill_layers the same for several layers' caches in one
 *                             launch
 *   wf_lmhead_accept_entropy  LM head reduced to argmax and entropy per row,
 *                             then greedy acceptance and the entropy route
 *
 * and the tree-shaped variant of the step, for autoregressive drafters that
 * propose a tree of candidates (Sec. 3.1; EAGLE-3 trees of depth 8, top-k
 * 10, 60 draft tokens, App. A):
 *
 *   wf_verify_attn_tree       verify attention under a per-row ancestor mask
 *   wf_lmhead_accept_tree     LM head as above, then the deepest accepted
 *                             tree node, its root path and the route
 *   wf_kv_compact_path        moves the accepted path's K/V rows together
 *
 * and the learned routing policy, the alternative to the entropy rule:
 *
 *   wf_router_neural          two-layer MLP on the final hidden state ->
 *                             predicted acceptance-length gain and route
 *
 * and the drafter side of a switch (Sec. 3.4):
 *
 *   wf_drafter_catchup        lazy catch-up of a drafter's KV cache over the
 *                             backlog: KV-only prefill, then the full layer
 *                             for the last backlog token
 *   wf_drafter_forward        the drafter's full layer (attention + SwiGLU
 *                             MLP) for a few tokens
 *   wf_tile_weights           one-time copy of a weight into the tiled
 *                             layout the WF_BF16_TILED calls stream
 *   wf_switch_init/commit     host-side lazy catch-up bookkeeping: which
 *                             backlog is due after each round
 *
 * Conventions shared by every call
 *   - Every tensor pointer is DEVICE memory owned by the caller, 16-byte
 *     aligned, densely packed in the layout stated.  The library never
 *     allocates, frees or synchronises, and keeps no global state (the one
 *     exception, wf_verify_attn_noalloc, holds a static device array).
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream).  Outputs are valid once the stream reaches that point.
 *   - Arguments are validated on the host before anything is launched; on a
 *     non-OK status nothing was enqueued.  A failed kernel launch returns
 *     WF_ERR_HIP.
 *   - Workspaces are caller-owned scratch of at least the size the matching
 *     *_workspace_bytes query returns, ZERO-FILLED before their first use.
 *     Each starts with a 4 MiB zero block of arrival counters and exchange
 *     slots, through which workgroups of one call combine results; partial
 *     results follow that block.  Every call leaves the zero block at zero
 *     again, so a workspace zeroed once serves any later call, of any kind
 *     and any sizes.  Two calls that overlap in time must not share one.
 *   - Reductions use a fixed order, so repeated calls on the same inputs and
 *     the same split count return bit-identical results.
 *   - Row-major throughout; "[a][b][c]" lists dimensions slowest first.
 */
#ifndef WF_H
#define WF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    WF_OK = 0,
    WF_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, bad size or range  */
    WF_ERR_UNSUPPORTED = 2,   /* valid but not implemented (e.g. head_dim)    */
    WF_ERR_WORKSPACE = 3,     /* workspace missing or smaller than required   */
    WF_ERR_HIP = 4,           /* the HIP runtime rejected a kernel launch     */
    /* not statuses: they make every int32 value a valid wf_status_t, so a
     * caller may pass any int (unknown codes have a status string too) */
    WF_STATUS_RANGE_MIN_ = -2147483647 - 1,
    WF_STATUS_RANGE_MAX_ = 2147483647
} wf_status_t;

typedef enum {
    WF_F32 = 0,               /* IEEE fp32 storage and arithmetic             */
    WF_BF16 = 1,              /* bf16 storage, fp32 accumulation              */
    WF_BF16_TILED = 2,        /* as WF_BF16, with the WEIGHT matrices (W_k,
                                 W_v, W_lm, the drafter layer's projections)
                                 in the tiled layout that wf_tile_weights
                                 writes; activations, norm gains, caches and
                                 outputs stay row-major.  Accepted by the
                                 KV-only prefill, drafter and LM-head calls
                                 (the LM head where its bf16 kernels for
                                 gamma <= 16 and d in {4096, 5120}, or
                                 d % 512 == 0, apply; else
                                 WF_ERR_UNSUPPORTED) and nowhere else
                                 (WF_ERR_INVALID_ARG).  Results are bit-for-bit
                                 those of WF_BF16 on the untiled weights.     */
    /* not dtypes: every int32 value is a valid wf_dtype_t (an unknown code
     * is rejected with WF_ERR_INVALID_ARG) */
    WF_DTYPE_RANGE_MIN_ = -2147483647 - 1,
    WF_DTYPE_RANGE_MAX_ = 2147483647
} wf_dtype_t;

/* Version of this ABI (bumped on any signature or semantic change). */
int32_t wf_abi_version(void);

/* Static description of a status code; never NULL. */
const char *wf_status_string(wf_status_t s);

/* ------------------------------------------------------------------------
 * wf_verify_attn -- target attention over the verify block (Sec. 3.2: the
 * candidate tokens return to the target for one parallel verification
 * pass; the round then continues from the last accepted token).
 *
 * Block row i (0 <= i < gamma) sits at position ctx_len + i.  Row 0 is the
 * last committed token, rows 1..gamma-1 are the drafts, whether they came
 * from an autoregressive chain or a diffusion block.  Verification is causal
 * inside the block: row i attends to the ctx_len cached keys and to block
 * keys ctx_len .. ctx_len+i, so row i equals a single-token decode on prefix
 * ctx_len+i and gamma == 1 is ordinary decoding.  Query head h reads KV head
 * h / (n_q_heads / n_kv_heads) (consecutive query heads share a KV head).
 *
 *   out[i][h][:] = sum_j softmax_j(softmax_scale * <q[i][h], K[g][j]>) V[g][j]
 *
 * q        [gamma][n_q_heads][head_dim], RoPE already applied.
 * k_cache  [n_kv_heads][cap][head_dim], post-RoPE keys.  Rows
 *          [0, ctx_len+gamma) must be valid: the caller appends the block's
 *          own K/V at rows ctx_len.. before the call.  Rows beyond are never
 *          read.
 * v_cache  [n_kv_heads][cap][head_dim].
 * out      [gamma][n_q_heads][head_dim], dtype dt (bf16 rounded to nearest
 *          even once from fp32).
 * Limits:  1 <= gamma <= 64; ctx_len >= 0; ctx_len + gamma <= cap;
 *          n_q_heads % n_kv_heads == 0; n_q_heads <= 256;
 *          head_dim in {64, 128} (else WF_ERR_UNSUPPORTED).
 * num_splits  0 selects the split of the key range automatically; a
 *          positive value forces that many key splits per KV head (results
 *          agree to fp32 rounding for any split count).  At most 1024.
 * workspace  >= wf_verify_attn_workspace_bytes(...) bytes with the same
 *          num_splits.
 * ---------------------------------------------------------------------- */
wf_status_t wf_verify_attn(wf_dtype_t dt, const void *q, const void *k_cache,
                           const void *v_cache, void *out, int32_t gamma,
                           int32_t ctx_len, int32_t cap, int32_t n_q_heads,
                           int32_t n_kv_heads, int32_t head_dim,
                           float softmax_scale, int32_t num_splits,
                           void *workspace, size_t workspace_bytes,
                           void *stream);

/* Workspace for wf_verify_attn and wf_verify_attn_tree (0 for invalid
 * arguments). */
size_t wf_verify_attn_workspace_bytes(wf_dtype_t dt, int32_t gamma,
                                      int32_t ctx_len, int32_t n_q_heads,
                                      int32_t n_kv_heads, int32_t head_dim,
                                      int32_t num_splits);

/* ------------------------------------------------------------------------
 * wf_verify_attn_noalloc -- wf_verify_attn without a workspace argument,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 *
 * Same arguments, limits, kernels and results as wf_verify_attn (bit for bit
 * at the same num_splits), minus the workspace.  The split partials go to a
 * static device array of WF_NOALLOC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends; a call whose workspace query
 * (wf_verify_attn_workspace_bytes, same arguments) exceeds that size returns
 * WF_ERR_WORKSPACE without launching anything (the 32 MiB below hold the
 * 4 MiB zero block and 28 MiB of partials: 16 rows x 64 query heads at
 * head_dim 128 take 264 KiB per key split, so up to 108 splits; the
 * automatic plan uses 32).  The first
 * call on a device looks up the array's address there (with that device
 * current) and clears its zero block with a kernel on `stream`; no call
 * allocates or frees.  Every call on one GPU uses that GPU's single array:
 * calls that overlap in time on one GPU (different streams, threads) race,
 * so the caller orders them.
 * ---------------------------------------------------------------------- */
#define WF_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

wf_status_t wf_verify_attn_noalloc(wf_dtype_t dt, const void *q, const void *k_cache,
                                   const void *v_cache, void *out, int32_t gamma,
                                   int32_t ctx_len, int32_t cap, int32_t n_q_heads,
                                   int32_t n_kv_heads, int32_t head_dim,
                                   float softmax_scale, int32_t num_splits,
                                   void *stream);

/* ------------------------------------------------------------------------
 * wf_verify_attn_tree -- target attention over a draft tree (Sec. 3.1: an
 * autoregressive drafter proposes a tree of candidates; Sec. 3.2: the target
 * verifies them all in one parallel pass).
 *
 * Block row i is tree node i: row 0 is the root (the last committed token)
 * and every node's parent has a smaller index.  Node i's K/V sit at cache
 * row ctx_len + i (its RoPE position, ctx_len + depth(i), is the caller's).
 * Row i attends to the ctx_len cached keys and to the block keys
 * ctx_len + j for j == i and for every j with bit j of tree_mask[i] set;
 * with tree_mask[i] = the ancestors of i this is causal attention along
 * node i's root path, and a chain (parent of j = j-1) gives exactly
 * wf_verify_attn.  Bits at or above gamma are ignored.
 *
 * tree_mask  [gamma] uint64, device memory, 16-byte aligned.
 * Everything else as for wf_verify_attn (same limits, same workspace
 * query); block rows a row does not see still have to hold finite values.
 * ---------------------------------------------------------------------- */
wf_status_t wf_verify_attn_tree(wf_dtype_t dt, const void *q,
                                const void *k_cache, const void *v_cache,
                                void *out, const uint64_t *tree_mask,
                                int32_t gamma, int32_t ctx_len, int32_t cap,
                                int32_t n_q_heads, int32_t n_kv_heads,
                                int32_t head_dim, float softmax_scale,
                                int32_t num_splits, void *workspace,
                                size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * wf_kv_only_prefill -- lazy catch-up of a drafter's KV cache (Sec. 3.4).
 * On a drafter switch, the tokens accepted while that drafter was inactive
 * (the backlog) are prefilled in one batch, and for them only the attention
 * layer's K/V are formed: no MLP, no LM head.  Token t is at position
 * start_pos + t:
 *
 *   K[g][start_pos+t][:] = RoPE(W_k[g*D:(g+1)*D][:] x[t], start_pos + t)
 *   V[g][start_pos+t][:] =      W_v[g*D:(g+1)*D][:] x[t]
 *
 * RoPE is the rotate-half form: for i < D/2, theta_i = rope_base^(-2i/D)
 * and the pair (k_i, k_{i+D/2}) turns by (start_pos+t)*theta_i radians
 * (angles formed in fp64).
 *
 * x         [n_tok][d_in], the layer input after RMSNorm.
 * w_k, w_v  [n_kv_heads*head_dim][d_in] each (output feature major);
 *           with WF_BF16_TILED their tiled copies (wf_tile_weights).
 * k_cache, v_cache  [n_kv_heads][cap][head_dim]; only rows
 *           [start_pos, start_pos+n_tok) are written (bf16 for both bf16
 *           dtypes, else fp32).
 * Limits:   0 <= n_tok <= 4096 (0 is a no-op); start_pos >= 0;
 *           start_pos + n_tok <= cap; head_dim in {64, 128};
 *           d_in >= 1, and d_in % 32 == 0 for the bf16 dtypes.
 * workspace >= wf_kv_only_prefill_workspace_bytes(...) bytes (may be NULL
 *           when that is 0: fp32, or no tokens).  The bf16 path splits the
 *           input dimension across a power-of-two number of workgroups whose
 *           sums meet up a fixed binary tree (deterministic), using exchange
 *           slots in the workspace's zero block.
 * ---------------------------------------------------------------------- */
wf_status_t wf_kv_only_prefill(wf_dtype_t dt, const void *x, const void *w_k,
                               const void *w_v, void *k_cache, void *v_cache,
                               int32_t n_tok, int32_t start_pos, int32_t cap,
                               int32_t d_in, int32_t n_kv_heads,
                               int32_t head_dim, double rope_base,
                               void *workspace, size_t workspace_bytes,
                               void *stream);

/* Workspace for wf_kv_only_prefill (0 when none is needed or for invalid
 * arguments). */
size_t wf_kv_only_prefill_workspace_bytes(wf_dtype_t dt, int32_t n_tok,
                                          int32_t d_in, int32_t n_kv_heads,
                                          int32_t head_dim);

/* The same catch-up for n_layers caches in one launch (Sec. 3.4: the
 * backlog is processed in one batch; the layers' K/V projections are
 * independent of each other once their inputs are known).  Layer l reads
 * x + l*x_layer_stride, w_k/w_v + l*w_layer_stride and writes
 * k_cache/v_cache + l*cache_layer_stride (strides in ELEMENTS; all other
 * arguments and the per-layer result exactly as wf_kv_only_prefill's).
 * Limits as wf_kv_only_prefill's, and 1 <= n_layers <= 1024; with
 * n_layers > 1 the strides must be at least one layer's x [n_tok][d_in],
 * W [n_kv_heads*head_dim][d_in] and cache [n_kv_heads][cap][head_dim] (no
 * two layers overlap) and keep every layer 16-byte aligned, else
 * WF_ERR_INVALID_ARG.  With many layers the launch has enough workgroups
 * without splitting the input dimension, so the bf16 sums may be formed in
 * a different (still fixed) order than a single-layer call's.
 * workspace >= wf_kv_only_prefill_layers_workspace_bytes(...) bytes. */
wf_status_t wf_kv_only_prefill_layers(wf_dtype_t dt, const void *x,
                                      const void *w_k, const void *w_v,
                                      void *k_cache, void *v_cache,
                                      int32_t n_tok, int32_t start_pos,
                                      int32_t cap, int32_t d_in,
                                      int32_t n_kv_heads, int32_t head_dim,
                                      double rope_base, int32_t n_layers,
                                      size_t x_layer_stride,
                                      size_t w_layer_stride,
                                      size_t cache_layer_stride,
                                      void *workspace, size_t workspace_bytes,
                                      void *stream);
size_t wf_kv_only_prefill_layers_workspace_bytes(wf_dtype_t dt, int32_t n_tok,
                                                 int32_t d_in,
                                                 int32_t n_kv_heads,
                                                 int32_t head_dim,
                                                 int32_t n_layers);

/* ------------------------------------------------------------------------
 * wf_lmhead_accept_entropy -- LM head, greedy acceptance and entropy route.
 *
 * For every verify row i the target's next-token logits z_i = W h_i are
 * reduced on the fly (never written out) to
 *   argmax_out[i]  = lowest index attaining max_v z_i[v]
 *   entropy_out[i] = -sum_v p_i(v) log p_i(v), p_i = softmax(z_i), in nats
 * (Sec. 3.3.1: an O(|V|) reduction over the next-token distribution).
 * Then greedy verification accepts the longest prefix of drafts the target
 * agrees with, and the entropy at the final accepted position picks the
 * next drafter (Sec. 3.3.1 rule: autoregressive iff H_t > tau):
 *   n     = number of j in 0.. with draft[j] == argmax[j] for all earlier j,
 *           at most gamma-1
 *   accept_out = { n, bonus token argmax[n], route (1 = AR, 0 = diffusion)
 *                  = entropy[n] > tau_entropy }
 *
 * h         [gamma][d] final-norm hidden states of the verify rows.
 * w_lm      [vocab][d] LM-head weight (one row per vocabulary entry).
 * logits    logits-only mode: [gamma][vocab] fp32 given directly, with
 *           h == w_lm == NULL; dt and d are then ignored.  Otherwise NULL.
 * draft     [gamma-1] int32: draft[j] is the token at block row j+1, checked
 *           against the argmax of row j.  May be NULL only when gamma == 1.
 * argmax_out [gamma] int32, entropy_out [gamma] fp32, accept_out [3] int32.
 * w_lm with WF_BF16_TILED: its tiled copy (wf_tile_weights; rows padded to
 *           a multiple of 16, so the buffer holds ceil(vocab/16)*16 rows).
 * Limits:   1 <= gamma <= 64; 1 <= vocab <= 2^30; d >= 1, and
 *           d % 32 == 0 for the bf16 dtypes; WF_BF16_TILED needs
 *           gamma <= 16 with d in {4096, 5120}, or d % 512 == 0
 *           (else WF_ERR_UNSUPPORTED).
 * workspace >= wf_lmhead_workspace_bytes(gamma, vocab) bytes.
 * ---------------------------------------------------------------------- */
wf_status_t wf_lmhead_accept_entropy(wf_dtype_t dt, const void *h,
                                     const void *w_lm, const float *logits,
                                     const int32_t *draft, int32_t gamma,
                                     int32_t d, int32_t vocab,
                                     float tau_entropy, int32_t *argmax_out,
                                     float *entropy_out, int32_t *accept_out,
                                     void *workspace, size_t workspace_bytes,
                                     void *stream);

/* Workspace for wf_lmhead_accept_entropy and wf_lmhead_accept_tree (0 for
 * invalid arguments). */
size_t wf_lmhead_workspace_bytes(int32_t gamma, int32_t vocab);

/* ------------------------------------------------------------------------
 * wf_lmhead_accept_tree -- LM head and greedy acceptance on a draft tree
 * (the tree of Sec. 3.1 verified as in Sec. 3.2; route rule of Sec. 3.3.1).
 *
 * argmax_out and entropy_out per row (tree node) exactly as for
 * wf_lmhead_accept_entropy.  Then: the root (node 0) is accepted; node
 * j >= 1 is accepted iff its parent p = parents[j] satisfies 0 <= p < j, p
 * is accepted and tokens[j] == argmax[p] (a node with an out-of-range parent
 * is never accepted).  The accepted node b of greatest depth (lowest index
 * among equals) ends the accepted path:
 *   accept_out = { n = depth(b) (accepted drafts), bonus = argmax[b],
 *                  route = entropy[b] > tau_entropy (1 = AR), b }
 *   path_out[t] = node at depth t on b's root path for t <= n, -1 after.
 *
 * tokens    [gamma] int32: the drafted token of each node (tokens[0], the
 *           root's, is not compared).
 * parents   [gamma] int32: parent index of each node (parents[0] ignored).
 * accept_out [4] int32; path_out [gamma] int32.  Other arguments, limits
 * and the workspace as for wf_lmhead_accept_entropy.
 * ---------------------------------------------------------------------- */
wf_status_t wf_lmhead_accept_tree(wf_dtype_t dt, const void *h,
                                  const void *w_lm, const float *logits,
                                  const int32_t *tokens, const int32_t *parents,
                                  int32_t gamma, int32_t d, int32_t vocab,
                                  float tau_entropy, int32_t *argmax_out,
                                  float *entropy_out, int32_t *accept_out,
                                  int32_t *path_out, void *workspace,
                                  size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * wf_kv_compact_path -- after tree acceptance, move the accepted path's K/V
 * rows to consecutive cache rows after the prefix, so the cache again holds
 * the committed sequence in order, in every layer at once:
 *   K_l[g][ctx_len + t] <- K_l[g][ctx_len + path[t]]   (and V), t = 0..n
 * with n = accept[0].  Both are read on the device (accept_out and path_out
 * of wf_lmhead_accept_tree), so the call can follow it on the same stream
 * without a host round trip.  A path entry outside [t, gamma) leaves row t
 * unchanged; rows other than ctx_len .. ctx_len+n are never written.
 *
 * k_cache, v_cache  layer 0's [n_kv_heads][cap][head_dim] cache, dtype dt;
 *          layer l's starts l * layer_stride elements further on.
 * accept  device int32, at least 1 entry; path  [gamma] device int32.
 * Limits: 1 <= gamma <= 64; ctx_len >= 0; ctx_len + gamma <= cap;
 *         head_dim in {64, 128}; 1 <= n_layers <= 1024; for n_layers > 1,
 *         layer_stride >= n_kv_heads * cap * head_dim and a multiple of 16
 *         bytes (ignored when n_layers == 1).
 * ---------------------------------------------------------------------- */
wf_status_t wf_kv_compact_path(wf_dtype_t dt, void *k_cache, void *v_cache,
                               const int32_t *accept, const int32_t *path,
                               int32_t gamma, int32_t ctx_len, int32_t cap,
                               int32_t n_kv_heads, int32_t head_dim,
                               int32_t n_layers, size_t layer_stride,
                               void *stream);

/* ------------------------------------------------------------------------
 * wf_router_neural -- the neural routing policy (Sec. 3.3.2; architecture
 * in the appendix on the neural router).  A two-layer MLP regressor on the
 * target's final hidden state predicts the acceptance-length gain of the
 * autoregressive drafter over the diffusion drafter, and the next round uses
 * the autoregressive drafter iff the gain exceeds tau_neural:
 *   delta_out[r] = w2 . GELU(W1 h[r] + b1) + b2   for every row r,
 *   GELU(x) = 0.5 x (1 + erf(x / sqrt 2))  (exact form; no dropout),
 *   route_out[0] = delta_out[row[0]] > tau_neural   (1 = AR, 0 = diffusion).
 *
 * h        [gamma][d] final-norm hidden states of the verify rows (the
 *          LM head's input).
 * w1 [m][d], b1 [m], w2 [m], b2 [1]: the router's weights, dtype dt like h
 *          (the paper's router has m = d/8).
 * row      device int32: the row to route on, usually the final accepted
 *          position written by the acceptance call (accept_out + 0 for
 *          chains and blocks, accept_out + 3 for trees); clamped to
 *          [0, gamma).
 * delta_out [gamma] fp32; route_out [1] int32.
 * Limits:  1 <= gamma <= 64; d >= 1 and m >= 1 (m <= 65536); for WF_BF16
 *          d % 32 == 0 and m % 16 == 0.  h and w1 16-byte aligned.
 * workspace >= wf_router_workspace_bytes(dt, gamma, d, m) bytes.
 * ---------------------------------------------------------------------- */
wf_status_t wf_router_neural(wf_dtype_t dt, const void *h, const void *w1,
                             const void *b1, const void *w2, const void *b2,
                             const int32_t *row, int32_t gamma, int32_t d,
                             int32_t m, float tau_neural, float *delta_out,
                             int32_t *route_out, void *workspace,
                             size_t workspace_bytes, void *stream);

/* Workspace for wf_router_neural (0 for invalid arguments). */
size_t wf_router_workspace_bytes(wf_dtype_t dt, int32_t gamma, int32_t d,
                                 int32_t m);

/* ------------------------------------------------------------------------
 * wf_lmhead_accept_route_neural -- the LM-head call of a chain/block round
 * (wf_lmhead_accept_entropy: argmax, entropy, greedy acceptance) with the
 * neural routing policy of Sec. 3.3.2 in place of the entropy rule: both
 * read the same final hidden states h, so the router's hidden layer W1 h is
 * formed in the same pass as the logits -- W1's m rows stream after the
 * vocabulary as extra 16-row blocks of the LM-head kernel -- and the finish
 * forms delta[r] = w2 . GELU(W1 h[r] + b1) + b2 (exact erf GELU) for every
 * row and routes on the final accepted row n: accept_out[2] = delta[n] >
 * tau_neural (strict), so routing adds no launch of its own.
 *
 * Arguments as wf_lmhead_accept_entropy (h, w_lm, draft, gamma, d, vocab,
 * argmax_out, entropy_out, accept_out; no logits-only mode) and as
 * wf_router_neural (w1 [m][d] in the layout dt names for the weights -- tiled
 * for WF_BF16_TILED, like w_lm -- b1, w2 [m], b2 [1] in the activations'
 * storage; delta_out [gamma] fp32).  The pass carries the router for bf16
 * weights with gamma <= 16, d in {4096, 5120} and m % 16 == 0; other shapes
 * run the LM head and then wf_router_neural's kernels on row n (not for
 * WF_BF16_TILED: WF_ERR_UNSUPPORTED).
 * workspace >= wf_lmhead_route_neural_workspace_bytes(...) bytes, zeroed
 * before first use (as every workspace).
 * ---------------------------------------------------------------------- */
wf_status_t wf_lmhead_accept_route_neural(wf_dtype_t dt, const void *h, const void *w_lm,
                                          const int32_t *draft, int32_t gamma, int32_t d,
                                          int32_t vocab, const void *w1, const void *b1,
                                          const void *w2, const void *b2, int32_t m,
                                          float tau_neural, int32_t *argmax_out,
                                          float *entropy_out, int32_t *accept_out,
                                          float *delta_out, void *workspace,
                                          size_t workspace_bytes, void *stream);

/* Workspace for wf_lmhead_accept_route_neural (0 for invalid arguments). */
size_t wf_lmhead_route_neural_workspace_bytes(wf_dtype_t dt, int32_t gamma, int32_t vocab,
                                              int32_t d, int32_t m);

/* ------------------------------------------------------------------------
 * Drafter layer and lazy catch-up (Sec. 3.4: "Lazy Catch-up" defers the
 * inactive drafter's cache updates until the router switches to it, then
 * processes the backlog in one batch; "KV-only Prefill" forms only the
 * attention layer's K/V for the backlog -- all of it but the last token,
 * whose hidden state the next draft starts from).
 *
 * A drafter layer (one pre-norm decoder layer, bf16 weights in nn.Linear
 * layout; pointers are device memory, the struct itself host memory read
 * during the call):
 *   xn  = RMSNorm(r) * attn_norm;  q, k, v = W_q xn, W_k xn, W_v xn with
 *   rotate-half RoPE on q and k at the token's position (theta_i =
 *   rope_base^(-2i/D), angles in fp64);  k, v -> cache rows;
 *   a   = causal grouped-query attention over the cache (scale 1/sqrt(D));
 *   h1  = r + W_o a;  xn2 = RMSNorm(h1) * mlp_norm;
 *   out = h1 + W_down (SiLU(W_gate xn2) * (W_up xn2)).
 * Activations are stored in bf16 between these steps.
 * ---------------------------------------------------------------------- */
typedef struct wf_decoder_layer {
    const void *attn_norm;   /* [hidden] */
    const void *w_q;         /* [n_q_heads*head_dim][hidden] */
    const void *w_k;         /* [n_kv_heads*head_dim][hidden] */
    const void *w_v;         /* [n_kv_heads*head_dim][hidden] */
    const void *w_o;         /* [hidden][n_q_heads*head_dim] */
    const void *mlp_norm;    /* [hidden] */
    const void *w_gate;      /* [inter][hidden] */
    const void *w_up;        /* [inter][hidden] */
    const void *w_down;      /* [hidden][inter] */
    int32_t hidden, n_q_heads, n_kv_heads, head_dim, inter;
    float rms_eps;
    double rope_base;
} wf_decoder_layer_t;

/* The full layer for n_tok tokens at positions pos .. pos+n_tok-1 (causal
 * among them).  r [n_tok][hidden] is the layer input (pre-norm residual
 * stream); the tokens' K/V are written to cache rows pos .. pos+n_tok-1 and
 * attention reads rows [0, pos + t]; out [n_tok][hidden].
 * Limits: dt == WF_BF16 or WF_BF16_TILED (the seven projections tiled;
 *         else WF_ERR_UNSUPPORTED); 1 <= n_tok <= 64;
 *         pos >= 0; pos + n_tok <= cap; head_dim in {64, 128};
 *         n_q_heads % n_kv_heads == 0; hidden, inter and
 *         n_q_heads*head_dim multiples of 32; weights, r, out and the
 *         caches 16-byte aligned.
 * workspace >= wf_drafter_forward_workspace_bytes(...) bytes, zero-filled
 *         before first use like every workspace (its zero block comes
 *         first). */
wf_status_t wf_drafter_forward(wf_dtype_t dt, const wf_decoder_layer_t *layer,
                               const void *r, int32_t n_tok, int32_t pos,
                               void *k_cache, void *v_cache, int32_t cap,
                               void *out, void *workspace,
                               size_t workspace_bytes, void *stream);
size_t wf_drafter_forward_workspace_bytes(wf_dtype_t dt,
                                          const wf_decoder_layer_t *layer,
                                          int32_t n_tok, int32_t pos);

/* Lazy catch-up over a backlog of n_backlog tokens whose layer inputs are
 * r [n_backlog][hidden], starting at cache row pos: RMSNorm(r[t]) *
 * attn_norm for the whole backlog in one batch and KV-only prefill in one
 * batch per 4096 tokens (cache rows pos .. pos+n_backlog-1), then the rest
 * of the layer -- attention, W_o, the MLP -- for the last token only;
 * out [hidden] is its output.  The cache rows and out equal those of
 * wf_drafter_forward over the whole backlog (to rounding).  Limits as for
 * wf_drafter_forward, with 1 <= n_backlog <= 2^20 and pos + n_backlog <= cap,
 * so any backlog wf_switch_commit hands out (up to the cache capacity) is
 * accepted.
 * workspace >= wf_drafter_catchup_workspace_bytes(...) bytes. */
wf_status_t wf_drafter_catchup(wf_dtype_t dt, const wf_decoder_layer_t *layer,
                               const void *r, int32_t n_backlog, int32_t pos,
                               void *k_cache, void *v_cache, int32_t cap,
                               void *out, void *workspace,
                               size_t workspace_bytes, void *stream);
size_t wf_drafter_catchup_workspace_bytes(wf_dtype_t dt,
                                          const wf_decoder_layer_t *layer,
                                          int32_t n_backlog, int32_t pos);

/* ------------------------------------------------------------------------
 * Tiled weight layout (WF_BF16_TILED).  A bf16 weight W [rows][cols]
 * (nn.Linear layout, cols % 32 == 0) is stored as 1 KB tiles of 16 rows x
 * 32 columns: tile (rb, c), rb < ceil(rows/16), c < cols/32, starts at
 * element (rb * cols/32 + c) * 512, and inside it element
 * (16*q + r) * 8 + e holds W[16*rb + r][32*c + 8*q + e] (r < 16, q < 4,
 * e < 8); rows past `rows` are zero.  Each tile is exactly one MFMA operand
 * load of a wave (lane 16*q + r takes 16 contiguous bytes), so the kernels
 * stream a weight in contiguous 1 KB pieces instead of 64-byte pieces of 16
 * rows.  A one-time transform of static weights (at model load), like any
 * inference engine's weight preprocessing.
 * ---------------------------------------------------------------------- */
/* Bytes of the tiled copy of a bf16 [rows][cols] weight (0 if rows < 1,
 * cols < 32 or cols % 32 != 0). */
size_t wf_tiled_weight_bytes(int32_t rows, int32_t cols);

/* Writes the tiled copy of the bf16 weight w [rows][cols] into `tiled`
 * (device, tiled_bytes >= wf_tiled_weight_bytes(rows, cols), 16-byte
 * aligned, must not overlap w).  Layer stacks: tile each layer's matrix into
 * its own slot (the tiled size equals the untiled one when rows % 16 == 0).
 * WF_ERR_INVALID_ARG on null/misaligned pointers or bad sizes,
 * WF_ERR_WORKSPACE if tiled_bytes is too small. */
wf_status_t wf_tile_weights(const void *w, int32_t rows, int32_t cols,
                            void *tiled, size_t tiled_bytes, void *stream);

/* ------------------------------------------------------------------------
 * wf_read_probe -- measurement support, not a step of the method: reads
 * [src, src + bytes) once with a plain streaming kernel (workgroups x 256
 * threads striding through the buffer together, 32 KB per workgroup and
 * round, 16-byte loads, 8 in flight per thread) and writes an XOR of what it
 * read to sink, so the loads cannot be dropped.  Timing it over a buffer larger than the 256 MB last-level
 * cache gives the HBM read rate a plain stream reaches, the ceiling the
 * benchmark compares the kernels with.  src, sink: device, 16-byte aligned;
 * bytes a positive multiple of 16; 1 <= workgroups <= 65536;
 * sink_bytes >= workgroups * 4096 (else WF_ERR_WORKSPACE).
 * ---------------------------------------------------------------------- */
wf_status_t wf_read_probe(const void *src, size_t bytes, void *sink, size_t sink_bytes,
                          int32_t workgroups, void *stream);

/* ------------------------------------------------------------------------
 * wf_read_probe_series -- measurement support, not a step of the method:
 * reps rounds over the n_bufs buffers [base + i * stride, + bytes),
 * i = 0 .. n_bufs - 1, each read once per round by the kernel of
 * wf_read_probe with `depth` (4 or 8) loads in flight per thread, all
 * launched back to back from the library (a caller's own launch rate would
 * otherwise limit short reads).  Timed over buffers that together exceed
 * the 256 MB last-level cache, it gives the time a plain read of `bytes`
 * takes on its own: the floor for a kernel that must move that many bytes,
 * launch, first-byte latency and drain included.  base, sink: device,
 * 16-byte aligned; bytes a positive multiple of 16; stride >= bytes and a
 * multiple of 16; n_bufs, reps >= 1; 1 <= workgroups <= 65536; sink_bytes
 * >= workgroups * 4096 (else WF_ERR_WORKSPACE).  Asynchronous on stream.
 * ---------------------------------------------------------------------- */
wf_status_t wf_read_probe_series(const void *base, size_t bytes, size_t stride,
                                 int32_t n_bufs, int32_t reps, void *sink, size_t sink_bytes,
                                 int32_t workgroups, int32_t depth, void *stream);

/* ------------------------------------------------------------------------
 * Lazy catch-up bookkeeping (Sec. 3.4 and its lazy catch-up study in
 * Sec. 4): a host-side record of how far the autoregressive drafter's KV
 * cache lags the committed sequence.  Only that drafter's cache can fall
 * behind: it is the one whose per-token K/V the next draft attends over.
 * Host memory only; no GPU work.  Under lazy catch-up nothing is due while
 * the diffusion drafter is active, and the whole backlog is due in one batch
 * when the router switches back; the naive scheme it is compared with keeps
 * the cache current every round.  The caller runs each due backlog through
 * wf_drafter_catchup (r = the backlog tokens' layer inputs, pos = start).
 * ---------------------------------------------------------------------- */
#define WF_DRAFTER_AR 0          /* autoregressive drafter (its cache lags)  */
#define WF_DRAFTER_DIFFUSION 1   /* diffusion (parallel) drafter             */

typedef struct wf_switch_state {
    int32_t active;        /* drafter of the next round: WF_DRAFTER_*        */
    int32_t lazy;          /* 1: lazy catch-up; 0: update every round        */
    int32_t committed;     /* tokens in the sequence (prompt + accepted)     */
    int32_t ar_cache_len;  /* rows in the AR drafter's KV cache              */
    int32_t switches;      /* rounds that switched to the AR drafter         */
    int32_t max_backlog;   /* largest backlog handed out so far              */
    int64_t caught_up;     /* tokens handed out for catch-up so far          */
    int64_t catchups;      /* backlogs handed out so far (catch-up calls)    */
} wf_switch_state_t;

/* Start of a sequence: both drafters have processed the prompt_len prompt
 * tokens; `active` drafts the first round.  WF_ERR_INVALID_ARG on a null
 * state, prompt_len < 0, active or lazy out of range. */
wf_status_t wf_switch_init(wf_switch_state_t *s, int32_t active, int32_t lazy,
                           int32_t prompt_len);

/* After a verify round: n_new >= 1 tokens joined the sequence (the accepted
 * drafts plus the bonus token, i.e. accept_out[0] + 1) and the router chose
 * next_drafter for the next round.  *start and *count receive the backlog
 * now due -- cache rows and positions start .. start+count-1 -- with
 * count = 0 when none is.  Lazy: due iff next_drafter is WF_DRAFTER_AR, and
 * then it is every token since the cache last caught up; naive: the round's
 * n_new tokens are due every round.  The state records the backlog as
 * handed out (the caller must run it before the AR drafter drafts again).
 * WF_ERR_INVALID_ARG (state unchanged) on null pointers, n_new < 1,
 * next_drafter out of range, or a sequence length past INT32_MAX. */
wf_status_t wf_switch_commit(wf_switch_state_t *s, int32_t n_new,
                             int32_t next_drafter, int32_t *start,
                             int32_t *count);

#ifdef __cplusplus
}
#endif

#endif /* WF_H */
