/*
 * wfref.c -- the CPU oracle for the WhiFlash target-verification step.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, fp64 restatement of
 * what the verification step computes, used to judge the GPU library.  Only
 * the test suite, the smoke check and the CPU-baseline leg of the benchmark
 * may load it; the product path never does.  It shares no code, header,
 * table or helper with the GPU library.
 *
 * Paper: "WhiFlash: Accelerating Speculative Decoding with Token-Level
 * Cross-Paradigm Routing" (arXiv 2606.07710).
 *
 * Every function below is the plain definition written out: no tiling, no
 * online softmax, no split of the key range, no fused reductions.  All
 * arithmetic is fp64; inputs are read from their stored precision
 * (fp32, bf16 or fp64) exactly, bit for bit.
 *
 * Parallelism: OpenMP over independent output rows only; the order of every
 * sum is the plain ascending index order, so results do not depend on the
 * thread count.
 *
 * Pins: each function is checked in tests/test_oracle_*.py against closed
 * forms, invariants, brute force and library routines (torch / numpy /
 * scipy on the CPU).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Storage codes of the inputs handed to the oracle. */
enum { WFREF_F32 = 0, WFREF_BF16 = 1, WFREF_F64 = 2 };

/* Read element idx of an array stored as fp32, bf16 (raw 16-bit pattern =
 * the upper half of an IEEE fp32) or fp64, widened exactly to double. */
static double elem(const void *base, int dtype, size_t idx)
{
    if (dtype == WFREF_F32)
        return (double)((const float *)base)[idx];
    if (dtype == WFREF_F64)
        return ((const double *)base)[idx];
    uint32_t bits = ((uint32_t)((const uint16_t *)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static int valid_dtype(int dtype)
{
    return dtype == WFREF_F32 || dtype == WFREF_BF16 || dtype == WFREF_F64;
}

int wfref_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ *
 * Verification attention (Sec. 3.2: the drafted candidates go back to the
 * target model, which checks them all in one forward pass).
 *
 * Block row i of the gamma-row verify block sits at sequence position
 * ctx_len + i.  Its query for head h attends causally to every cached key
 * j in [0, ctx_len) and to the block's own keys ctx_len .. ctx_len + i.
 * Grouped-query mapping: q-head h reads kv-head h / (n_q_heads/n_kv_heads).
 *
 *   s_j   = scale * <q[i,h,:], K[g,j,:]>
 *   p_j   = exp(s_j - max_j s_j) / sum_j exp(s_j - max_j s_j)
 *   out   = sum_j p_j * V[g,j,:]
 *
 * Layouts: q [gamma][n_q_heads][head_dim]; k_cache, v_cache
 * [n_kv_heads][cap][head_dim]; out [gamma][n_q_heads][head_dim] (fp64).
 * ------------------------------------------------------------------------ */
static void attend_one(int dtype, const void *q, const void *k_cache,
                       const void *v_cache, int ctx_len, int cap,
                       int n_q_heads, int n_kv_heads, int head_dim,
                       double scale, int i, int h, double *scores,
                       double *out_row)
{
    const int group = n_q_heads / n_kv_heads;
    const int g = h / group;
    const int n_keys = ctx_len + i + 1;
    const size_t q_off = ((size_t)i * n_q_heads + h) * head_dim;
    const size_t kv_head_off = (size_t)g * cap * head_dim;

    double smax = -INFINITY;
    for (int j = 0; j < n_keys; ++j) {
        double dot = 0.0;
        for (int d = 0; d < head_dim; ++d)
            dot += elem(q, dtype, q_off + d) *
                   elem(k_cache, dtype, kv_head_off + (size_t)j * head_dim + d);
        scores[j] = scale * dot;
        if (scores[j] > smax)
            smax = scores[j];
    }
    double denom = 0.0;
    for (int j = 0; j < n_keys; ++j) {
        scores[j] = exp(scores[j] - smax);
        denom += scores[j];
    }
    for (int d = 0; d < head_dim; ++d)
        out_row[d] = 0.0;
    for (int j = 0; j < n_keys; ++j) {
        const double p = scores[j] / denom;
        for (int d = 0; d < head_dim; ++d)
            out_row[d] += p * elem(v_cache, dtype,
                                   kv_head_off + (size_t)j * head_dim + d);
    }
}

static int attn_args_ok(int dtype, int gamma, int ctx_len, int cap,
                        int n_q_heads, int n_kv_heads, int head_dim)
{
    if (!valid_dtype(dtype) || gamma < 1 || ctx_len < 0 || head_dim < 1)
        return 0;
    if (n_kv_heads < 1 || n_q_heads < 1 || n_q_heads % n_kv_heads != 0)
        return 0;
    if ((long long)ctx_len + gamma > cap)
        return 0;
    return 1;
}

int wfref_verify_attn(int dtype, const void *q, const void *k_cache,
                      const void *v_cache, double *out, int gamma, int ctx_len,
                      int cap, int n_q_heads, int n_kv_heads, int head_dim,
                      double scale)
{
    if (!attn_args_ok(dtype, gamma, ctx_len, cap, n_q_heads, n_kv_heads,
                      head_dim))
        return 1;
    const int n_pairs = gamma * n_q_heads;
    int fail = 0;
#pragma omp parallel
    {
        double *scores = malloc(sizeof(double) * (size_t)(ctx_len + gamma));
        if (!scores) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int pr = 0; pr < n_pairs; ++pr) {
                const int i = pr / n_q_heads, h = pr % n_q_heads;
                attend_one(dtype, q, k_cache, v_cache, ctx_len, cap, n_q_heads,
                           n_kv_heads, head_dim, scale, i, h, scores,
                           out + (size_t)pr * head_dim);
            }
        }
        free(scores);
    }
    return fail ? 2 : 0;
}

/* The same definition evaluated only at the listed (row, head) pairs:
 * rows_heads holds n_pairs pairs (i, h); out is [n_pairs][head_dim]. */
int wfref_verify_attn_rows(int dtype, const void *q, const void *k_cache,
                           const void *v_cache, double *out, int gamma,
                           int ctx_len, int cap, int n_q_heads, int n_kv_heads,
                           int head_dim, double scale, int n_pairs,
                           const int32_t *rows_heads)
{
    if (!attn_args_ok(dtype, gamma, ctx_len, cap, n_q_heads, n_kv_heads,
                      head_dim))
        return 1;
    for (int p = 0; p < n_pairs; ++p)
        if (rows_heads[2 * p] < 0 || rows_heads[2 * p] >= gamma ||
            rows_heads[2 * p + 1] < 0 || rows_heads[2 * p + 1] >= n_q_heads)
            return 1;
    int fail = 0;
#pragma omp parallel
    {
        double *scores = malloc(sizeof(double) * (size_t)(ctx_len + gamma));
        if (!scores) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int p = 0; p < n_pairs; ++p)
                attend_one(dtype, q, k_cache, v_cache, ctx_len, cap, n_q_heads,
                           n_kv_heads, head_dim, scale, rows_heads[2 * p],
                           rows_heads[2 * p + 1], scores,
                           out + (size_t)p * head_dim);
        }
        free(scores);
    }
    return fail ? 2 : 0;
}

/* ------------------------------------------------------------------------ *
 * Tree verification.  An autoregressive drafter proposes a tree of
 * candidates rather than a chain (Sec. 3.1; the EAGLE-3 setting of App. A:
 * depth 8, top-k 10, 60 draft tokens), and the target checks every node in
 * the same single parallel pass (Sec. 3.2).
 *
 * Block row i is tree node i.  Row 0 is the root (the last committed
 * token); every other node's parent has a smaller index.  Row i attends to
 * the ctx_len cached keys and to the block keys ctx_len + j of the nodes j
 * it may see: j == i, or bit j of mask[i] set (0 <= j < gamma <= 64).
 * With mask[i] = the ancestors of node i this is ordinary causal attention
 * along node i's root path; for a chain (node j's parent is j-1) it is the
 * block-causal verify attention above.
 *
 *   keys(i) = {0 .. ctx_len-1} U {ctx_len + j : j == i or mask[i] bit j}
 *   out[i,h,:] = sum_{j in keys(i)} softmax_j(scale <q[i,h], K[g,j]>) V[g,j]
 * ------------------------------------------------------------------------ */
static void attend_mask_one(int dtype, const void *q, const void *k_cache,
                            const void *v_cache, int ctx_len, int cap,
                            int gamma, int n_q_heads, int n_kv_heads,
                            int head_dim, double scale, uint64_t row_mask,
                            int i, int h, int *keys, double *scores,
                            double *out_row)
{
    const int group = n_q_heads / n_kv_heads;
    const int g = h / group;
    const size_t q_off = ((size_t)i * n_q_heads + h) * head_dim;
    const size_t kv_head_off = (size_t)g * cap * head_dim;

    int n_keys = 0;
    for (int j = 0; j < ctx_len; ++j)
        keys[n_keys++] = j;
    for (int j = 0; j < gamma; ++j)
        if (j == i || ((row_mask >> j) & 1u))
            keys[n_keys++] = ctx_len + j;

    double smax = -INFINITY;
    for (int t = 0; t < n_keys; ++t) {
        const size_t krow = kv_head_off + (size_t)keys[t] * head_dim;
        double dot = 0.0;
        for (int d = 0; d < head_dim; ++d)
            dot += elem(q, dtype, q_off + d) * elem(k_cache, dtype, krow + d);
        scores[t] = scale * dot;
        if (scores[t] > smax)
            smax = scores[t];
    }
    double denom = 0.0;
    for (int t = 0; t < n_keys; ++t) {
        scores[t] = exp(scores[t] - smax);
        denom += scores[t];
    }
    for (int d = 0; d < head_dim; ++d)
        out_row[d] = 0.0;
    for (int t = 0; t < n_keys; ++t) {
        const double p = scores[t] / denom;
        const size_t vrow = kv_head_off + (size_t)keys[t] * head_dim;
        for (int d = 0; d < head_dim; ++d)
            out_row[d] += p * elem(v_cache, dtype, vrow + d);
    }
}

int wfref_verify_attn_mask(int dtype, const void *q, const void *k_cache,
                           const void *v_cache, double *out,
                           const uint64_t *mask, int gamma, int ctx_len,
                           int cap, int n_q_heads, int n_kv_heads,
                           int head_dim, double scale)
{
    if (!attn_args_ok(dtype, gamma, ctx_len, cap, n_q_heads, n_kv_heads,
                      head_dim) || gamma > 64 || !mask)
        return 1;
    const int n_pairs = gamma * n_q_heads;
    int fail = 0;
#pragma omp parallel
    {
        double *scores = malloc(sizeof(double) * (size_t)(ctx_len + gamma));
        int *keys = malloc(sizeof(int) * (size_t)(ctx_len + gamma));
        if (!scores || !keys) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int pr = 0; pr < n_pairs; ++pr) {
                const int i = pr / n_q_heads, h = pr % n_q_heads;
                attend_mask_one(dtype, q, k_cache, v_cache, ctx_len, cap,
                                gamma, n_q_heads, n_kv_heads, head_dim, scale,
                                mask[i], i, h, keys, scores,
                                out + (size_t)pr * head_dim);
            }
        }
        free(scores);
        free(keys);
    }
    return fail ? 2 : 0;
}

/* ------------------------------------------------------------------------ *
 * Rotary position embedding, rotate-half pairing (the paper names no
 * variant; this is the pairing of the Qwen3 / Llama-3.1 targets it uses).
 * For i < head_dim/2, theta_i = base^(-2i/head_dim), phi = pos * theta_i:
 *   (v_i, v_{i+D/2}) -> (v_i cos phi - v_{i+D/2} sin phi,
 *                        v_{i+D/2} cos phi + v_i sin phi)
 * Angles are formed in fp64.
 * ------------------------------------------------------------------------ */
void wfref_rope_inplace(double *v, int head_dim, double pos, double base)
{
    const int half = head_dim / 2;
    for (int i = 0; i < half; ++i) {
        const double theta = pow(base, -2.0 * (double)i / (double)head_dim);
        const double phi = pos * theta;
        const double c = cos(phi), s = sin(phi);
        const double a = v[i], b = v[i + half];
        v[i] = a * c - b * s;
        v[i + half] = b * c + a * s;
    }
}

/* ------------------------------------------------------------------------ *
 * KV-only prefill (Sec. 3.4, "KV-only Prefill"): for catch-up tokens only
 * the attention layer's keys and values are formed; no MLP, no LM head.
 * Token t sits at position start_pos + t:
 *   k = W_k[g*D:(g+1)*D, :] x_t ;  K[g, t] = RoPE(k, start_pos + t)
 *   v = W_v[g*D:(g+1)*D, :] x_t ;  V[g, t] = v
 * x [n_tok][d_in]; w_k, w_v [n_kv_heads*head_dim][d_in] (row = output
 * feature); k_out, v_out [n_kv_heads][n_tok][head_dim] (fp64).
 * ------------------------------------------------------------------------ */
int wfref_kv_only_prefill(int dtype, const void *x, const void *w_k,
                          const void *w_v, double *k_out, double *v_out,
                          int n_tok, int start_pos, int d_in, int n_kv_heads,
                          int head_dim, double rope_base)
{
    if (!valid_dtype(dtype) || n_tok < 0 || start_pos < 0 || d_in < 1 ||
        n_kv_heads < 1 || head_dim < 2 || head_dim % 2 != 0)
        return 1;
    const int n_units = n_tok * n_kv_heads;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < n_units; ++u) {
        const int t = u / n_kv_heads, g = u % n_kv_heads;
        double *krow = k_out + ((size_t)g * n_tok + t) * head_dim;
        double *vrow = v_out + ((size_t)g * n_tok + t) * head_dim;
        for (int e = 0; e < head_dim; ++e) {
            const size_t wrow = ((size_t)g * head_dim + e) * d_in;
            double ak = 0.0, av = 0.0;
            for (int c = 0; c < d_in; ++c) {
                const double xv = elem(x, dtype, (size_t)t * d_in + c);
                ak += elem(w_k, dtype, wrow + c) * xv;
                av += elem(w_v, dtype, wrow + c) * xv;
            }
            krow[e] = ak;
            vrow[e] = av;
        }
        wfref_rope_inplace(krow, head_dim, (double)start_pos + t, rope_base);
    }
    return 0;
}

/* ------------------------------------------------------------------------ *
 * LM head, argmax and entropy per verify row (Sec. 3.3.1: the router reads
 * the entropy of the target's next-token distribution over the vocabulary).
 *   z[v]    = <h[i,:], W[v,:]>            (or z given directly)
 *   argmax  = lowest index attaining max_v z[v]
 *   p[v]    = exp(z[v] - max z) / sum_u exp(z[u] - max z)
 *   H       = -sum_v p[v] log p[v]   (natural log, 0 log 0 = 0)
 *   margin  = max z - second-largest z (0 when the max is attained twice)
 * h [gamma][d]; w [vocab][d]; logits [gamma][vocab] fp32 (logits mode: h
 * and w NULL).  logits_out, when not NULL, receives z in fp64.
 * ------------------------------------------------------------------------ */
int wfref_lmhead_rows(int dtype, const void *h, const void *w,
                      const float *logits, int gamma, int d, int vocab,
                      int32_t *argmax_out, double *entropy_out,
                      double *margin_out, double *logits_out)
{
    if (gamma < 1 || vocab < 1)
        return 1;
    const int logits_mode = (logits != NULL);
    if (!logits_mode && (!valid_dtype(dtype) || !h || !w || d < 1))
        return 1;
    double *z = logits_out;
    int own = 0;
    if (!z) {
        z = malloc(sizeof(double) * (size_t)gamma * vocab);
        if (!z)
            return 2;
        own = 1;
    }
    if (logits_mode) {
        for (size_t e = 0; e < (size_t)gamma * vocab; ++e)
            z[e] = (double)logits[e];
    } else {
#pragma omp parallel for schedule(static)
        for (int v = 0; v < vocab; ++v)
            for (int i = 0; i < gamma; ++i) {
                double acc = 0.0;
                for (int c = 0; c < d; ++c)
                    acc += elem(h, dtype, (size_t)i * d + c) *
                           elem(w, dtype, (size_t)v * d + c);
                z[(size_t)i * vocab + v] = acc;
            }
    }
    for (int i = 0; i < gamma; ++i) {
        const double *zi = z + (size_t)i * vocab;
        int best = 0;
        for (int v = 1; v < vocab; ++v)
            if (zi[v] > zi[best])
                best = v;
        double second = -INFINITY;
        for (int v = 0; v < vocab; ++v)
            if (v != best && zi[v] > second)
                second = zi[v];
        const double zmax = zi[best];
        double denom = 0.0;
        for (int v = 0; v < vocab; ++v)
            denom += exp(zi[v] - zmax);
        double ent = 0.0;
        for (int v = 0; v < vocab; ++v) {
            const double p = exp(zi[v] - zmax) / denom;
            if (p > 0.0)
                ent -= p * log(p);
        }
        argmax_out[i] = best;
        entropy_out[i] = ent;
        if (margin_out)
            margin_out[i] = (vocab > 1) ? zmax - second : INFINITY;
    }
    if (own)
        free(z);
    return 0;
}

/* ------------------------------------------------------------------------ *
 * Greedy acceptance and the entropy route (Sec. 3.3.1 routing rule; greedy
 * verification as used throughout the evaluation, Sec. 4).
 *   draft[j] is the drafted token at block row j+1; it is accepted iff it
 *   equals the target's argmax at row j and every earlier draft was accepted.
 *   n      = number of accepted drafts (0 .. gamma-1)
 *   bonus  = argmax[n]   (the target's own token after the accepted prefix)
 *   H_t    = entropy[n]  (distribution at the final accepted position)
 *   route  = 1 (autoregressive drafter) if H_t > tau, else 0 (diffusion)
 * out3 = {n, bonus, route}; *h_t receives H_t.
 * ------------------------------------------------------------------------ */
int wfref_accept(const int32_t *argmax, const double *entropy,
                 const int32_t *draft, int gamma, double tau, int32_t *out3,
                 double *h_t)
{
    if (gamma < 1 || (gamma > 1 && !draft))
        return 1;
    int n = 0;
    while (n < gamma - 1 && draft[n] == argmax[n])
        ++n;
    out3[0] = n;
    out3[1] = argmax[n];
    out3[2] = (entropy[n] > tau) ? 1 : 0;
    if (h_t)
        *h_t = entropy[n];
    return 0;
}

/* ------------------------------------------------------------------------ *
 * Greedy acceptance on a draft tree and the entropy route (the tree of
 * Sec. 3.1 verified as in Sec. 3.2; rule of Sec. 3.3.1).
 *   The root (node 0) is accepted.  Node j >= 1 with parent p = parents[j]
 *   is accepted iff 0 <= p < j, p is accepted and tokens[j] == argmax[p]
 *   (the target, having seen p's path, would itself emit tokens[j]).  A node
 *   whose parent index is out of range is never accepted.
 *   depth(0) = 0, depth(j) = depth(parents[j]) + 1.
 *   b     = the accepted node of greatest depth (lowest index among equals)
 *   n     = depth(b), the number of accepted drafts
 *   bonus = argmax[b]; H_t = entropy[b]; route = H_t > tau (1 = AR)
 * out4 = {n, bonus, route, b}; path[t] = the node at depth t on b's root
 * path for t <= n, -1 for t > n; *h_t receives H_t.  tokens[0] and
 * parents[0] are not read.
 * ------------------------------------------------------------------------ */
int wfref_accept_tree(const int32_t *argmax, const double *entropy,
                      const int32_t *tokens, const int32_t *parents,
                      int gamma, double tau, int32_t *out4, int32_t *path,
                      double *h_t)
{
    if (gamma < 1 || gamma > 64 || (gamma > 1 && (!tokens || !parents)))
        return 1;
    int accepted[64], depth[64];
    accepted[0] = 1;
    depth[0] = 0;
    for (int j = 1; j < gamma; ++j) {
        const int p = parents[j];
        if (p < 0 || p >= j) {
            accepted[j] = 0;
            depth[j] = 0;
            continue;
        }
        depth[j] = depth[p] + 1;
        accepted[j] = accepted[p] && tokens[j] == argmax[p];
    }
    int b = 0;
    for (int j = 1; j < gamma; ++j)
        if (accepted[j] && depth[j] > depth[b])
            b = j;
    const int n = depth[b];
    for (int t = 0; t < gamma; ++t)
        path[t] = -1;
    for (int v = b, t = n; t >= 0; --t) {
        path[t] = v;
        v = (t > 0) ? parents[v] : v;
    }
    out4[0] = n;
    out4[1] = argmax[b];
    out4[2] = (entropy[b] > tau) ? 1 : 0;
    out4[3] = b;
    if (h_t)
        *h_t = entropy[b];
    return 0;
}

/* ------------------------------------------------------------------------ *
 * Neural routing policy (Sec. 3.3.2; architecture in the appendix on the
 * neural router): a two-layer MLP regressor on the target's final hidden
 * state predicts the acceptance-length gain of the autoregressive drafter
 * over the diffusion drafter,
 *   delta = w2 . GELU(W1 h + b1) + b2,   GELU(x) = x * Phi(x)
 *         = 0.5 x (1 + erf(x / sqrt 2))   (exact form; dropout is off at
 *                                          inference),
 * with W1 [m][d], m = d/8, and the route is the autoregressive drafter iff
 * delta > tau_neural.  Evaluated here for every row of h [gamma][d];
 * storage code dtype for h, W1, b1, w2 and b2 alike.  delta_out [gamma].
 * ------------------------------------------------------------------------ */
int wfref_router_mlp(int dtype, const void *h, const void *w1, const void *b1,
                     const void *w2, const void *b2, int gamma, int d, int m,
                     double *delta_out)
{
    if (!valid_dtype(dtype) || gamma < 1 || d < 1 || m < 1)
        return 1;
#pragma omp parallel for schedule(static)
    for (int r = 0; r < gamma; ++r) {
        double acc = elem(b2, dtype, 0);
        for (int i = 0; i < m; ++i) {
            double z = elem(b1, dtype, i);
            for (int k = 0; k < d; ++k)
                z += elem(w1, dtype, (size_t)i * d + k) *
                     elem(h, dtype, (size_t)r * d + k);
            const double g = 0.5 * z * (1.0 + erf(z / sqrt(2.0)));
            acc += elem(w2, dtype, i) * g;
        }
        delta_out[r] = acc;
    }
    return 0;
}

/* ------------------------------------------------------------------------ *
 * RMSNorm of M rows: y = x / sqrt(mean(x^2) + eps) * gain (fp64).
 * ------------------------------------------------------------------------ */
int wfref_rmsnorm(int dtype, const void *x, const void *gain, int M, int d,
                  double eps, double *y)
{
    if (!valid_dtype(dtype) || M < 1 || d < 1)
        return 1;
    for (int m = 0; m < M; ++m) {
        double ss = 0.0;
        for (int c = 0; c < d; ++c) {
            const double xv = elem(x, dtype, (size_t)m * d + c);
            ss += xv * xv;
        }
        const double inv = 1.0 / sqrt(ss / d + eps);
        for (int c = 0; c < d; ++c)
            y[(size_t)m * d + c] =
                elem(x, dtype, (size_t)m * d + c) * inv * elem(gain, dtype, c);
    }
    return 0;
}

/* ------------------------------------------------------------------------ *
 * One full decoder layer of a drafter for M tokens at positions
 * pos .. pos+M-1, against a cache whose rows [0, pos) hold the earlier
 * tokens.  Lazy catch-up (Sec. 3.4) runs it only for the last backlog
 * token -- the one whose hidden state the next draft needs -- and forms the
 * other backlog tokens' K/V alone; a full catch-up runs it for all of them.
 *   xn  = RMSNorm(r) * g1
 *   q, k, v = Wq xn, Wk xn, Wv xn; RoPE on q and k at the token's position
 *   cache rows pos + t <- (k, v)
 *   a   = causal grouped-query attention of q over cache rows [0, pos + t]
 *   h1  = r + Wo a
 *   xn2 = RMSNorm(h1) * g2
 *   out = h1 + Wd (SiLU(Wg xn2) * (Wu xn2)),  SiLU(x) = x / (1 + exp(-x))
 * r [M][d], weights in nn.Linear layout (Wq [Hq*D][d], Wk/Wv [Hkv*D][d],
 * Wo [d][Hq*D], Wg/Wu [inter][d], Wd [d][inter]) and the gains share the
 * storage code; k_cache, v_cache are fp64 [Hkv][cap][D] and are updated
 * in place; out [M][d] fp64.
 * ------------------------------------------------------------------------ */
int wfref_decoder_forward(int dtype, const void *r, int M, int pos,
                          const void *g1, const void *wq, const void *wk,
                          const void *wv, const void *wo, const void *g2,
                          const void *wg, const void *wu, const void *wd,
                          int d, int n_q_heads, int n_kv_heads, int head_dim,
                          int inter, double rms_eps, double rope_base,
                          double *k_cache, double *v_cache, int cap,
                          double *out)
{
    if (!valid_dtype(dtype) || M < 1 || pos < 0 || pos + M > cap || d < 1 ||
        n_kv_heads < 1 || n_q_heads % n_kv_heads != 0 || head_dim % 2 != 0 ||
        inter < 1)
        return 1;
    const int qd = n_q_heads * head_dim;
    const int group = n_q_heads / n_kv_heads;
    const double scale = 1.0 / sqrt((double)head_dim);
    double *xn = malloc(sizeof(double) * (size_t)M * d);
    double *q = malloc(sizeof(double) * (size_t)M * qd);
    double *a = malloc(sizeof(double) * (size_t)M * qd);
    double *h1 = malloc(sizeof(double) * (size_t)M * d);
    double *xn2 = malloc(sizeof(double) * (size_t)d);
    double *act = malloc(sizeof(double) * (size_t)inter);
    double *s = malloc(sizeof(double) * (size_t)(pos + M));
    int rc = 0;
    if (!xn || !q || !a || !h1 || !xn2 || !act || !s) {
        rc = 2;
        goto done;
    }
    wfref_rmsnorm(dtype, r, g1, M, d, rms_eps, xn);
    for (int t = 0; t < M; ++t) {
        const double *x = xn + (size_t)t * d;
        for (int o = 0; o < qd; ++o) {
            double acc = 0.0;
            for (int c = 0; c < d; ++c)
                acc += elem(wq, dtype, (size_t)o * d + c) * x[c];
            q[(size_t)t * qd + o] = acc;
        }
        for (int h = 0; h < n_q_heads; ++h)
            wfref_rope_inplace(q + (size_t)t * qd + (size_t)h * head_dim, head_dim,
                               (double)(pos + t), rope_base);
        for (int g = 0; g < n_kv_heads; ++g) {
            double *kr = k_cache + ((size_t)g * cap + pos + t) * head_dim;
            double *vr = v_cache + ((size_t)g * cap + pos + t) * head_dim;
            for (int e = 0; e < head_dim; ++e) {
                double ak = 0.0, av = 0.0;
                for (int c = 0; c < d; ++c) {
                    ak += elem(wk, dtype, ((size_t)g * head_dim + e) * d + c) * x[c];
                    av += elem(wv, dtype, ((size_t)g * head_dim + e) * d + c) * x[c];
                }
                kr[e] = ak;
                vr[e] = av;
            }
            wfref_rope_inplace(kr, head_dim, (double)(pos + t), rope_base);
        }
    }
    for (int t = 0; t < M; ++t)
        for (int h = 0; h < n_q_heads; ++h) {
            const int g = h / group;
            const double *qr = q + (size_t)t * qd + (size_t)h * head_dim;
            const int n = pos + t + 1;
            double smax = -INFINITY;
            for (int j = 0; j < n; ++j) {
                const double *kr = k_cache + ((size_t)g * cap + j) * head_dim;
                double dot = 0.0;
                for (int e = 0; e < head_dim; ++e)
                    dot += qr[e] * kr[e];
                s[j] = scale * dot;
                if (s[j] > smax)
                    smax = s[j];
            }
            double denom = 0.0;
            for (int j = 0; j < n; ++j) {
                s[j] = exp(s[j] - smax);
                denom += s[j];
            }
            double *ar = a + (size_t)t * qd + (size_t)h * head_dim;
            for (int e = 0; e < head_dim; ++e)
                ar[e] = 0.0;
            for (int j = 0; j < n; ++j) {
                const double *vr = v_cache + ((size_t)g * cap + j) * head_dim;
                for (int e = 0; e < head_dim; ++e)
                    ar[e] += (s[j] / denom) * vr[e];
            }
        }
    for (int t = 0; t < M; ++t) {
        const double *ar = a + (size_t)t * qd;
        double *hr = h1 + (size_t)t * d;
        for (int o = 0; o < d; ++o) {
            double acc = 0.0;
            for (int c = 0; c < qd; ++c)
                acc += elem(wo, dtype, (size_t)o * qd + c) * ar[c];
            hr[o] = elem(r, dtype, (size_t)t * d + o) + acc;
        }
        double ss = 0.0;
        for (int c = 0; c < d; ++c)
            ss += hr[c] * hr[c];
        const double inv = 1.0 / sqrt(ss / d + rms_eps);
        for (int c = 0; c < d; ++c)
            xn2[c] = hr[c] * inv * elem(g2, dtype, c);
        for (int i = 0; i < inter; ++i) {
            double zg = 0.0, zu = 0.0;
            for (int c = 0; c < d; ++c) {
                zg += elem(wg, dtype, (size_t)i * d + c) * xn2[c];
                zu += elem(wu, dtype, (size_t)i * d + c) * xn2[c];
            }
            act[i] = zg / (1.0 + exp(-zg)) * zu;
        }
        for (int o = 0; o < d; ++o) {
            double acc = 0.0;
            for (int i = 0; i < inter; ++i)
                acc += elem(wd, dtype, (size_t)o * inter + i) * act[i];
            out[(size_t)t * d + o] = hr[o] + acc;
        }
    }
done:
    free(xn);
    free(q);
    free(a);
    free(h1);
    free(xn2);
    free(act);
    free(s);
    return rc;
}

/* ------------------------------------------------------------------------ *
 * One full decoder attention layer over a fresh sequence of T tokens
 * (positions pos0 .. pos0+T-1), used only to pin the KV-only prefill: the
 * keys and values it records must equal what KV-only prefill produces for
 * the same normalised inputs (Sec. 3.4: catch-up needs only the KV cache).
 *   xn    = RMSNorm(x) * gain          (eps inside the square root)
 *   q,k,v = W_q xn, W_k xn, W_v xn;  q,k rotated by RoPE at their position
 *   out   = causal grouped-query softmax attention, scale 1/sqrt(head_dim)
 * x [T][d]; gain [d]; w_q [n_q_heads*D][d]; w_k, w_v [n_kv_heads*D][d].
 * Outputs (fp64): xn_out [T][d]; k_out, v_out [n_kv_heads][T][D];
 * q_out [T][n_q_heads][D] (post-RoPE); attn_out [T][n_q_heads][D].
 * Inputs use the given storage code for x, gain and the weights.
 * ------------------------------------------------------------------------ */
int wfref_layer_forward(int dtype, const void *x, const void *gain,
                        const void *w_q, const void *w_k, const void *w_v,
                        int T, int pos0, int d, int n_q_heads, int n_kv_heads,
                        int head_dim, double rms_eps, double rope_base,
                        double *xn_out, double *q_out, double *k_out,
                        double *v_out, double *attn_out)
{
    if (!valid_dtype(dtype) || T < 1 || d < 1 || n_kv_heads < 1 ||
        n_q_heads % n_kv_heads != 0 || head_dim % 2 != 0)
        return 1;
    for (int t = 0; t < T; ++t) {
        double ss = 0.0;
        for (int c = 0; c < d; ++c) {
            const double xv = elem(x, dtype, (size_t)t * d + c);
            ss += xv * xv;
        }
        const double inv = 1.0 / sqrt(ss / d + rms_eps);
        for (int c = 0; c < d; ++c)
            xn_out[(size_t)t * d + c] =
                elem(x, dtype, (size_t)t * d + c) * inv * elem(gain, dtype, c);
    }
    for (int t = 0; t < T; ++t) {
        const double *xr = xn_out + (size_t)t * d;
        for (int h = 0; h < n_q_heads; ++h) {
            double *qr = q_out + ((size_t)t * n_q_heads + h) * head_dim;
            for (int e = 0; e < head_dim; ++e) {
                double acc = 0.0;
                for (int c = 0; c < d; ++c)
                    acc += elem(w_q, dtype, ((size_t)h * head_dim + e) * d + c) *
                           xr[c];
                qr[e] = acc;
            }
            wfref_rope_inplace(qr, head_dim, (double)pos0 + t, rope_base);
        }
        for (int g = 0; g < n_kv_heads; ++g) {
            double *kr = k_out + ((size_t)g * T + t) * head_dim;
            double *vr = v_out + ((size_t)g * T + t) * head_dim;
            for (int e = 0; e < head_dim; ++e) {
                double ak = 0.0, av = 0.0;
                for (int c = 0; c < d; ++c) {
                    ak += elem(w_k, dtype, ((size_t)g * head_dim + e) * d + c) *
                          xr[c];
                    av += elem(w_v, dtype, ((size_t)g * head_dim + e) * d + c) *
                          xr[c];
                }
                kr[e] = ak;
                vr[e] = av;
            }
            wfref_rope_inplace(kr, head_dim, (double)pos0 + t, rope_base);
        }
    }
    const int group = n_q_heads / n_kv_heads;
    const double scale = 1.0 / sqrt((double)head_dim);
    double *s = malloc(sizeof(double) * (size_t)T);
    if (!s)
        return 2;
    for (int t = 0; t < T; ++t)
        for (int h = 0; h < n_q_heads; ++h) {
            const int g = h / group;
            const double *qr = q_out + ((size_t)t * n_q_heads + h) * head_dim;
            double smax = -INFINITY;
            for (int j = 0; j <= t; ++j) {
                const double *kr = k_out + ((size_t)g * T + j) * head_dim;
                double dot = 0.0;
                for (int e = 0; e < head_dim; ++e)
                    dot += qr[e] * kr[e];
                s[j] = scale * dot;
                if (s[j] > smax)
                    smax = s[j];
            }
            double denom = 0.0;
            for (int j = 0; j <= t; ++j) {
                s[j] = exp(s[j] - smax);
                denom += s[j];
            }
            double *orow = attn_out + ((size_t)t * n_q_heads + h) * head_dim;
            for (int e = 0; e < head_dim; ++e)
                orow[e] = 0.0;
            for (int j = 0; j <= t; ++j) {
                const double *vr = v_out + ((size_t)g * T + j) * head_dim;
                for (int e = 0; e < head_dim; ++e)
                    orow[e] += (s[j] / denom) * vr[e];
            }
        }
    free(s);
    return 0;
}
