// drafter.hip -- the drafter side of a switch (Sec. 3.4 of the WhiFlash
// paper).  Lazy catch-up brings the incoming drafter's KV cache up to date
// over the backlog in one batch: KV-only prefill for every backlog token but
// the last, which runs the drafter's full layer -- attention and a SwiGLU
// MLP -- because the next draft starts from its hidden state.  The full
// layer for M tokens at positions pos .. pos+M-1:
//
//   xn  = RMSNorm(r) * g1                     rmsnorm_bf16
//   K/V = RoPE(Wk xn), Wv xn  -> cache rows    the KV-only prefill kernel
//   q   = RoPE(Wq xn)                          skinny linear + reduce_rope_bf16
//   a   = causal GQA attention over the cache  the verify-attention kernels
//   h1  = r + Wo a                             skinny linear + reduce_store_bf16
//   xn2 = RMSNorm(h1) * g2                     rmsnorm_bf16
//   act = SiLU(Wg xn2) * (Wu xn2)              one skinny linear over [Wg; Wu]
//                                              + reduce_swiglu_bf16
//   out = h1 + Wd act                          skinny linear + reduce_store_bf16
//
// Activations are rounded to bf16 between the steps, as a bf16 model stores
// them; every sum runs in fp32 in a fixed order.
//
// For a single token (the catch-up's last) each projection carries its
// epilogue instead: q = RoPE(Wq xn) on the KV-only prefill kernel (its
// split-K exchange tree spreads the 32 MB over the chip), h1 = r + Wo a and
// out = h1 + Wd act in one kernel each, and [Wg; Wu] with the MLP's RMSNorm
// folded into its loads and SwiGLU into its epilogue -- 8 launches per
// catch-up instead of 13.
#include <cmath>

#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kNormThreads = 256;
constexpr int kMaxHalfDim = 64;

struct RopeParams {
    double theta[kMaxHalfDim];   // base^(-2i/D), i < D/2, formed on the host in fp64
};

// One workgroup per row.  Each thread takes 8-element chunks c, c + 256,
// ... of the row with 16-byte loads, kRowBatch of them issued before any is
// used; the sum of squares runs in a fixed order (chunk order within a
// thread, then the wave butterfly, then the waves in order).  The scaling
// pass reads the row again (a cache hit) with the gains.
constexpr int kRowBatch = 4;

__device__ __forceinline__ u32x4 load_u32x4(const uint16_t *p) {
    return *reinterpret_cast<const u32x4 *>(p);
}

__device__ __forceinline__ float lo_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f32(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Workgroup r normalises row min(r, n_rows - 1); y (row-major) gets rows
// below n_rows, y_tiled (if given) every row of the grid in 16-token x
// 32-dim tiles of 1 KB in the MFMA operand's lane order -- the layout the
// KV-only prefill reads with one contiguous load per tile (the grid then
// covers n_rows rounded up to 16; the pad rows repeat the last row).
__global__ __launch_bounds__(kNormThreads) void rmsnorm_bf16(const uint16_t *__restrict__ x,
                                                             const uint16_t *__restrict__ g,
                                                             float eps, uint16_t *__restrict__ y,
                                                             int d, int n_rows,
                                                             uint16_t *__restrict__ y_tiled) {
    __shared__ float part[kNormThreads / kWave];
    const int row = blockIdx.x;
    const uint16_t *xr = x + (size_t)min(row, n_rows - 1) * d;
    const int n_chunks = d / 8;
    float ss = 0.f;
    for (int c0 = threadIdx.x; c0 < n_chunks; c0 += kNormThreads * kRowBatch) {
        u32x4 v[kRowBatch];
#pragma unroll
        for (int u = 0; u < kRowBatch; ++u)
            if (c0 + u * kNormThreads < n_chunks)
                v[u] = load_u32x4(xr + 8 * (c0 + u * kNormThreads));
#pragma unroll
        for (int u = 0; u < kRowBatch; ++u)
            if (c0 + u * kNormThreads < n_chunks) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = lo_f32(v[u][e]), b = hi_f32(v[u][e]);
                    ss = fmaf(a, a, ss);
                    ss = fmaf(b, b, ss);
                }
            }
    }
    ss = wave_sum(ss);
    if (threadIdx.x % kWave == 0)
        part[threadIdx.x / kWave] = ss;
    __syncthreads();
    float tot = part[0];
#pragma unroll
    for (int w = 1; w < kNormThreads / kWave; ++w)
        tot += part[w];
    const float inv = 1.f / sqrtf(tot / (float)d + eps);
    uint16_t *yr = row < n_rows ? y + (size_t)row * d : nullptr;
    // tile (row / 16, chunk c) holds lane (row % 16) + 16 * (8-dim group
    // within the chunk) at 16 bytes per lane
    uint16_t *yt = y_tiled ? y_tiled + (size_t)(row / 16) * (d / 32) * 512 + (row % 16) * 8
                           : nullptr;
    for (int c0 = threadIdx.x; c0 < n_chunks; c0 += kNormThreads * kRowBatch) {
        u32x4 v[kRowBatch], gv[kRowBatch];
#pragma unroll
        for (int u = 0; u < kRowBatch; ++u)
            if (c0 + u * kNormThreads < n_chunks) {
                v[u] = load_u32x4(xr + 8 * (c0 + u * kNormThreads));
                gv[u] = load_u32x4(g + 8 * (c0 + u * kNormThreads));
            }
#pragma unroll
        for (int u = 0; u < kRowBatch; ++u)
            if (c0 + u * kNormThreads < n_chunks) {
                u32x4 o;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    o[e] = pack_bf16x2(lo_f32(v[u][e]) * inv * lo_f32(gv[u][e]),
                                       hi_f32(v[u][e]) * inv * hi_f32(gv[u][e]));
                const int cc = c0 + u * kNormThreads;          // 8-element chunk
                if (yr)
                    *reinterpret_cast<u32x4 *>(yr + 8 * cc) = o;
                if (yt)
                    *reinterpret_cast<u32x4 *>(yt + (size_t)(cc / 4) * 512 + (cc % 4) * 128) = o;
            }
    }
}

// The slices of one output in order; all loads are issued before the first
// add (one memory round trip, not ks).
__device__ __forceinline__ float sum_slices(const float *zpart, int ks, int n_out, int rows,
                                            int f, int r) {
    float v[kLinearMaxSlices];
#pragma unroll
    for (int k = 0; k < kLinearMaxSlices; ++k)
        v[k] = k < ks ? zpart[((size_t)k * n_out + f) * rows + r] : 0.f;
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kLinearMaxSlices; ++k)
        if (k < ks)
            s += v[k];
    return s;
}

// y[r][f] = bf16(sum of slices (+ res[r][f]))
__global__ __launch_bounds__(256) void reduce_store_bf16(const float *__restrict__ zpart, int ks,
                                                         int n_out, int rows,
                                                         const uint16_t *__restrict__ res,
                                                         uint16_t *__restrict__ y) {
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)rows * n_out)
        return;
    const int r = (int)(idx / n_out), f = (int)(idx % n_out);
    float s = sum_slices(zpart, ks, n_out, rows, f, r);
    if (res)
        s += bf16_to_f32(res[idx]);
    y[idx] = f32_to_bf16(s);
}

// q[r][h][i], q[r][h][i + D/2] = RoPE at position pos + r of the pair's sums
// (angle formed and reduced modulo 2*pi in fp64, sine and cosine in fp32)
__global__ __launch_bounds__(256) void reduce_rope_bf16(const float *__restrict__ zpart, int ks,
                                                        int n_heads, int head_dim, int rows,
                                                        int pos, RopeParams rp,
                                                        uint16_t *__restrict__ q) {
    const int half = head_dim / 2;
    const int n_out = n_heads * head_dim;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)rows * n_heads * half)
        return;
    const int i = (int)(idx % half);
    const int h = (int)((idx / half) % n_heads);
    const int r = (int)(idx / ((long long)half * n_heads));
    float lo = sum_slices(zpart, ks, n_out, rows, h * head_dim + i, r);
    float hi = sum_slices(zpart, ks, n_out, rows, h * head_dim + i + half, r);
    constexpr double kTwoPi = 6.283185307179586;
    constexpr double kInvTwoPi = 0.15915494309189535;
    const double phi = (double)(pos + r) * rp.theta[i];
    const double red = fma(-rint(phi * kInvTwoPi), kTwoPi, phi);
    float sf, cf;
    sincosf((float)red, &sf, &cf);
    const float a = lo, b = hi;
    lo = a * cf - b * sf;
    hi = b * cf + a * sf;
    uint16_t *qr = q + ((size_t)r * n_heads + h) * head_dim;
    qr[i] = f32_to_bf16(lo);
    qr[i + half] = f32_to_bf16(hi);
}

// act[r][i] = bf16(SiLU(gate) * up); features [0, inter) are the gate
// projection, [inter, 2 inter) the up projection
__global__ __launch_bounds__(256) void reduce_swiglu_bf16(const float *__restrict__ zpart, int ks,
                                                          int inter, int rows,
                                                          uint16_t *__restrict__ act) {
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)rows * inter)
        return;
    const int r = (int)(idx / inter), i = (int)(idx % inter);
    const float gt = sum_slices(zpart, ks, 2 * inter, rows, i, r);
    const float up = sum_slices(zpart, ks, 2 * inter, rows, inter + i, r);
    act[idx] = f32_to_bf16(gt / (1.f + expf(-gt)) * up);
}

inline unsigned blocks_for(long long n) { return (unsigned)((n + 255) / 256); }

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace of the full layer: the attention call's (its zero block first,
// which the prefill call shares), then the bf16 activations and the fp32
// linear slices.
struct DrafterLayout {
    size_t attn, xn, q, a, h1, xn2, act, zpart, total;
    AttnPlan plan;
};

DrafterLayout drafter_layout(const wf_decoder_layer_t &L, int M, int pos) {
    DrafterLayout o{};
    const int qd = L.n_q_heads * L.head_dim;
    o.plan = plan_attn(WF_BF16, M, pos, L.n_q_heads, L.n_kv_heads, L.head_dim, 0);
    size_t at = align256(attn_workspace_bytes(o.plan, M, L.n_q_heads, L.head_dim));
    o.attn = 0;
    o.xn = at;
    at = align256(at + (size_t)M * L.hidden * 2);
    o.q = at;
    at = align256(at + (size_t)M * qd * 2);
    o.a = at;
    at = align256(at + (size_t)M * qd * 2);
    o.h1 = at;
    at = align256(at + (size_t)M * L.hidden * 2);
    o.xn2 = at;
    at = align256(at + (size_t)M * L.hidden * 2);
    o.act = at;
    at = align256(at + (size_t)M * L.inter * 2);
    o.zpart = at;
    const size_t zq = (size_t)linear_slices(L.hidden, qd) * qd;
    const size_t zo = (size_t)linear_slices(qd, L.hidden) * L.hidden;
    const size_t zgu = (size_t)linear_slices(L.hidden, 2 * L.inter) * 2 * L.inter;
    const size_t zd = (size_t)linear_slices(L.inter, L.hidden) * L.hidden;
    const size_t zmax = std::max(std::max(zq, zo), std::max(zgu, zd));
    o.total = align256(at + zmax * M * sizeof(float));
    return o;
}

}  // namespace

size_t drafter_forward_workspace_bytes(const wf_decoder_layer_t &L, int M, int pos) {
    return drafter_layout(L, M, pos).total;
}

// Catch-up workspace: the last token's full-layer workspace, then the
// backlog's normalised rows (row-major, for the last token's projections),
// then the same rows in 16 x 32 tiles for the KV-only prefill.
size_t drafter_catchup_workspace_bytes(const wf_decoder_layer_t &L, int n, int pos) {
    return align256(drafter_forward_workspace_bytes(L, 1, pos + n - 1)) +
           align256((size_t)n * L.hidden * 2) + (size_t)((n + 15) / 16) * 16 * L.hidden * 2;
}

namespace {

// The full layer for M tokens.  xn_given: the tokens' RMSNorm(r) * g1 with
// their K/V already in the cache (the catch-up normalises and prefills the
// whole backlog in one batch), else both are formed here.
wf_status_t drafter_forward(const wf_decoder_layer_t &L, const uint16_t *rb, int M, int pos,
                            void *k_cache, void *v_cache, int cap, void *out,
                            void *workspace, hipStream_t stream, bool tiled,
                            const uint16_t *xn_given, bool q_ready = false) {
    const wf_dtype_t wdt = tiled ? WF_BF16_TILED : WF_BF16;
    const DrafterLayout o = drafter_layout(L, M, pos);
    char *ws = static_cast<char *>(workspace);
    auto *xn = reinterpret_cast<uint16_t *>(ws + o.xn);
    auto *q = reinterpret_cast<uint16_t *>(ws + o.q);
    auto *a = reinterpret_cast<uint16_t *>(ws + o.a);
    auto *h1 = reinterpret_cast<uint16_t *>(ws + o.h1);
    auto *xn2 = reinterpret_cast<uint16_t *>(ws + o.xn2);
    auto *act = reinterpret_cast<uint16_t *>(ws + o.act);
    auto *zp = reinterpret_cast<float *>(ws + o.zpart);
    const int d = L.hidden, qd = L.n_q_heads * L.head_dim, I = L.inter;
    auto W = [](const void *p) { return static_cast<const uint16_t *>(p); };
    wf_status_t st;

    if (xn_given) {
        xn = const_cast<uint16_t *>(xn_given);
    } else {
        rmsnorm_bf16<<<M, kNormThreads, 0, stream>>>(rb, W(L.attn_norm), L.rms_eps, xn, d, M,
                                                      nullptr);
        st = launch_prefill(wdt, xn, L.w_k, L.w_v, k_cache, v_cache, M, pos, cap, d,
                            L.n_kv_heads, L.head_dim, L.rope_base, workspace, stream);
        if (st != WF_OK)
            return st;
    }
    if (M == 1) {
        // One token (the catch-up's last): every projection carries its
        // epilogue -- RoPE, a residual, or the MLP's RMSNorm and SwiGLU --
        // so the layer is five launches after the K/V: W_q, attention (two),
        // W_o, [W_gate; W_up], W_down.
        // (q_ready: the caller has already formed q in the layout's slot)
        if (!q_ready &&
            (st = launch_q_rope(xn, W(L.w_q), q, d, L.n_q_heads, L.head_dim, pos,
                                L.rope_base, workspace, stream, tiled)) != WF_OK)
            return st;
        st = launch_attn(WF_BF16, q, k_cache, v_cache, a, 1, pos, cap, L.n_q_heads,
                         L.n_kv_heads, L.head_dim, (float)(1.0 / std::sqrt((double)L.head_dim)),
                         nullptr, o.plan, workspace, stream);
        if (st != WF_OK)
            return st;
        if ((st = launch_linear_resid(a, W(L.w_o), rb, qd, d, h1, stream, tiled)) != WF_OK)
            return st;
        if ((st = launch_linear_norm_swiglu(h1, W(L.mlp_norm), L.rms_eps, W(L.w_gate),
                                            W(L.w_up), d, I, act, stream, tiled)) != WF_OK)
            return st;
        return launch_linear_resid(act, W(L.w_down), h1, I, d, static_cast<uint16_t *>(out),
                                   stream, tiled);
    }
    // q = RoPE(Wq xn)
    if ((st = launch_linear_partial(xn, W(L.w_q), nullptr, qd, 0, M, d, zp, stream, tiled)) != WF_OK)
        return st;
    RopeParams rp{};
    for (int i = 0; i < L.head_dim / 2; ++i)
        rp.theta[i] = std::pow(L.rope_base, -2.0 * (double)i / (double)L.head_dim);
    reduce_rope_bf16<<<blocks_for((long long)M * qd / 2), 256, 0, stream>>>(
        zp, linear_slices(d, qd), L.n_q_heads, L.head_dim, M, pos, rp, q);
    // a = attention over the cache, causal among the M tokens
    st = launch_attn(WF_BF16, q, k_cache, v_cache, a, M, pos, cap, L.n_q_heads, L.n_kv_heads,
                     L.head_dim, (float)(1.0 / std::sqrt((double)L.head_dim)), nullptr, o.plan,
                     workspace, stream);
    if (st != WF_OK)
        return st;
    // h1 = r + Wo a (the slices summed over many workgroups), then
    // xn2 = RMSNorm(h1) * g2.  (One workgroup per row doing both took
    // 13 us: a single CU summing the slices of a whole row is latency-bound.)
    if ((st = launch_linear_partial(a, W(L.w_o), nullptr, d, 0, M, qd, zp, stream, tiled)) != WF_OK)
        return st;
    reduce_store_bf16<<<blocks_for((long long)M * d), 256, 0, stream>>>(
        zp, linear_slices(qd, d), d, M, rb, h1);
    rmsnorm_bf16<<<M, kNormThreads, 0, stream>>>(h1, W(L.mlp_norm), L.rms_eps, xn2, d, M,
                                                  nullptr);
    // act = SiLU(Wg xn2) * (Wu xn2): in one launch where the input
    // dimension is not split, else slices and a separate SwiGLU pass
    st = launch_linear_swiglu(xn2, W(L.w_gate), W(L.w_up), I, M, d, act, stream, tiled);
    if (st == WF_ERR_UNSUPPORTED) {
        if ((st = launch_linear_partial(xn2, W(L.w_gate), W(L.w_up), I, I, M, d, zp, stream,
                                        tiled)) != WF_OK)
            return st;
        reduce_swiglu_bf16<<<blocks_for((long long)M * I), 256, 0, stream>>>(
            zp, linear_slices(d, 2 * I), I, M, act);
    } else if (st != WF_OK) {
        return st;
    }
    // out = h1 + Wd act
    if ((st = launch_linear_partial(act, W(L.w_down), nullptr, d, 0, M, I, zp, stream, tiled)) != WF_OK)
        return st;
    reduce_store_bf16<<<blocks_for((long long)M * d), 256, 0, stream>>>(
        zp, linear_slices(I, d), d, M, h1, static_cast<uint16_t *>(out));
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace

wf_status_t launch_drafter_forward(const wf_decoder_layer_t &L, const void *r, int M, int pos,
                                   void *k_cache, void *v_cache, int cap, void *out,
                                   void *workspace, hipStream_t stream, bool tiled) {
    return drafter_forward(L, static_cast<const uint16_t *>(r), M, pos, k_cache, v_cache, cap,
                           out, workspace, stream, tiled, nullptr);
}

// Catch-up: RMSNorm and KV-only prefill of the whole backlog in one batch
// each (the last token's K/V included), then the rest of the layer for the
// last token from its normalised row.
wf_status_t launch_drafter_catchup(const wf_decoder_layer_t &L, const void *r, int n, int pos,
                                   void *k_cache, void *v_cache, int cap, void *out,
                                   void *workspace, hipStream_t stream, bool tiled) {
    const int d = L.hidden;
    const auto *rb = static_cast<const uint16_t *>(r);
    const DrafterLayout lay = drafter_layout(L, 1, pos + n - 1);
    char *tail = static_cast<char *>(workspace) + align256(lay.total);
    auto *xnb = reinterpret_cast<uint16_t *>(tail);
    auto *xnt = reinterpret_cast<uint16_t *>(tail + align256((size_t)n * d * 2));
    const uint16_t *x_last = xnb + (size_t)(n - 1) * d;
    rmsnorm_bf16<<<(n + 15) / 16 * 16, kNormThreads, 0, stream>>>(
        rb, static_cast<const uint16_t *>(L.attn_norm), L.rms_eps, xnb, d, n, xnt);
    // A backlog of one batch: its K/V and the last token's q in one launch
    // (they only share the normalised rows).
    bool q_ready = false;
    if (n <= kCatchupChunk) {
        const wf_status_t st = launch_prefill_and_q(
            tiled, xnt, L.w_k, L.w_v, k_cache, v_cache, n, pos, cap, d, L.n_kv_heads, x_last,
            static_cast<const uint16_t *>(L.w_q),
            reinterpret_cast<uint16_t *>(static_cast<char *>(workspace) + lay.q), L.n_q_heads,
            L.head_dim, pos + n - 1, L.rope_base, workspace, stream);
        if (st != WF_OK && st != WF_ERR_UNSUPPORTED)
            return st;
        q_ready = st == WF_OK;
    }
    // otherwise the whole backlog's K/V in batches of at most kCatchupChunk
    // tokens (one KV-only prefill each), reading the tiled rows (a batch
    // starts on a 16-row tile boundary), and q in the layer below
    for (int c0 = 0; !q_ready && c0 < n; c0 += kCatchupChunk) {
        const int m = std::min(kCatchupChunk, n - c0);
        const wf_status_t st = launch_prefill(tiled ? WF_BF16_TILED : WF_BF16,
                                              xnt + (size_t)c0 * d, L.w_k, L.w_v, k_cache,
                                              v_cache, m, pos + c0, cap, d, L.n_kv_heads,
                                              L.head_dim, L.rope_base, workspace, stream,
                                              1, 0, 0, 0, true);
        if (st != WF_OK)
            return st;
    }
    return drafter_forward(L, rb + (size_t)(n - 1) * d, 1, pos + n - 1, k_cache, v_cache, cap,
                           out, workspace, stream, tiled, x_last, q_ready);
}

}  // namespace wf
