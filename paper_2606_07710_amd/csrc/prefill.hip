// prefill.hip -- KV-only prefill of catch-up tokens (Sec. 3.4 of the
// WhiFlash paper: after a drafter switch the incoming drafter's cache is
// caught up on the backlog in one batch, forming only the attention
// layer's keys and values -- no MLP, no LM head).
//
//   K[g][p+t] = RoPE(W_k[g] x_t, p+t),   V[g][p+t] = W_v[g] x_t
//
// bf16 path: the work unit is (KV head, K or V, pair of 16-feature blocks f
// and f + head_dim/2).  Pairing the two halves of the rotate-half RoPE puts
// both elements of every rotation pair in the same lane of the MFMA
// accumulators, so RoPE is a register epilogue.  The input dimension is
// split across workgroups so a handful of units still spreads over the whole
// chip; each slice writes an fp32 partial, and a second kernel sums the
// slices in order, rotates and writes the cache rows.  Tokens are the MFMA N dimension (blocks of 16).
// RoPE angles are formed in fp64: at positions ~65K an fp32 angle would be
// off by ~4e-3 rad.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kPfMaxChunksPerWave = 8;   // 32-wide chunks per wave per k-slice
constexpr int kPfTargetWorkgroups = 512;

struct PrefillParams {
    const void *x;
    const void *w_k;
    const void *w_v;
    void *k_cache;
    void *v_cache;
    int n_tok, start_pos, cap, d_in, n_kv_heads;
    double rope_base;
    float *ws;                 // bf16 path: split-K partials
    int chunks_per_split;      // 32-wide chunks of d_in per k-slice
};

__device__ __forceinline__ void rope_pair(float &lo, float &hi, int i, int dh,
                                          int pos, double base) {
    const double theta = pow(base, -2.0 * (double)i / (double)dh);
    const double phi = (double)pos * theta;
    double s, c;
    sincos(phi, &s, &c);
    const float cf = (float)c, sf = (float)s;
    const float a = lo, b = hi;
    lo = a * cf - b * sf;
    hi = b * cf + a * sf;
}

// Split-K: workgroup (unit, k-slice, token block) computes D[feature][token]
// over its slice of the input dimension for the unit's two 16-feature blocks
// (f and f + head_dim/2 of one head, K or V), writes the fp32 partial to
// ws[unit][token block][kslice][2][16][TOK].
template <int DH, int NBT>
__global__ __launch_bounds__(256) void prefill_partial_bf16(PrefillParams a) {
    constexpr int PAIRS = DH / 32;       // 16-feature block pairs per head
    constexpr int TOK = 16 * NBT;
    constexpr int WAVES = 4;
    constexpr int MAXC = kPfMaxChunksPerWave;
    __shared__ float zs[WAVES][2][16][TOK + 1];

    const int unit = blockIdx.x;         // (g, kind, pair)
    const int ks = blockIdx.y;
    const int tb = blockIdx.z;
    const int pair = unit % PAIRS;
    const int kind = (unit / PAIRS) % 2; // 0 = K, 1 = V
    const int g = unit / (2 * PAIRS);
    const int t0 = tb * TOK;

    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;

    const uint16_t *w = static_cast<const uint16_t *>(kind ? a.w_v : a.w_k);
    const uint16_t *x = static_cast<const uint16_t *>(a.x);
    const int f_lo = g * DH + 16 * pair;           // first feature, low half
    const int c_begin = ks * a.chunks_per_split;   // 32-wide chunks of d_in
    const uint16_t *wp0 = w + (size_t)(f_lo + m16) * a.d_in + c4 * 8;
    const uint16_t *wp1 = w + (size_t)(f_lo + DH / 2 + m16) * a.d_in + c4 * 8;
    // Tokens past n_tok read the last token instead: they only feed MFMA
    // output columns that are never stored.
    const uint16_t *xp[NBT];
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb)
        xp[nb] = x + (size_t)min(t0 + nb * 16 + m16, a.n_tok - 1) * a.d_in + c4 * 8;

    // every load of this wave's chunks is issued before the first MFMA
    bf16x8 wr[MAXC][2], xr[MAXC][NBT];
#pragma unroll
    for (int u = 0; u < MAXC; ++u) {
        const int c = wave + WAVES * u;
        if (c < a.chunks_per_split) {
            const int off = (c_begin + c) * 32;
            wr[u][0] = load_bf16x8(wp0 + off);
            wr[u][1] = load_bf16x8(wp1 + off);
#pragma unroll
            for (int nb = 0; nb < NBT; ++nb)
                xr[u][nb] = load_bf16x8(xp[nb] + off);
        }
    }
    f32x4 acc[2][NBT];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
            acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < MAXC; ++u) {
        if (wave + WAVES * u < a.chunks_per_split) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int nb = 0; nb < NBT; ++nb)
                    acc[mb][nb] = mfma16x16x32(wr[u][mb], xr[u][nb], acc[mb][nb]);
        }
    }
    // lane (m16, c4) holds D[feature 4*c4 + i][token nb*16 + m16]
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                zs[wave][mb][4 * c4 + i][nb * 16 + m16] = acc[mb][nb][i];
    __syncthreads();
    // sum the waves in a fixed order and write the partial
    const int ksplit = gridDim.y;
    const size_t ub = (size_t)unit * gridDim.z + tb;           // (unit, token block)
    float *part = a.ws + ub * ksplit * (2 * 16 * TOK);
    float *dst = part + (size_t)ks * (2 * 16 * TOK);
    for (int idx = threadIdx.x; idx < 2 * 16 * TOK; idx += blockDim.x) {
        const int mb = idx / (16 * TOK);
        const int e = (idx / TOK) % 16;
        const int tl = idx % TOK;
        float v = zs[0][mb][e][tl];
#pragma unroll
        for (int ww = 1; ww < WAVES; ++ww)
            v += zs[ww][mb][e][tl];
        dst[idx] = v;
    }

    // The last k-slice workgroup of this (unit, token block) to finish sums
    // the slices in slice order, applies RoPE to K and writes the cache rows.
}

// Workgroup (unit, token block) sums the unit's k-slice partials in slice
// order, applies RoPE to K and writes the cache rows.
template <int DH, int NBT>
__global__ __launch_bounds__(256) void prefill_finish_bf16(PrefillParams a, int ksplit) {
    constexpr int PAIRS = DH / 32;
    constexpr int TOK = 16 * NBT;
    const int unit = blockIdx.x;
    const int tb = blockIdx.y;
    const int pair = unit % PAIRS;
    const int kind = (unit / PAIRS) % 2;
    const int g = unit / (2 * PAIRS);
    const int t0 = tb * TOK;
    const size_t ub = (size_t)unit * gridDim.y + tb;
    const float *part = a.ws + ub * ksplit * (2 * 16 * TOK);
    uint16_t *cache = static_cast<uint16_t *>(kind ? a.v_cache : a.k_cache);
    for (int idx = threadIdx.x; idx < 16 * TOK; idx += blockDim.x) {
        const int e = idx / TOK;
        const int tl = idx % TOK;
        const int t = t0 + tl;
        if (t >= a.n_tok)
            continue;
        // slices in ascending order; loads batched so they are in flight
        // together (clamped, masked at the add)
        constexpr int KB = 16;
        float lo = 0.f, hi = 0.f;
        for (int k0 = 0; k0 < ksplit; k0 += KB) {
            float vl[KB], vh[KB];
#pragma unroll
            for (int b = 0; b < KB; ++b) {
                const int k = min(k0 + b, ksplit - 1);
                vl[b] = part[k * (2 * 16 * TOK) + e * TOK + tl];
                vh[b] = part[k * (2 * 16 * TOK) + 16 * TOK + e * TOK + tl];
            }
#pragma unroll
            for (int b = 0; b < KB; ++b)
                if (k0 + b < ksplit) {
                    lo += vl[b];
                    hi += vh[b];
                }
        }
        const int pos = a.start_pos + t;
        if (kind == 0)
            rope_pair(lo, hi, 16 * pair + e, DH, pos, a.rope_base);
        uint16_t *row = cache + ((size_t)g * a.cap + pos) * DH;
        row[16 * pair + e] = f32_to_bf16(lo);
        row[DH / 2 + 16 * pair + e] = f32_to_bf16(hi);
    }
}

// fp32 path: one thread per (token, KV head, rotation pair, K or V).
__global__ __launch_bounds__(256) void prefill_f32(PrefillParams a, int dh) {
    const int half = dh / 2;
    const long long total = (long long)a.n_tok * a.n_kv_heads * half * 2;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int i = (int)(idx % half);
    const int kind = (int)((idx / half) % 2);
    const int g = (int)((idx / (2 * half)) % a.n_kv_heads);
    const int t = (int)(idx / (2LL * half * a.n_kv_heads));
    const float *x = static_cast<const float *>(a.x) + (size_t)t * a.d_in;
    const float *w = static_cast<const float *>(kind ? a.w_v : a.w_k);
    const float *w_lo = w + (size_t)(g * dh + i) * a.d_in;
    const float *w_hi = w + (size_t)(g * dh + i + half) * a.d_in;
    float lo = 0.f, hi = 0.f;
    for (int c = 0; c < a.d_in; ++c) {
        lo = fmaf(w_lo[c], x[c], lo);
        hi = fmaf(w_hi[c], x[c], hi);
    }
    const int pos = a.start_pos + t;
    if (kind == 0)
        rope_pair(lo, hi, i, dh, pos, a.rope_base);
    float *row = static_cast<float *>(kind ? a.v_cache : a.k_cache) + ((size_t)g * a.cap + pos) * dh;
    row[i] = lo;
    row[i + half] = hi;
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

PrefillPlan plan_prefill(int n_tok, int d_in, int n_kv_heads, int head_dim) {
    PrefillPlan p{};
    p.nbt = std::min(4, std::max(1, cdiv(n_tok, 16)));
    p.token_blocks = std::max(1, cdiv(n_tok, 16 * p.nbt));
    p.units = n_kv_heads * 2 * (head_dim / 32);
    const int chunks = d_in / 32;
    // enough k-slices to cover the chip, each wave owning 1..8 chunks
    int ks = std::max(1, cdiv(kPfTargetWorkgroups, p.units * p.token_blocks));
    ks = std::min(ks, std::max(1, chunks / 4));                   // >= 4 chunks per slice
    ks = std::max(ks, cdiv(chunks, 4 * kPfMaxChunksPerWave));    // <= 32 chunks per slice
    p.chunks_per_split = cdiv(chunks, ks);
    p.ksplit = cdiv(chunks, p.chunks_per_split);
    return p;
}

size_t prefill_workspace_bytes(wf_dtype_t dt, int n_tok, int d_in, int n_kv_heads,
                               int head_dim) {
    if (dt != WF_BF16 || n_tok == 0)
        return 0;
    const PrefillPlan p = plan_prefill(n_tok, d_in, n_kv_heads, head_dim);
    const size_t part = (size_t)p.units * p.token_blocks * p.ksplit * 2 * 16 * (16 * p.nbt) * sizeof(float);
    return kCounterBytes + part;
}

wf_status_t launch_prefill(wf_dtype_t dt, const void *x, const void *w_k,
                           const void *w_v, void *k_cache, void *v_cache,
                           int n_tok, int start_pos, int cap, int d_in,
                           int n_kv_heads, int head_dim, double rope_base,
                           void *workspace, hipStream_t stream) {
    PrefillParams a{x, w_k, w_v, k_cache, v_cache, n_tok, start_pos, cap, d_in,
                    n_kv_heads, rope_base, nullptr, 0};
    if (dt == WF_BF16) {
        const PrefillPlan p = plan_prefill(n_tok, d_in, n_kv_heads, head_dim);
        a.chunks_per_split = p.chunks_per_split;
        a.ws = reinterpret_cast<float *>(static_cast<char *>(workspace) + kCounterBytes);
        dim3 grid(p.units, p.ksplit, p.token_blocks), block(256);
        dim3 fgrid(p.units, p.token_blocks);
#define WF_PF_CASE(DHV, NBV)                                                        \
    if (head_dim == DHV && p.nbt == NBV) {                                          \
        prefill_partial_bf16<DHV, NBV><<<grid, block, 0, stream>>>(a);              \
        prefill_finish_bf16<DHV, NBV><<<fgrid, block, 0, stream>>>(a, p.ksplit);    \
    } else
        WF_PF_CASE(128, 1) WF_PF_CASE(128, 2) WF_PF_CASE(128, 3) WF_PF_CASE(128, 4)
        WF_PF_CASE(64, 1) WF_PF_CASE(64, 2) WF_PF_CASE(64, 3) WF_PF_CASE(64, 4)
        { return WF_ERR_UNSUPPORTED; }
#undef WF_PF_CASE
    } else {
        const long long total = (long long)n_tok * n_kv_heads * head_dim;
        const unsigned blocks = (unsigned)((total + 255) / 256);
        prefill_f32<<<blocks, 256, 0, stream>>>(a, head_dim);
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
