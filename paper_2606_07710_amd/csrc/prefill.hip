// prefill.hip -- KV-only prefill of catch-up tokens (Sec. 3.4 of the
// WhiFlash paper: after a drafter switch the incoming drafter's cache is
// caught up on the backlog in one batch, forming only the attention
// layer's keys and values -- no MLP, no LM head).
//
//   K[g][p+t] = RoPE(W_k[g] x_t, p+t),   V[g][p+t] = W_v[g] x_t
//
// bf16 path: one workgroup per (KV head, K or V, pair of 16-feature blocks
// f and f + head_dim/2).  Pairing the two halves of the rotate-half RoPE in
// one workgroup puts both elements of every rotation pair in the same lane
// of the MFMA accumulators, so RoPE is a register-only epilogue.  Eight
// waves split the input dimension; their partial sums meet in LDS in a fixed
// order.  Tokens are the MFMA N dimension (blocks of 16, up to 64 per
// launch row of the grid).
// RoPE angles are formed in fp64: at positions ~65K an fp32 angle would be
// off by ~4e-3 rad.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kPfWaves = 8;
constexpr int kPfPrefetch = 4;

struct PrefillParams {
    const void *x;
    const void *w_k;
    const void *w_v;
    void *k_cache;
    void *v_cache;
    int n_tok, start_pos, cap, d_in, n_kv_heads;
    double rope_base;
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

template <int DH, int NBT>
__global__ __launch_bounds__(512) void prefill_bf16(PrefillParams a) {
    constexpr int PAIRS = DH / 32;       // 16-feature block pairs per head
    constexpr int TOK = 16 * NBT;
    __shared__ float zs[2][16][TOK + 1];

    const int unit = blockIdx.x;         // (g, kind, pair)
    const int pair = unit % PAIRS;
    const int kind = (unit / PAIRS) % 2; // 0 = K, 1 = V
    const int g = unit / (2 * PAIRS);
    const int t0 = blockIdx.y * TOK;

    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;

    const uint16_t *w = static_cast<const uint16_t *>(kind ? a.w_v : a.w_k);
    const uint16_t *x = static_cast<const uint16_t *>(a.x);
    const int f_lo = g * DH + 16 * pair;           // first feature, low half
    const uint16_t *wp[2] = {
        w + (size_t)(f_lo + m16) * a.d_in + c4 * 8,
        w + (size_t)(f_lo + DH / 2 + m16) * a.d_in + c4 * 8};
    // Tokens past n_tok read the last token instead: they only feed MFMA
    // output columns that are never stored, and nothing waits on a load early.
    const uint16_t *xp[NBT];
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb)
        xp[nb] = x + (size_t)min(t0 + nb * 16 + m16, a.n_tok - 1) * a.d_in + c4 * 8;

    f32x4 acc[2][NBT];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
            acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nchunks = a.d_in / 32;
    const int cpw = (wave < nchunks) ? (nchunks - wave + kPfWaves - 1) / kPfWaves : 0;
    bf16x8 wb[kPfPrefetch][2], xb[kPfPrefetch][NBT];
    auto load_chunk = [&](int u, bf16x8 (&wr)[2], bf16x8 (&xr)[NBT]) {
        const int off = (wave + kPfWaves * u) * 32;
        wr[0] = load_bf16x8(wp[0] + off);
        wr[1] = load_bf16x8(wp[1] + off);
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
            xr[nb] = load_bf16x8(xp[nb] + off);
    };
    auto mac = [&](const bf16x8 (&wr)[2], const bf16x8 (&xr)[NBT]) {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int nb = 0; nb < NBT; ++nb)
                acc[mb][nb] = mfma16x16x32(wr[mb], xr[nb], acc[mb][nb]);
    };
    // Branch-free steady state (exact wait counting, kPfPrefetch chunks in
    // flight), peeled last group, then any remainder chunks.
    const int ngroups = cpw / kPfPrefetch;
    if (ngroups > 0) {
#pragma unroll
        for (int p = 0; p < kPfPrefetch; ++p) {
            load_chunk(p, wb[p], xb[p]);
            __builtin_amdgcn_sched_barrier(0);   // issue chunk by chunk
        }
        for (int gi = 0; gi < ngroups - 1; ++gi) {
#pragma unroll
            for (int p = 0; p < kPfPrefetch; ++p) {
                mac(wb[p], xb[p]);
                load_chunk((gi + 1) * kPfPrefetch + p, wb[p], xb[p]);
                // keep each refill right behind the MFMAs that free its
                // registers, so kPfPrefetch chunks stay in flight
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int p = 0; p < kPfPrefetch; ++p)
            mac(wb[p], xb[p]);
    }
    for (int u = ngroups * kPfPrefetch; u < cpw; ++u) {
        load_chunk(u, wb[0], xb[0]);
        mac(wb[0], xb[0]);
    }

    // lane (m16, c4) holds D[feature 4*c4 + i][token nb*16 + m16]
#pragma unroll 1
    for (int ww = 0; ww < kPfWaves; ++ww) {
        if (wave == ww) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int nb = 0; nb < NBT; ++nb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float &dst = zs[mb][4 * c4 + i][nb * 16 + m16];
                        dst = (ww > 0) ? dst + acc[mb][nb][i] : acc[mb][nb][i];
                    }
        }
        __syncthreads();
    }

    // epilogue: thread per (feature e of the block, token)
    uint16_t *cache = static_cast<uint16_t *>(kind ? a.v_cache : a.k_cache);
    for (int idx = threadIdx.x; idx < 16 * TOK; idx += blockDim.x) {
        const int e = idx % 16;
        const int tl = idx / 16;
        const int t = t0 + tl;
        if (t >= a.n_tok)
            continue;
        float lo = zs[0][e][tl], hi = zs[1][e][tl];
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

wf_status_t launch_prefill(wf_dtype_t dt, const void *x, const void *w_k,
                           const void *w_v, void *k_cache, void *v_cache,
                           int n_tok, int start_pos, int cap, int d_in,
                           int n_kv_heads, int head_dim, double rope_base,
                           hipStream_t stream) {
    PrefillParams a{x, w_k, w_v, k_cache, v_cache, n_tok, start_pos, cap, d_in,
                    n_kv_heads, rope_base};
    if (dt == WF_BF16) {
        const int nbt = std::min(4, cdiv(n_tok, 16));
        const int tok_per_row = 16 * nbt;
        dim3 grid(n_kv_heads * 2 * (head_dim / 32), cdiv(n_tok, tok_per_row));
        dim3 block(512);
#define WF_PF_CASE(DHV, NBV)                                        \
    if (head_dim == DHV && nbt == NBV) {                            \
        prefill_bf16<DHV, NBV><<<grid, block, 0, stream>>>(a);      \
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
