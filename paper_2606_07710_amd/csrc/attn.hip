// attn.hip -- verification attention of a gamma-row draft block against the
// KV cache (parallel target verification, Sec. 3.2 of the WhiFlash paper).
//
// Split-KV design for batch 1 on MI355X.  Every workgroup owns one KV head g
// and one contiguous slice ("split") of the key range, and processes all
// G*gamma query rows of that head at once, so every K/V byte is fetched from
// HBM exactly once.  Inside the workgroup four waves stream interleaved
// 32-key tiles; each keeps an fp32 online-softmax state per row.  The waves
// merge through LDS and the workgroup writes one fp32 partial (unnormalised
// output row, running max, running sum) per (split, row).  A second kernel
// combines the splits in a fixed order.
//
// bf16 path, per 32-key tile and wave (16x16x32 bf16 MFMA):
//   S^T = K * Q^T : A = 16 keys x 32 dims straight from global memory,
//                   B = Q^T held in registers for the whole kernel.
//   P   = exp2((S - m) * scale * log2 e), online max/sum per row.
//   O^T += V^T * P^T : B = P^T comes out of the S^T accumulator already in
//                   operand layout (the key order inside a tile is chosen so
//                   each lane owns 8 consecutive keys of its row); A = V^T is
//                   read from a per-wave LDS copy of the V tile, stored with
//                   an XOR swizzle so the transposing reads hit 32 distinct
//                   banks.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kTileKeys = 32;
constexpr int kAttnWaves = 4;

struct AttnParams {
    const uint16_t *q16;      // bf16 path
    const uint16_t *k16;
    const uint16_t *v16;
    const float *q32;         // fp32 path
    const float *k32;
    const float *v32;
    float *ws_acc;            // [splits][gamma*n_q_heads][head_dim]
    float *ws_ml;             // [splits][gamma*n_q_heads][2]
    int gamma, ctx_len, cap, n_q_heads, n_kv_heads, group, rows, n_keys;
    int splits, keys_per_split, n_row_groups;
    float sl2;                // softmax_scale * log2(e)
};

// ---------------------------------------------------------------------------
// bf16 split-KV partial kernel.  DH = head_dim, NB = 16-row blocks per row
// group (rows handled per wave = 16*NB).
// ---------------------------------------------------------------------------
template <int DH, int NB>
__global__ __launch_bounds__(256) void attn_partial_bf16(AttnParams a) {
    constexpr int KC = DH / 32;          // 32-dim chunks of a key row
    constexpr int MD = DH / 16;          // 16-dim output blocks
    constexpr int GR = DH / 8;           // 16-byte granules per key row
    constexpr int VLD = kTileKeys * GR / kWave;  // V loads per lane per tile
    constexpr int ROWS = 16 * NB;

    __shared__ __attribute__((aligned(16))) uint16_t vtile[kAttnWaves][kTileKeys * DH];
    __shared__ __attribute__((aligned(16))) float osum[ROWS * DH];
    __shared__ float mls[kAttnWaves][ROWS][2];

    // ---- which (kv head, split, row group) this workgroup owns -------------
    int unit, rg;
    if (a.n_row_groups == 1) {
        unit = blockIdx.x;
        rg = 0;
    } else {
        // keep the row groups of one (head, split) on one XCD, adjacent in
        // its dispatch order, so the second reader of a K/V tile hits L2
        const int xcd = blockIdx.x & 7, w = blockIdx.x >> 3;
        rg = w % a.n_row_groups;
        unit = (w / a.n_row_groups) * 8 + xcd;
    }
    if (unit >= a.n_kv_heads * a.splits)
        return;
    const int g = unit % a.n_kv_heads;
    const int split = unit / a.n_kv_heads;

    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;

    const int k_begin = split * a.keys_per_split;
    const int k_end = min(a.n_keys, k_begin + a.keys_per_split);
    const int n_tiles = (k_end > k_begin) ? (k_end - k_begin + kTileKeys - 1) / kTileKeys : 0;

    // ---- Q^T operands and per-row causal limits ------------------------------
    bf16x8 qf[NB][KC];
    int lim[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int r = rg * ROWS + nb * 16 + m16;
        if (r < a.rows) {
            const int i = r / a.group;
            const int h = g * a.group + (r % a.group);
            const uint16_t *qp = a.q16 + ((size_t)i * a.n_q_heads + h) * DH + c4 * 8;
#pragma unroll
            for (int kk = 0; kk < KC; ++kk)
                qf[nb][kk] = load_bf16x8(qp + kk * 32);
            lim[nb] = a.ctx_len + i;
        } else {
#pragma unroll
            for (int kk = 0; kk < KC; ++kk)
                qf[nb][kk] = zero_bf16x8();
            lim[nb] = 0x7fffffff;        // padding row: no mask, never stored
        }
    }

    f32x4 o[MD][NB];
    float mrow[NB], lrow[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        mrow[nb] = -INFINITY;
        lrow[nb] = 0.f;
#pragma unroll
        for (int md = 0; md < MD; ++md)
            o[md][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    const size_t head_off = (size_t)g * a.cap * DH;
    const uint16_t *kbase = a.k16 + head_off;
    const uint16_t *vbase = a.v16 + head_off;
    uint16_t *vt = vtile[wave];
    const int last_key = a.n_keys - 1;

    // Key of A-row m (16 rows) in M-block mb of a tile: tile base +
    // 8*(m/4) + 4*mb + m%4, so S^T lane (m16, c4) ends up owning the 8
    // consecutive keys 8*c4 .. 8*c4+7 of its row.
    const int krow0 = 8 * (m16 >> 2) + (m16 & 3);

    bf16x8 kn[2][KC], vn[VLD];
    auto load_tile = [&](int t, bf16x8 (&kr)[2][KC], bf16x8 (&vr)[VLD]) {
        const int kb = k_begin + t * kTileKeys;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const int key = min(kb + krow0 + 4 * mb, last_key);
            const uint16_t *p = kbase + (size_t)key * DH + c4 * 8;
#pragma unroll
            for (int kk = 0; kk < KC; ++kk)
                kr[mb][kk] = load_bf16x8(p + kk * 32);
        }
#pragma unroll
        for (int r = 0; r < VLD; ++r) {
            const int chunk = r * kWave + lane;
            const int key = kb + chunk / GR;
            const int gi = chunk % GR;
            bf16x8 val = load_bf16x8(vbase + (size_t)min(key, last_key) * DH + gi * 8);
            vr[r] = (key <= last_key) ? val : zero_bf16x8();
        }
    };

    int t = wave;
    if (t < n_tiles)
        load_tile(t, kn, vn);
    for (; t < n_tiles; t += kAttnWaves) {
        bf16x8 kc[2][KC], vc[VLD];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int kk = 0; kk < KC; ++kk)
                kc[mb][kk] = kn[mb][kk];
#pragma unroll
        for (int r = 0; r < VLD; ++r)
            vc[r] = vn[r];
        if (t + kAttnWaves < n_tiles)
            load_tile(t + kAttnWaves, kn, vn);

        // S^T = K Q^T
        f32x4 s[2][NB];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < KC; ++kk)
                    acc = mfma16x16x32(kc[mb][kk], qf[nb][kk], acc);
                s[mb][nb] = acc;
            }

        // V tile -> LDS (granule swizzle: gi ^ 2*((key/8)%4))
#pragma unroll
        for (int r = 0; r < VLD; ++r) {
            const int chunk = r * kWave + lane;
            const int kl = chunk / GR;
            const int gi = chunk % GR;
            const int gs = gi ^ (2 * ((kl >> 3) & 3));
            *reinterpret_cast<u32x4 *>(vt + kl * DH + gs * 8) = __builtin_bit_cast(u32x4, vc[r]);
        }

        // causal mask + online softmax
        const int kb = k_begin + t * kTileKeys;
        const bool need_mask = (kb + kTileKeys - 1) > a.ctx_len;
        bf16x8 pb[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            float mx = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int key = kb + 8 * c4 + 4 * mb + i;
                    if (need_mask && key > lim[nb])
                        s[mb][nb][i] = -INFINITY;
                    mx = fmaxf(mx, s[mb][nb][i]);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
            mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
            const float mnew = fmaxf(mrow[nb], mx);
            const float muse = (mnew == -INFINITY) ? 0.f : mnew;
            const float alpha = exp2f((mrow[nb] - muse) * a.sl2);
            const float moff = -muse * a.sl2;
            mrow[nb] = mnew;
            float psum = 0.f;
            float p[8];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float e = exp2f(fmaf(s[mb][nb][i], a.sl2, moff));
                    p[4 * mb + i] = e;
                    psum += e;
                }
            lrow[nb] = fmaf(lrow[nb], alpha, psum);
#pragma unroll
            for (int md = 0; md < MD; ++md)
                o[md][nb] *= alpha;
            uint32_t pw[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                pw[j] = (uint32_t)f32_to_bf16(p[2 * j]) |
                        ((uint32_t)f32_to_bf16(p[2 * j + 1]) << 16);
            u32x4 pv = {pw[0], pw[1], pw[2], pw[3]};
            pb[nb] = __builtin_bit_cast(bf16x8, pv);
        }

        // O^T += V^T P^T   (A operand: V[8*c4 + j][16*md + m16], j = 0..7)
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int md = 0; md < MD; ++md) {
            const int gi = 2 * md + (m16 >> 3);
            const int gs = gi ^ (2 * c4);
            const uint16_t *src = vt + (8 * c4) * DH + gs * 8 + (m16 & 7);
            uint32_t w[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                w[j] = (uint32_t)src[(2 * j) * DH] | ((uint32_t)src[(2 * j + 1) * DH] << 16);
            u32x4 av = {w[0], w[1], w[2], w[3]};
            const bf16x8 va = __builtin_bit_cast(bf16x8, av);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                o[md][nb] = mfma16x16x32(va, pb[nb], o[md][nb]);
        }
        __builtin_amdgcn_wave_barrier();
    }

    // ---- per-wave row sums (the 4 K-groups of a row hold disjoint keys) -----
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        float l = lrow[nb];
        l += __shfl_xor(l, 16, kWave);
        l += __shfl_xor(l, 32, kWave);
        lrow[nb] = l;
        if (c4 == 0) {
            mls[wave][nb * 16 + m16][0] = mrow[nb];
            mls[wave][nb * 16 + m16][1] = l;
        }
    }
    __syncthreads();

    // ---- merge the four waves in a fixed order through LDS ------------------
    float fac[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int r = nb * 16 + m16;
        float mm = -INFINITY;
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w)
            mm = fmaxf(mm, mls[w][r][0]);
        const float muse = (mm == -INFINITY) ? 0.f : mm;
        fac[nb] = (mrow[nb] == -INFINITY) ? 0.f : exp2f((mrow[nb] - muse) * a.sl2);
    }
#pragma unroll 1
    for (int w = 0; w < kAttnWaves; ++w) {
        if (wave == w) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int md = 0; md < MD; ++md) {
                    float *dst = osum + (nb * 16 + m16) * DH + md * 16 + 4 * c4;
                    f32x4 v = o[md][nb] * fac[nb];
                    if (w > 0)
                        v += *reinterpret_cast<f32x4 *>(dst);
                    *reinterpret_cast<f32x4 *>(dst) = v;
                }
        }
        __syncthreads();
    }

    // ---- write the workgroup partial ----------------------------------------
    const int pairs = a.gamma * a.n_q_heads;
    for (int idx = threadIdx.x; idx < ROWS * (DH / 4); idx += blockDim.x) {
        const int rl = idx / (DH / 4);
        const int d4 = idx % (DH / 4);
        const int r = rg * ROWS + rl;
        if (r >= a.rows)
            continue;
        const int i = r / a.group;
        const int h = g * a.group + (r % a.group);
        const size_t pr = (size_t)split * pairs + (size_t)i * a.n_q_heads + h;
        reinterpret_cast<f32x4 *>(a.ws_acc + pr * DH)[d4] =
            reinterpret_cast<const f32x4 *>(osum + rl * DH)[d4];
        if (d4 == 0) {
            float mm = -INFINITY, ll = 0.f;
#pragma unroll
            for (int w = 0; w < kAttnWaves; ++w)
                mm = fmaxf(mm, mls[w][rl][0]);
            const float muse = (mm == -INFINITY) ? 0.f : mm;
#pragma unroll
            for (int w = 0; w < kAttnWaves; ++w) {
                const float mw = mls[w][rl][0];
                const float f = (mw == -INFINITY) ? 0.f : exp2f((mw - muse) * a.sl2);
                ll = fmaf(mls[w][rl][1], f, ll);
            }
            a.ws_ml[pr * 2] = mm;
            a.ws_ml[pr * 2 + 1] = ll;
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 split-KV partial kernel (plain VALU; one wave per (split, row, head)).
// ---------------------------------------------------------------------------
template <int DH>
__global__ __launch_bounds__(64) void attn_partial_f32(AttnParams a) {
    constexpr int E = DH / kWave;        // output dims per lane
    __shared__ float qs[DH];
    const int split = blockIdx.x;
    const int pr = blockIdx.y;           // i * n_q_heads + h
    const int i = pr / a.n_q_heads, h = pr % a.n_q_heads;
    const int g = h / a.group;
    const int lane = threadIdx.x;

    const float *qp = a.q32 + (size_t)pr * DH;
    for (int d = lane; d < DH; d += kWave)
        qs[d] = qp[d];
    __syncthreads();

    const int k_begin = split * a.keys_per_split;
    const int k_end = min(min(a.n_keys, k_begin + a.keys_per_split), a.ctx_len + i + 1);
    const float *kbase = a.k32 + (size_t)g * a.cap * DH;
    const float *vbase = a.v32 + (size_t)g * a.cap * DH;

    float m = -INFINITY, l = 0.f, acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e)
        acc[e] = 0.f;

    for (int kb = k_begin; kb < k_end; kb += kWave) {
        const int j = kb + lane;
        float sc = -INFINITY;
        if (j < k_end) {
            const float *kr = kbase + (size_t)j * DH;
            float dot = 0.f;
            for (int d = 0; d < DH; ++d)
                dot = fmaf(qs[d], kr[d], dot);
            sc = dot;
        }
        const float mnew = fmaxf(m, wave_max(sc));
        const float alpha = (m == -INFINITY) ? 0.f : exp2f((m - mnew) * a.sl2);
        const float p = (j < k_end) ? exp2f((sc - mnew) * a.sl2) : 0.f;
        l = fmaf(l, alpha, wave_sum(p));
#pragma unroll
        for (int e = 0; e < E; ++e)
            acc[e] *= alpha;
        const int cnt = min(kWave, k_end - kb);
        for (int tt = 0; tt < cnt; ++tt) {
            const float pt = __shfl(p, tt, kWave);
            const float *vr = vbase + (size_t)(kb + tt) * DH;
#pragma unroll
            for (int e = 0; e < E; ++e)
                acc[e] = fmaf(pt, vr[lane + e * kWave], acc[e]);
        }
        m = mnew;
    }

    const size_t prs = (size_t)split * a.gamma * a.n_q_heads + pr;
#pragma unroll
    for (int e = 0; e < E; ++e)
        a.ws_acc[prs * DH + lane + e * kWave] = acc[e];
    if (lane == 0) {
        a.ws_ml[prs * 2] = m;
        a.ws_ml[prs * 2 + 1] = l;
    }
}

// ---------------------------------------------------------------------------
// Split merge: out = sum_s w_s acc_s / sum_s w_s l_s, w_s = exp(m_s - max m),
// splits combined in ascending order.  One wave per (row, q head).
// ---------------------------------------------------------------------------
template <int DH, bool OUT_BF16>
__global__ __launch_bounds__(64) void attn_merge(const float *__restrict__ ws_acc,
                                                 const float *__restrict__ ws_ml,
                                                 void *out, int pairs, int splits,
                                                 float sl2) {
    constexpr int E = DH / kWave;
    const int pr = blockIdx.x;
    const int lane = threadIdx.x;
    float mloc = -INFINITY;
    for (int s = lane; s < splits; s += kWave)
        mloc = fmaxf(mloc, ws_ml[((size_t)s * pairs + pr) * 2]);
    const float mm = wave_max(mloc);
    const float muse = (mm == -INFINITY) ? 0.f : mm;
    float acc[E], lsum = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e)
        acc[e] = 0.f;
    for (int s = 0; s < splits; ++s) {
        const size_t ps = (size_t)s * pairs + pr;
        const float ms = ws_ml[ps * 2];
        const float w = (ms == -INFINITY) ? 0.f : exp2f((ms - muse) * sl2);
        lsum = fmaf(w, ws_ml[ps * 2 + 1], lsum);
#pragma unroll
        for (int e = 0; e < E; ++e)
            acc[e] = fmaf(w, ws_acc[ps * DH + lane + e * kWave], acc[e]);
    }
    const float inv = 1.f / lsum;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const float v = acc[e] * inv;
        const size_t oi = (size_t)pr * DH + lane + e * kWave;
        if (OUT_BF16)
            static_cast<uint16_t *>(out)[oi] = f32_to_bf16(v);
        else
            static_cast<float *>(out)[oi] = v;
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

// Split plan shared by the workspace query and the launcher.
AttnPlan plan_attn(wf_dtype_t dt, int gamma, int ctx_len, int n_q_heads,
                   int n_kv_heads, int head_dim, int num_splits) {
    AttnPlan p{};
    const int group = n_q_heads / n_kv_heads;
    const int rows = group * gamma;
    const int n_keys = ctx_len + gamma;
    const int n_tiles = cdiv(n_keys, kTileKeys);
    p.rows = rows;
    if (dt == WF_BF16) {
        p.nb = rows <= 16 ? 1 : rows <= 32 ? 2 : 4;
        p.n_row_groups = cdiv(rows, 16 * p.nb);
    } else {
        p.nb = 0;
        p.n_row_groups = 1;
    }
    int splits = num_splits;
    if (splits <= 0) {
        // aim for ~2 workgroups per CU of the 256-CU chip, but give every
        // wave of a workgroup at least two tiles to stream
        const int target = 512 / (n_kv_heads * p.n_row_groups);
        const int max_by_work = std::max(1, n_tiles / (2 * kAttnWaves));
        splits = std::max(1, std::min(target, max_by_work));
    }
    splits = std::min(splits, n_tiles);
    // keys per split: whole tiles, then drop splits left empty by rounding
    const int tiles_per_split = cdiv(n_tiles, splits);
    p.keys_per_split = tiles_per_split * kTileKeys;
    p.splits = cdiv(n_keys, p.keys_per_split);
    return p;
}

size_t attn_workspace_bytes(const AttnPlan &p, int gamma, int n_q_heads, int head_dim) {
    const size_t pairs = (size_t)gamma * n_q_heads;
    return (size_t)p.splits * pairs * (head_dim + 2) * sizeof(float);
}

wf_status_t launch_attn(wf_dtype_t dt, const void *q, const void *k_cache,
                        const void *v_cache, void *out, int gamma, int ctx_len,
                        int cap, int n_q_heads, int n_kv_heads, int head_dim,
                        float softmax_scale, const AttnPlan &p, void *workspace,
                        hipStream_t stream) {
    AttnParams a{};
    const size_t pairs = (size_t)gamma * n_q_heads;
    a.ws_acc = static_cast<float *>(workspace);
    a.ws_ml = a.ws_acc + (size_t)p.splits * pairs * head_dim;
    a.gamma = gamma;
    a.ctx_len = ctx_len;
    a.cap = cap;
    a.n_q_heads = n_q_heads;
    a.n_kv_heads = n_kv_heads;
    a.group = n_q_heads / n_kv_heads;
    a.rows = p.rows;
    a.n_keys = ctx_len + gamma;
    a.splits = p.splits;
    a.keys_per_split = p.keys_per_split;
    a.n_row_groups = p.n_row_groups;
    a.sl2 = softmax_scale * kLog2e;

    if (dt == WF_BF16) {
        a.q16 = static_cast<const uint16_t *>(q);
        a.k16 = static_cast<const uint16_t *>(k_cache);
        a.v16 = static_cast<const uint16_t *>(v_cache);
        const int units = n_kv_heads * p.splits;
        int blocks = units;
        if (p.n_row_groups > 1)
            blocks = cdiv(units, 8) * 8 * p.n_row_groups;
        dim3 grid(blocks), block(256);
#define WF_ATTN_CASE(DHV, NBV)                                               \
    if (head_dim == DHV && p.nb == NBV) {                                    \
        attn_partial_bf16<DHV, NBV><<<grid, block, 0, stream>>>(a);          \
    } else
        WF_ATTN_CASE(128, 1) WF_ATTN_CASE(128, 2) WF_ATTN_CASE(128, 4)
        WF_ATTN_CASE(64, 1) WF_ATTN_CASE(64, 2) WF_ATTN_CASE(64, 4)
        { return WF_ERR_UNSUPPORTED; }
#undef WF_ATTN_CASE
    } else {
        a.q32 = static_cast<const float *>(q);
        a.k32 = static_cast<const float *>(k_cache);
        a.v32 = static_cast<const float *>(v_cache);
        dim3 grid(p.splits, (unsigned)pairs), block(64);
        if (head_dim == 128)
            attn_partial_f32<128><<<grid, block, 0, stream>>>(a);
        else
            attn_partial_f32<64><<<grid, block, 0, stream>>>(a);
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;

    dim3 mgrid((unsigned)pairs), mblock(64);
    const bool ob = (dt == WF_BF16);
    if (head_dim == 128) {
        if (ob)
            attn_merge<128, true><<<mgrid, mblock, 0, stream>>>(a.ws_acc, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
        else
            attn_merge<128, false><<<mgrid, mblock, 0, stream>>>(a.ws_acc, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
    } else {
        if (ob)
            attn_merge<64, true><<<mgrid, mblock, 0, stream>>>(a.ws_acc, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
        else
            attn_merge<64, false><<<mgrid, mblock, 0, stream>>>(a.ws_acc, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
