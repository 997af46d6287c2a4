// attn.hip -- verification attention of a gamma-row draft block against the
// KV cache (parallel target verification, Sec. 3.2 of the WhiFlash paper).
//
// Split-KV design for batch 1 on MI355X.  Every workgroup owns one KV head g
// and one contiguous slice ("split") of the key range, and processes the
// G*gamma query rows of that head (up to 64 per workgroup), so every K/V
// byte is fetched from HBM once.  Its waves form KS key streams x RG row
// groups; each keeps an fp32 online-softmax state per row.  The streams
// merge through LDS and the workgroup writes one partial per (split, row):
// the unnormalised output row (bf16 on the bf16 path, fp32 otherwise) and
// the fp32 running max and sum.  A second kernel combines the splits in a
// fixed order.
//
// bf16 path, per 32-key tile and wave (16x16x32 bf16 MFMA):
//   S^T = K * Q^T : A = 16 keys x 32 dims from the LDS copy of the K tile,
//                   B = Q^T held in registers for the whole kernel.
//   P   = exp2((S - m) * scale * log2 e), online max/sum per row.
//   O^T += V^T * P^T : B = P^T comes out of the S^T accumulator already in
//                   operand layout (each lane owns 8 consecutive keys of its
//                   row); A = V^T comes from transposing reads of the LDS
//                   copy of the V tile.
#include <type_traits>

#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kTileKeys = 32;

struct AttnParams {
    const uint16_t *q16;      // bf16 path
    const uint16_t *k16;
    const uint16_t *v16;
    const float *q32;         // fp32 path
    const float *k32;
    const float *v32;
    void *ws_o;               // [splits][gamma*n_q_heads][head_dim], unnormalised
                              // partial outputs: bf16 (bf16 path) or fp32
    float *ws_ml;             // [splits][gamma*n_q_heads][2]: running max, sum
    // Tree verification: bit j of tree_mask[i] lets block row i see block
    // row j (row i always sees itself); nullptr = block-causal.
    const uint64_t *tree_mask;
    int gamma, ctx_len, cap, n_q_heads, n_kv_heads, group, rows, n_keys;
    int splits, keys_per_split, n_row_groups;
    float sl2;                // softmax_scale * log2(e)
};

// ---------------------------------------------------------------------------
// bf16 split-KV partial kernel.
//
// Workgroup = KS key streams x RG row groups of waves.  Stream s handles the
// tiles s, s+KS, ... of the workgroup's key split; the RG waves of a stream
// share each tile and own 16*NBW query rows apiece.  Tiles travel HBM -> LDS
// with global_load_lds (no VGPR staging) into a two-deep ring per stream:
// while a step computes on one ring half, the next step's tiles land in the
// other.  All waves advance in lockstep, one barrier per step.
//
// LDS tile = K rows then V rows (row = head_dim bf16).  Both are swizzled so
// the MFMA operand reads are bank-conflict free:
//   K: 16-byte granule g of local key k sits at granule g ^ (k mod GRAN);
//      operand reads are ds_read_b128 of (key 16*mb + m16, granule 4*kk + c4).
//   V: 32-byte segment j of local key k sits at segment j ^ (k mod SEGS);
//      the V^T operand is two ds_read_b64_tr_b16: source lane q of lane group
//      c4 points at dims 16*md + 4*(q%4) of key 16*h + 4*c4 + q/4, and the
//      transpose hands lane q the 4 keys of dim 16*md + q.
// With the natural key order (M-block mb row m = key 16*mb + m) the S^T
// accumulator of lane (m16, c4) holds keys 16*mb + 4*c4 + i of its row --
// exactly the P^T operand the transposed V^T pairs with.
// ---------------------------------------------------------------------------
template <int DH>
struct TileGeom {
    static constexpr int kRowBytes = DH * 2;
    static constexpr int kHalfBytes = kTileKeys * kRowBytes;     // K or V part
    static constexpr int kTileBytes = 2 * kHalfBytes;
    static constexpr int kLoadsPerHalf = kHalfBytes / 1024;       // 1 KB per wave load
    static constexpr int kGran = kRowBytes / 16;
    static constexpr int kSegs = kRowBytes / 32;
};

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define WF_LDS(T) __attribute__((address_space(3))) T

template <int N>
using ic = std::integral_constant<int, N>;

// 32-bit LDS byte address of a __shared__ object.
__device__ __forceinline__ unsigned lds_addr(const void *p) {
    return (unsigned)(uintptr_t)(const WF_LDS(char) *)p;
}

// s_waitcnt vmcnt(n) for the few counts the pipeline needs (n must be a
// compile-time immediate).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt immediate out of range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// HBM -> LDS copy of 16 bytes per lane: lane L's 16 bytes at `src` land at
// LDS byte lds + 16*L (lds wave-uniform).  Written as inline assembly so
// the compiler does not know these loads write LDS: it would otherwise make
// every LDS read wait for all of them.  Completion is tracked by the
// explicit vmcnt waits of the pipeline.
__device__ __forceinline__ void lds_dma16(const void *src, unsigned lds) {
    asm volatile("s_mov_b32 m0, %1\n\t"
                 "s_nop 0\n\t"
                 "global_load_lds_dwordx4 %0, off"
                 :
                 : "v"(src), "s"(lds)
                 : "memory", "m0");
}

// The same copy addressed as a wave-uniform 64-bit base (SGPRs) plus a
// 32-bit per-lane byte offset: no per-lane address arithmetic at issue.
// NT: with the non-temporal hint, for tiles that only this workgroup reads.
template <bool NT = false>
__device__ __forceinline__ void lds_dma16_so(const char *base, unsigned voff, unsigned lds) {
    if constexpr (NT)
        asm volatile("s_mov_b32 m0, %2\n\t"
                     "s_nop 0\n\t"
                     "global_load_lds_dwordx4 %0, %1 nt"
                     :
                     : "v"(voff), "s"(base), "s"(lds)
                     : "memory", "m0");
    else
        asm volatile("s_mov_b32 m0, %2\n\t"
                     "s_nop 0\n\t"
                     "global_load_lds_dwordx4 %0, %1"
                     :
                     : "v"(voff), "s"(base), "s"(lds)
                     : "memory", "m0");
}

// NT: the K/V tiles are copied with the non-temporal hint; the launch sets
// it when one row group covers each head, so a workgroup is the only reader
// of its tiles (several row groups share them through L2).
template <int DH, int NBW, int RG, int KS, int NBUF, bool NT>
__global__ __launch_bounds__(64 * KS * RG) void attn_partial_bf16(AttnParams a) {
    using TG = TileGeom<DH>;
    constexpr int KC = DH / 32;
    constexpr int MD = DH / 16;
    constexpr int ROWS_W = 16 * NBW;
    constexpr int ROWS_WG = ROWS_W * RG;
    constexpr int NLOAD = 2 * TG::kLoadsPerHalf;      // wave loads per tile
    constexpr int LPW = NLOAD / RG;                   // loads per wave per stage
    static_assert(NLOAD % RG == 0, "tile loads must split evenly over row groups");
    static_assert(NBUF >= 2 && NBUF <= 4, "ring depth 2..4");
    constexpr int STAGE_BYTES = KS * TG::kTileBytes;  // one tile per stream

    // Stream-merge regions at the end reuse ring buffers 0 and 1.  Rows are
    // padded by 4 floats so the 16 rows of a wave's accumulator tile fall in
    // distinct banks.
    constexpr int OST = DH + 4;
    constexpr int REGION_BYTES = KS > 1 ? ROWS_WG * OST * 4 : 0;
    constexpr int MAX_RS = STAGE_BYTES > REGION_BYTES ? STAGE_BYTES : REGION_BYTES;
    // Streams 1..KS-1 hand their accumulators to stream 0 through NREG
    // regions: two (fewer merge rounds) when there are two or more such
    // streams and the regions fit.
    constexpr int NREG = (KS >= 3 && 2 * MAX_RS + (NBUF - 2) * STAGE_BYTES +
                          KS * ROWS_WG * 8 + 16 <= 160 * 1024) ? 2 : 1;
    constexpr int RING0_BYTES = STAGE_BYTES > REGION_BYTES ? STAGE_BYTES : REGION_BYTES;
    constexpr int RING1_BYTES = NREG < 2 ? STAGE_BYTES : RING0_BYTES;
    static_assert(RING0_BYTES + RING1_BYTES + (NBUF - 2) * STAGE_BYTES +
                  KS * ROWS_WG * 8 + 16 <= 160 * 1024, "LDS budget");
    // The ring buffers are separate objects, so the compiler can tell reads
    // of one buffer from the LDS-DMA writes still landing in the others.
    __shared__ __attribute__((aligned(1024))) char ring0[RING0_BYTES];
    __shared__ __attribute__((aligned(1024))) char ring1[RING1_BYTES];
    __shared__ __attribute__((aligned(1024))) char ring2[NBUF > 2 ? STAGE_BYTES : 16];
    __shared__ __attribute__((aligned(1024))) char ring3[NBUF > 3 ? STAGE_BYTES : 16];
    __shared__ float mls[KS][ROWS_WG][2];
    __shared__ int overflow;
    if (threadIdx.x == 0)
        overflow = 0;                        // published by the first barrier
    auto ring = [&](auto bi) -> char * {
        constexpr int B = decltype(bi)::value;
        if constexpr (B == 0)
            return ring0;
        else if constexpr (B == 1)
            return ring1;
        else if constexpr (B == 2)
            return ring2;
        else
            return ring3;
    };

    // ---- which (kv head, split, row group) this workgroup owns -------------
    int unit, rgw;
    if (a.n_row_groups == 1) {
        unit = blockIdx.x;
        rgw = 0;
    } else {
        // keep the row groups of one (head, split) on one XCD, adjacent in
        // its dispatch order, so the second reader of a K/V tile hits L2
        const int xcd = blockIdx.x & 7, w = blockIdx.x >> 3;
        rgw = w % a.n_row_groups;
        unit = (w / a.n_row_groups) * 8 + xcd;
    }
    if (unit >= a.n_kv_heads * a.splits)
        return;
    const int g = unit % a.n_kv_heads;
    const int split = unit / a.n_kv_heads;

    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;
    const int stream = wave % KS;
    const int rgi = wave / KS;

    // splits own near-equal runs of whole tiles: [s*T/S, (s+1)*T/S)
    const int tiles_total = (a.n_keys + kTileKeys - 1) / kTileKeys;
    const int t_first = (int)((long long)split * tiles_total / a.splits);
    const int t_last = (int)((long long)(split + 1) * tiles_total / a.splits);
    const int k_begin = t_first * kTileKeys;
    const int n_tiles = t_last - t_first;
    const int n_steps = (n_tiles + KS - 1) / KS;
    const int last_key = a.n_keys - 1;
    const float sl2 = a.sl2;

    const size_t head_off = (size_t)g * a.cap * DH;
    const char *kg = reinterpret_cast<const char *>(a.k16 + head_off);
    const char *vg = reinterpret_cast<const char *>(a.v16 + head_off);

    // Issue this wave's LPW loads of its stream's tile of stage `st` into
    // ring buffer `bi`.  Load j < kLoadsPerHalf fills K rows, the rest V
    // rows; lane L of load j writes LDS bytes 16*(64*j' + L) of its half
    // (j' = j mod kLoadsPerHalf).  A stream whose tile lies past the split
    // (ragged last stage) loads the split's last tile again, so every wave
    // issues the same number of loads per stage; that copy is never used.
    // Each lane's byte offset within a tile is the same for every tile, so
    // it is formed once; only a tile reaching past the last key clamps its
    // keys one by one.
    auto src_off = [&](int jr, int kl_cap) -> unsigned {
        const int j = rgi + jr * RG;
        const bool is_v = j >= TG::kLoadsPerHalf;
        const int jj = is_v ? j - TG::kLoadsPerHalf : j;
        const int gidx = jj * kWave + lane;            // granule in the half
        const int kl = gidx / TG::kGran;                // local key
        const int pg = gidx % TG::kGran;                // physical granule
        int lg;                                         // logical granule
        if (!is_v) {
            lg = pg ^ (kl & (TG::kGran - 1));
        } else {
            const int seg = (pg >> 1) ^ (kl & (TG::kSegs - 1));
            lg = 2 * seg + (pg & 1);
        }
        return (unsigned)(min(kl, kl_cap) * TG::kRowBytes + lg * 16);
    };
    // (kept in registers only for up to 8 loads per wave and stage; with
    // more, the extra registers cost more than the address arithmetic)
    constexpr bool kKeepOff = LPW <= 8;
    unsigned voff[kKeepOff ? LPW : 1];
#pragma unroll
    for (int jr = 0; jr < (kKeepOff ? LPW : 1); ++jr)
        voff[jr] = src_off(jr, kTileKeys - 1);
    auto issue = [&](auto bi, int st) __attribute__((always_inline)) {
        const int t = min(KS * st + stream, n_tiles - 1);
        const int kb = k_begin + t * kTileKeys;
        const unsigned slot = lds_addr(ring(bi)) + stream * TG::kTileBytes;
        const size_t tile_off = (size_t)kb * TG::kRowBytes;
        auto go = [&](auto clamp_tag, auto nt_tag) __attribute__((always_inline)) {
#pragma unroll
            for (int jr = 0; jr < LPW; ++jr) {
                const int j = rgi + jr * RG;
                const bool is_v = j >= TG::kLoadsPerHalf;
                const int jj = is_v ? j - TG::kLoadsPerHalf : j;
                unsigned off;
                if constexpr (decltype(clamp_tag)::value)
                    off = src_off(jr, last_key - kb);
                else if constexpr (kKeepOff)
                    off = voff[jr];
                else
                    off = src_off(jr, kTileKeys - 1);
                lds_dma16_so<decltype(nt_tag)::value>(
                    (is_v ? vg : kg) + tile_off, off, slot + (is_v ? TG::kHalfBytes : 0) + jj * 1024);
            }
        };
        if (kb + kTileKeys - 1 <= last_key)
            go(std::false_type{}, std::integral_constant<bool, NT>{});
        else
            go(std::true_type{}, std::integral_constant<bool, NT>{});
    };

    // ---- Q^T operands and causal limits of this wave's rows ------------------
    const int row0 = rgw * ROWS_WG + rgi * ROWS_W;
    const bool tree = a.tree_mask != nullptr;   // kernel argument: uniform
    const uint64_t gbits = a.gamma >= 64 ? ~0ull : (1ull << a.gamma) - 1ull;
    bf16x8 qf[NBW][KC];
    int lim[NBW];
    uint64_t tm[NBW];                 // tree mode: block rows the row sees
    auto load_q = [&]() {
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
            const int r = row0 + nb * 16 + m16;
            const int rc = min(r, a.rows - 1);
            const int i = rc / a.group;
            const int h = g * a.group + (rc % a.group);
            const uint16_t *qp = a.q16 + ((size_t)i * a.n_q_heads + h) * DH + c4 * 8;
#pragma unroll
            for (int kk = 0; kk < KC; ++kk)
                qf[nb][kk] = load_bf16x8(qp + kk * 32);
            // padding rows (r >= rows) reuse a real row's query and are never
            // stored; they must not be masked harder than it
            lim[nb] = a.ctx_len + i;
            tm[nb] = tree ? ((a.tree_mask[i] | (1ull << i)) & gbits) : 0ull;
        }
    };

    f32x4 o[MD][NBW];
    float mref[NBW], lrow[NBW];
    float moff[NBW];                  // -mref * sl2 (0 while mref is -inf)

    // Operands of a tile from LDS:
    //   K: ds_read_b128 of (key 16*mb + m16, granule 4*kk + c4).
    //   V^T: two transposing reads per 16 dims.
    auto read_k = [&](auto bi, bf16x8 (&kop)[2][KC]) __attribute__((always_inline)) {
        const WF_LDS(char) *kt = (const WF_LDS(char) *)ring(bi) + stream * TG::kTileBytes;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const int kl = 16 * mb + m16;
#pragma unroll
            for (int kk = 0; kk < KC; ++kk) {
                const int pg = (4 * kk + c4) ^ (kl & (TG::kGran - 1));
                kop[mb][kk] = __builtin_bit_cast(
                    bf16x8, *(const WF_LDS(u32x4) *)(kt + kl * TG::kRowBytes + pg * 16));
            }
        }
    };
    auto read_vt = [&](auto bi, bf16x8 (&vop)[MD]) __attribute__((always_inline)) {
        const WF_LDS(char) *vt = (const WF_LDS(char) *)ring(bi) + stream * TG::kTileBytes +
                                 TG::kHalfBytes;
        const int q4 = m16 & 3, qk = m16 >> 2;
#pragma unroll
        for (int md = 0; md < MD; ++md) {
            v4i16 half[2];
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const int kl = 16 * hh + 4 * c4 + qk;
                const int ps = md ^ (kl & (TG::kSegs - 1));
                half[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (WF_LDS(v4i16) *)(vt + kl * TG::kRowBytes + ps * 32 + q4 * 8));
            }
            typedef short v8i16 __attribute__((ext_vector_type(8)));
            const v8i16 both = __builtin_shufflevector(half[0], half[1], 0, 1, 2, 3, 4, 5, 6, 7);
            vop[md] = __builtin_bit_cast(bf16x8, both);
        }
    };

    auto compute = [&](auto bi, int t, auto rescale_tag) __attribute__((always_inline)) {
        constexpr bool RESCALE = decltype(rescale_tag)::value;
        bf16x8 kop[2][KC], vop[MD];
        read_k(bi, kop);
        read_vt(bi, vop);
        // S^T = K Q^T
        f32x4 s[2][NBW];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                s[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < KC; ++kk)
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    s[mb][nb] = mfma16x16x32(kop[mb][kk], qf[nb][kk], s[mb][nb]);
        }
        // mask: only tiles reaching into the block (block-causal: past its
        // first row, which every row sees; tree: from its first row on)
        const int kb = k_begin + t * kTileKeys;
        if (tree) {
            if (kb + kTileKeys - 1 >= a.ctx_len) {
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
                    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int j = kb + 16 * mb + 4 * c4 + i - a.ctx_len;
                            bool vis;
                            if constexpr (NBW == 1) {
                                // branch-free (selects, no exec-mask
                                // branches): j < gamma <= 64 bounds the shift
                                const bool bit = ((tm[nb] >> (j & 63)) & 1ull) != 0;
                                vis = (j < 0) | ((j < a.gamma) & bit);
                            } else {
                                // (the select form's extra registers make
                                // the two-block waves spill)
                                vis = j < 0 || (j < a.gamma && ((tm[nb] >> j) & 1ull));
                            }
                            s[mb][nb][i] = vis ? s[mb][nb][i] : -INFINITY;
                        }
            }
        } else if (kb + kTileKeys - 1 > a.ctx_len) {
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = kb + 16 * mb + 4 * c4 + i;
                        s[mb][nb][i] = (key > lim[nb]) ? -INFINITY : s[mb][nb][i];
                    }
        }
        // lane-local maxima over the lane's 8 keys of each row
        auto lane_max = [&](int nb) {
            return fmaxf(fmaxf(fmaxf(s[0][nb][0], s[0][nb][1]), fmaxf(s[0][nb][2], s[0][nb][3])),
                         fmaxf(fmaxf(s[1][nb][0], s[1][nb][1]), fmaxf(s[1][nb][2], s[1][nb][3])));
        };
        auto row_max = [&](float m) {
            m = fmaxf(m, __shfl_xor(m, 16, kWave));
            return fmaxf(m, __shfl_xor(m, 32, kWave));
        };
        if constexpr (RESCALE) {
            float mx[NBW];
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                mx[nb] = row_max(lane_max(nb));
            bool grow = false;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                grow |= (mx[nb] - mref[nb]) * sl2 > 8.f;
            if (__ballot(grow)) {
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) {
                    const float nr = ((mx[nb] - mref[nb]) * sl2 > 8.f) ? mx[nb] : mref[nb];
                    const float alpha = (nr == mref[nb]) ? 1.f : fast_exp2((mref[nb] - nr) * sl2);
                    lrow[nb] *= alpha;
#pragma unroll
                    for (int md = 0; md < MD; ++md)
                        o[md][nb] *= alpha;
                    mref[nb] = nr;
                    moff[nb] = (nr == -INFINITY) ? 0.f : -nr * sl2;
                }
            }
        } else {
            // The reference maximum of a row is its maximum over the first
            // tile with a visible key (O and l are still zero until then);
            // only that tile needs the lane maxima and the cross-lane
            // reduction.
            bool unset = false;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                unset |= mref[nb] == -INFINITY;
            if (__ballot(unset)) {
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) {
                    const float m = row_max(lane_max(nb));
                    if (mref[nb] == -INFINITY) {
                        mref[nb] = m;
                        moff[nb] = (m == -INFINITY) ? 0.f : -m * sl2;
                    }
                }
            }
        }
        // P = exp2((S - mref) * scale * log2 e) in the P^T operand layout
        bf16x8 pb[NBW];
        bool over = false;
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
            float p[8];
            float psum = 0.f;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float e = fast_exp2(fmaf(s[mb][nb][i], sl2, moff[nb]));
                    p[4 * mb + i] = e;
                    psum += e;
                }
            // Without rescaling, a weight above 2^64 means a score outgrew
            // the row's reference maximum by more than 64 log2 units; the
            // lane's sum of its non-negative weights exceeds 2^64 whenever
            // one of them does (and is +inf if one overflowed), so testing
            // the sum catches every such growth.
            if constexpr (!RESCALE)
                over |= psum > 0x1p64f;
            lrow[nb] += psum;
            u32x4 pv = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                        pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
            pb[nb] = __builtin_bit_cast(bf16x8, pv);
        }
        if constexpr (!RESCALE) {
            if (__ballot(over))
                overflow = 1;                // the workgroup reruns rescaling
        }
        // O^T += V^T P^T
#pragma unroll
        for (int md = 0; md < MD; ++md)
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                o[md][nb] = mfma16x16x32(vop[md], pb[nb], o[md][nb]);
    };

    // One pipeline step: stage st sits in ring buffer bi.  Up to NBUF-1
    // stages are in flight; the wait leaves the later ones outstanding.
    // After the barrier stage st is complete in LDS (each wave waited for
    // its own loads of it) and every wave is done with the buffer of stage
    // st-1 (its reads returned before they fed the MFMAs), which then
    // receives stage st+NBUF-1.  The barrier is a bare s_barrier: the
    // compiler-generated fence of __syncthreads() would wait for the loads
    // of every later stage as well.
    auto step = [&](auto bi, int st, auto rescale_tag) __attribute__((always_inline)) {
        constexpr int B = decltype(bi)::value;
        const int later = min(NBUF - 2, n_steps - 1 - st);   // stages issued after st
        if (later >= 2)
            wait_vmcnt<2 * LPW>();
        else if (later == 1)
            wait_vmcnt<LPW>();
        else
            wait_vmcnt<0>();
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (st + NBUF - 1 < n_steps)
            issue(ic<(B + NBUF - 1) % NBUF>{}, st + NBUF - 1);
        const int t = KS * st + stream;
        if (t < n_tiles)
            compute(bi, t, rescale_tag);
    };

    // One pass over the split; the step loop is unrolled by the ring depth so
    // every step names its ring buffer at compile time.
    auto pass = [&](auto rescale_tag, bool first_pass) __attribute__((always_inline)) {
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
            mref[nb] = -INFINITY;
            moff[nb] = 0.f;
            lrow[nb] = 0.f;
#pragma unroll
            for (int md = 0; md < MD; ++md)
                o[md][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        if (first_pass)
            load_q();
        issue(ic<0>{}, 0);
        if (NBUF > 2 && 1 < n_steps)
            issue(ic<1 % NBUF>{}, 1);
        if (NBUF > 3 && 2 < n_steps)
            issue(ic<2 % NBUF>{}, 2);
        if (first_pass) {
            // The Q loads precede every DMA; once they are in, tie the
            // registers so the compiler sees no load pending on them in
            // the step loop (it would otherwise drain all DMA there).
            const int issued = min(NBUF - 1, n_steps);
            if (issued >= 3)
                wait_vmcnt<3 * LPW>();
            else if (issued == 2)
                wait_vmcnt<2 * LPW>();
            else
                wait_vmcnt<LPW>();
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
                for (int kk = 0; kk < KC; ++kk)
                    asm volatile("" : "+v"(qf[nb][kk]));
        }
        for (int st = 0; st < n_steps; st += NBUF) {
            step(ic<0>{}, st, rescale_tag);
            if (st + 1 >= n_steps)
                break;
            step(ic<1>{}, st + 1, rescale_tag);
            if constexpr (NBUF > 2) {
                if (st + 2 >= n_steps)
                    break;
                step(ic<2 % NBUF>{}, st + 2, rescale_tag);
            }
            if constexpr (NBUF > 3) {
                if (st + 3 >= n_steps)
                    break;
                step(ic<3 % NBUF>{}, st + 3, rescale_tag);
            }
        }
        __syncthreads();
    };

    pass(std::false_type{}, true);
    if (overflow)                            // uniform: read after a barrier
        pass(std::true_type{}, false);

    // ---- per-wave row sums (the 4 K-groups of a row hold disjoint keys) -----
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        float l = lrow[nb];
        l += __shfl_xor(l, 16, kWave);
        l += __shfl_xor(l, 32, kWave);
        lrow[nb] = l;
        if (KS > 1 && c4 == 0) {
            mls[stream][rgi * ROWS_W + nb * 16 + m16][0] = mref[nb];
            mls[stream][rgi * ROWS_W + nb * 16 + m16][1] = l;
        }
    }
    // (one key stream: each row's state is complete in its wave's registers)
    if constexpr (KS > 1)
        __syncthreads();

    // ---- merge the KS streams of each row ------------------------------------
    // Stream s >= 1 adds its rescaled accumulator into region (s-1) % NREG in
    // round (s-1) / NREG (round 0 stores); stream 0 then adds the regions to
    // its own registers, in region order, and writes the partial straight
    // from registers -- a fixed summation order.
    auto oreg = [&](int r) { return (WF_LDS(float) *)(r ? ring1 : ring0); };
    float fac[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        if constexpr (KS == 1) {
            fac[nb] = 1.f;               // a row without visible keys has o == 0
            continue;
        }
        const int r = rgi * ROWS_W + nb * 16 + m16;
        float mm = -INFINITY;
#pragma unroll
        for (int st = 0; st < KS; ++st)
            mm = fmaxf(mm, mls[st][r][0]);
        const float muse = (mm == -INFINITY) ? 0.f : mm;
        fac[nb] = (mref[nb] == -INFINITY) ? 0.f : fast_exp2((mref[nb] - muse) * sl2);
    }
    // Two key streams whose merged rows fit a ring buffer as bf16: each
    // stream owns half the head dims (stream s: dim blocks [s*MD/2,
    // (s+1)*MD/2)) and hands the other half, rescaled, to the other stream
    // through ring0; each adds the half it receives to its own rescaled half
    // (the same two terms as the single hand-off, rounded once more or less
    // where the compiler fuses the multiply into the add), stages its merged
    // half as bf16 rows, and then every wave of the workgroup writes the
    // rows out as 16-byte pieces (draft trees, 64-row workgroups: 23.35 ->
    // 22.80 us per call at 244 rows and 8K keys; 32B shapes, 128-row
    // workgroups: 60.3 -> 59.8 us at 64K keys; with 16 or 32 rows the extra
    // barrier is not paid back, so those keep the single hand-off below).
    constexpr int SRB = DH * 2 + 16;                 // padded staged row bytes
    // (the staged rows fill ring1, or ring1 and ring2 half and half)
    constexpr int SHALF = ROWS_WG * SRB <= RING1_BYTES ? ROWS_WG : ROWS_WG / 2;
    constexpr bool SPLIT2 = KS == 2 && MD % 2 == 0 && ROWS_WG >= 64 &&
                            SHALF * SRB <= RING1_BYTES &&
                            (SHALF == ROWS_WG || (NBUF > 2 && SHALF * SRB <= STAGE_BYTES));
    if constexpr (SPLIT2) {
        constexpr int MH = MD / 2;
        WF_LDS(float) *reg = oreg(0);
        auto srow = [&](int row) {                   // staged row address
            if constexpr (SHALF == ROWS_WG)
                return (WF_LDS(char) *)ring1 + row * SRB;
            else
                return (WF_LDS(char) *)(row < SHALF ? ring1 : ring2) + (row % SHALF) * SRB;
        };
        auto give = [&](auto base_tag) __attribute__((always_inline)) {
            constexpr int B = decltype(base_tag)::value;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                const int rl = rgi * ROWS_W + nb * 16 + m16;
#pragma unroll
                for (int mh = 0; mh < MH; ++mh)
                    *(WF_LDS(f32x4) *)(reg + rl * OST + (B + mh) * 16 + 4 * c4) =
                        o[B + mh][nb] * fac[nb];
            }
        };
        auto take = [&](auto base_tag) __attribute__((always_inline)) {
            constexpr int B = decltype(base_tag)::value;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                const int rl = rgi * ROWS_W + nb * 16 + m16;
#pragma unroll
                for (int mh = 0; mh < MH; ++mh) {
                    const int md = B + mh;
                    const f32x4 v = o[md][nb] * fac[nb] +
                                    *(WF_LDS(const f32x4) *)(reg + rl * OST + md * 16 + 4 * c4);
                    *(WF_LDS(u32x2) *)(srow(rl) + (md * 16 + 4 * c4) * 2) =
                        u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                }
            }
        };
        if (stream == 0)
            give(ic<MH>{});
        else
            give(ic<0>{});
        __syncthreads();
        if (stream == 0)
            take(ic<0>{});
        else
            take(ic<MH>{});
        const int pairs = a.gamma * a.n_q_heads;
        if (stream == 0 && c4 == 0) {
            // the row's (max, sum) over both streams
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                const int rl = rgi * ROWS_W + nb * 16 + m16;
                const int r = rgw * ROWS_WG + rl;
                if (r >= a.rows)
                    continue;
                const size_t pr = (size_t)split * pairs + (size_t)(r / a.group) * a.n_q_heads +
                                  g * a.group + (r % a.group);
                float mm = -INFINITY, ll = 0.f;
#pragma unroll
                for (int st = 0; st < KS; ++st)
                    mm = fmaxf(mm, mls[st][rl][0]);
                const float muse = (mm == -INFINITY) ? 0.f : mm;
#pragma unroll
                for (int st = 0; st < KS; ++st) {
                    const float mw = mls[st][rl][0];
                    const float f = (mw == -INFINITY) ? 0.f : fast_exp2((mw - muse) * sl2);
                    ll = fmaf(mls[st][rl][1], f, ll);
                }
                a.ws_ml[pr * 2] = mm;
                a.ws_ml[pr * 2 + 1] = ll;
            }
        }
        __syncthreads();
        // whole rows of consecutive (row, head) pairs, 16 bytes per lane
        constexpr int PPR = DH / 8;                  // 16-byte pieces per row
        for (int pc = threadIdx.x; pc < ROWS_WG * PPR; pc += 64 * KS * RG) {
            const int row = pc / PPR, col = pc % PPR;
            const int r = rgw * ROWS_WG + row;
            if (r < a.rows) {
                const size_t pr = (size_t)split * pairs + (size_t)(r / a.group) * a.n_q_heads +
                                  g * a.group + (r % a.group);
                reinterpret_cast<u32x4 *>(static_cast<uint16_t *>(a.ws_o) + pr * DH)[col] =
                    *(const WF_LDS(u32x4) *)(srow(row) + col * 16);
            }
        }
        return;
    }
    if constexpr (KS > 1) {
        constexpr int ROUNDS = (KS - 1 + NREG - 1) / NREG;
#pragma unroll 1
        for (int round = 0; round < ROUNDS; ++round) {
            if (stream >= 1 && (stream - 1) / NREG == round) {
                WF_LDS(float) *reg = oreg((stream - 1) % NREG);
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
                    for (int md = 0; md < MD; ++md) {
                        WF_LDS(float) *dst = reg + (rgi * ROWS_W + nb * 16 + m16) * OST + md * 16 + 4 * c4;
                        f32x4 v = o[md][nb] * fac[nb];
                        if (round > 0)
                            v += *(WF_LDS(f32x4) *)dst;
                        *(WF_LDS(f32x4) *)dst = v;
                    }
            }
            __syncthreads();
        }
    }
    if (stream != 0)
        return;

    // ---- write the workgroup partial (stream 0 waves) ------------------------
    // Lane (m16, c4) holds dims md*16 + 4*c4 .. +3 of row nb*16 + m16.
    constexpr int NR = KS - 1 < NREG ? KS - 1 : NREG;   // regions in use
    const int pairs = a.gamma * a.n_q_heads;
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int rl = rgi * ROWS_W + nb * 16 + m16;
        const int r = rgw * ROWS_WG + rl;
        if (r >= a.rows)
            continue;
        const int i = r / a.group;
        const int h = g * a.group + (r % a.group);
        const size_t pr = (size_t)split * pairs + (size_t)i * a.n_q_heads + h;
        uint2 *dst = reinterpret_cast<uint2 *>(static_cast<uint16_t *>(a.ws_o) + pr * DH);
        if constexpr (KS == 1 && NBW == 1) {
            // one key stream, 16 rows per wave: stage the bf16 rows in the
            // (idle) ring so they leave in 16-byte pieces below
            constexpr int RB = DH * 2 + 16;              // padded row bytes
            static_assert(2 * 16 * RB <= STAGE_BYTES, "staging exceeds a ring slot");
            static_assert(RG <= 4, "two waves per ring buffer");
            WF_LDS(char) *stg = (WF_LDS(char) *)(rgi < 2 ? ring0 : ring1) + (rgi & 1) * 16 * RB;
#pragma unroll
            for (int md = 0; md < MD; ++md) {
                f32x4 v = o[md][nb] * fac[nb];
                *(WF_LDS(u32x2) *)(stg + m16 * RB + (md * 16 + 4 * c4) * 2) =
                    u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
            }
        } else {
#pragma unroll
        for (int md = 0; md < MD; ++md) {
            f32x4 v = o[md][nb] * fac[nb];
#pragma unroll
            for (int rr = 0; rr < NR; ++rr)
                v += *(WF_LDS(const f32x4) *)(oreg(rr) + rl * OST + md * 16 + 4 * c4);
            // bf16 partials: the split merge weighs them by at most 1 and
            // the output is rounded to bf16 anyway
            dst[md * 4 + c4] = uint2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        }
        }
        if (KS == 1 && c4 == 0) {
            a.ws_ml[pr * 2] = mref[nb];
            a.ws_ml[pr * 2 + 1] = lrow[nb];
        } else if (c4 == 0) {
            float mm = -INFINITY, ll = 0.f;
#pragma unroll
            for (int st = 0; st < KS; ++st)
                mm = fmaxf(mm, mls[st][rl][0]);
            const float muse = (mm == -INFINITY) ? 0.f : mm;
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const float mw = mls[st][rl][0];
                const float f = (mw == -INFINITY) ? 0.f : fast_exp2((mw - muse) * sl2);
                ll = fmaf(mls[st][rl][1], f, ll);
            }
            a.ws_ml[pr * 2] = mm;
            a.ws_ml[pr * 2 + 1] = ll;
        }
    }
    if constexpr (KS == 1 && NBW == 1) {
        // the wave's 16 staged rows leave as 16-byte pieces: each store
        // writes whole rows of consecutive (row, head) pairs
        constexpr int RB = DH * 2 + 16;
        constexpr int PPR = DH / 8;                    // 16-byte pieces per row
        const WF_LDS(char) *stg = (const WF_LDS(char) *)(rgi < 2 ? ring0 : ring1) + (rgi & 1) * 16 * RB;
        const int pairs2 = a.gamma * a.n_q_heads;
#pragma unroll
        for (int pc = lane; pc < 16 * PPR; pc += kWave) {
            const int row = pc / PPR, col = pc % PPR;
            const int r = rgw * ROWS_WG + rgi * ROWS_W + row;
            if (r < a.rows) {
                const int i = r / a.group;
                const int h = g * a.group + (r % a.group);
                const size_t pr = (size_t)split * pairs2 + (size_t)i * a.n_q_heads + h;
                reinterpret_cast<u32x4 *>(static_cast<uint16_t *>(a.ws_o) + pr * DH)[col] =
                    *(const WF_LDS(u32x4) *)(stg + row * RB + col * 16);
            }
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
    const bool tree = a.tree_mask != nullptr;
    const uint64_t gbits = a.gamma >= 64 ? ~0ull : (1ull << a.gamma) - 1ull;
    const uint64_t tm = tree ? ((a.tree_mask[i] | (1ull << i)) & gbits) : 0ull;
    const int k_end = min(min(a.n_keys, k_begin + a.keys_per_split),
                          tree ? a.n_keys : a.ctx_len + i + 1);
    const float *kbase = a.k32 + (size_t)g * a.cap * DH;
    const float *vbase = a.v32 + (size_t)g * a.cap * DH;

    float m = -INFINITY, l = 0.f, acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e)
        acc[e] = 0.f;

    for (int kb = k_begin; kb < k_end; kb += kWave) {
        const int j = kb + lane;
        const int jb = j - a.ctx_len;
        const bool vis = j < k_end && (!tree || jb < 0 || ((tm >> jb) & 1ull));
        float sc = -INFINITY;
        if (vis) {
            const float *kr = kbase + (size_t)j * DH;
            float dot = 0.f;
#pragma unroll 16
            for (int d = 0; d < DH; ++d)
                dot = fmaf(qs[d], kr[d], dot);
            sc = dot;
        }
        const float mnew = fmaxf(m, wave_max(sc));
        const float alpha = (m == -INFINITY) ? 0.f : exp2f((m - mnew) * a.sl2);
        const float p = vis ? exp2f((sc - mnew) * a.sl2) : 0.f;
        l = fmaf(l, alpha, wave_sum(p));
#pragma unroll
        for (int e = 0; e < E; ++e)
            acc[e] *= alpha;
        // every key up to cnt is a cache row in range; a masked key has
        // p = 0 and adds nothing (no branch, so the loads can be batched)
        const int cnt = min(kWave, k_end - kb);
#pragma unroll 16
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
        static_cast<float *>(a.ws_o)[prs * DH + lane + e * kWave] = acc[e];
    if (lane == 0) {
        a.ws_ml[prs * 2] = m;
        a.ws_ml[prs * 2 + 1] = l;
    }
}

// ---------------------------------------------------------------------------
// Split merge: out = sum_s w_s acc_s / sum_s w_s l_s, w_s = exp(m_s - max m).
// One wave per (row, q head).  Lane L owns float4 column L % (head_dim/4)
// of the splits L / (head_dim/4), + G, + 2G, ... (G split groups per wave),
// accumulated in ascending order; the groups are then added with a fixed
// butterfly.  The first batch of partial loads is issued before the weights
// are formed, so a merge over up to G*kMergeBatch splits is one round trip.
// ---------------------------------------------------------------------------
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
constexpr int kMergeBatch = 16;          // float4 loads in flight per lane
constexpr int kMaxSplits = 1024;

// BF16: partials and output in bf16 (else fp32).
template <int DH, bool BF16>
__global__ __launch_bounds__(64) void attn_merge(const void *__restrict__ ws_o,
                                                 const float *__restrict__ ws_ml,
                                                 void *out, int pairs, int splits,
                                                 float sl2) {
    constexpr int Q = DH / 4;                // 4-element columns of a row
    constexpr int G = kWave / Q;             // split groups per wave
    constexpr int B = kMergeBatch;
    __shared__ float wsh[kMaxSplits];
    const int pr = blockIdx.x;
    const int lane = threadIdx.x;
    const int d4 = lane % Q;
    const int grp = lane / Q;
    const size_t sstride = (size_t)pairs * Q;    // column stride between splits

    auto load_batch = [&](int s0, f32x4 (&v)[B]) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const size_t idx = (size_t)min(s0 + G * b, splits - 1) * sstride +
                               (size_t)pr * Q + d4;
            if constexpr (BF16) {
                // (each partial is read once: non-temporal)
            const u32x2 pt = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(ws_o) + idx);
            const uint2 pk = {pt.x, pt.y};
                v[b] = f32x4{bf16_to_f32((uint16_t)pk.x), bf16_to_f32((uint16_t)(pk.x >> 16)),
                             bf16_to_f32((uint16_t)pk.y), bf16_to_f32((uint16_t)(pk.y >> 16))};
            } else {
                v[b] = reinterpret_cast<const f32x4 *>(ws_o)[idx];
            }
        }
    };
    f32x4 v[B];
    load_batch(grp, v);

    // weights of every split (lane j: splits j, j + 64, ...)
    float mloc = -INFINITY;
    for (int s = lane; s < splits; s += kWave)
        mloc = fmaxf(mloc, ws_ml[((size_t)s * pairs + pr) * 2]);
    const float mm = wave_max(mloc);
    const float muse = (mm == -INFINITY) ? 0.f : mm;
    float lpart = 0.f;
    for (int s = lane; s < splits; s += kWave) {
        const size_t ps = (size_t)s * pairs + pr;
        const float ms = ws_ml[ps * 2];
        const float w = (ms == -INFINITY) ? 0.f : fast_exp2((ms - muse) * sl2);
        wsh[s] = w;
        lpart = fmaf(w, ws_ml[ps * 2 + 1], lpart);
    }
    const float inv = 1.f / wave_sum(lpart);
    __syncthreads();

    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = grp;; s0 += G * B) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int sp = s0 + G * b;
            if (sp < splits)
                acc += wsh[sp] * v[b];
        }
        if (s0 + G * B >= splits)
            break;
        load_batch(s0 + G * B, v);
    }
#pragma unroll
    for (int off = Q; off < kWave; off *= 2) {
        f32x4 o;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            o[c] = __shfl_xor(acc[c], off, kWave);
        acc += o;
    }
    if (grp == 0) {
        const size_t oi = (size_t)pr * DH + 4 * d4;
        const f32x4 r = acc * inv;
        if (BF16) {
            uint2 pk = {pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3])};
            *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(out) + oi) = pk;
        } else {
            *reinterpret_cast<f32x4 *>(static_cast<float *>(out) + oi) = r;
        }
    }
}

// Split merge for up to G*kMergeBatch splits (every plan of the bf16 path
// at head_dim 128 uses at most 32): WPB waves per workgroup, one per
// (row, q head).  Lane (group grp, column d4) loads, in one batch, the
// partial columns of its splits grp, grp + G, ... together with their
// (max, sum) pairs, so the whole merge is one memory round trip: the group
// maxima meet in a butterfly over the G groups, each lane weighs its own
// splits in ascending order, and the weighted columns and sums meet in a
// second fixed butterfly (every lane of a column ends with the same bits).
template <int DH, bool BF16, int WPB>
__global__ __launch_bounds__(64 * WPB) void attn_merge_one(const void *__restrict__ ws_o,
                                                           const float *__restrict__ ws_ml,
                                                           void *out, int pairs, int splits,
                                                           float sl2) {
    constexpr int Q = DH / 4;
    constexpr int G = kWave / Q;
    constexpr int B = kMergeBatch;
    const int pr = blockIdx.x * WPB + wave_id();
    if (pr >= pairs)
        return;
    const int lane = threadIdx.x % kWave;
    const int d4 = lane % Q;
    const int grp = lane / Q;
    const size_t sstride = (size_t)pairs * Q;
    f32x4 v[B];
    float2 ml[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const int sp = min(grp + G * b, splits - 1);
        const size_t idx = (size_t)sp * sstride + (size_t)pr * Q + d4;
        if constexpr (BF16) {
            // (each partial is read once: non-temporal)
            const u32x2 pt = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(ws_o) + idx);
            const uint2 pk = {pt.x, pt.y};
            v[b] = f32x4{bf16_to_f32((uint16_t)pk.x), bf16_to_f32((uint16_t)(pk.x >> 16)),
                         bf16_to_f32((uint16_t)pk.y), bf16_to_f32((uint16_t)(pk.y >> 16))};
        } else {
            v[b] = reinterpret_cast<const f32x4 *>(ws_o)[idx];
        }
        ml[b] = reinterpret_cast<const float2 *>(ws_ml)[(size_t)sp * pairs + pr];
    }
    float mx = -INFINITY;
#pragma unroll
    for (int b = 0; b < B; ++b)
        if (grp + G * b < splits)
            mx = fmaxf(mx, ml[b].x);
#pragma unroll
    for (int off = Q; off < kWave; off *= 2)
        mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
    const float muse = (mx == -INFINITY) ? 0.f : mx;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float lsum = 0.f;
#pragma unroll
    for (int b = 0; b < B; ++b) {
        if (grp + G * b < splits) {
            const float w = (ml[b].x == -INFINITY) ? 0.f : fast_exp2((ml[b].x - muse) * sl2);
            lsum = fmaf(w, ml[b].y, lsum);
            acc += w * v[b];
        }
    }
#pragma unroll
    for (int off = Q; off < kWave; off *= 2) {
        f32x4 o;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            o[c] = __shfl_xor(acc[c], off, kWave);
        acc += o;
        lsum += __shfl_xor(lsum, off, kWave);
    }
    if (grp == 0) {
        const size_t oi = (size_t)pr * DH + 4 * d4;
        const f32x4 r = acc * (1.f / lsum);
        if constexpr (BF16) {
            *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(out) + oi) =
                uint2{pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3])};
        } else {
            *reinterpret_cast<f32x4 *>(static_cast<float *>(out) + oi) = r;
        }
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
        p.part_bytes = 2;
        // rows per wave 16*nb; rg row groups x ks key streams per workgroup
        // (at most 8 waves, so each wave may hold up to 256 registers)
        // and a ring of nbuf stages of ks tiles (LDS: nbuf*ks tiles)
        // (65-128 rows, e.g. 64 q heads over 8 KV heads with a 16-token
        // block: one 128-row workgroup per (head, split), 60 against 72 us
        // at 64K keys with two 64-row ones; more rows, e.g. a draft tree's
        // 244: 64-row workgroups in several row groups, 26.1 against
        // 27.8 us at 8K keys with 128-row ones)
        // (up to 64 rows: one key stream of four 16-row waves, 31.3 against
        // 32.2 us with two streams at 32K keys; up to 32 rows: two streams
        // and a three-stage ring, 13.5 against 14.9 us with four streams at
        // 8K keys, 30.1 against 31.7 us at 32K keys for 16 rows)
        if (rows <= 16) {
            p.nb = 1; p.rg = 1; p.ks = 2; p.nbuf = 3;
        } else if (rows <= 32) {
            p.nb = 1; p.rg = 2; p.ks = 2; p.nbuf = 3;
        } else if (rows <= 64) {
            p.nb = 1; p.rg = 4; p.ks = 1; p.nbuf = 3;
        } else if (rows > 128) {
            p.nb = 1; p.rg = 4; p.ks = 2; p.nbuf = 3;
        } else {
            p.nb = 2; p.rg = 4; p.ks = 2; p.nbuf = 3;
        }
        p.n_row_groups = cdiv(rows, 16 * p.nb * p.rg);
    } else {
        p.part_bytes = 4;
        p.nb = 0;
        p.rg = 1;
        p.ks = 1;
        p.nbuf = 0;
        p.n_row_groups = 1;
    }
    int splits = num_splits;
    if (splits <= 0) {
        // one workgroup per CU of the 256-CU chip, but give every key
        // stream of a workgroup at least two tiles (fp32: one wave per
        // split and pair, at least one 64-key block each); a single
        // token over 4K keys: 32 splits per head, 9.4 against 10.6 us
        // with 16
        const int target = std::max(1, 256 / (n_kv_heads * p.n_row_groups));
        const int max_by_work = dt == WF_BF16
                                    ? std::max(1, n_tiles / (2 * p.ks))
                                    : std::max(1, cdiv(n_keys, kWave));
        splits = std::max(1, std::min(target, max_by_work));
    }
    splits = std::min(splits, n_tiles);
    if (dt == WF_BF16) {
        // the bf16 kernel deals whole tiles out evenly: [s*T/S, (s+1)*T/S)
        p.splits = splits;
        p.keys_per_split = 0;
    } else {
        // fp32: contiguous key ranges of whole tiles; drop splits left empty
        const int tiles_per_split = cdiv(n_tiles, splits);
        p.keys_per_split = tiles_per_split * kTileKeys;
        p.splits = cdiv(n_keys, p.keys_per_split);
    }
    return p;
}

// Workspace: counter block, then [splits][pairs][2] fp32 (max, sum), then
// the [splits][pairs][head_dim] partial outputs (p.part_bytes each).
size_t attn_workspace_bytes(const AttnPlan &p, int gamma, int n_q_heads, int head_dim) {
    const size_t pairs = (size_t)gamma * n_q_heads;
    return kCounterBytes + (size_t)p.splits * pairs * (2 * sizeof(float) + (size_t)head_dim * p.part_bytes);
}

wf_status_t launch_attn(wf_dtype_t dt, const void *q, const void *k_cache,
                        const void *v_cache, void *out, int gamma, int ctx_len,
                        int cap, int n_q_heads, int n_kv_heads, int head_dim,
                        float softmax_scale, const uint64_t *tree_mask,
                        const AttnPlan &p, void *workspace, hipStream_t stream) {
    AttnParams a{};
    a.tree_mask = tree_mask;
    const size_t pairs = (size_t)gamma * n_q_heads;
    a.ws_ml = reinterpret_cast<float *>(static_cast<char *>(workspace) + kCounterBytes);
    a.ws_o = a.ws_ml + (size_t)p.splits * pairs * 2;
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
        dim3 grid(blocks), block(64 * p.ks * p.rg);
#define WF_ATTN_CASE(DHV, NBV, RGV, KSV, NBUFV)                                      \
    if (head_dim == DHV && p.nb == NBV && p.rg == RGV && p.ks == KSV &&               \
        p.nbuf == NBUFV) {                                                            \
        if (p.n_row_groups == 1)                                                      \
            attn_partial_bf16<DHV, NBV, RGV, KSV, NBUFV, true><<<grid, block, 0, stream>>>(a);  \
        else                                                                          \
            attn_partial_bf16<DHV, NBV, RGV, KSV, NBUFV, false><<<grid, block, 0, stream>>>(a); \
    } else
        WF_ATTN_CASE(128, 1, 1, 2, 3) WF_ATTN_CASE(128, 1, 2, 2, 3)
        WF_ATTN_CASE(128, 1, 4, 1, 3) WF_ATTN_CASE(128, 1, 4, 2, 3)
        WF_ATTN_CASE(128, 2, 4, 2, 3)
        WF_ATTN_CASE(64, 1, 1, 2, 3) WF_ATTN_CASE(64, 1, 2, 2, 3)
        WF_ATTN_CASE(64, 1, 4, 1, 3) WF_ATTN_CASE(64, 1, 4, 2, 3)
        WF_ATTN_CASE(64, 2, 4, 2, 3)
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

    const bool ob = (dt == WF_BF16);
    constexpr int kMergeWpb = 1;
    if (p.splits <= (kWave / (head_dim / 4)) * kMergeBatch) {
        dim3 g1((unsigned)cdiv((int)pairs, kMergeWpb)), b1(64 * kMergeWpb);
        if (head_dim == 128) {
            if (ob)
                attn_merge_one<128, true, kMergeWpb><<<g1, b1, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
            else
                attn_merge_one<128, false, kMergeWpb><<<g1, b1, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
        } else {
            if (ob)
                attn_merge_one<64, true, kMergeWpb><<<g1, b1, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
            else
                attn_merge_one<64, false, kMergeWpb><<<g1, b1, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
        }
        return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
    }
    dim3 mgrid((unsigned)pairs), mblock(64);
    if (head_dim == 128) {
        if (ob)
            attn_merge<128, true><<<mgrid, mblock, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
        else
            attn_merge<128, false><<<mgrid, mblock, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
    } else {
        if (ob)
            attn_merge<64, true><<<mgrid, mblock, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
        else
            attn_merge<64, false><<<mgrid, mblock, 0, stream>>>(a.ws_o, a.ws_ml, out, (int)pairs, p.splits, a.sl2);
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
