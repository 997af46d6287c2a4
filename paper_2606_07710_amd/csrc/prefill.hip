// prefill.hip -- KV-only prefill of catch-up tokens (Sec. 3.4 of the
// WhiFlash paper: after a drafter switch the incoming drafter's cache is
// caught up on the backlog in one batch, forming only the attention
// layer's keys and values -- no MLP, no LM head).
//
//   K[g][p+t] = RoPE(W_k[g] x_t, p+t),   V[g][p+t] = W_v[g] x_t
//
// bf16 path: the work unit is (KV head, K or V, one or two pairs of
// 16-feature blocks f and f + head_dim/2).  Pairing the two halves of the
// rotate-half RoPE puts
// both elements of every rotation pair in the same thread after the
// reduction, so RoPE is a register epilogue.  The input dimension is split
// across a power-of-two number of workgroups so a handful of units still
// spreads over the whole chip; the slices' sums meet up a fixed binary tree
// of device-scope atomic exchanges (deterministic: every node adds exactly
// two values), and the thread that leaves the root rotates and writes the
// cache pair.  Tokens are the MFMA N dimension (blocks of 16).
// RoPE angles are formed in fp64: at positions ~65K an fp32 angle would be
// off by ~4e-3 rad.
#include <cmath>

#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kPfMaxChunksPerWave = 8;   // 32-wide chunks per wave per k-slice
constexpr int kPfWideMaxChunks = 4;      // the same for two-pair units (more operand registers)
constexpr int kPfWideMinTokens = 65;     // two-pair units from this many tokens of one layer on
constexpr int kPfWideMinTokensBesideQ = 384;   // the same beside the catch-up's q projection
constexpr int kPfWideNbt3Tokens = 160;   // three 16-token blocks per workgroup up to here, then four
constexpr int kPfTargetWorkgroups = 256;
constexpr int kMaxHalfDim = 64;          // head_dim <= 128

struct PrefillParams {
    const void *x;
    const void *w_k;
    const void *w_v;
    void *k_cache;
    void *v_cache;
    int n_tok, start_pos, cap, d_in, n_kv_heads;
    double theta[kMaxHalfDim];  // RoPE frequencies base^(-2i/D), i < D/2
    unsigned long long *slots; // bf16 path: k-slice exchange slots, zero between calls
    int chunks_per_split;      // 32-wide chunks of d_in per k-slice
    int token_blocks;          // blockIdx.z = layer * token_blocks + token block
    long long x_ls, w_ls, c_ls; // element strides between layers (x, W_k|W_v, caches)
    int w_tiled;               // W_k, W_v in 16x32 tiles of 1 KB (bf16 path)
    int kinds;                 // 2: K and V; 1: K only (a rotated projection, e.g. q)
    int rope_shift;            // RoPE position = cache row position + rope_shift
    int x_tiled;               // x in 16-token x 32-dim tiles of 1 KB, token rows
                               // padded to a multiple of 16 (bf16 path)
};

// Rotation of the pair (lo, hi) = (k_i, k_{i+D/2}) by pos * theta_i, with
// theta_i = base^(-2i/D) precomputed on the host in fp64.  The angle is
// formed and reduced modulo 2*pi in fp64 (at pos ~65K an fp32 angle would be
// off by ~4e-3 rad); the reduced angle, in [-pi, pi], is exact to ~1e-16 and
// its sine and cosine are taken in fp32 (~1e-7).
__device__ __forceinline__ void rope_pair(float &lo, float &hi, double theta, int pos) {
    constexpr double kTwoPi = 6.283185307179586;
    const double phi = (double)pos * theta;
    const double r = fma(-rint(phi / kTwoPi), kTwoPi, phi);
    float sf, cf;
    sincosf((float)r, &sf, &cf);
    const float a = lo, b = hi;
    lo = a * cf - b * sf;
    hi = b * cf + a * sf;
}

// Split-K: workgroup (unit, k-slice, token block) computes D[feature][token]
// over its slice of the input dimension for the unit's 16-feature blocks
// (f and f + head_dim/2 of each of its pairs, one head, K or V); the slices
// then meet through the exchange tree below.
// The body takes its workgroup's grid coordinates explicitly, so one launch
// can run two such problems side by side (prefill_pair_bf16).
// A unit holds PPU consecutive pairs: its 2*PPU feature blocks are the low
// halves of those pairs (blocks 0..PPU-1) and then their high halves.
template <int DH, int NBT, int MAXC, int PPU>
__device__ __forceinline__ void prefill_body(const PrefillParams &a, int unit, int ks, int bz,
                                             int n_units, int ksplit) {
    constexpr int PAIRS = DH / 32;       // 16-feature block pairs per head
    static_assert(PAIRS % PPU == 0, "a unit's pairs must tile the head");
    constexpr int UPH = PAIRS / PPU;     // units per head and kind
    constexpr int MB = 2 * PPU;          // 16-feature blocks per unit
    constexpr int TOK = 16 * NBT;
    constexpr int WAVES = 4;
    __shared__ float zs[WAVES][MB][16][TOK + 1];

    const int tb = bz % a.token_blocks;
    const int layer = bz / a.token_blocks;
    const int pair0 = (unit % UPH) * PPU;                     // the unit's first pair
    const int kind = a.kinds == 2 ? (unit / UPH) % 2 : 0;     // 0 = K, 1 = V
    const int g = unit / (a.kinds * UPH);
    const int t0 = tb * TOK;

    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;

    const uint16_t *w = static_cast<const uint16_t *>(kind ? a.w_v : a.w_k) + layer * a.w_ls;
    const uint16_t *x = static_cast<const uint16_t *>(a.x) + layer * a.x_ls;
    const int c_begin = ks * a.chunks_per_split;   // 32-wide chunks of d_in
    // chunks of this slice (the last slices of a power-of-two split may be
    // short or empty)
    const int n_c = max(0, min(a.chunks_per_split, a.d_in / 32 - c_begin));
    // W operand of chunk c: row-major, lane (m16, c4) reads 16 bytes of row
    // m16 (64 contiguous bytes per row and load); tiled, the wave reads the
    // chunk's 1 KB tile contiguously
    const uint16_t *wp[MB];
    const int wstep = a.w_tiled ? 512 : 32;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        // first feature of block mb
        const int f = g * DH + 16 * (pair0 + mb % PPU) + (mb < PPU ? 0 : DH / 2);
        if (a.w_tiled)
            wp[mb] = w + (size_t)(f / 16) * (size_t)(a.d_in / 32) * 512 + lane * 8;
        else
            wp[mb] = w + (size_t)(f + m16) * a.d_in + c4 * 8;
    }
    // Tokens past n_tok read the last token (row-major) or the padded
    // rows of the last 16-token tile (tiled) instead: they only feed MFMA
    // output columns that are never stored.  A tiled x gives every load one
    // contiguous 1 KB tile (16 tokens x 32 dims in the operand's lane order)
    // instead of 64 bytes from each of 16 rows.
    const uint16_t *xp[NBT];
    int xstep;
    if (a.x_tiled) {
        const size_t kch = (size_t)(a.d_in / 32);
        const int last_blk = (a.n_tok + 15) / 16 - 1;
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
            xp[nb] = x + (size_t)min(t0 / 16 + nb, last_blk) * kch * 512 + lane * 8;
        xstep = 512;
    } else {
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
            xp[nb] = x + (size_t)min(t0 + nb * 16 + m16, a.n_tok - 1) * a.d_in + c4 * 8;
        xstep = 32;
    }

    f32x4 acc[MB][NBT];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
            acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // wave-strided chunks c = wave, wave + 4, ...; batches of MAXC chunks
    // whose loads are all issued before the batch's first MFMA (a single
    // token's projection takes all of a wave's chunks in one batch: one
    // memory round trip instead of two)
    for (int cb = wave; cb < n_c; cb += WAVES * MAXC) {
        bf16x8 wr[MAXC][MB], xr[MAXC][NBT];
#pragma unroll
        for (int u = 0; u < MAXC; ++u) {
            const int c = cb + WAVES * u;
            if (c < n_c) {
                const size_t off = (size_t)(c_begin + c) * xstep;
                const size_t woff = (size_t)(c_begin + c) * wstep;
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    wr[u][mb] = load_bf16x8(wp[mb] + woff);
#pragma unroll
                for (int nb = 0; nb < NBT; ++nb)
                    xr[u][nb] = load_bf16x8(xp[nb] + off);
            }
        }
#pragma unroll
        for (int u = 0; u < MAXC; ++u) {
            if (cb + WAVES * u < n_c) {
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                    for (int nb = 0; nb < NBT; ++nb)
                        acc[mb][nb] = mfma16x16x32(wr[u][mb], xr[u][nb], acc[mb][nb]);
            }
        }
    }
    // lane (m16, c4) holds D[feature 4*c4 + i][token nb*16 + m16]
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                zs[wave][mb][4 * c4 + i][nb * 16 + m16] = acc[mb][nb][i];
    __syncthreads();
    // Thread (e, token) sums the waves in order for its rotation pair
    // (feature 16*pair + e of the low half and its partner in the high
    // half; e runs fastest across threads, so a wave's cache writes cover
    // whole 32-byte runs of 4 rows instead of 2 bytes of 64 rows: 6.6 ->
    // 6.45 us at 16 tokens, 15.5 -> 14.6 at 80), then combines the k-slices up a fixed binary tree: leaf
    // ksplit + k, node i with children 2i and 2i+1, one 64-bit exchange slot
    // per internal node and pair.  The first slice to reach a node parks its
    // (lo, hi) there; the second takes it, adds (a commutative fp32 add, so
    // the result does not depend on who came first), resets the slot and
    // climbs on.  Whoever leaves the root finishes the pair: RoPE for K,
    // bf16 cache write.  Slot 0 means empty; a parked pair is stored as
    // (bits(hi) << 32) | (bits(lo) + 1), never 0 for arithmetic results.
    // A thread holds NI pairs (idx = tid + 256 i) and climbs with all of
    // them at once: one exchange round trip per tree level, not per pair.
    constexpr int NP = 16 * PPU * TOK;   // rotation pairs per workgroup
    constexpr int NI = NP / 256;
    static_assert(NP % 256 == 0, "pairs per workgroup must fill the 256 threads");
    const size_t ub =                                          // (layer, unit, token block)
        ((size_t)layer * n_units + unit) * a.token_blocks + tb;
    unsigned long long *slots = a.slots + ub * (size_t)(ksplit - 1) * NP;
    uint16_t *cache = static_cast<uint16_t *>(kind ? a.v_cache : a.k_cache) + layer * a.c_ls;
    float lo[NI], hi[NI];
    bool mine[NI];
#pragma unroll
    for (int n = 0; n < NI; ++n) {
        const int idx = threadIdx.x + 256 * n;
        const int pl = idx / (16 * TOK);           // the unit's pair
        const int e = idx % 16;
        const int tl = (idx / 16) % TOK;
        lo[n] = zs[0][pl][e][tl];
        hi[n] = zs[0][PPU + pl][e][tl];
#pragma unroll
        for (int ww = 1; ww < WAVES; ++ww) {
            lo[n] += zs[ww][pl][e][tl];
            hi[n] += zs[ww][PPU + pl][e][tl];
        }
        mine[n] = true;
    }
    for (unsigned node = (unsigned)(ksplit + ks); node > 1; node /= 2) {
        unsigned long long *level = slots + (size_t)(node / 2 - 1) * NP + threadIdx.x;
        unsigned long long old[NI];
#pragma unroll
        for (int n = 0; n < NI; ++n) {
            const unsigned long long packed =
                ((unsigned long long)__float_as_uint(hi[n]) << 32) |
                (unsigned long long)(__float_as_uint(lo[n]) + 1u);
            old[n] = mine[n] ? __hip_atomic_exchange(level + 256 * n, packed, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)
                             : 0ull;
        }
        bool any = false;
#pragma unroll
        for (int n = 0; n < NI; ++n) {
            if (!mine[n])
                continue;
            if (old[n] == 0ull) {
                mine[n] = false;       // the sibling finishes this node
                continue;
            }
            lo[n] += __uint_as_float((unsigned)old[n] - 1u);
            hi[n] += __uint_as_float((unsigned)(old[n] >> 32));
            __hip_atomic_store(level + 256 * n, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            any = true;
        }
        if (!any)
            break;
    }
#pragma unroll
    for (int n = 0; n < NI; ++n) {
        const int idx = threadIdx.x + 256 * n;
        const int pair = pair0 + idx / (16 * TOK);
        const int e = idx % 16;
        const int t = t0 + (idx / 16) % TOK;
        if (!mine[n] || t >= a.n_tok)
            continue;
        const int pos = a.start_pos + t;
        float l = lo[n], h = hi[n];
        if (kind == 0)
            rope_pair(l, h, a.theta[16 * pair + e], pos + a.rope_shift);
        uint16_t *row = cache + ((size_t)g * a.cap + pos) * DH;
        row[16 * pair + e] = f32_to_bf16(l);
        row[DH / 2 + 16 * pair + e] = f32_to_bf16(h);
    }
}

template <int DH, int NBT, int MAXC = kPfMaxChunksPerWave, int PPU = 1>
__global__ __launch_bounds__(256) void prefill_bf16(PrefillParams a) {
    prefill_body<DH, NBT, MAXC, PPU>(a, blockIdx.x, blockIdx.y, blockIdx.z, gridDim.x, gridDim.y);
}

// Two independent projections in one launch: workgroups [0, n1) run the
// first problem's grid (units1 x ks1 x z1, flattened), the rest the
// second's.  Each keeps its own exchange slots (disjoint parts of the zero
// block).  The drafter catch-up runs the backlog's K/V and the last token's
// q this way: one launch instead of two back to back.
template <int DH, int NBT1, int MAXC1, int PPU1, int NBT2, int MAXC2>
__global__ __launch_bounds__(256) void prefill_pair_bf16(PrefillParams a1, PrefillParams a2,
                                                         int units1, int ks1, int z1,
                                                         int units2, int ks2) {
    const int b = blockIdx.x;
    const int n1 = units1 * ks1 * z1;
    if (b < n1) {
        prefill_body<DH, NBT1, MAXC1, PPU1>(a1, b % units1, (b / units1) % ks1,
                                            b / (units1 * ks1), units1, ks1);
    } else {
        const int c = b - n1;
        prefill_body<DH, NBT2, MAXC2, 1>(a2, c % units2, (c / units2) % ks2, c / (units2 * ks2),
                                         units2, ks2);
    }
}

// fp32 path: one wave per (token, KV head, rotation pair, K or V).  Lane
// l takes the input dims l, l + 64, ... (coalesced loads) in order; the two
// dot products then meet in a fixed butterfly, and lane 0 rotates and
// writes the pair.
__global__ __launch_bounds__(256) void prefill_f32(PrefillParams a, int dh) {
    const int half = dh / 2;
    const long long total = (long long)a.n_tok * a.n_kv_heads * half * 2;
    const long long idx = ((long long)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    const int lane = threadIdx.x % kWave;
    if (idx >= total)
        return;                          // whole waves: idx is wave-uniform
    const int i = (int)(idx % half);
    const int kind = (int)((idx / half) % 2);
    const int g = (int)((idx / (2 * half)) % a.n_kv_heads);
    const int t = (int)(idx / (2LL * half * a.n_kv_heads));
    const float *x = static_cast<const float *>(a.x) + (size_t)t * a.d_in;
    const float *w = static_cast<const float *>(kind ? a.w_v : a.w_k);
    const float *w_lo = w + (size_t)(g * dh + i) * a.d_in;
    const float *w_hi = w + (size_t)(g * dh + i + half) * a.d_in;
    float lo = 0.f, hi = 0.f;
#pragma unroll 4
    for (int c = lane; c < a.d_in; c += kWave) {
        const float xv = x[c];
        lo = fmaf(w_lo[c], xv, lo);
        hi = fmaf(w_hi[c], xv, hi);
    }
    lo = wave_sum(lo);
    hi = wave_sum(hi);
    if (lane != 0)
        return;
    const int pos = a.start_pos + t;
    if (kind == 0)
        rope_pair(lo, hi, a.theta[i], pos);
    float *row = static_cast<float *>(kind ? a.v_cache : a.k_cache) + ((size_t)g * a.cap + pos) * dh;
    row[i] = lo;
    row[i + half] = hi;
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

// Exchange slots: (ksplit - 1) internal tree nodes x 16*16*ppu*nbt pairs
// per (unit, token block), inside the workspace's zero block.
static size_t prefill_slot_bytes(const PrefillPlan &p, int n_layers) {
    return (size_t)n_layers * p.units * p.token_blocks * (p.ksplit - 1) *
           (16 * 16 * p.ppu * p.nbt) * sizeof(unsigned long long);
}

PrefillPlan plan_prefill(int n_tok, int d_in, int n_kv_heads, int head_dim, int n_layers,
                         int kinds, bool beside_q) {
    PrefillPlan p{};
    const int pairs = head_dim / 32;
    // One layer with more than four token blocks (a switch's backlog): units
    // of two pairs, so each workgroup reads its slice of the activations for
    // twice the features (the activation reads across all units halve) and
    // the grid keeps more k-slices; otherwise one pair per unit.  Measured
    // (8B shapes): 80 tokens 14.6 -> 12.8 us, 160 21.3 -> 15.3, 1024 69 ->
    // 43, 4096 271 -> 160; at 40 tokens two-pair units were slower (their
    // eight k-slices add a third exchange level).  Sharing a launch with the
    // catch-up's q projection, whose workgroups take the CUs' second slots,
    // they pay from about 384 tokens on (catch-up: 128 tokens 97.3 against
    // 100.2 us with one-pair units, 512 tokens 108.4 against 113.7).
    const int wide_min = beside_q ? kPfWideMinTokensBesideQ : kPfWideMinTokens;
    p.ppu = (n_layers == 1 && n_tok >= wide_min && pairs % 2 == 0) ? 2 : 1;
    if (p.ppu == 2) {
        p.nbt = n_tok <= kPfWideNbt3Tokens ? 3 : 4;
    } else {
        // as few token blocks as four 16-token blocks each allow, the
        // 16-token blocks dealt out evenly over them (80 tokens: 48 + 32,
        // not 64 + 16; the 80-token catch-up 96.2-97.6 -> 95.1-95.3 us)
        const int blocks16 = std::max(1, cdiv(n_tok, 16));
        p.nbt = cdiv(blocks16, cdiv(blocks16, 4));
    }
    p.token_blocks = std::max(1, cdiv(n_tok, 16 * p.nbt));
    p.units = n_kv_heads * kinds * (pairs / p.ppu);
    const int chunks = d_in / 32;
    // a power-of-two number of k-slices: enough to cover the chip, at least
    // 4 chunks per slice, and the exchange slots inside the 4 MiB zero block
    // (one pair per unit: layers * units * token_blocks * (ksplit - 1) < 256
    // keeps them under 2 MiB).  Several layers in one launch need fewer
    // slices (none from 256 (layer, unit, token block) triples up).
    const long long base = (long long)p.units * p.token_blocks * n_layers;
    int ks = 1;
    for (;;) {
        PrefillPlan q = p;
        q.ksplit = ks * 2;
        if (ks * 2 * base > kPfTargetWorkgroups || chunks / (ks * 2) < 4 ||
            prefill_slot_bytes(q, n_layers) > kCounterBytes)
            break;
        ks *= 2;
    }
    p.chunks_per_split = cdiv(chunks, ks);
    p.ksplit = ks;
    return p;
}

bool prefill_fits(int n_tok, int d_in, int n_kv_heads, int head_dim, int n_layers) {
    const PrefillPlan p = plan_prefill(n_tok, d_in, n_kv_heads, head_dim, n_layers);
    return prefill_slot_bytes(p, n_layers) <= kCounterBytes &&
           (long long)p.token_blocks * n_layers <= 65535;
}

size_t prefill_workspace_bytes(wf_dtype_t dt, int n_tok, int d_in, int n_kv_heads,
                               int head_dim) {
    if (dt != WF_BF16 || n_tok == 0)
        return 0;
    return kCounterBytes;
}

wf_status_t launch_prefill(wf_dtype_t dt, const void *x, const void *w_k,
                           const void *w_v, void *k_cache, void *v_cache,
                           int n_tok, int start_pos, int cap, int d_in,
                           int n_kv_heads, int head_dim, double rope_base,
                           void *workspace, hipStream_t stream, int n_layers,
                           long long x_ls, long long w_ls, long long c_ls, bool x_tiled) {
    const bool tiled = dt == WF_BF16_TILED;
    if (tiled)
        dt = WF_BF16;
    if (x_tiled && dt != WF_BF16)
        return WF_ERR_UNSUPPORTED;
    PrefillParams a{x, w_k, w_v, k_cache, v_cache, n_tok, start_pos, cap, d_in,
                    n_kv_heads, {}, nullptr, 0, 1, x_ls, w_ls, c_ls, tiled ? 1 : 0, 2, 0,
                    x_tiled ? 1 : 0};
    for (int i = 0; i < head_dim / 2; ++i)
        a.theta[i] = std::pow(rope_base, -2.0 * (double)i / (double)head_dim);
    if (dt == WF_BF16) {
        const PrefillPlan p = plan_prefill(n_tok, d_in, n_kv_heads, head_dim, n_layers);
        a.chunks_per_split = p.chunks_per_split;
        a.token_blocks = p.token_blocks;
        a.slots = static_cast<unsigned long long *>(workspace);
        dim3 grid(p.units, p.ksplit, p.token_blocks * n_layers), block(256);
#define WF_PF_CASE(DHV, NBV)                                                        \
    if (head_dim == DHV && p.nbt == NBV && p.ppu == 1) {                            \
        prefill_bf16<DHV, NBV><<<grid, block, 0, stream>>>(a);                      \
    } else
#define WF_PF_WIDE(DHV, NBV)                                                        \
    if (head_dim == DHV && p.nbt == NBV && p.ppu == 2) {                            \
        prefill_bf16<DHV, NBV, kPfWideMaxChunks, 2><<<grid, block, 0, stream>>>(a); \
    } else
        WF_PF_CASE(128, 1) WF_PF_CASE(128, 2) WF_PF_CASE(128, 3) WF_PF_CASE(128, 4)
        WF_PF_CASE(64, 1) WF_PF_CASE(64, 2) WF_PF_CASE(64, 3) WF_PF_CASE(64, 4)
        WF_PF_WIDE(128, 3) WF_PF_WIDE(128, 4) WF_PF_WIDE(64, 3) WF_PF_WIDE(64, 4)
        { return WF_ERR_UNSUPPORTED; }
#undef WF_PF_WIDE
#undef WF_PF_CASE
    } else {
        const long long total = (long long)n_tok * n_kv_heads * head_dim;   // waves
        const unsigned blocks = (unsigned)((total * kWave + 255) / 256);
        for (int l = 0; l < n_layers; ++l) {
            PrefillParams al = a;
            al.x = static_cast<const float *>(x) + l * x_ls;
            al.w_k = static_cast<const float *>(w_k) + l * w_ls;
            al.w_v = static_cast<const float *>(w_v) + l * w_ls;
            al.k_cache = static_cast<float *>(k_cache) + l * c_ls;
            al.v_cache = static_cast<float *>(v_cache) + l * c_ls;
            prefill_f32<<<blocks, 256, 0, stream>>>(al, head_dim);
        }
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

// The drafter catch-up's first two projections in one launch: the KV-only
// prefill of the backlog's n_tok tiled rows (as launch_prefill with a tiled
// x) and q = RoPE(W_q x_last) of the last token (as launch_q_rope), the
// first set of exchange slots at the start of the zero block, the second at
// its end.  WF_ERR_UNSUPPORTED when the two sets do not fit side by side (the
// caller then launches the two one after the other).
wf_status_t launch_prefill_and_q(bool tiled, const uint16_t *x_rows, const void *w_k,
                                 const void *w_v, void *k_cache, void *v_cache, int n_tok,
                                 int start_pos, int cap, int d_in, int n_kv_heads,
                                 const uint16_t *x_last, const uint16_t *w_q, uint16_t *q,
                                 int n_q_heads, int head_dim, int q_pos, double rope_base,
                                 void *workspace, hipStream_t stream) {
    PrefillParams a1{x_rows, w_k, w_v, k_cache, v_cache, n_tok, start_pos, cap, d_in,
                     n_kv_heads, {}, nullptr, 0, 1, 0, 0, 0, tiled ? 1 : 0, 2, 0, 1};
    PrefillParams a2{x_last, w_q, w_q, q, q, 1, 0, 1, d_in, n_q_heads, {}, nullptr, 0, 1, 0, 0, 0,
                     tiled ? 1 : 0, 1, q_pos, 0};
    for (int i = 0; i < head_dim / 2; ++i)
        a1.theta[i] = a2.theta[i] = std::pow(rope_base, -2.0 * (double)i / (double)head_dim);
    const PrefillPlan p1 = plan_prefill(n_tok, d_in, n_kv_heads, head_dim, 1, 2, true);
    const PrefillPlan p2 = plan_prefill(1, d_in, n_q_heads, head_dim, 1, 1);
    const size_t q_off = (kCounterBytes - prefill_slot_bytes(p2, 1)) / 256 * 256;
    if (prefill_slot_bytes(p2, 1) > kCounterBytes || prefill_slot_bytes(p1, 1) > q_off)
        return WF_ERR_UNSUPPORTED;
    a1.chunks_per_split = p1.chunks_per_split;
    a1.token_blocks = p1.token_blocks;
    a1.slots = static_cast<unsigned long long *>(workspace);
    a2.chunks_per_split = p2.chunks_per_split;
    a2.token_blocks = p2.token_blocks;
    a2.slots = reinterpret_cast<unsigned long long *>(static_cast<char *>(workspace) + q_off);
    const long long n1 = (long long)p1.units * p1.ksplit * p1.token_blocks;
    const long long n2 = (long long)p2.units * p2.ksplit * p2.token_blocks;
    const dim3 grid((unsigned)(n1 + n2)), block(256);
    const bool wide2 = p2.chunks_per_split > 4 * kPfMaxChunksPerWave;
    constexpr int M8 = kPfMaxChunksPerWave, M16 = 2 * kPfMaxChunksPerWave;
    constexpr int MW = kPfWideMaxChunks;
#define WF_PAIR_CASE(DHV, NBV, MC, PPUV)                                                    \
    if (head_dim == DHV && p1.nbt == NBV && p1.ppu == PPUV) {                               \
        if (wide2)                                                                          \
            prefill_pair_bf16<DHV, NBV, MC, PPUV, 1, M16><<<grid, block, 0, stream>>>(      \
                a1, a2, p1.units, p1.ksplit, p1.token_blocks, p2.units, p2.ksplit);         \
        else                                                                                \
            prefill_pair_bf16<DHV, NBV, MC, PPUV, 1, M8><<<grid, block, 0, stream>>>(       \
                a1, a2, p1.units, p1.ksplit, p1.token_blocks, p2.units, p2.ksplit);         \
    } else
    WF_PAIR_CASE(128, 1, M8, 1) WF_PAIR_CASE(128, 2, M8, 1) WF_PAIR_CASE(128, 3, M8, 1)
    WF_PAIR_CASE(128, 4, M8, 1) WF_PAIR_CASE(64, 1, M8, 1) WF_PAIR_CASE(64, 2, M8, 1)
    WF_PAIR_CASE(64, 3, M8, 1) WF_PAIR_CASE(64, 4, M8, 1)
    WF_PAIR_CASE(128, 3, MW, 2) WF_PAIR_CASE(128, 4, MW, 2)
    WF_PAIR_CASE(64, 3, MW, 2) WF_PAIR_CASE(64, 4, MW, 2)
    { return WF_ERR_UNSUPPORTED; }
#undef WF_PAIR_CASE
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

// q = RoPE(W_q x) for one token: the K half of the kernel above with the
// query heads as its heads, written to q [n_heads][head_dim] (a one-row
// "cache") and rotated at position pos.  The split over the input
// dimension and the exchange tree spread its units over the whole chip.
wf_status_t launch_q_rope(const uint16_t *x, const uint16_t *w_q, uint16_t *q, int d_in,
                          int n_heads, int head_dim, int pos, double rope_base,
                          void *workspace, hipStream_t stream, bool tiled) {
    PrefillParams a{x, w_q, w_q, q, q, 1, 0, 1, d_in, n_heads, {}, nullptr, 0, 1, 0, 0, 0,
                    tiled ? 1 : 0, 1, pos, 0};
    for (int i = 0; i < head_dim / 2; ++i)
        a.theta[i] = std::pow(rope_base, -2.0 * (double)i / (double)head_dim);
    const PrefillPlan p = plan_prefill(1, d_in, n_heads, head_dim, 1, 1);
    if (prefill_slot_bytes(p, 1) > kCounterBytes)
        return WF_ERR_UNSUPPORTED;
    a.chunks_per_split = p.chunks_per_split;
    a.token_blocks = p.token_blocks;
    a.slots = static_cast<unsigned long long *>(workspace);
    dim3 grid(p.units, p.ksplit, p.token_blocks), block(256);
    const bool wide = p.chunks_per_split > 4 * kPfMaxChunksPerWave;   // > 8 chunks per wave
    if (head_dim == 128 && wide)
        prefill_bf16<128, 1, 2 * kPfMaxChunksPerWave><<<grid, block, 0, stream>>>(a);
    else if (head_dim == 128)
        prefill_bf16<128, 1><<<grid, block, 0, stream>>>(a);
    else if (head_dim == 64 && wide)
        prefill_bf16<64, 1, 2 * kPfMaxChunksPerWave><<<grid, block, 0, stream>>>(a);
    else if (head_dim == 64)
        prefill_bf16<64, 1><<<grid, block, 0, stream>>>(a);
    else
        return WF_ERR_UNSUPPORTED;
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace wf
