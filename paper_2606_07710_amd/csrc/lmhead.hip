// lmhead.hip -- LM head reduced on the fly to argmax and softmax entropy per
// verify row, then greedy acceptance and the entropy route (Sec. 3.3.1 of
// the WhiFlash paper: the router reads the entropy of the target's
// next-token distribution at the final accepted position; greedy
// verification keeps the longest draft prefix the target agrees with).
//
// Stage 1 (one workgroup per vocabulary tile): z = h W^T for the tile's
// vocabulary rows, reduced immediately to one mergeable row state
// (max, argmax, sum of the other exponentials, sum of p*log-terms) per
// (row, tile).  Logits never reach memory.
//   bf16: 16x16x32 bf16 MFMA skinny GEMM; 8 waves split the hidden dimension
//   and stream W with a 4-deep prefetch; partial logits meet in LDS.
//   fp32: plain VALU dot products.
//   logits-only mode: the tile reads given fp32 logits.
// Stage 2 (one workgroup per row): merge the row's tile states in a fixed
// order and emit argmax and entropy; the last row to finish then emits the
// accept length, bonus token and route.
#include <type_traits>

#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kLmTile = 64;          // vocabulary rows per matmul tile
constexpr int kLmMB = kLmTile / 16;  // 16-row MFMA blocks per tile
constexpr int kLmWaves = 8;
constexpr int kLmPrefetch = 4;       // 32-dim chunks in flight per wave
// The persistent kernel keeps fewer chunks in flight: its 8 waves x 2 chunks
// x 4 blocks (64 KB per CU) already cover the memory latency, and a shorter
// queue shortens the pipeline fill (measured: 229 us against 234 at 4 and
// 240 at 1 per call on the 8B head).
constexpr int kLmStreamPrefetch = 2;
constexpr int kLogitsTile = 256;     // vocabulary entries per logits tile
constexpr int kMaxGamma = 64;
constexpr int kLmStreamGrid = 256;      // persistent grid: one workgroup per CU

// ---- shared epilogue: tile logits in LDS -> one state per row --------------
// zs is [kMaxGamma][kLmTile + 4]; zs[r][v] holds row r's logit of v0 + v.
__device__ __forceinline__ void tile_states(const float (*zs)[kLmTile + 4],
                                            RowState *states, int tile,
                                            int n_tiles, int v0, int gamma,
                                            int vocab, int wave, int n_waves,
                                            int lane) {
    for (int r = wave; r < gamma; r += n_waves) {
        const int v = v0 + lane;
        RowState s = (v < vocab) ? state_single(zs[r][lane], v) : state_empty();
        s = wave_merge(s);
        if (lane == 0)
            states[(size_t)r * n_tiles + tile] = s;
    }
}

// Second kernel: workgroup r merges row r's tile states (thread t takes
// tiles t, t + 256, ... in order, then a fixed butterfly across the wave and
// the four waves in order) into argmax and entropy.  The last row workgroup
// to arrive (device-scope ticket) applies greedy acceptance and the entropy
// route; it resets the ticket counter for the next call.
constexpr int kFinishThreads = 256;
constexpr int kFinishBatch = 16;

struct LmFinish {
    RowState *states;        // [gamma][n_tiles]
    unsigned *fcnt;          // ticket counter, zero between calls
    const int32_t *draft;    // chain: [gamma-1] drafts; tree: [gamma] node tokens
    const int32_t *parents;  // tree: [gamma] parent of each node; chain: nullptr
    int32_t *path_out;       // tree: [gamma] accepted root path
    int32_t *argmax_out;
    float *entropy_out;
    int32_t *accept_out;
    int gamma, n_tiles;
    float tau;
    // Neural routing policy folded into the pass (nullptr w1: the entropy
    // rule).  W1 [m][d] streams as m/16 extra 16-row blocks after the
    // vocabulary; their "logits" z = W1 h go to zr [gamma][m], and the
    // finish forms delta[r] = w2 . GELU(z[r] + b1) + b2 and routes on
    // delta[n] > tau_neural.
    const uint16_t *w1;
    const uint16_t *b1, *w2, *b2;   // bf16
    float *zr;
    float *delta_out;
    int m;
    float tau_neural;
};

__device__ __forceinline__ float gelu_erf(float x) {
    return 0.5f * x * (1.f + erff(x * 0.70710678118654752f));
}

// Greedy acceptance on a draft tree, run by the last row workgroup once
// every row's argmax is out.  Node j (one lane each, gamma <= 64) walks its
// root path: it is accepted iff every node v on it has a parent p < v whose
// argmax equals v's token.  The accepted node of greatest depth (lowest
// index among equals) ends the accepted path; it gives the accept length,
// bonus token and route, and lane 0 writes its root path.
__device__ __forceinline__ void tree_accept(const LmFinish &f, int wave, int lane) {
    __shared__ int s_par[kMaxGamma], s_tok[kMaxGamma], s_am[kMaxGamma];
    if (wave == 0 && lane < f.gamma) {
        s_par[lane] = f.parents[lane];
        s_tok[lane] = f.draft[lane];
        s_am[lane] = f.argmax_out[lane];
    }
    __syncthreads();
    if (wave != 0)
        return;
    bool ok = lane < f.gamma;
    int depth = 0;
    // indices fall strictly along the walk, so it ends within `lane` steps
    for (int v = lane; ok && v > 0; ++depth) {
        const int p = s_par[v];
        if (p < 0 || p >= v || s_tok[v] != s_am[p])
            ok = false;
        v = p;
    }
    int key = ok ? (depth << 6) | (63 - lane) : -1;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        key = max(key, __shfl_xor(key, off, kWave));
    const int b = 63 - (key & 63);      // the root is always accepted: key >= 0
    const int n = key >> 6;
    if (lane > n && lane < f.gamma)
        f.path_out[lane] = -1;
    if (lane == 0) {
        for (int t = n, v = b; t >= 0; --t) {
            f.path_out[t] = v;
            v = s_par[v];
        }
        f.accept_out[0] = n;
        f.accept_out[1] = s_am[b];
        f.accept_out[2] = (f.entropy_out[b] > f.tau) ? 1 : 0;
        f.accept_out[3] = b;
        *f.fcnt = 0u;
    }
}

__global__ __launch_bounds__(kFinishThreads) void lm_finish_rows(LmFinish f) {
    __shared__ RowState ws[kFinishThreads / kWave];
    const int r = blockIdx.x;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const RowState *row = f.states + (size_t)r * f.n_tiles;
    // batches of kFinishBatch loads in flight per thread (clamped addresses,
    // masked merges), merged in ascending tile order
    RowState s = state_empty();
    for (int base = threadIdx.x; base < f.n_tiles; base += kFinishThreads * kFinishBatch) {
        RowState buf[kFinishBatch];
#pragma unroll
        for (int b = 0; b < kFinishBatch; ++b)
            buf[b] = row[min(base + b * kFinishThreads, f.n_tiles - 1)];
#pragma unroll
        for (int b = 0; b < kFinishBatch; ++b)
            if (base + b * kFinishThreads < f.n_tiles)
                s = state_merge(s, buf[b]);
    }
    s = wave_merge(s);
    if (lane == 0)
        ws[wave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        RowState m = ws[0];
#pragma unroll
        for (int w = 1; w < kFinishThreads / kWave; ++w)
            m = state_merge(m, ws[w]);
        f.argmax_out[r] = m.a;
        f.entropy_out[r] = state_entropy(m);
    }
    if (f.w1) {
        // delta[r] = b2 + sum_u w2[u] GELU(z[r][u] + b1[u]): thread t takes
        // units t, t + 256, ... in order, then a fixed butterfly and the
        // waves in order
        __shared__ float dsum[kFinishThreads / kWave];
        float acc = 0.f;
        for (int u = threadIdx.x; u < f.m; u += kFinishThreads)
            acc = fmaf(bf16_to_f32(f.w2[u]),
                       gelu_erf(f.zr[(size_t)r * f.m + u] + bf16_to_f32(f.b1[u])), acc);
        acc = wave_sum(acc);
        if (lane == 0)
            dsum[wave] = acc;
        __syncthreads();
        if (threadIdx.x == 0) {
            float dl = bf16_to_f32(f.b2[0]);
#pragma unroll
            for (int w = 0; w < kFinishThreads / kWave; ++w)
                dl += dsum[w];
            f.delta_out[r] = dl;
        }
    }
    if (!arrive_last(f.fcnt, (unsigned)f.gamma))
        return;
    if (f.parents) {
        tree_accept(f, wave, lane);
        return;
    }
    if (threadIdx.x == 0) {
        int n = 0;
        while (n < f.gamma - 1 && f.draft[n] == f.argmax_out[n])
            ++n;
        f.accept_out[0] = n;
        f.accept_out[1] = f.argmax_out[n];
        f.accept_out[2] = f.w1 ? (f.delta_out[n] > f.tau_neural ? 1 : 0)
                               : (f.entropy_out[n] > f.tau ? 1 : 0);
        *f.fcnt = 0u;
    }
}

template <int NBL>
__global__ __launch_bounds__(512) void lm_tiles_bf16(const uint16_t *__restrict__ h,
                                                     const uint16_t *__restrict__ w,
                                                     LmFinish f, int d, int vocab) {
    RowState *states = f.states;
    const int gamma = f.gamma, n_tiles = f.n_tiles;
    __shared__ __attribute__((aligned(16))) float zs[kMaxGamma][kLmTile + 4];
    const int tile = blockIdx.x;
    const int v0 = tile * kLmTile;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;

    const uint16_t *wp[kLmMB];
#pragma unroll
    for (int mb = 0; mb < kLmMB; ++mb)
        wp[mb] = w + (size_t)min(v0 + 16 * mb + m16, vocab - 1) * d + c4 * 8;
    // Rows past gamma read row gamma-1 instead: they only feed MFMA output
    // columns that are never used, and nothing waits on a load early.
    const uint16_t *hp[NBL];
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
        hp[nb] = h + (size_t)min(nb * 16 + m16, gamma - 1) * d + c4 * 8;

    f32x4 acc[kLmMB][NBL];
#pragma unroll
    for (int mb = 0; mb < kLmMB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBL; ++nb)
            acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nchunks = d / 32;
    const int cpw = (wave < nchunks) ? (nchunks - wave + kLmWaves - 1) / kLmWaves : 0;

    bf16x8 wb[kLmPrefetch][kLmMB], hb[kLmPrefetch][NBL];
    auto load_chunk = [&](int u, bf16x8 (&wr)[kLmMB], bf16x8 (&hr)[NBL]) {
        const int off = (wave + kLmWaves * u) * 32;
#pragma unroll
        for (int mb = 0; mb < kLmMB; ++mb)
            wr[mb] = load_bf16x8_nt(wp[mb] + off);
#pragma unroll
        for (int nb = 0; nb < NBL; ++nb)
            hr[nb] = load_bf16x8(hp[nb] + off);
    };
    auto mac = [&](const bf16x8 (&wr)[kLmMB], const bf16x8 (&hr)[NBL]) {
#pragma unroll
        for (int mb = 0; mb < kLmMB; ++mb)
#pragma unroll
            for (int nb = 0; nb < NBL; ++nb)
                acc[mb][nb] = mfma16x16x32(wr[mb], hr[nb], acc[mb][nb]);
    };
    // Steady state without branches, so the compiler's wait counting stays
    // exact and kLmPrefetch chunks stay in flight: consume a group of chunks
    // while refilling the same registers with the next group.
    const int ngroups = cpw / kLmPrefetch;
    if (ngroups > 0) {
#pragma unroll
        for (int p = 0; p < kLmPrefetch; ++p) {
            load_chunk(p, wb[p], hb[p]);
            __builtin_amdgcn_sched_barrier(0);   // issue chunk by chunk
        }
        for (int gi = 0; gi < ngroups - 1; ++gi) {
#pragma unroll
            for (int p = 0; p < kLmPrefetch; ++p) {
                mac(wb[p], hb[p]);
                load_chunk((gi + 1) * kLmPrefetch + p, wb[p], hb[p]);
                // keep each refill right behind the MFMAs that free its
                // registers, so kLmPrefetch chunks stay in flight
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int p = 0; p < kLmPrefetch; ++p)
            mac(wb[p], hb[p]);
    }
    for (int u = ngroups * kLmPrefetch; u < cpw; ++u) {
        load_chunk(u, wb[0], hb[0]);
        mac(wb[0], hb[0]);
    }

    // partial logits of the 8 waves meet in LDS in a fixed order
#pragma unroll 1
    for (int ww = 0; ww < kLmWaves; ++ww) {
        if (wave == ww) {
#pragma unroll
            for (int nb = 0; nb < NBL; ++nb) {
                const int r = nb * 16 + m16;
                if (r < gamma) {
#pragma unroll
                    for (int mb = 0; mb < kLmMB; ++mb) {
                        f32x4 *dst = reinterpret_cast<f32x4 *>(&zs[r][16 * mb + 4 * c4]);
                        f32x4 v = acc[mb][nb];
                        if (ww > 0)
                            v += *dst;
                        *dst = v;
                    }
                }
            }
        }
        __syncthreads();
    }
    tile_states(zs, states, tile, n_tiles, v0, gamma, vocab, wave, kLmWaves, lane);
}

// Persistent bf16 LM head for up to 16 verify rows and a hidden size of
// CPW * 32 * 8: workgroup b owns the 16-row vocabulary blocks b, b + G,
// b + 2G, ... (G workgroups) and walks them in tiles of kLmMB blocks, so at
// any moment the grid streams one contiguous stretch of W (measured 213-215
// against 218-220 us per call with one contiguous run per workgroup).  Each of the 8 waves owns a
// contiguous CPW*32-dim slice of the hidden dimension, keeps its slice of h
// in registers for the whole run, and streams W with kLmStreamPrefetch chunks in
// flight; the prefetch runs on across tile boundaries, so the stream never
// drains.  Per tile the 8 partial logit blocks meet in LDS (double
// buffered: one barrier per tile) and every row's tile state is folded
// into a running state in ascending vocabulary order; the workgroup writes
// one state per row at the end.
template <int CPW>
__global__ __launch_bounds__(512) void lm_stream_bf16(const uint16_t *__restrict__ h,
                                                      const uint16_t *__restrict__ w,
                                                      LmFinish f, int vocab, int tiled) {
    constexpr int D = CPW * 32 * kLmWaves;
    constexpr int P = kLmStreamPrefetch;
    static_assert(CPW % P == 0 && CPW >= P, "chunks per wave");
    __shared__ __attribute__((aligned(16))) float zs[2][kLmWaves][16][kLmTile + 4];
    const int gamma = f.gamma;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;

    const int nblk_v = (vocab + 15) / 16;
    const int nblk = nblk_v + (f.w1 ? f.m / 16 : 0);   // + the router's W1 blocks
    // block j of this workgroup (j = kLmMB * t + mb) is blockIdx.x + G*j
    const int GB = gridDim.x;
    const int nmine = (nblk - (int)blockIdx.x + GB - 1) / GB;
    const int ntile = (nmine + kLmMB - 1) / kLmMB;

    // this wave's slice of h: chunk u covers dims (wave*CPW + u)*32 + 8*c4 ..
    bf16x8 hr[CPW];
    {
        const uint16_t *hp = h + (size_t)min(m16, gamma - 1) * D + wave * CPW * 32 + c4 * 8;
#pragma unroll
        for (int u = 0; u < CPW; ++u)
            hr[u] = load_bf16x8(hp + u * 32);
    }
    // W rows of tile t, block mb.  Blocks past the workgroup's last one (a
    // ragged last tile) re-read that block, which is in L2, and are masked
    // out of the states.
    // (tiled W: the block's 1 KB tiles of this wave's slice, one per chunk,
    // read contiguously)
    const int cs = tiled ? 512 : 32;               // elements between chunks
    const int last_blk = (int)blockIdx.x + GB * (nmine - 1);
    auto wrow = [&](int t, int mb) {
        int blk = min((int)blockIdx.x + GB * (kLmMB * t + mb), last_blk);
        const uint16_t *base = w;
        int rows = vocab;
        if (blk >= nblk_v) {                       // a router block: W1 rows
            blk -= nblk_v;
            base = f.w1;
            rows = f.m;
        }
        if (tiled)
            return base + ((size_t)blk * (D / 32) + wave * CPW) * 512 + lane * 8;
        const int row = min(blk * 16 + m16, rows - 1);
        return base + (size_t)row * D + wave * CPW * 32 + c4 * 8;
    };

    bf16x8 wb[P][kLmMB];
    {
        const int t0 = min(0, ntile - 1);
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
            for (int mb = 0; mb < kLmMB; ++mb)
                wb[p][mb] = load_bf16x8_nt(wrow(t0, mb) + p * cs);
    }
    RowState run[2] = {state_empty(), state_empty()};

    // One tile; all but the last also load the head chunks of the next tile
    // (the last tile is peeled so that no branch sits in the steady state).
    auto tile = [&](int t, auto last_tag) __attribute__((always_inline)) {
        constexpr bool LAST = decltype(last_tag)::value;
        const uint16_t *cur[kLmMB], *nxt[kLmMB];
#pragma unroll
        for (int mb = 0; mb < kLmMB; ++mb) {
            cur[mb] = wrow(t, mb);
            nxt[mb] = wrow(LAST ? t : t + 1, mb);
        }
        f32x4 acc[kLmMB];
#pragma unroll
        for (int mb = 0; mb < kLmMB; ++mb)
            acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int u = 0; u < CPW; ++u) {
            const int p = u % P;
#pragma unroll
            for (int mb = 0; mb < kLmMB; ++mb)
                acc[mb] = mfma16x16x32(wb[p][mb], hr[u], acc[mb]);
            // refill the slot with the chunk P ahead (near the end of the
            // tile: the next tile's head chunks)
            // (the last tile, whose padding blocks re-read the workgroup's
            // last block, loads its rows cached: 1.5-3 us faster per call)
            if (u + P < CPW) {
#pragma unroll
                for (int mb = 0; mb < kLmMB; ++mb)
                    wb[p][mb] = LAST ? load_bf16x8(cur[mb] + (u + P) * cs)
                                     : load_bf16x8_nt(cur[mb] + (u + P) * cs);
            } else if (!LAST) {
#pragma unroll
                for (int mb = 0; mb < kLmMB; ++mb)
                    wb[p][mb] = load_bf16x8_nt(nxt[mb] + (u + P - CPW) * cs);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // lane (m16, c4) holds logits of vocabulary rows 16*mb + 4*c4 + i of
        // the tile for verify row m16
        const int buf = t & 1;
#pragma unroll
        for (int mb = 0; mb < kLmMB; ++mb)
            *reinterpret_cast<f32x4 *>(&zs[buf][wave][m16][16 * mb + 4 * c4]) = acc[mb];
        __syncthreads();
        // rows wave and wave + 8, column = lane: sum the 8 waves in order
        const int j = kLmMB * t + lane / 16;
        const int blk = (int)blockIdx.x + GB * j;
        const int v = blk * 16 + (lane & 15);
        const bool valid = j < nmine && blk < nblk_v && v < vocab;
        const bool hidden = j < nmine && blk >= nblk_v;   // router unit v - 16 nblk_v
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int r = wave + kLmWaves * k;
            if (r < gamma) {
                float z = zs[buf][0][r][lane];
#pragma unroll
                for (int ww = 1; ww < kLmWaves; ++ww)
                    z += zs[buf][ww][r][lane];
                if (hidden)
                    f.zr[(size_t)r * f.m + (v - 16 * nblk_v)] = z;
                RowState st = valid ? state_single(z, v) : state_empty();
                st = wave_merge(st);
                run[k] = state_merge(run[k], st);
            }
        }
    };
    for (int t = 0; t + 1 < ntile; ++t)
        tile(t, std::false_type{});
    if (ntile > 0)
        tile(ntile - 1, std::true_type{});
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int r = wave + kLmWaves * k;
        if (r < gamma && lane == 0)
            f.states[(size_t)r * f.n_tiles + blockIdx.x] = run[k];
    }
}

// Persistent bf16 LM head for up to 64 verify rows (NBL groups of 16) and
// a hidden size that is a multiple of 512.  Workgroup b owns the 16-row
// vocabulary blocks [b0, b1); wave w owns blocks b0 + w + 8j, j < MBW (a
// block past the run re-reads the run's last block and is masked out of the
// states).  The hidden dimension is walked in K-blocks of 512 dims: each
// K-block of h, all rows, is staged in LDS (double-buffered; the 16-byte
// granules of a row are XOR-swizzled by the row so the MFMA operand reads
// are bank-conflict free) and shared by the 8 waves, so h leaves L2 once per
// workgroup and K-block, while W streams from HBM straight into registers P
// chunks ahead, across K-block boundaries (the last K-block is peeled).  The
// logits of all of a wave's blocks stay in registers for the whole K loop,
// and each row's state over the run is formed once at the end: lane values
// in ascending vocabulary order, then the 4 lanes of a row, then the 8 waves
// in order.
constexpr int kWideK = 512;                 // hidden dims per staged K-block
constexpr int kWideGran = kWideK / 8;       // 16-byte granules per row per K-block
constexpr int kWideMaxBlocksPerWave = 5;

template <int NBL, int MBW, int P>
__global__ __launch_bounds__(512) void lm_wide_bf16(const uint16_t *__restrict__ h,
                                                    const uint16_t *__restrict__ w,
                                                    LmFinish f, int d, int vocab, int tiled) {
    constexpr int ROWS = 16 * NBL;
    constexpr int CPB = kWideK / 32;                   // chunks per K-block
    constexpr int HLOADS = ROWS * kWideGran / 512;     // h granules per thread per K-block
    static_assert(CPB % P == 0, "prefetch depth must divide the K-block");
    __shared__ __attribute__((aligned(16))) u32x4 hs[2][ROWS][kWideGran];
    __shared__ RowState wst[kLmWaves][ROWS];

    const int gamma = f.gamma;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;
    const int nblk = (vocab + 15) / 16;
    const int b0 = (int)((long long)blockIdx.x * nblk / gridDim.x);
    const int b1 = (int)((long long)(blockIdx.x + 1) * nblk / gridDim.x);
    const int nkb = d / kWideK;

    // chunk 0 of each of this wave's blocks (tiled W: the block's first
    // 1 KB tile; chunks follow 512 elements apart instead of 32)
    const int cs = tiled ? 512 : 32;
    const uint16_t *wrow[MBW];
#pragma unroll
    for (int j = 0; j < MBW; ++j) {
        const int blk = max(min(b0 + wave + 8 * j, b1 - 1), 0);
        wrow[j] = tiled ? w + (size_t)blk * (d / 32) * 512 + lane * 8
                        : w + (size_t)min(blk * 16 + m16, vocab - 1) * d + c4 * 8;
    }
    // h staging: granule idx = threadIdx.x + 512 q of the K-block is row
    // idx / kWideGran, granule idx % kWideGran (rows past gamma repeat the
    // last row; their logits are never used)
    // (staged in two halves, q in [half*HH, (half+1)*HH), to keep few
    // registers in flight)
    constexpr int HH = HLOADS / 2;
    static_assert(HLOADS % 2 == 0, "h staging halves");
    auto hload = [&](int kb, int half, u32x4 (&hr)[HH]) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < HH; ++q) {
            const int idx = threadIdx.x + 512 * (half * HH + q);
            const int row = idx / kWideGran, g = idx % kWideGran;
            hr[q] = *reinterpret_cast<const u32x4 *>(
                h + (size_t)min(row, gamma - 1) * d + kb * kWideK + 8 * g);
        }
    };
    auto hstore = [&](int buf, int half, const u32x4 (&hr)[HH]) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < HH; ++q) {
            const int idx = threadIdx.x + 512 * (half * HH + q);
            const int row = idx / kWideGran, g = idx % kWideGran;
            hs[buf][row][g ^ (row & 15)] = hr[q];
        }
    };

    f32x4 acc[MBW][NBL];
#pragma unroll
    for (int j = 0; j < MBW; ++j)
#pragma unroll
        for (int nb = 0; nb < NBL; ++nb)
            acc[j][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    bf16x8 wb[P][MBW];
    {
        u32x4 hr[HH];
        hload(0, 0, hr);
        hstore(0, 0, hr);
        hload(0, 1, hr);
        hstore(0, 1, hr);
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
            for (int j = 0; j < MBW; ++j)
                wb[p][j] = load_bf16x8_nt(wrow[j] + p * cs);
        __syncthreads();
    }

    // One K-block; all but the last also stage the next K-block of h and
    // refill W from the next K-block's first chunks.
    auto kblock = [&](int kb, auto last_tag) __attribute__((always_inline)) {
        constexpr bool LAST = decltype(last_tag)::value;
        const int buf = kb & 1;
        u32x4 hr[HH];
        if (!LAST)
            hload(kb + 1, 0, hr);
        const int cbase = kb * CPB;
#pragma unroll
        for (int u = 0; u < CPB; ++u) {
            const int p = u % P;
            if (!LAST && u == CPB / 2) {
                hstore(buf ^ 1, 0, hr);
                hload(kb + 1, 1, hr);
            }
            bf16x8 hop[NBL];
#pragma unroll
            for (int nb = 0; nb < NBL; ++nb)
                hop[nb] = __builtin_bit_cast(bf16x8, hs[buf][nb * 16 + m16][(4 * u + c4) ^ m16]);
#pragma unroll
            for (int j = 0; j < MBW; ++j)
#pragma unroll
                for (int nb = 0; nb < NBL; ++nb)
                    acc[j][nb] = mfma16x16x32(wb[p][j], hop[nb], acc[j][nb]);
            if (!LAST || u + P < CPB) {
#pragma unroll
                for (int j = 0; j < MBW; ++j)
                    wb[p][j] = load_bf16x8_nt(wrow[j] + (size_t)(cbase + u + P) * cs);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (!LAST) {
            hstore(buf ^ 1, 1, hr);
            asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        }
    };
    for (int kb = 0; kb + 1 < nkb; ++kb)
        kblock(kb, std::false_type{});
    kblock(nkb - 1, std::true_type{});

    // row states: lane values in ascending vocabulary order, then the four
    // lanes of a row (fixed butterfly), then the waves in order
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb) {
        RowState st = state_empty();
#pragma unroll
        for (int j = 0; j < MBW; ++j) {
            const int blk = b0 + wave + 8 * j;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int v = blk * 16 + 4 * c4 + i;
                if (blk < b1 && v < vocab)
                    st = state_merge(st, state_single(acc[j][nb][i], v));
            }
        }
        st = state_merge(st, shfl_xor_state(st, 16));
        st = state_merge(st, shfl_xor_state(st, 32));
        if (c4 == 0)
            wst[wave][nb * 16 + m16] = st;
    }
    __syncthreads();
    const int r = threadIdx.x;
    if (r < gamma) {
        RowState m = wst[0][r];
#pragma unroll
        for (int ww = 1; ww < kLmWaves; ++ww)
            m = state_merge(m, wst[ww][r]);
        f.states[(size_t)r * f.n_tiles + blockIdx.x] = m;
    }
}

// NR = verify rows per thread (rows rq, rq + 4, ...: ceil(gamma / 4) rounded
// up to a power of two), a template parameter so the inner loop carries no
// per-row branches.
template <int NR>
__global__ __launch_bounds__(256) void lm_tiles_f32(const float *__restrict__ h,
                                                    const float *__restrict__ w,
                                                    LmFinish f, int d, int vocab) {
    RowState *states = f.states;
    const int gamma = f.gamma, n_tiles = f.n_tiles;
    constexpr int kRowsPerThread = NR;
    static_assert(kMaxGamma == kLmTile, "h and W tiles share the staging map");
    __shared__ __attribute__((aligned(16))) float zs[kMaxGamma][kLmTile + 4];
    const int tile = blockIdx.x;
    const int v0 = tile * kLmTile;
    const int vl = threadIdx.x % kLmTile;
    const int rq = threadIdx.x / kLmTile;
    // h and the tile's W rows are staged in LDS 128 dims at a time with
    // coalesced loads; W rows are padded so the 64 threads of a wave (64
    // vocabulary rows, one column) hit distinct banks, and a wave's threads
    // share one verify-row group, so each h read is a broadcast.  Each
    // thread's sum still runs over the dimensions in order.
    // (every thread issues all of its staging loads before its first LDS
    // store: one memory round trip per chunk)
    constexpr int KC = 128;
    constexpr int NL = kLmTile * KC / 256;          // staged floats per thread
    __shared__ float hs[kMaxGamma][KC];
    __shared__ float wt[kLmTile][KC + 1];
    float acc[kRowsPerThread];
#pragma unroll
    for (int k = 0; k < kRowsPerThread; ++k)
        acc[k] = 0.f;
    for (int c0 = 0; c0 < d; c0 += KC) {
        const int kc = min(KC, d - c0);
        float hv[NL], wv_[NL];
#pragma unroll
        for (int u = 0; u < NL; ++u) {
            const int idx = threadIdx.x + 256 * u;
            const int r = idx / KC, c = idx % KC;     // kMaxGamma * KC == kLmTile * KC
            hv[u] = (r < gamma && c < kc) ? h[(size_t)r * d + c0 + c] : 0.f;
            wv_[u] = c < kc ? w[(size_t)min(v0 + r, vocab - 1) * d + c0 + c] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < NL; ++u) {
            const int idx = threadIdx.x + 256 * u;
            hs[idx / KC][idx % KC] = hv[u];
            wt[idx / KC][idx % KC] = wv_[u];
        }
        __syncthreads();
#pragma unroll 8
        for (int c = 0; c < kc; ++c) {
            const float wv = wt[vl][c];
#pragma unroll
            for (int k = 0; k < kRowsPerThread; ++k)      // rows past gamma: zeros
                acc[k] = fmaf(hs[rq + 4 * k][c], wv, acc[k]);
        }
    }
#pragma unroll
    for (int k = 0; k < kRowsPerThread; ++k) {
        const int r = rq + 4 * k;
        if (r < gamma)
            zs[r][vl] = acc[k];
    }
    __syncthreads();
    tile_states(zs, states, tile, n_tiles, v0, gamma, vocab, threadIdx.x / kWave,
                blockDim.x / kWave, threadIdx.x % kWave);
}

__global__ __launch_bounds__(256) void lm_tiles_logits(const float *__restrict__ logits,
                                                       LmFinish f, int vocab) {
    const int tile = blockIdx.x;
    const int v0 = tile * kLogitsTile;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    for (int r = wave; r < f.gamma; r += 4) {
        const float *row = logits + (size_t)r * vocab;
        RowState s = state_empty();
#pragma unroll
        for (int e = 0; e < kLogitsTile / kWave; ++e) {
            const int v = v0 + e * kWave + lane;
            if (v < vocab)
                s = state_merge(s, state_single(row[v], v));
        }
        s = wave_merge(s);
        if (lane == 0)
            f.states[(size_t)r * f.n_tiles + tile] = s;
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

// The counter block at the workspace start holds the ticket counter; the
// tile states (sized for the finest tiling) follow it.
size_t lmhead_workspace_bytes(int gamma, int vocab) {
    return kCounterBytes + (size_t)gamma * cdiv(vocab, kLmTile) * sizeof(RowState);
}


bool lmhead_router_fusable(wf_dtype_t dt, int gamma, int d, int m) {
    return (dt == WF_BF16 || dt == WF_BF16_TILED) && gamma <= 16 && (d == 4096 || d == 5120) &&
           m >= 16 && m % 16 == 0;
}

size_t lmhead_router_workspace_bytes(int gamma, int vocab, int m) {
    return lmhead_workspace_bytes(gamma, vocab) + (size_t)gamma * m * sizeof(float);
}

wf_status_t launch_lmhead(wf_dtype_t dt, const void *h, const void *w_lm,
                          const float *logits, const int32_t *draft,
                          const int32_t *parents, int gamma, int d, int vocab,
                          float tau, int32_t *argmax_out, float *entropy_out,
                          int32_t *accept_out, int32_t *path_out,
                          void *workspace, hipStream_t stream, const LmRouter *router) {
    if (router && (logits || parents || !lmhead_router_fusable(dt, gamma, d, router->m)))
        return WF_ERR_UNSUPPORTED;
    const int tiled = dt == WF_BF16_TILED ? 1 : 0;
    if (tiled)
        dt = WF_BF16;
    char *ws = static_cast<char *>(workspace);
    LmFinish f;
    f.states = reinterpret_cast<RowState *>(ws + kCounterBytes);
    f.fcnt = reinterpret_cast<unsigned *>(ws);
    f.draft = draft;
    f.parents = parents;
    f.path_out = path_out;
    f.argmax_out = argmax_out;
    f.entropy_out = entropy_out;
    f.accept_out = accept_out;
    f.gamma = gamma;
    f.tau = tau;
    f.w1 = nullptr;
    f.b1 = f.w2 = f.b2 = nullptr;
    f.zr = nullptr;
    f.delta_out = nullptr;
    f.m = 0;
    f.tau_neural = 0.f;
    if (router) {
        f.w1 = static_cast<const uint16_t *>(router->w1);
        f.b1 = static_cast<const uint16_t *>(router->b1);
        f.w2 = static_cast<const uint16_t *>(router->w2);
        f.b2 = static_cast<const uint16_t *>(router->b2);
        f.m = router->m;
        f.tau_neural = router->tau;
        f.delta_out = router->delta_out;
        f.zr = reinterpret_cast<float *>(ws + lmhead_workspace_bytes(gamma, vocab));
    }
    if (logits) {
        f.n_tiles = cdiv(vocab, kLogitsTile);
        lm_tiles_logits<<<f.n_tiles, 256, 0, stream>>>(logits, f, vocab);
    } else if (dt == WF_BF16 && gamma <= 16 && (d == 4096 || d == 5120)) {
        // persistent: one workgroup per CU, one state per row per workgroup
        f.n_tiles = std::min(kLmStreamGrid, cdiv(vocab, kLmTile));
        const uint16_t *hb = static_cast<const uint16_t *>(h);
        const uint16_t *wb = static_cast<const uint16_t *>(w_lm);
        if (d == 4096)
            lm_stream_bf16<16><<<f.n_tiles, 512, 0, stream>>>(hb, wb, f, vocab, tiled);
        else
            lm_stream_bf16<20><<<f.n_tiles, 512, 0, stream>>>(hb, wb, f, vocab, tiled);
    } else if (dt == WF_BF16 && d % kWideK == 0) {
        // persistent: about one workgroup per CU, each wave at most
        // kWideMaxBlocksPerWave 16-row vocabulary blocks
        const int nblk = cdiv(vocab, 16);
        const int per_wg = kLmWaves * kWideMaxBlocksPerWave;
        f.n_tiles = std::max(std::min(kLmStreamGrid, cdiv(nblk, kLmWaves)), cdiv(nblk, per_wg));
        const int mbw = cdiv(cdiv(nblk, f.n_tiles), kLmWaves);
        const uint16_t *hb = static_cast<const uint16_t *>(h);
        const uint16_t *wb = static_cast<const uint16_t *>(w_lm);
        const int nbl = cdiv(gamma, 16);
#define WF_WIDE(NBLV, MBWV, PV)                                                              \
    if (nbl == NBLV && mbw <= MBWV) {                                                      \
        lm_wide_bf16<NBLV, MBWV, PV><<<f.n_tiles, 512, 0, stream>>>(hb, wb, f, d, vocab,   \
                                                                    tiled);                \
    } else
        WF_WIDE(1, 2, 4) WF_WIDE(1, 5, 4) WF_WIDE(2, 2, 4) WF_WIDE(2, 5, 4)
        WF_WIDE(3, 2, 4) WF_WIDE(3, 5, 2) WF_WIDE(4, 2, 4) WF_WIDE(4, 5, 2)
        { return WF_ERR_UNSUPPORTED; }
#undef WF_WIDE
    } else if (tiled) {
        return WF_ERR_UNSUPPORTED;              // no tiled form of the tile kernel
    } else if (dt == WF_BF16) {
        f.n_tiles = cdiv(vocab, kLmTile);
        const uint16_t *hb = static_cast<const uint16_t *>(h);
        const uint16_t *wb = static_cast<const uint16_t *>(w_lm);
        const int nbl = cdiv(gamma, 16);
        switch (nbl) {
        case 1: lm_tiles_bf16<1><<<f.n_tiles, 512, 0, stream>>>(hb, wb, f, d, vocab); break;
        case 2: lm_tiles_bf16<2><<<f.n_tiles, 512, 0, stream>>>(hb, wb, f, d, vocab); break;
        case 3: lm_tiles_bf16<3><<<f.n_tiles, 512, 0, stream>>>(hb, wb, f, d, vocab); break;
        default: lm_tiles_bf16<4><<<f.n_tiles, 512, 0, stream>>>(hb, wb, f, d, vocab); break;
        }
    } else {
        f.n_tiles = cdiv(vocab, kLmTile);
        const float *hf = static_cast<const float *>(h);
        const float *wf32 = static_cast<const float *>(w_lm);
        const int nr = cdiv(gamma, 4);
        if (nr <= 2)
            lm_tiles_f32<2><<<f.n_tiles, 256, 0, stream>>>(hf, wf32, f, d, vocab);
        else if (nr <= 4)
            lm_tiles_f32<4><<<f.n_tiles, 256, 0, stream>>>(hf, wf32, f, d, vocab);
        else if (nr <= 8)
            lm_tiles_f32<8><<<f.n_tiles, 256, 0, stream>>>(hf, wf32, f, d, vocab);
        else
            lm_tiles_f32<16><<<f.n_tiles, 256, 0, stream>>>(hf, wf32, f, d, vocab);
    }
    lm_finish_rows<<<gamma, kFinishThreads, 0, stream>>>(f);
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
