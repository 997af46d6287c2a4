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
// Stage 2 (one workgroup): per row, merge the tile states in ascending tile
// order, emit argmax and entropy, then the accept length, bonus token and
// route.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kLmTile = 64;          // vocabulary rows per matmul tile
constexpr int kLmMB = kLmTile / 16;  // 16-row MFMA blocks per tile
constexpr int kLmWaves = 8;
constexpr int kLmPrefetch = 4;       // 32-dim chunks in flight per wave
constexpr int kLogitsTile = 256;     // vocabulary entries per logits tile
constexpr int kMaxGamma = 64;

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

template <int NBL>
__global__ __launch_bounds__(512) void lm_tiles_bf16(const uint16_t *__restrict__ h,
                                                     const uint16_t *__restrict__ w,
                                                     RowState *__restrict__ states,
                                                     int gamma, int d, int vocab,
                                                     int n_tiles) {
    __shared__ __attribute__((aligned(16))) float zs[kMaxGamma][kLmTile + 4];
    const int tile = blockIdx.x;
    const int v0 = tile * kLmTile;
    const int wave = threadIdx.x / kWave;
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
            wr[mb] = load_bf16x8(wp[mb] + off);
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

__global__ __launch_bounds__(256) void lm_tiles_f32(const float *__restrict__ h,
                                                    const float *__restrict__ w,
                                                    RowState *__restrict__ states,
                                                    int gamma, int d, int vocab,
                                                    int n_tiles) {
    constexpr int kRowsPerThread = kMaxGamma / 4;
    __shared__ __attribute__((aligned(16))) float zs[kMaxGamma][kLmTile + 4];
    const int tile = blockIdx.x;
    const int v0 = tile * kLmTile;
    const int vl = threadIdx.x % kLmTile;
    const int rq = threadIdx.x / kLmTile;
    const float *wr = w + (size_t)min(v0 + vl, vocab - 1) * d;
    float acc[kRowsPerThread];
#pragma unroll
    for (int k = 0; k < kRowsPerThread; ++k)
        acc[k] = 0.f;
    for (int c = 0; c < d; ++c) {
        const float wv = wr[c];
#pragma unroll
        for (int k = 0; k < kRowsPerThread; ++k) {
            const int r = rq + 4 * k;
            if (r < gamma)
                acc[k] = fmaf(h[(size_t)r * d + c], wv, acc[k]);
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
                                                       RowState *__restrict__ states,
                                                       int gamma, int vocab,
                                                       int n_tiles) {
    const int tile = blockIdx.x;
    const int v0 = tile * kLogitsTile;
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    for (int r = wave; r < gamma; r += 4) {
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
            states[(size_t)r * n_tiles + tile] = s;
    }
}

__global__ __launch_bounds__(1024) void lm_finish(const RowState *__restrict__ states,
                                                  int n_tiles,
                                                  const int32_t *__restrict__ draft,
                                                  int gamma, float tau,
                                                  int32_t *__restrict__ argmax_out,
                                                  float *__restrict__ entropy_out,
                                                  int32_t *__restrict__ accept_out) {
    __shared__ int32_t am[kMaxGamma];
    __shared__ float ent[kMaxGamma];
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const int n_waves = blockDim.x / kWave;
    for (int r = wave; r < gamma; r += n_waves) {
        const RowState *row = states + (size_t)r * n_tiles;
        RowState s = state_empty();
        for (int t = lane; t < n_tiles; t += kWave)
            s = state_merge(s, row[t]);
        s = wave_merge(s);
        if (lane == 0) {
            const float H = state_entropy(s);
            argmax_out[r] = s.a;
            entropy_out[r] = H;
            am[r] = s.a;
            ent[r] = H;
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int n = 0;
        while (n < gamma - 1 && draft[n] == am[n])
            ++n;
        accept_out[0] = n;
        accept_out[1] = am[n];
        accept_out[2] = (ent[n] > tau) ? 1 : 0;
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

size_t lmhead_workspace_bytes(int gamma, int vocab) {
    return (size_t)gamma * cdiv(vocab, kLmTile) * sizeof(RowState);
}

wf_status_t launch_lmhead(wf_dtype_t dt, const void *h, const void *w_lm,
                          const float *logits, const int32_t *draft, int gamma,
                          int d, int vocab, float tau, int32_t *argmax_out,
                          float *entropy_out, int32_t *accept_out,
                          void *workspace, hipStream_t stream) {
    RowState *states = static_cast<RowState *>(workspace);
    int n_tiles;
    if (logits) {
        n_tiles = cdiv(vocab, kLogitsTile);
        lm_tiles_logits<<<n_tiles, 256, 0, stream>>>(logits, states, gamma, vocab, n_tiles);
    } else if (dt == WF_BF16) {
        n_tiles = cdiv(vocab, kLmTile);
        const uint16_t *hb = static_cast<const uint16_t *>(h);
        const uint16_t *wb = static_cast<const uint16_t *>(w_lm);
        const int nbl = cdiv(gamma, 16);
        switch (nbl) {
        case 1: lm_tiles_bf16<1><<<n_tiles, 512, 0, stream>>>(hb, wb, states, gamma, d, vocab, n_tiles); break;
        case 2: lm_tiles_bf16<2><<<n_tiles, 512, 0, stream>>>(hb, wb, states, gamma, d, vocab, n_tiles); break;
        case 3: lm_tiles_bf16<3><<<n_tiles, 512, 0, stream>>>(hb, wb, states, gamma, d, vocab, n_tiles); break;
        default: lm_tiles_bf16<4><<<n_tiles, 512, 0, stream>>>(hb, wb, states, gamma, d, vocab, n_tiles); break;
        }
    } else {
        n_tiles = cdiv(vocab, kLmTile);
        lm_tiles_f32<<<n_tiles, 256, 0, stream>>>(static_cast<const float *>(h),
                                                 static_cast<const float *>(w_lm),
                                                 states, gamma, d, vocab, n_tiles);
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    lm_finish<<<1, 1024, 0, stream>>>(states, n_tiles, draft, gamma, tau, argmax_out,
                                      entropy_out, accept_out);
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
