// gemv.hip -- skinny linear layers y = W x for a handful of rows x (at most
// 64: the verify rows of the neural router, the tokens of a drafter layer),
// split over the input dimension so that even a few hundred output features
// spread over the chip.  Workgroup (t, k) owns output features 16t .. 16t+15
// and the k-th slice of the input; its 8 waves take interleaved 32-wide
// chunks of the slice with all loads of a batch issued before its first
// MFMA (16x16x32 bf16: A = 16 features x 32 inputs, B = 32 inputs x 16
// rows), and their partial sums meet in LDS in wave order.  The result is
// one fp32 partial per slice, zpart[k][feature][row]; the caller's epilogue
// kernel adds the slices in order.  Two weight matrices may share a launch
// (features [0, n_a) from w_a, [n_a, n_a + n_b) from w_b), as the gate and
// up projections of a SwiGLU MLP do.  Weights row-major or in 16x32 tiles
// of 1 KB (one contiguous wave load per chunk).
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kGemvWaves = 8;
constexpr int kGemvBatch = 8;          // 32-wide chunks per wave per load batch
constexpr int kGemvTargetWorkgroups = 1024;
constexpr int kComputeUnits = 256;

// FB 16-feature blocks per workgroup: with many rows each workgroup reads
// its slice of x for FB blocks at once (x would otherwise be re-read by
// every 16-feature workgroup); fewer chunks per load batch keep the
// operands in registers, and the 8 waves' sums meet in LDS RB blocks at a
// time.  Every accumulator still takes its chunks in the same order, so
// the result does not depend on FB.
//
// SWI (one slice, w_a = W_gate and w_b = W_up, both n_a features): the
// first FB/2 blocks of workgroup b are gate blocks FB/2 * b + j and the
// rest the matching up blocks, and the epilogue stores
// act[r][f] = bf16(SiLU(gate) * up) instead of the fp32 sums: the same
// values, rounded the same way, as the sums followed by the separate
// SwiGLU kernel.
template <int NBL, int FB, bool SWI = false>
__global__ __launch_bounds__(kGemvWaves * kWave) void linear_partial_bf16(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ w_a,
    const uint16_t *__restrict__ w_b, int n_a, float *__restrict__ zpart, int rows,
    int k_in, int n_out, int chunks_per_slice, int tiled, uint16_t *__restrict__ act) {
    static_assert(!SWI || (FB % 2 == 0), "gate and up blocks come in pairs");
    constexpr int BATCH = FB == 1 ? kGemvBatch : FB <= 4 ? kGemvBatch / 2 : 2;
    constexpr int RB = (SWI || FB > 4) ? 2 : FB;
    constexpr int HB = FB / 2;
    __shared__ float zs[kGemvWaves][16 * RB][16 * NBL + 1];
    const int f00 = 16 * FB * blockIdx.x;
    const int ks = blockIdx.y;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;
    const int c_begin = ks * chunks_per_slice;
    const int n_c = max(0, min(chunks_per_slice, k_in / 32 - c_begin));

    // W operand of chunk c for block fb: row-major, 16 bytes of row
    // f0 + m16 per lane; tiled, the 1 KB tile of the 16-feature block
    // (n_a % 16 == 0, so a block never straddles the two matrices)
    const uint16_t *wp[FB];
    const int wstep = tiled ? 512 : 32;
#pragma unroll
    for (int fb = 0; fb < FB; ++fb) {
        const int f0 = SWI ? 16 * (HB * (int)blockIdx.x + fb % HB) + (fb < HB ? 0 : n_a)
                           : f00 + 16 * fb;
        if (tiled) {
            const int blk = f0 < n_a ? f0 / 16 : (f0 - n_a) / 16;
            wp[fb] = (f0 < n_a ? w_a : w_b) + ((size_t)blk * (k_in / 32) + c_begin) * 512 +
                     lane * 8;
        } else {
            const int f = f0 + m16;
            const uint16_t *wrow =
                f < n_a ? w_a + (size_t)f * k_in : w_b + (size_t)(f - n_a) * k_in;
            wp[fb] = wrow + (size_t)c_begin * 32 + c4 * 8;
        }
    }
    // rows past `rows` read the last row: their columns are never used
    const uint16_t *xp[NBL];
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
        xp[nb] = x + (size_t)min(16 * nb + m16, rows - 1) * k_in + (size_t)c_begin * 32 + c4 * 8;

    f32x4 acc[FB][NBL];
#pragma unroll
    for (int fb = 0; fb < FB; ++fb)
#pragma unroll
        for (int nb = 0; nb < NBL; ++nb)
            acc[fb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int cb = wave; cb < n_c; cb += kGemvWaves * BATCH) {
        bf16x8 wr[BATCH][FB], xr[BATCH][NBL];
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
            const int c = cb + kGemvWaves * u;
            if (c < n_c) {
#pragma unroll
                for (int fb = 0; fb < FB; ++fb)
                    wr[u][fb] = load_bf16x8_nt(wp[fb] + (size_t)c * wstep);
#pragma unroll
                for (int nb = 0; nb < NBL; ++nb)
                    xr[u][nb] = load_bf16x8(xp[nb] + c * 32);
            }
        }
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
            if (cb + kGemvWaves * u < n_c) {
#pragma unroll
                for (int fb = 0; fb < FB; ++fb)
#pragma unroll
                    for (int nb = 0; nb < NBL; ++nb)
                        acc[fb][nb] = mfma16x16x32(wr[u][fb], xr[u][nb], acc[fb][nb]);
            }
        }
    }
#pragma unroll
    for (int pb = 0; pb < FB / RB; ++pb) {
        if (pb)
            __syncthreads();
#pragma unroll
        for (int fr = 0; fr < RB; ++fr)
#pragma unroll
            for (int nb = 0; nb < NBL; ++nb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    zs[wave][16 * fr + 4 * c4 + i][16 * nb + m16] =
                        acc[SWI ? pb + HB * fr : pb * RB + fr][nb][i];
        __syncthreads();
        if constexpr (SWI) {
            // gate block pb in zs rows 0..15, its up block in 16..31; 16
            // consecutive features per row, so the stores form 32-byte runs
            const int g0 = 16 * (HB * (int)blockIdx.x + pb);
            for (int idx = threadIdx.x; idx < 16 * rows; idx += blockDim.x) {
                const int u = idx % 16, r = idx / 16;
                float zg = zs[0][u][r], zu = zs[0][16 + u][r];
#pragma unroll
                for (int ww = 1; ww < kGemvWaves; ++ww) {
                    zg += zs[ww][u][r];
                    zu += zs[ww][16 + u][r];
                }
                // (0 + z: the sum over one slice, as the slice sum forms it)
                const float gt = 0.f + zg, up = 0.f + zu;
                act[(size_t)r * n_a + g0 + u] = f32_to_bf16(gt / (1.f + expf(-gt)) * up);
            }
            continue;
        }
        for (int idx = threadIdx.x; idx < 16 * RB * rows; idx += blockDim.x) {
            const int u = idx / rows, r = idx % rows;
            float z = zs[0][u][r];
#pragma unroll
            for (int ww = 1; ww < kGemvWaves; ++ww)
                z += zs[ww][u][r];
            zpart[((size_t)ks * n_out + f00 + 16 * RB * pb + u) * rows + r] = z;
        }
    }
}

// Skinny linear layer with its epilogue in the same kernel, for a single
// token (one row): workgroup t owns one or two 16-feature blocks and the
// whole input dimension, so no partial sums leave the workgroup.  The 8
// waves take interleaved 32-wide chunks (all loads of a batch issued before
// its first MFMA), their sums meet in LDS in wave order, and the epilogue
// writes bf16 outputs:
//   kEpiResid   y = res + W x                      (block t)
//   kEpiSwiglu  act = SiLU(Wg x') * (Wu x')       (gate block t, up block t),
//               x' = RMSNorm(x) * gain, folded in: W (x * gain) is formed from
//               x * gain in bf16 and scaled by the row's 1/rms, whose sum of
//               squares the workgroup forms from the same loads of x.
enum EpiMode { kEpiResid = 0, kEpiSwiglu = 1 };

struct EpiParams {
    const uint16_t *x;      // [k_in] (kEpiSwiglu: the un-normalised row)
    const uint16_t *w_a;    // blocks A
    const uint16_t *w_b;    // kEpiSwiglu: the up projection
    const uint16_t *res;    // kEpiResid: [n_out]
    const uint16_t *gain;   // kEpiSwiglu: RMSNorm gains [k_in]
    uint16_t *y;            // [n_out]
    float eps;
    int k_in, n_out, tiled;
};

template <int MODE>
__global__ __launch_bounds__(kGemvWaves * kWave) void linear_epi_bf16(EpiParams a) {
    constexpr int NBLK = MODE == kEpiResid ? 1 : 2;
    __shared__ float zs[kGemvWaves][16 * NBLK];
    __shared__ float sq[kGemvWaves];
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;
    const int n_c = a.k_in / 32;

    // blocks of this workgroup and their matrices
    int blk[NBLK];
    const uint16_t *wm[NBLK];
    if constexpr (MODE == kEpiResid) {
        blk[0] = blockIdx.x;
        wm[0] = a.w_a;
    } else {
        blk[0] = blk[1] = blockIdx.x;
        wm[0] = a.w_a;
        wm[1] = a.w_b;
    }
    const uint16_t *wp[NBLK];
    int wstep;
#pragma unroll
    for (int j = 0; j < NBLK; ++j)
        wp[j] = a.tiled ? wm[j] + (size_t)blk[j] * n_c * 512 + lane * 8
                        : wm[j] + (size_t)(16 * blk[j] + m16) * a.k_in + c4 * 8;
    wstep = a.tiled ? 512 : 32;
    const uint16_t *xp = a.x + c4 * 8;          // the row, as the B operand (column 0..15 alike)
    const uint16_t *gp = a.gain + c4 * 8;

    f32x4 acc[NBLK];
#pragma unroll
    for (int j = 0; j < NBLK; ++j)
        acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    float ss = 0.f;
    // (two blocks: half the batch, so the same bytes are in flight and the
    // registers leave room for two workgroups per compute unit)
    constexpr int BATCH = NBLK == 1 ? kGemvBatch : kGemvBatch / 2;
    for (int cb = wave; cb < n_c; cb += kGemvWaves * BATCH) {
        bf16x8 wr[BATCH][NBLK], xr[BATCH];
        u32x4 gr[BATCH];
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
            const int c = cb + kGemvWaves * u;
            if (c < n_c) {
#pragma unroll
                for (int j = 0; j < NBLK; ++j)
                    wr[u][j] = load_bf16x8_nt(wp[j] + (size_t)c * wstep);
                xr[u] = load_bf16x8(xp + c * 32);
                if constexpr (MODE == kEpiSwiglu)
                    gr[u] = *reinterpret_cast<const u32x4 *>(gp + c * 32);
            }
        }
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
            if (cb + kGemvWaves * u < n_c) {
                bf16x8 xo = xr[u];
                if constexpr (MODE == kEpiSwiglu) {
                    // x * gain in bf16, and the row's sum of squares (each
                    // lane of column 0 counts its 8 elements once)
                    const u32x4 xv = __builtin_bit_cast(u32x4, xr[u]);
                    u32x4 o;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float x0 = __uint_as_float(xv[e] << 16);
                        const float x1 = __uint_as_float(xv[e] & 0xffff0000u);
                        const float g0 = __uint_as_float(gr[u][e] << 16);
                        const float g1 = __uint_as_float(gr[u][e] & 0xffff0000u);
                        if (m16 == 0) {
                            ss = fmaf(x0, x0, ss);
                            ss = fmaf(x1, x1, ss);
                        }
                        o[e] = pack_bf16x2(x0 * g0, x1 * g1);
                    }
                    xo = __builtin_bit_cast(bf16x8, o);
                }
#pragma unroll
                for (int j = 0; j < NBLK; ++j)
                    acc[j] = mfma16x16x32(wr[u][j], xo, acc[j]);
            }
        }
    }
    // lane (m16, c4) holds features 4*c4 + i of column m16 (every column
    // is the same row; column 0 is kept)
    if (m16 == 0) {
#pragma unroll
        for (int j = 0; j < NBLK; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                zs[wave][16 * j + 4 * c4 + i] = acc[j][i];
    }
    if constexpr (MODE == kEpiSwiglu) {
        ss += __shfl_xor(ss, 16, kWave);
        ss += __shfl_xor(ss, 32, kWave);
        if (lane == 0)
            sq[wave] = ss;
    }
    __syncthreads();
    const int e = threadIdx.x;
    if (e >= 16)
        return;
    float z[NBLK];
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
        z[j] = zs[0][16 * j + e];
#pragma unroll
        for (int ww = 1; ww < kGemvWaves; ++ww)
            z[j] += zs[ww][16 * j + e];
    }
    if constexpr (MODE == kEpiResid) {
        const int f = 16 * blk[0] + e;
        a.y[f] = f32_to_bf16(z[0] + bf16_to_f32(a.res[f]));
    } else {
        float tot = sq[0];
#pragma unroll
        for (int ww = 1; ww < kGemvWaves; ++ww)
            tot += sq[ww];
        const float inv = 1.f / sqrtf(tot / (float)a.k_in + a.eps);
        const float gt = z[0] * inv, up = z[1] * inv;
        a.y[16 * blk[0] + e] = f32_to_bf16(gt / (1.f + expf(-gt)) * up);
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

wf_status_t launch_linear_resid(const uint16_t *x, const uint16_t *w, const uint16_t *res,
                                int k_in, int n_out, uint16_t *y, hipStream_t stream,
                                bool tiled) {
    EpiParams a{};
    a.x = x;
    a.w_a = w;
    a.res = res;
    a.y = y;
    a.k_in = k_in;
    a.n_out = n_out;
    a.tiled = tiled ? 1 : 0;
    linear_epi_bf16<kEpiResid><<<n_out / 16, kGemvWaves * kWave, 0, stream>>>(a);
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

wf_status_t launch_linear_norm_swiglu(const uint16_t *x, const uint16_t *gain, float eps,
                                      const uint16_t *w_gate, const uint16_t *w_up, int k_in,
                                      int inter, uint16_t *act, hipStream_t stream,
                                      bool tiled) {
    EpiParams a{};
    a.x = x;
    a.gain = gain;
    a.eps = eps;
    a.w_a = w_gate;
    a.w_b = w_up;
    a.y = act;
    a.k_in = k_in;
    a.n_out = inter;
    a.tiled = tiled ? 1 : 0;
    linear_epi_bf16<kEpiSwiglu><<<inter / 16, kGemvWaves * kWave, 0, stream>>>(a);
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

int linear_slices(int k_in, int n_out) {
    const int chunks = k_in / 32;
    const int tiles = n_out / 16;
    // up to four workgroups per compute unit, at least 4 chunks per slice
    int ks = 1;
    while (tiles * ks * 2 <= kGemvTargetWorkgroups && chunks / (ks * 2) >= 4 &&
           ks * 2 <= kLinearMaxSlices)
        ks *= 2;
    return ks;
}

wf_status_t launch_linear_partial(const uint16_t *x, const uint16_t *w_a,
                                  const uint16_t *w_b, int n_a, int n_b, int rows,
                                  int k_in, float *zpart, hipStream_t stream, bool tiled) {
    const int t = tiled ? 1 : 0;
    const int n_out = n_a + n_b;
    const int ks = linear_slices(k_in, n_out);
    const int cps = cdiv(k_in / 32, ks);
    const dim3 block(kGemvWaves * kWave);
    const int nbl = cdiv(rows, 16);
    // From 12 rows on, several feature blocks per workgroup: x is then read
    // once per 64 or 96 features instead of once per 16 (64 rows of a
    // 4096-wide x weigh as much as the workgroup's weights); below that the
    // extra workgroups of single blocks pay more.  Among the block counts
    // that divide the features, take the one with the fewest operand bytes
    // per compute unit (W rows and x rows of a slice, per workgroup), counting
    // whole rounds of one workgroup per CU: 1536 blocks and 64 rows as 768
    // workgroups of 2 cost 3 x (32 + 64) rows, as 384 of 4 2 x (64 + 64), as
    // 256 of 6 1 x (96 + 64) (measured 201, 184 and 166 us for the
    // 64-token drafter layer).
    const int tiles = n_out / 16;
    int fb = 1;
    if (rows >= 12) {
        auto cost = [&](int f) {
            return cdiv(tiles / f * ks, kComputeUnits) * (16 * f + 16 * nbl);
        };
        for (int f : {2, 4, 6})
            if (tiles % f == 0 && (fb == 1 || cost(f) <= cost(fb)))
                fb = f;
    }
    const dim3 grid(tiles / fb, ks);
#define WF_LIN(NBLV, FBV)                                                                 \
    if (nbl == NBLV && fb == FBV) {                                                       \
        linear_partial_bf16<NBLV, FBV><<<grid, block, 0, stream>>>(                       \
            x, w_a, w_b, n_a, zpart, rows, k_in, n_out, cps, t, nullptr);                 \
    } else
    WF_LIN(1, 1) WF_LIN(1, 2) WF_LIN(1, 4) WF_LIN(1, 6)
    WF_LIN(2, 1) WF_LIN(2, 2) WF_LIN(2, 4) WF_LIN(2, 6)
    WF_LIN(3, 1) WF_LIN(3, 2) WF_LIN(3, 4) WF_LIN(3, 6)
    WF_LIN(4, 1) WF_LIN(4, 2) WF_LIN(4, 4) WF_LIN(4, 6)
    { return WF_ERR_UNSUPPORTED; }
#undef WF_LIN
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

wf_status_t launch_linear_swiglu(const uint16_t *x, const uint16_t *w_gate,
                                 const uint16_t *w_up, int inter, int rows, int k_in,
                                 uint16_t *act, hipStream_t stream, bool tiled) {
    const int tiles = 2 * inter / 16;
    const int nbl = cdiv(rows, 16);
    if (rows < 12 || rows > 64 || inter % 16 || k_in % 32 || linear_slices(k_in, 2 * inter) != 1)
        return WF_ERR_UNSUPPORTED;
    // the block count of the split launch's rule, among those whose gate
    // half divides the gate blocks
    auto cost = [&](int f) { return cdiv(tiles / f, kComputeUnits) * (16 * f + 16 * nbl); };
    int fb = 0;
    for (int f : {2, 4, 6})
        if ((inter / 16) % (f / 2) == 0 && (fb == 0 || cost(f) <= cost(fb)))
            fb = f;
    if (fb == 0)
        return WF_ERR_UNSUPPORTED;
    const dim3 grid(tiles / fb, 1);
    const dim3 block(kGemvWaves * kWave);
    const int t = tiled ? 1 : 0;
    const int cps = k_in / 32;
#define WF_SWI(NBLV, FBV)                                                                 \
    if (nbl == NBLV && fb == FBV) {                                                       \
        linear_partial_bf16<NBLV, FBV, true><<<grid, block, 0, stream>>>(                 \
            x, w_gate, w_up, inter, nullptr, rows, k_in, 2 * inter, cps, t, act);         \
    } else
    WF_SWI(1, 2) WF_SWI(1, 4) WF_SWI(1, 6) WF_SWI(2, 2) WF_SWI(2, 4) WF_SWI(2, 6)
    WF_SWI(3, 2) WF_SWI(3, 4) WF_SWI(3, 6) WF_SWI(4, 2) WF_SWI(4, 4) WF_SWI(4, 6)
    { return WF_ERR_UNSUPPORTED; }
#undef WF_SWI
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace wf
