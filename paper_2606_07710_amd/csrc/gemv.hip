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

template <int NBL>
__global__ __launch_bounds__(kGemvWaves * kWave) void linear_partial_bf16(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ w_a,
    const uint16_t *__restrict__ w_b, int n_a, float *__restrict__ zpart, int rows,
    int k_in, int n_out, int chunks_per_slice, int tiled) {
    __shared__ float zs[kGemvWaves][16][16 * NBL + 1];
    const int f0 = 16 * blockIdx.x;
    const int ks = blockIdx.y;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;
    const int c_begin = ks * chunks_per_slice;
    const int n_c = max(0, min(chunks_per_slice, k_in / 32 - c_begin));

    // W operand of chunk c: row-major, 16 bytes of row f0 + m16 per lane;
    // tiled, the 1 KB tile of the 16-feature block (n_a % 16 == 0, so a
    // block never straddles the two matrices)
    const uint16_t *wp;
    int wstep;
    if (tiled) {
        const int blk = f0 < n_a ? f0 / 16 : (f0 - n_a) / 16;
        wp = (f0 < n_a ? w_a : w_b) + ((size_t)blk * (k_in / 32) + c_begin) * 512 + lane * 8;
        wstep = 512;
    } else {
        const int f = f0 + m16;
        const uint16_t *wrow = f < n_a ? w_a + (size_t)f * k_in : w_b + (size_t)(f - n_a) * k_in;
        wp = wrow + (size_t)c_begin * 32 + c4 * 8;
        wstep = 32;
    }
    // rows past `rows` read the last row: their columns are never used
    const uint16_t *xp[NBL];
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
        xp[nb] = x + (size_t)min(16 * nb + m16, rows - 1) * k_in + (size_t)c_begin * 32 + c4 * 8;

    f32x4 acc[NBL];
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
        acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int cb = wave; cb < n_c; cb += kGemvWaves * kGemvBatch) {
        bf16x8 wr[kGemvBatch], xr[kGemvBatch][NBL];
#pragma unroll
        for (int u = 0; u < kGemvBatch; ++u) {
            const int c = cb + kGemvWaves * u;
            if (c < n_c) {
                wr[u] = load_bf16x8(wp + (size_t)c * wstep);
#pragma unroll
                for (int nb = 0; nb < NBL; ++nb)
                    xr[u][nb] = load_bf16x8(xp[nb] + c * 32);
            }
        }
#pragma unroll
        for (int u = 0; u < kGemvBatch; ++u) {
            if (cb + kGemvWaves * u < n_c) {
#pragma unroll
                for (int nb = 0; nb < NBL; ++nb)
                    acc[nb] = mfma16x16x32(wr[u], xr[u][nb], acc[nb]);
            }
        }
    }
    // lane (m16, c4) holds features 4*c4 + i of row 16*nb + m16
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            zs[wave][4 * c4 + i][16 * nb + m16] = acc[nb][i];
    __syncthreads();
    for (int idx = threadIdx.x; idx < 16 * rows; idx += blockDim.x) {
        const int u = idx / rows, r = idx % rows;
        float z = zs[0][u][r];
#pragma unroll
        for (int ww = 1; ww < kGemvWaves; ++ww)
            z += zs[ww][u][r];
        zpart[((size_t)ks * n_out + f0 + u) * rows + r] = z;
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

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
    const dim3 grid(n_out / 16, ks);
    const dim3 block(kGemvWaves * kWave);
    switch (cdiv(rows, 16)) {
    case 1: linear_partial_bf16<1><<<grid, block, 0, stream>>>(x, w_a, w_b, n_a, zpart, rows, k_in, n_out, cps, t); break;
    case 2: linear_partial_bf16<2><<<grid, block, 0, stream>>>(x, w_a, w_b, n_a, zpart, rows, k_in, n_out, cps, t); break;
    case 3: linear_partial_bf16<3><<<grid, block, 0, stream>>>(x, w_a, w_b, n_a, zpart, rows, k_in, n_out, cps, t); break;
    default: linear_partial_bf16<4><<<grid, block, 0, stream>>>(x, w_a, w_b, n_a, zpart, rows, k_in, n_out, cps, t); break;
    }
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace wf
