// router.hip -- the neural routing policy (Sec. 3.3.2 of the WhiFlash paper;
// its architecture is given in the appendix on the neural router): a
// two-layer MLP regressor on the target model's final hidden state predicts
// the acceptance-length gain of the autoregressive drafter over the
// diffusion drafter, and the next round uses the autoregressive drafter iff
// that gain exceeds tau_neural:
//
//   delta[r] = w2 . GELU(W1 h[r] + b1) + b2,   GELU(x) = 0.5 x (1 + erf(x/sqrt 2))
//
// (W1 [m][d] with m = d/8; dropout is off at inference).  delta is formed
// for every verify row -- reading W1 once costs the same for all rows -- and
// the route is taken at the row a device-side index names (the final
// accepted position from the acceptance call), so no host round trip sits
// between acceptance and routing.
//
// Kernel 1: workgroup g owns hidden units 16g .. 16g+15.  bf16: the 8 waves
// split the input dimension into interleaved 32-wide chunks, z = W1 h runs
// on 16x16x32 MFMA (A = 16 units x 32 dims, B = 32 dims x 16 rows), the
// waves' partial sums meet in LDS in wave order, and each row's 16 units
// are folded into one partial of delta in unit order.  fp32: one thread per
// (unit, row) and a plain dot product; one partial per unit.
// Kernel 2 (one workgroup): delta[r] = b2 + the partials in order, then the
// route.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kRouterWaves = 8;
constexpr int kRouterBatch = 8;       // 32-wide chunks per wave per load batch
constexpr int kRouterMaxGamma = 64;

__device__ __forceinline__ float gelu_exact(float x) {
    return 0.5f * x * (1.f + erff(x * 0.70710678118654752f));
}

template <int NBL>
__global__ __launch_bounds__(kRouterWaves * kWave) void router_hidden_bf16(
    const uint16_t *__restrict__ h, const uint16_t *__restrict__ w1,
    const uint16_t *__restrict__ b1, const uint16_t *__restrict__ w2,
    float *__restrict__ parts, int gamma, int d) {
    __shared__ float zs[kRouterWaves][16][16 * NBL + 1];
    const int u0 = 16 * blockIdx.x;
    const int wave = wave_id();
    const int lane = threadIdx.x % kWave;
    const int m16 = lane & 15;
    const int c4 = lane >> 4;
    const int nchunks = d / 32;

    const uint16_t *wp = w1 + (size_t)(u0 + m16) * d + c4 * 8;
    // rows past gamma read row gamma-1: their columns are never used
    const uint16_t *hp[NBL];
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
        hp[nb] = h + (size_t)min(16 * nb + m16, gamma - 1) * d + c4 * 8;

    f32x4 acc[NBL];
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
        acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int cb = wave; cb < nchunks; cb += kRouterWaves * kRouterBatch) {
        bf16x8 wr[kRouterBatch], hr[kRouterBatch][NBL];
#pragma unroll
        for (int u = 0; u < kRouterBatch; ++u) {
            const int c = cb + kRouterWaves * u;
            if (c < nchunks) {
                wr[u] = load_bf16x8(wp + c * 32);
#pragma unroll
                for (int nb = 0; nb < NBL; ++nb)
                    hr[u][nb] = load_bf16x8(hp[nb] + c * 32);
            }
        }
#pragma unroll
        for (int u = 0; u < kRouterBatch; ++u) {
            if (cb + kRouterWaves * u < nchunks) {
#pragma unroll
                for (int nb = 0; nb < NBL; ++nb)
                    acc[nb] = mfma16x16x32(wr[u], hr[u][nb], acc[nb]);
            }
        }
    }
    // lane (m16, c4) holds z of units 4*c4 + i for row 16*nb + m16
#pragma unroll
    for (int nb = 0; nb < NBL; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            zs[wave][4 * c4 + i][16 * nb + m16] = acc[nb][i];
    __syncthreads();
    const int r = threadIdx.x;
    if (r < gamma) {
        float p = 0.f;
        for (int u = 0; u < 16; ++u) {
            float z = zs[0][u][r];
#pragma unroll
            for (int ww = 1; ww < kRouterWaves; ++ww)
                z += zs[ww][u][r];
            z += bf16_to_f32(b1[u0 + u]);
            p = fmaf(bf16_to_f32(w2[u0 + u]), gelu_exact(z), p);
        }
        parts[(size_t)blockIdx.x * gamma + r] = p;
    }
}

__global__ __launch_bounds__(256) void router_hidden_f32(
    const float *__restrict__ h, const float *__restrict__ w1,
    const float *__restrict__ b1, const float *__restrict__ w2,
    float *__restrict__ parts, int gamma, int d, int m) {
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)m * gamma)
        return;
    const int u = (int)(idx / gamma), r = (int)(idx % gamma);
    const float *wr = w1 + (size_t)u * d;
    const float *hr = h + (size_t)r * d;
    float z = b1[u];
    for (int k = 0; k < d; ++k)
        z = fmaf(wr[k], hr[k], z);
    parts[(size_t)u * gamma + r] = w2[u] * gelu_exact(z);
}

template <bool BF16>
__global__ __launch_bounds__(kRouterMaxGamma) void router_finish(
    const float *__restrict__ parts, const void *b2, const int32_t *row,
    float tau, float *delta_out, int32_t *route_out, int gamma, int n_parts) {
    __shared__ float ds[kRouterMaxGamma];
    const int r = threadIdx.x;
    if (r < gamma) {
        float s = BF16 ? bf16_to_f32(*static_cast<const uint16_t *>(b2))
                       : *static_cast<const float *>(b2);
        for (int g = 0; g < n_parts; ++g)
            s += parts[(size_t)g * gamma + r];
        delta_out[r] = s;
        ds[r] = s;
    }
    __syncthreads();
    if (r == 0) {
        const int sel = min(max(*row, 0), gamma - 1);
        *route_out = (ds[sel] > tau) ? 1 : 0;
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

size_t router_workspace_bytes(int gamma, int m) {
    return kCounterBytes + (size_t)gamma * m * sizeof(float);
}

wf_status_t launch_router(wf_dtype_t dt, const void *h, const void *w1,
                          const void *b1, const void *w2, const void *b2,
                          const int32_t *row, int gamma, int d, int m, float tau,
                          float *delta_out, int32_t *route_out, void *workspace,
                          hipStream_t stream) {
    float *parts = reinterpret_cast<float *>(static_cast<char *>(workspace) + kCounterBytes);
    int n_parts;
    if (dt == WF_BF16) {
        n_parts = m / 16;
        const auto *hh = static_cast<const uint16_t *>(h);
        const auto *ww1 = static_cast<const uint16_t *>(w1);
        const auto *bb1 = static_cast<const uint16_t *>(b1);
        const auto *ww2 = static_cast<const uint16_t *>(w2);
        switch (cdiv(gamma, 16)) {
        case 1: router_hidden_bf16<1><<<n_parts, kRouterWaves * kWave, 0, stream>>>(hh, ww1, bb1, ww2, parts, gamma, d); break;
        case 2: router_hidden_bf16<2><<<n_parts, kRouterWaves * kWave, 0, stream>>>(hh, ww1, bb1, ww2, parts, gamma, d); break;
        case 3: router_hidden_bf16<3><<<n_parts, kRouterWaves * kWave, 0, stream>>>(hh, ww1, bb1, ww2, parts, gamma, d); break;
        default: router_hidden_bf16<4><<<n_parts, kRouterWaves * kWave, 0, stream>>>(hh, ww1, bb1, ww2, parts, gamma, d); break;
        }
        router_finish<true><<<1, kRouterMaxGamma, 0, stream>>>(parts, b2, row, tau, delta_out,
                                                               route_out, gamma, n_parts);
    } else {
        n_parts = m;
        const long long threads = (long long)m * gamma;
        router_hidden_f32<<<(unsigned)((threads + 255) / 256), 256, 0, stream>>>(
            static_cast<const float *>(h), static_cast<const float *>(w1),
            static_cast<const float *>(b1), static_cast<const float *>(w2), parts, gamma,
            d, m);
        router_finish<false><<<1, kRouterMaxGamma, 0, stream>>>(parts, b2, row, tau, delta_out,
                                                                route_out, gamma, n_parts);
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
