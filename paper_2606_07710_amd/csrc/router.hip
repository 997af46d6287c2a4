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
// Kernel 1 forms z = W1 h without the bias.  bf16: the skinny linear layer
// of gemv.hip, split over the input dimension so the few hundred hidden
// units still spread over the chip (one fp32 partial per slice).  fp32: one
// thread per (unit, row), a plain dot product over all of d (one slice).
// Kernel 2 (one workgroup per 16 hidden units): z = b1 + the slices in
// order, GELU, times w2, and the 16 units of each row summed in unit order.
// Kernel 3 (one workgroup): delta = b2 + the unit groups in order, then the
// route.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kRouterMaxGamma = 64;

__device__ __forceinline__ float gelu_exact(float x) {
    return 0.5f * x * (1.f + erff(x * 0.70710678118654752f));
}

__global__ __launch_bounds__(256) void router_hidden_f32(
    const float *__restrict__ h, const float *__restrict__ w1,
    float *__restrict__ zpart, int gamma, int d, int m) {
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)m * gamma)
        return;
    const int u = (int)(idx / gamma), r = (int)(idx % gamma);
    const float *wr = w1 + (size_t)u * d;
    const float *hr = h + (size_t)r * d;
    float z = 0.f;
    for (int k = 0; k < d; ++k)
        z = fmaf(wr[k], hr[k], z);
    zpart[(size_t)u * gamma + r] = z;
}

template <bool BF16>
__device__ __forceinline__ float ld_param(const void *p, int i) {
    return BF16 ? bf16_to_f32(static_cast<const uint16_t *>(p)[i])
                : static_cast<const float *>(p)[i];
}

// part [cdiv(m,16)][gamma]: w2 . GELU(z) over the group's 16 units
template <bool BF16>
__global__ __launch_bounds__(256) void router_units(const float *__restrict__ zpart,
                                                    const void *b1, const void *w2,
                                                    float *__restrict__ part, int gamma,
                                                    int m, int n_slices) {
    __shared__ float cs[16][kRouterMaxGamma + 1];
    const int u0 = 16 * blockIdx.x;
    const int u = threadIdx.x / 16;
    const int rr = threadIdx.x % 16;
    const bool unit_ok = u0 + u < m;
    const float bias = unit_ok ? ld_param<BF16>(b1, u0 + u) : 0.f;
    const float w2u = unit_ok ? ld_param<BF16>(w2, u0 + u) : 0.f;
#pragma unroll
    for (int q = 0; q < kRouterMaxGamma / 16; ++q) {
        const int r = rr + 16 * q;
        if (r < gamma) {
            float zs[kLinearMaxSlices];
#pragma unroll
            for (int k = 0; k < kLinearMaxSlices; ++k)
                zs[k] = (unit_ok && k < n_slices)
                            ? zpart[((size_t)k * m + u0 + u) * gamma + r] : 0.f;
            float z = bias;
#pragma unroll
            for (int k = 0; k < kLinearMaxSlices; ++k)
                if (k < n_slices)
                    z += zs[k];
            cs[u][r] = unit_ok ? w2u * gelu_exact(z) : 0.f;
        }
    }
    __syncthreads();
    const int r = threadIdx.x;
    if (r < gamma) {
        float p = 0.f;
#pragma unroll
        for (int uu = 0; uu < 16; ++uu)
            p += cs[uu][r];
        part[(size_t)blockIdx.x * gamma + r] = p;
    }
}

template <bool BF16>
__global__ __launch_bounds__(kRouterMaxGamma) void router_finish(
    const float *__restrict__ part, const void *b2, const int32_t *row, float tau,
    float *delta_out, int32_t *route_out, int gamma, int n_groups) {
    constexpr int kBatch = 16;
    __shared__ float ds[kRouterMaxGamma];
    const int r = threadIdx.x;
    if (r < gamma) {
        float s = ld_param<BF16>(b2, 0);
        for (int g0 = 0; g0 < n_groups; g0 += kBatch) {
            float v[kBatch];
#pragma unroll
            for (int b = 0; b < kBatch; ++b)
                v[b] = (g0 + b < n_groups) ? part[(size_t)(g0 + b) * gamma + r] : 0.f;
#pragma unroll
            for (int b = 0; b < kBatch; ++b)
                if (g0 + b < n_groups)
                    s += v[b];
        }
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

size_t router_workspace_bytes(wf_dtype_t dt, int gamma, int d, int m) {
    const int ks = dt == WF_BF16 ? linear_slices(d, m) : 1;
    return kCounterBytes + ((size_t)ks * m + (size_t)cdiv(m, 16)) * gamma * sizeof(float);
}

wf_status_t launch_router(wf_dtype_t dt, const void *h, const void *w1,
                          const void *b1, const void *w2, const void *b2,
                          const int32_t *row, int gamma, int d, int m, float tau,
                          float *delta_out, int32_t *route_out, void *workspace,
                          hipStream_t stream) {
    float *zpart = reinterpret_cast<float *>(static_cast<char *>(workspace) + kCounterBytes);
    const int groups = cdiv(m, 16);
    int ks = 1;
    if (dt == WF_BF16) {
        ks = linear_slices(d, m);
        const wf_status_t st = launch_linear_partial(static_cast<const uint16_t *>(h),
                                                     static_cast<const uint16_t *>(w1),
                                                     nullptr, m, 0, gamma, d, zpart, stream);
        if (st != WF_OK)
            return st;
    } else {
        const long long threads = (long long)m * gamma;
        router_hidden_f32<<<(unsigned)((threads + 255) / 256), 256, 0, stream>>>(
            static_cast<const float *>(h), static_cast<const float *>(w1), zpart, gamma, d, m);
    }
    float *part = zpart + (size_t)ks * m * gamma;
    if (dt == WF_BF16) {
        router_units<true><<<groups, 256, 0, stream>>>(zpart, b1, w2, part, gamma, m, ks);
        router_finish<true><<<1, kRouterMaxGamma, 0, stream>>>(part, b2, row, tau, delta_out,
                                                               route_out, gamma, groups);
    } else {
        router_units<false><<<groups, 256, 0, stream>>>(zpart, b1, w2, part, gamma, m, ks);
        router_finish<false><<<1, kRouterMaxGamma, 0, stream>>>(part, b2, row, tau, delta_out,
                                                                route_out, gamma, groups);
    }
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
