// compact.hip -- KV-cache compaction after tree verification.  Once the
// target has accepted a root path of the draft tree (autoregressive drafters
// propose trees, Sec. 3.1, verified in one parallel pass, Sec. 3.2), the K/V
// rows of the path's nodes move to consecutive rows right after the cached
// prefix, so the cache holds the committed sequence in order again and the
// next round appends after it:
//
//   K[g][ctx_len + t] <- K[g][ctx_len + path[t]],  t = 0..n   (same for V)
//
// n = accept[0] is read on the device, so the call can follow the acceptance
// on the same stream without a host round trip.  One launch covers every
// layer of a cache laid out with a fixed stride between layers.  Sources and
// destinations overlap, so each workgroup (layer, KV head, K or V) stages its
// rows in LDS before writing any of them.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

constexpr int kMaxPathRows = 64;
constexpr int kMaxRowU4 = 32;          // 16-byte units per row: 128 x fp32

__global__ __launch_bounds__(256) void compact_rows(char *k_cache, char *v_cache,
                                                    const int32_t *accept,
                                                    const int32_t *path, int gamma,
                                                    int ctx_len, int cap, int row_u4,
                                                    size_t layer_bytes) {
    __shared__ u32x4 stage[kMaxPathRows * kMaxRowU4];
    __shared__ int src_row[kMaxPathRows];
    const int g = blockIdx.x;
    char *base = (blockIdx.y ? v_cache : k_cache) + (size_t)blockIdx.z * layer_bytes +
                 (size_t)g * cap * row_u4 * 16;
    const int n = min(max(accept[0], 0), gamma - 1);
    // the node at depth t has index >= t; anything else is left in place
    if ((int)threadIdx.x <= n) {
        const int t = threadIdx.x;
        const int p = path[t];
        src_row[t] = (p >= t && p < gamma) ? p : -1;
    }
    __syncthreads();
    const int total = (n + 1) * row_u4;
    for (int idx = threadIdx.x; idx < total; idx += blockDim.x) {
        const int t = idx / row_u4, u = idx % row_u4;
        const int s = src_row[t];
        if (s >= 0)
            stage[idx] = reinterpret_cast<const u32x4 *>(base + (size_t)(ctx_len + s) * row_u4 * 16)[u];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < total; idx += blockDim.x) {
        const int t = idx / row_u4, u = idx % row_u4;
        const int s = src_row[t];
        if (s >= 0 && s != t)
            reinterpret_cast<u32x4 *>(base + (size_t)(ctx_len + t) * row_u4 * 16)[u] = stage[idx];
    }
}

}  // namespace

wf_status_t launch_compact(wf_dtype_t dt, void *k_cache, void *v_cache,
                           const int32_t *accept, const int32_t *path,
                           int gamma, int ctx_len, int cap, int n_kv_heads,
                           int head_dim, int n_layers, size_t layer_stride,
                           hipStream_t stream) {
    const int elem = dt == WF_BF16 ? 2 : 4;
    const int row_bytes = head_dim * elem;
    const int row_u4 = row_bytes / 16;
    if (gamma > kMaxPathRows || row_u4 > kMaxRowU4 || row_bytes % 16 != 0)
        return WF_ERR_UNSUPPORTED;
    compact_rows<<<dim3(n_kv_heads, 2, n_layers), 256, 0, stream>>>(
        static_cast<char *>(k_cache), static_cast<char *>(v_cache), accept, path,
        gamma, ctx_len, cap, row_u4, layer_stride * elem);
    if (hipGetLastError() != hipSuccess)
        return WF_ERR_HIP;
    return WF_OK;
}

}  // namespace wf
