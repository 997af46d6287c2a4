// noalloc.hip -- wf_verify_attn_noalloc: verify attention without a
// caller-provided workspace, for callers that cannot allocate (code under
// HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
//
// The split partials live in `scratch`, a file-scope device array of
// WF_NOALLOC_SCRATCH_BYTES that every GPU the library runs on holds until
// the process ends.  Its layout is that of a verify-attention workspace (the
// zero block, then the partials), so the call runs exactly the kernels of
// wf_verify_attn.  Host code never passes the array's name to a kernel: on
// the first call on a device, with that device current, the device address
// is looked up once with hipGetSymbolAddress and kept per device, and the
// zero block is cleared by a fill kernel on the caller's stream (the kernels
// leave it at zero after every call).  Nothing here allocates.  All calls on
// one GPU share its array: calls that overlap in time on one GPU race.
#include <mutex>

#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {
namespace {

constexpr size_t kScratchBytes = WF_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static_assert(kScratchBytes > kCounterBytes && kScratchBytes % 256 == 0,
              "scratch holds the zero block and the partials");

__device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` per device, found once with that device
// current; null until then.
void *g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

__global__ __launch_bounds__(256) void zero_fill_u32x4(u32x4 *p, size_t n) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = z;
}

// Scratch of the current device, cleared on first use (on `stream`).
wf_status_t device_scratch(hipStream_t stream, void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return WF_ERR_HIP;
    if (dev >= kMaxDevices)
        return WF_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return WF_ERR_HIP;
        zero_fill_u32x4<<<256, 256, 0, stream>>>(static_cast<u32x4 *>(ptr),
                                                 kCounterBytes / sizeof(u32x4));
        if (hipGetLastError() != hipSuccess)
            return WF_ERR_HIP;
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return WF_OK;
}

}  // namespace
}  // namespace wf

extern "C" wf_status_t wf_verify_attn_noalloc(wf_dtype_t dt, const void *q,
                                              const void *k_cache, const void *v_cache,
                                              void *out, int32_t gamma, int32_t ctx_len,
                                              int32_t cap, int32_t n_q_heads,
                                              int32_t n_kv_heads, int32_t head_dim,
                                              float softmax_scale, int32_t num_splits,
                                              void *stream) {
    wf::AttnPlan p{};
    wf_status_t st = wf::validate_verify_attn(dt, q, k_cache, v_cache, out, gamma, ctx_len,
                                              cap, n_q_heads, n_kv_heads, head_dim,
                                              softmax_scale, num_splits, &p);
    if (st != WF_OK)
        return st;
    if (wf::attn_workspace_bytes(p, gamma, n_q_heads, head_dim) > wf::kScratchBytes)
        return WF_ERR_WORKSPACE;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    void *ws = nullptr;
    st = wf::device_scratch(s, &ws);
    if (st != WF_OK)
        return st;
    return wf::launch_attn(dt, q, k_cache, v_cache, out, gamma, ctx_len, cap, n_q_heads,
                           n_kv_heads, head_dim, softmax_scale, nullptr, p, ws, s);
}
