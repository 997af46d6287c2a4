// probe.hip -- streaming-read ceiling of the device memory (measurement
// support for the benchmark, not a step of the method).
//
// Each of `workgroups` workgroups reads one contiguous share of the buffer
// with 16-byte loads, kProbeDepth of them in flight per thread, and folds
// them into an XOR that it writes to the sink (so the loads cannot be
// dropped).  The bytes read over the kernel's duration give the rate a
// plain read stream reaches on the part; with a buffer larger than the
// 256 MB last-level cache, that rate is the HBM's.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeDepth = 8;

__global__ __launch_bounds__(kProbeThreads) void read_probe(const u32x4 *__restrict__ src,
                                                            size_t n16, size_t per_wg,
                                                            u32x4 *__restrict__ sink) {
    const size_t begin = (size_t)blockIdx.x * per_wg;
    const size_t end = begin + per_wg < n16 ? begin + per_wg : n16;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (size_t i = begin + threadIdx.x; i < end; i += (size_t)kProbeThreads * kProbeDepth) {
        u32x4 v[kProbeDepth];
#pragma unroll
        for (int u = 0; u < kProbeDepth; ++u) {
            const size_t j = i + (size_t)u * kProbeThreads;
            v[u] = j < end ? src[j] : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kProbeDepth; ++u)
            acc ^= v[u];
    }
    sink[(size_t)blockIdx.x * kProbeThreads + threadIdx.x] = acc;
}

}  // namespace

wf_status_t launch_read_probe(const void *src, size_t bytes, void *sink, int workgroups,
                              hipStream_t stream) {
    const size_t n16 = bytes / 16;
    const size_t per_wg = (n16 + workgroups - 1) / workgroups;
    read_probe<<<workgroups, kProbeThreads, 0, stream>>>(static_cast<const u32x4 *>(src), n16,
                                                         per_wg, static_cast<u32x4 *>(sink));
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace wf
