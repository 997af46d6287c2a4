// probe.hip -- streaming-read ceiling of the device memory (measurement
// support for the benchmark, not a step of the method).
//
// The workgroups stride through the buffer together: in each round
// workgroup b reads the 32 KB piece b of the round (16-byte loads, 8 in
// flight per thread), so the whole grid reads one contiguous stretch at a
// time -- on MI355X the fastest of the plain read patterns measured (grid
// stride, 512 workgroups: 6.3 TB/s; one contiguous share per workgroup:
// 5.9-6.1 TB/s).  Each thread folds what it read into an XOR that it
// writes to the sink, so the loads cannot be dropped.  The bytes read over
// the kernel's duration give the rate a plain read stream reaches on the
// part; with a buffer larger than the 256 MB last-level cache, that rate is
// the HBM's.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeDepth = 8;

__global__ __launch_bounds__(kProbeThreads) void read_probe(const u32x4 *__restrict__ src,
                                                            size_t n16,
                                                            u32x4 *__restrict__ sink) {
    constexpr size_t kPiece = (size_t)kProbeThreads * kProbeDepth;   // 16-byte units
    const size_t stride = (size_t)gridDim.x * kPiece;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (size_t i = (size_t)blockIdx.x * kPiece + threadIdx.x; i < n16; i += stride) {
        u32x4 v[kProbeDepth];
#pragma unroll
        for (int u = 0; u < kProbeDepth; ++u) {
            const size_t j = i + (size_t)u * kProbeThreads;
            v[u] = j < n16 ? src[j] : u32x4{0u, 0u, 0u, 0u};
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
    read_probe<<<workgroups, kProbeThreads, 0, stream>>>(static_cast<const u32x4 *>(src),
                                                         bytes / 16, static_cast<u32x4 *>(sink));
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace wf
