// probe.hip -- streaming-read ceiling of the device memory (measurement
// support for the benchmark, not a step of the method).
//
// The workgroups stride through the buffer together: in each round
// workgroup b reads piece b of the round (16-byte loads, 4 or 8 in flight
// per thread: 16 or 32 KB per workgroup), so the whole grid reads one
// contiguous stretch at a time -- on MI355X the fastest of the plain read patterns measured (grid
// stride, 512 workgroups: 6.3 TB/s; one contiguous share per workgroup:
// 5.9-6.1 TB/s).  Each thread folds what it read into an XOR that it
// writes to the sink, so the loads cannot be dropped.  The bytes read over
// the kernel's duration give the rate a plain read stream reaches on the
// part; with a buffer larger than the 256 MB last-level cache, that rate is
// the HBM's.  A series of such reads over buffers that together exceed
// that cache, launched back to back, gives the time a plain read of a given
// size takes on its own -- the floor for any kernel that must move as many
// bytes (a short read pays the launch, the first-byte latency and the
// drain as well as the streaming).
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {
namespace {

constexpr int kProbeThreads = 256;

// D 16-byte loads in flight per thread; a round of the grid reads
// workgroups * 256 * D * 16 bytes.
template <int D>
__global__ __launch_bounds__(kProbeThreads) void read_probe(const u32x4 *__restrict__ src,
                                                            size_t n16,
                                                            u32x4 *__restrict__ sink) {
    constexpr size_t kPiece = (size_t)kProbeThreads * D;   // 16-byte units
    const size_t stride = (size_t)gridDim.x * kPiece;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (size_t i = (size_t)blockIdx.x * kPiece + threadIdx.x; i < n16; i += stride) {
        u32x4 v[D];
#pragma unroll
        for (int u = 0; u < D; ++u) {
            const size_t j = i + (size_t)u * kProbeThreads;
            v[u] = j < n16 ? src[j] : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < D; ++u)
            acc ^= v[u];
    }
    sink[(size_t)blockIdx.x * kProbeThreads + threadIdx.x] = acc;
}

wf_status_t launch_one(const void *src, size_t bytes, void *sink, int workgroups, int depth,
                       hipStream_t stream) {
    const auto *s = static_cast<const u32x4 *>(src);
    auto *k = static_cast<u32x4 *>(sink);
    if (depth == 4)
        read_probe<4><<<workgroups, kProbeThreads, 0, stream>>>(s, bytes / 16, k);
    else
        read_probe<8><<<workgroups, kProbeThreads, 0, stream>>>(s, bytes / 16, k);
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace

wf_status_t launch_read_probe(const void *src, size_t bytes, void *sink, int workgroups,
                              hipStream_t stream) {
    return launch_one(src, bytes, sink, workgroups, 8, stream);
}

// reps rounds over n_bufs buffers base + i * stride, launched back to back
// from this loop (a caller's own launch rate would limit short reads).
wf_status_t launch_read_probe_series(const void *base, size_t bytes, size_t stride, int n_bufs,
                                     int reps, void *sink, int workgroups, int depth,
                                     hipStream_t stream) {
    for (int r = 0; r < reps; ++r)
        for (int i = 0; i < n_bufs; ++i) {
            const wf_status_t st = launch_one(static_cast<const char *>(base) + (size_t)i * stride,
                                              bytes, sink, workgroups, depth, stream);
            if (st != WF_OK)
                return st;
        }
    return WF_OK;
}

}  // namespace wf
