// tile.hip -- the tiled bf16 weight layout.  A weight W [rows][cols] is cut
// into 16-row x 32-column tiles of 1 KB, each laid out exactly as one wave's
// MFMA operand load wants it (lane 16*q + r: row r, columns 8q .. 8q+7), so
// a kernel that walks W reads one contiguous 1 KB per wave load.  The copy
// runs once per weight; each thread moves one 16-byte granule.
#include "wf_api_internal.h"
#include "wf_device.h"

namespace wf {

namespace {

__global__ __launch_bounds__(256) void tile_weights_bf16(const uint16_t *__restrict__ w,
                                                         uint16_t *__restrict__ out, int rows,
                                                         int cols, long long granules) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= granules)
        return;
    const int kch = cols / 32;
    const long long tile = g / 64;
    const int lane = (int)(g % 64);
    const int rb = (int)(tile / kch), c = (int)(tile % kch);
    const int row = 16 * rb + (lane & 15);
    const int col = 32 * c + 8 * (lane >> 4);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < rows)
        v = *reinterpret_cast<const u32x4 *>(w + (size_t)row * cols + col);
    *reinterpret_cast<u32x4 *>(out + (size_t)g * 8) = v;
}

}  // namespace

size_t tiled_weight_bytes(int rows, int cols) {
    return (size_t)((rows + 15) / 16) * 16 * (size_t)cols * 2;
}

wf_status_t launch_tile_weights(const void *w, int rows, int cols, void *tiled,
                                hipStream_t stream) {
    const long long granules = (long long)((rows + 15) / 16) * (cols / 32) * 64;
    tile_weights_bf16<<<(unsigned)((granules + 255) / 256), 256, 0, stream>>>(
        static_cast<const uint16_t *>(w), static_cast<uint16_t *>(tiled), rows, cols, granules);
    return hipGetLastError() == hipSuccess ? WF_OK : WF_ERR_HIP;
}

}  // namespace wf
