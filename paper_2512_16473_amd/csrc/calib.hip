// Measurement yardstick: a plain contiguous HBM read with the access pattern of the
// decode weight kernels (16-byte nontemporal loads, 64 lanes covering 1 KiB per load).
// It computes nothing of the method; its rate on a device is the practical ceiling the
// weight-streaming kernels are compared with, next to the 8 TB/s specification.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kStreamBlock = 256;
constexpr uint32_t kStreamMagic = 0x9E3779B9u;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t fold(const u32x4_t v) { return v.x ^ v.y ^ v.z ^ v.w; }

// Grid-stride read of n 16-byte words, one load per lane per step: at any moment the
// resident waves read one narrow, contiguous window of memory. Of the patterns measured
// on gfx950 (several loads in flight per lane, spaced a grid apart or within a lane's
// own run of KiBs), this plain one with eight 256-thread work groups per compute unit
// read fastest at every size from 0.4 to 8 GiB. Each lane folds what it read; a lane
// whose fold equals kStreamMagic writes it to sink[0], so the loads cannot be removed
// and the kernel writes nothing in practice.
__global__ __launch_bounds__(kStreamBlock) void k_read_stream(const u32x4_t *p, size_t n, uint32_t *sink)
{
    const size_t stride = (size_t)gridDim.x * kStreamBlock;
    uint32_t acc = 0;
    for (size_t i = (size_t)blockIdx.x * kStreamBlock + threadIdx.x; i < n; i += stride)
        acc ^= fold(__builtin_nontemporal_load(p + i));
    if (acc == kStreamMagic) sink[0] = acc;
}

}  // namespace
}  // namespace moe

extern "C" {

int moe_read_stream(const void *buf, size_t bytes, uint32_t *sink, int grid, void *stream)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(grid >= 0, "moe_read_stream: grid=%d < 0", grid);
    MOE_REQUIRE(bytes % 16 == 0, "moe_read_stream: bytes=%zu is not a multiple of 16", bytes);
    if (bytes == 0) return MOE_OK;
    MOE_REQUIRE(buf && sink, "moe_read_stream: null pointer");
    MOE_REQUIRE(moe::aligned16(buf) && ((uintptr_t)sink & 3u) == 0,
                "moe_read_stream: buf must be 16-byte and sink 4-byte aligned");
    if (grid == 0) grid = 8 * moe::device_cu_count();
    (void)hipGetLastError();
    hipLaunchKernelGGL(moe::k_read_stream, dim3(grid), dim3(moe::kStreamBlock), 0, (hipStream_t)stream,
                       static_cast<const moe::u32x4_t *>(buf), bytes / 16, sink);
    MOE_HIP(hipGetLastError());
    return MOE_OK;
    MOE_GUARD_END
}

}  // extern "C"
