// Device helpers of the weight-streaming GEMV kernels: bf16 unpacking, nontemporal
// 16-byte loads, wave-wide sums and 8-wide dot products (HIP device code only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {
namespace stream_ops {

constexpr int kWave = 64;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

typedef const __attribute__((address_space(1))) u32x4_t global_u32x4_t;

// 16-byte load marked nontemporal (streamed weights are read exactly once), from the
// global address space: the slab pointers come through LDS tables, and without the cast
// the compiler emits flat loads, which also count against the LDS wait counter, so every
// wait for an LDS read would wait for the weight loads in flight as well.
__device__ __forceinline__ uint4 stream_load(const uint4 *p)
{
    const u32x4_t v = __builtin_nontemporal_load((global_u32x4_t *)(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// acc += dot(8 bf16 weights, 8 fp32 activations)
__device__ __forceinline__ float dot8(const uint4 w, const float *a, float acc)
{
    acc = fmaf(bf_lo(w.x), a[0], acc);
    acc = fmaf(bf_hi(w.x), a[1], acc);
    acc = fmaf(bf_lo(w.y), a[2], acc);
    acc = fmaf(bf_hi(w.y), a[3], acc);
    acc = fmaf(bf_lo(w.z), a[4], acc);
    acc = fmaf(bf_hi(w.z), a[5], acc);
    acc = fmaf(bf_lo(w.w), a[6], acc);
    acc = fmaf(bf_hi(w.w), a[7], acc);
    return acc;
}

__device__ __forceinline__ void load8(const float *src, float *dst)
{
    const float4 v0 = reinterpret_cast<const float4 *>(src)[0];
    const float4 v1 = reinterpret_cast<const float4 *>(src)[1];
    dst[0] = v0.x; dst[1] = v0.y; dst[2] = v0.z; dst[3] = v0.w;
    dst[4] = v1.x; dst[5] = v1.y; dst[6] = v1.z; dst[7] = v1.w;
}


}  // namespace stream_ops
}  // namespace moe
