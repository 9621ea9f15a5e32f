// gfx950 kernels of the MoE expert stage: router gating, the hit-expert SwiGLU
// FFN as two weight-streaming GEMV kernels, the split-K reduce + combine.
//
// Batch-1 decode reads every weight of a hit expert exactly once and does two
// flops per weight, so the FFN is bound by HBM bandwidth, not by the matrix cores.
// The kernels therefore stream each bf16 weight row with 16-byte loads per lane
// (a 64-lane wave covers 512 contiguous weights per load), keep the activation
// vector in registers for the whole life of the wave, reduce each row across the
// wave with cross-lane shuffles, and spread the rows of all hit experts evenly
// over every wave of the grid. The down projection splits its reduction (length f)
// into segments of at most kSegMax so the activation slice a wave holds stays in
// registers; the fixed-order sum of the segment partials is fused into the combine.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moe.h"
#include "moe_internal.h"

namespace moe {

namespace {

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;

__device__ __forceinline__ float bf_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

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

// Number of reduction segments and segment length of a down projection with
// reduction length fj (fj a multiple of 8).
__device__ __host__ __forceinline__ int seg_count(int fj) { return (fj + kSegMax - 1) / kSegMax; }
__device__ __host__ __forceinline__ int seg_len(int fj)
{
    const int s = seg_count(fj);
    return (((fj + s - 1) / s) + 7) & ~7;
}

// Per-block table of the active jobs, built by the first threads of the block.
struct JobLds {
    int slot[kMaxJobs];           // slot (routed) / 0 (shared) / -1 inactive
    int f[kMaxJobs];              // rows (gate/up) of the job, 0 if inactive
    int start[kMaxJobs + 1];      // prefix sum of work items per job
    const uint8_t *slab[kMaxJobs];
};

// items_of(j, fj): work items of an active job for the kernel at hand.
template <typename ItemsOf>
__device__ __forceinline__ void build_jobs(const FfnParams &p, JobLds &t, ItemsOf items_of)
{
    const int njobs = p.k + 1;
    if (threadIdx.x < njobs) {
        const int j = threadIdx.x;
        int slot = -1, fj = 0;
        const uint8_t *slab = nullptr;
        if (j < p.k) {
            const int s = p.sel[j];
            if (p.slotmap) slot = (s >= 0 && s < p.n) ? p.slotmap[s] : -1;
            else slot = s;
            if (slot >= p.nslots) slot = -1;
            if (slot >= 0) { fj = p.f; slab = p.pool + (uint64_t)slot * p.slab_stride; }
        } else if (p.shared && p.f_shared > 0) {
            slot = 0; fj = p.f_shared; slab = p.shared;
        }
        t.slot[j] = slot;
        t.f[j] = fj;
        t.slab[j] = slab;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int acc = 0;
        for (int j = 0; j < njobs; ++j) {
            t.start[j] = acc;
            if (t.slot[j] >= 0) acc += items_of(t.f[j]);
        }
        t.start[njobs] = acc;
    }
    __syncthreads();
}

__device__ __forceinline__ int find_job(const JobLds &t, int njobs, int it)
{
    int j = 0;
    while (j + 1 < njobs && t.start[j + 1] <= it) ++j;
    return j;
}

// ---------------------------------------------------------------------------
// Gate/up/SiLU: h_j[i] = SiLU(W1_j[i,:] x) * (W3_j[i,:] x) for every row i of
// every active job. CPL = 16-byte chunks per lane along d (d <= CPL * 512).
// ---------------------------------------------------------------------------
template <int CPL>
__global__ __launch_bounds__(kBlock) void k_gate_up(FfnParams p)
{
    __shared__ JobLds t;
    build_jobs(p, t, [](int fj) { return fj; });
    const int njobs = p.k + 1;
    if (blockIdx.x == 0 && threadIdx.x < njobs) p.jobslot[threadIdx.x] = t.slot[threadIdx.x];

    const int lane = threadIdx.x & (kWave - 1);
    const int nwaves = gridDim.x * kWavesPerBlock;
    const int wid = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int total = t.start[njobs];
    if (wid >= total) return;

    const int d = p.d;
    const int nch = d >> 3;
    float xr[CPL * 8];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const int ch = c * kWave + lane;
        if (ch < nch) load8(p.x + ch * 8, xr + c * 8);
        else
#pragma unroll
            for (int e = 0; e < 8; ++e) xr[c * 8 + e] = 0.f;
    }

    for (int it = wid; it < total; it += nwaves) {
        const int j = find_job(t, njobs, it);
        const int i = it - t.start[j];
        const int fj = t.f[j];
        const uint4 *r1 = reinterpret_cast<const uint4 *>(t.slab[j] + (uint64_t)i * d * 2);
        const uint4 *r3 = reinterpret_cast<const uint4 *>(t.slab[j] + ((uint64_t)fj * d + (uint64_t)i * d) * 2);
        uint4 a[CPL], b[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int ch = c * kWave + lane;
            if (ch < nch) { a[c] = r1[ch]; b[c] = r3[ch]; }
            else { a[c] = make_uint4(0, 0, 0, 0); b[c] = make_uint4(0, 0, 0, 0); }
        }
        float g0 = 0.f, g1 = 0.f, u0 = 0.f, u1 = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; c += 2) {
            g0 = dot8(a[c], xr + c * 8, g0);
            u0 = dot8(b[c], xr + c * 8, u0);
            if (c + 1 < CPL) {
                g1 = dot8(a[c + 1], xr + (c + 1) * 8, g1);
                u1 = dot8(b[c + 1], xr + (c + 1) * 8, u1);
            }
        }
        const float g = wave_sum(g0 + g1);
        const float u = wave_sum(u0 + u1);
        if (lane == 0) p.h[(size_t)j * p.hstride + i] = g / (1.0f + expf(-g)) * u;
    }
}

// ---------------------------------------------------------------------------
// Down: partial[j][s][i] = sum over segment s of W2_j[i, c] h_j[c].
// A work item is (job, segment, block of kRowsPerDownItem output rows); the wave
// holds its h segment in registers and streams the rows.
// ---------------------------------------------------------------------------
constexpr int kCplK = kSegMax / (8 * kWave);   // chunks per lane of one segment

__global__ __launch_bounds__(kBlock) void k_down(FfnParams p)
{
    __shared__ JobLds t;
    const int d = p.d;
    const int nrb = (d + kRowsPerDownItem - 1) / kRowsPerDownItem;
    build_jobs(p, t, [nrb](int fj) { return seg_count(fj) * nrb; });
    const int njobs = p.k + 1;

    const int lane = threadIdx.x & (kWave - 1);
    const int nwaves = gridDim.x * kWavesPerBlock;
    const int wid = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int total = t.start[njobs];

    for (int it = wid; it < total; it += nwaves) {
        const int j = find_job(t, njobs, it);
        const int local = it - t.start[j];
        const int s = local / nrb;
        const int rb = local - s * nrb;
        const int fj = t.f[j];
        const int seg = seg_len(fj);
        const int c0 = s * seg;
        const int len = min(seg, fj - c0);
        const int nch = len >> 3;

        float hr[kCplK * 8];
        const float *hj = p.h + (size_t)j * p.hstride + c0;
#pragma unroll
        for (int c = 0; c < kCplK; ++c) {
            const int ch = c * kWave + lane;
            if (ch < nch) load8(hj + ch * 8, hr + c * 8);
            else
#pragma unroll
                for (int e = 0; e < 8; ++e) hr[c * 8 + e] = 0.f;
        }

        const uint8_t *w2 = t.slab[j] + (uint64_t)2 * fj * d * 2;
        const int i0 = rb * kRowsPerDownItem;
        const int i1 = min(d, i0 + kRowsPerDownItem);
        float *out = p.partial + ((size_t)j * p.smax + s) * d;
        for (int i = i0; i < i1; i += 2) {
            const bool two = (i + 1 < i1);
            const uint4 *ra = reinterpret_cast<const uint4 *>(w2 + ((uint64_t)i * fj + c0) * 2);
            const uint4 *rb2 = reinterpret_cast<const uint4 *>(w2 + ((uint64_t)(two ? i + 1 : i) * fj + c0) * 2);
            uint4 a[kCplK], b[kCplK];
#pragma unroll
            for (int c = 0; c < kCplK; ++c) {
                const int ch = c * kWave + lane;
                if (ch < nch) { a[c] = ra[ch]; b[c] = rb2[ch]; }
                else { a[c] = make_uint4(0, 0, 0, 0); b[c] = make_uint4(0, 0, 0, 0); }
            }
            float s0 = 0.f, s1 = 0.f, q0 = 0.f, q1 = 0.f;
#pragma unroll
            for (int c = 0; c < kCplK; c += 2) {
                s0 = dot8(a[c], hr + c * 8, s0);
                q0 = dot8(b[c], hr + c * 8, q0);
                s1 = dot8(a[c + 1], hr + (c + 1) * 8, s1);
                q1 = dot8(b[c + 1], hr + (c + 1) * 8, q1);
            }
            const float ya = wave_sum(s0 + s1);
            const float yb = wave_sum(q0 + q1);
            if (lane == 0) {
                out[i] = ya;
                if (two) out[i + 1] = yb;
            }
        }
    }
}

// out[i] = sum_j weight_j * sum_s partial[j][s][i] (+ y_extra[i]); fixed order.
__global__ __launch_bounds__(kBlock) void k_reduce(FfnParams p, const float *y_extra, float *out)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= p.d) return;
    float acc = 0.f;
    for (int j = 0; j <= p.k; ++j) {
        if (p.jobslot[j] < 0) continue;
        const int fj = (j < p.k) ? p.f : p.f_shared;
        const int S = seg_count(fj);
        float s = 0.f;
        for (int q = 0; q < S; ++q) s += p.partial[((size_t)j * p.smax + q) * p.d + i];
        const float wj = (j < p.k) ? p.w[j] : 1.0f;
        acc = fmaf(wj, s, acc);
    }
    if (y_extra) acc += y_extra[i];
    out[i] = acc;
}

__global__ __launch_bounds__(kBlock) void k_combine(const float *a, const float *b, const float *c,
                                                    int d, float *out)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= d) return;
    float v = 0.f;
    if (a) v += a[i];
    if (b) v += b[i];
    if (c) v += c[i];
    out[i] = v;
}

// ---------------------------------------------------------------------------
// Router: one block per token. Logits accumulate the exact fp64 products of the
// fp32 inputs; selection and gate weights are computed in fp64 by wave 0.
// NaN logits are ranked as -inf so the selected ids are always valid.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_router(const float *X, const float *Wr, int d, int n,
                                                   int k, int32_t *idx, float *wout)
{
    __shared__ double logit[MOE_MAX_EXPERTS];
    const int t = blockIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const float *x = X + (size_t)t * d;
    for (int e = wv; e < n; e += kWavesPerBlock) {
        const float *w = Wr + (size_t)e * d;
        double acc = 0.0;
        for (int j = lane * 4; j < d; j += kWave * 4) {
            const float4 xv = *reinterpret_cast<const float4 *>(x + j);
            const float4 wvv = *reinterpret_cast<const float4 *>(w + j);
            acc += (double)wvv.x * (double)xv.x;
            acc += (double)wvv.y * (double)xv.y;
            acc += (double)wvv.z * (double)xv.z;
            acc += (double)wvv.w * (double)xv.w;
        }
        acc = wave_sum(acc);
        if (lane == 0) logit[e] = acc;
    }
    __syncthreads();
    if (wv != 0) return;

    constexpr int kPer = MOE_MAX_EXPERTS / kWave;
    double v[kPer];
    bool taken[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int e = q * kWave + lane;
        double l = (e < n) ? logit[e] : -INFINITY;
        if (l != l) l = -INFINITY;
        v[q] = l;
        taken[q] = (e >= n);
    }
    // Lane r keeps the r-th selected (logit, id): order is logit desc, id asc.
    double my_l = -INFINITY;
    int my_i = -1;
    for (int r = 0; r < k; ++r) {
        double bv = -INFINITY;
        int bi = 0x7fffffff;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int e = q * kWave + lane;
            if (!taken[q] && (v[q] > bv || (v[q] == bv && e < bi))) { bv = v[q]; bi = e; }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const double ov = __shfl_xor(bv, o, kWave);
            const int oi = __shfl_xor(bi, o, kWave);
            if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
        }
        if (lane == r) { my_l = bv; my_i = bi; }
#pragma unroll
        for (int q = 0; q < kPer; ++q)
            if (q * kWave + lane == bi) taken[q] = true;
    }
    // w_r = exp(l_r - l_0) / sum_{s<k} exp(l_s - l_0), the softmax restricted to
    // the selected set (equal to p_S / sum p_S).
    const double l0 = __shfl(my_l, 0, kWave);
    const double ex = (lane < k) ? exp(my_l - l0) : 0.0;
    const double z = wave_sum(ex);
    if (lane < k) {
        idx[(size_t)t * k + lane] = my_i;
        wout[(size_t)t * k + lane] = (float)(ex / z);
    }
}

template <int CPL>
hipError_t launch_gate_up_cpl(const FfnParams &p, int blocks, hipStream_t s)
{
    hipLaunchKernelGGL(k_gate_up<CPL>, dim3(blocks), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_gate_up(const FfnParams &p, int blocks, hipStream_t s)
{
    const int cpl = (p.d / 8 + kWave - 1) / kWave;
    switch (cpl) {
#define MOE_CPL_CASE(N) case N: return launch_gate_up_cpl<N>(p, blocks, s);
        MOE_CPL_CASE(1) MOE_CPL_CASE(2) MOE_CPL_CASE(3) MOE_CPL_CASE(4)
        MOE_CPL_CASE(5) MOE_CPL_CASE(6) MOE_CPL_CASE(7) MOE_CPL_CASE(8)
        MOE_CPL_CASE(9) MOE_CPL_CASE(10) MOE_CPL_CASE(11) MOE_CPL_CASE(12)
        MOE_CPL_CASE(13) MOE_CPL_CASE(14) MOE_CPL_CASE(15) MOE_CPL_CASE(16)
#undef MOE_CPL_CASE
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

int device_cu_count()
{
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cached[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cached[dev] = v;
    }
    return cached[dev];
}

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

size_t ffn_workspace_bytes(int max_jobs, int d, int f_max)
{
    (void)max_jobs;
    const size_t hstride = (size_t)((f_max + 63) & ~63);
    const size_t smax = (size_t)seg_count(f_max);
    return align256(sizeof(int32_t) * kMaxJobs) + align256(sizeof(float) * kMaxJobs * hstride) +
           align256(sizeof(float) * kMaxJobs * smax * (size_t)d);
}

void ffn_bind_workspace(FfnParams &p, void *ws, int max_jobs, int d, int f_max)
{
    (void)max_jobs;
    const size_t hstride = (size_t)((f_max + 63) & ~63);
    uint8_t *b = static_cast<uint8_t *>(ws);
    p.jobslot = reinterpret_cast<int32_t *>(b);
    b += align256(sizeof(int32_t) * kMaxJobs);
    p.h = reinterpret_cast<float *>(b);
    p.hstride = (int)hstride;
    b += align256(sizeof(float) * kMaxJobs * hstride);
    p.partial = reinterpret_cast<float *>(b);
    p.smax = seg_count(f_max);
}

hipError_t launch_router(const float *x, const float *wr, int T, int d, int n, int k, int32_t *idx,
                         float *w, hipStream_t s)
{
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_router, dim3(T), dim3(kBlock), 0, s, x, wr, d, n, k, idx, w);
    return hipGetLastError();
}

hipError_t launch_ffn_stream(const FfnParams &p, hipStream_t s, const FfnEvents *ev, hipEvent_t after_down)
{
    const int cus = device_cu_count();
    // Upper bounds of the work (every routed job active); waves with no item exit.
    const int fmax_rows = p.k * p.f + (p.shared ? p.f_shared : 0);
    const int nrb = (p.d + kRowsPerDownItem - 1) / kRowsPerDownItem;
    const int down_items = p.k * seg_count(p.f) * nrb + (p.shared ? seg_count(p.f_shared) * nrb : 0);
    auto blocks_for = [&](int items) {
        int b = (items + kWavesPerBlock - 1) / kWavesPerBlock;
        const int cap = cus * 8;
        if (b > cap) b = cap;
        return b < 1 ? 1 : b;
    };
    hipError_t e;
    if (ev && ev->start && (e = hipEventRecord(ev->start, s)) != hipSuccess) return e;
    if ((e = launch_gate_up(p, blocks_for(fmax_rows), s)) != hipSuccess) return e;
    if (ev && ev->mid && (e = hipEventRecord(ev->mid, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_down, dim3(blocks_for(down_items)), dim3(kBlock), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev && ev->end && (e = hipEventRecord(ev->end, s)) != hipSuccess) return e;
    if (after_down && (e = hipEventRecord(after_down, s)) != hipSuccess) return e;
    return hipSuccess;
}

hipError_t launch_ffn_reduce(const FfnParams &p, const float *y_extra, float *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_reduce, dim3((p.d + kBlock - 1) / kBlock), dim3(kBlock), 0, s, p, y_extra, out);
    return hipGetLastError();
}

hipError_t launch_combine(const float *a, const float *b, const float *c, int d, float *out, hipStream_t s)
{
    if (d <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_combine, dim3((d + kBlock - 1) / kBlock), dim3(kBlock), 0, s, a, b, c, d, out);
    return hipGetLastError();
}

}  // namespace moe
