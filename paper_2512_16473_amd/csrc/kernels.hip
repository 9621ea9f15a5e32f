// gfx950 kernels of the MoE expert stage: router gating, the hit-expert SwiGLU
// FFN as two weight-streaming GEMV kernels, and the fixed-order reduce + combine.
//
// Batch-1 decode reads every weight of a hit expert exactly once and does two
// flops per weight, so the FFN is bound by HBM bandwidth, not by the matrix cores.
// The kernels stream each bf16 weight row with 16-byte nontemporal loads per lane
// (a 64-lane wave covers 512 contiguous weights per load; the weights are used once,
// so they are not kept in the caches), keep the activation slice in registers for
// the life of the wave, reduce each row across the wave with cross-lane shuffles,
// and spread the rows of all hit experts evenly over every wave of the grid. The
// down projection splits its reduction (length f) into segments of at most kSegMax
// so the activation slice a wave holds stays in registers; each wave takes one
// contiguous, equal share of all (segment, row) pairs, and the segment partials,
// already scaled by the gate weight, are summed in a fixed order by the reduce.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "moe.h"
#include "moe_internal.h"
#include "stream_ops.h"

namespace moe {

namespace {

using namespace stream_ops;   // kWave, bf16 unpacking, loads, wave sums, dot8
constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kRouterBlock = 512;
constexpr int kMetaParts = 20;   // index in the workspace header of the partial count

// Reduction segments of a down projection with reduction length fj (a multiple of
// 8), and the segment length.
__device__ __host__ __forceinline__ int seg_count(int fj) { return (fj + kSegMax - 1) / kSegMax; }
__device__ __host__ __forceinline__ int seg_len(int fj)
{
    const int s = seg_count(fj);
    return (((fj + s - 1) / s) + 7) & ~7;
}

// Per-block table of the jobs, built by the first threads of the block from the
// selection (and the device expert->slot mirror). Inactive jobs own no work.
struct JobLds {
    const uint8_t *slab[kMaxJobs];
    float w[kMaxJobs];            // gate weight (1 for the shared expert)
    int slot[kMaxJobs];           // slot (routed) / 0 (shared) / -1 inactive
    int f[kMaxJobs];              // d_ffn of the job, 0 if inactive
    int row0[kMaxJobs + 1];       // prefix of gate/up rows over jobs
    int part0[kMaxJobs + 1];      // prefix of down segments over jobs (compact partial index)
};

__device__ __forceinline__ void build_jobs(const FfnParams &p, JobLds &t, bool need_w)
{
    const int njobs = p.k + 1;
    if (threadIdx.x < njobs) {
        const int j = threadIdx.x;
        int slot = -1, fj = 0;
        const uint8_t *slab = nullptr;
        float w = 1.0f;
        if (j < p.k) {
            const int s = p.sel[j];
            if (p.slotmap) slot = (s >= 0 && s < p.n) ? p.slotmap[s] : -1;
            else slot = s;
            if (slot >= p.nslots) slot = -1;
            if (slot >= 0) {
                fj = p.f;
                slab = p.pool + (uint64_t)slot * p.slab_stride;
                if (need_w) w = p.w[j];
            }
        } else if (p.shared && p.f_shared > 0) {
            slot = 0;
            fj = p.f_shared;
            slab = p.shared;
        }
        t.slot[j] = slot;
        t.f[j] = fj;
        t.slab[j] = slab;
        t.w[j] = w;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int rows = 0, parts = 0;
        for (int j = 0; j < njobs; ++j) {
            t.row0[j] = rows;
            t.part0[j] = parts;
            if (t.slot[j] >= 0) {
                rows += t.f[j];
                parts += seg_count(t.f[j]);
            }
        }
        t.row0[njobs] = rows;
        t.part0[njobs] = parts;
    }
    __syncthreads();
}

// Job owning item `it` of a prefix table (it < table[njobs]).
__device__ __forceinline__ int job_of(const int *table, int njobs, int it)
{
    int j = 0;
    while (j + 1 < njobs && table[j + 1] <= it) ++j;
    return j;
}

// ---------------------------------------------------------------------------
// Gate/up/SiLU: h_j[i] = SiLU(W1_j[i,:] x) * (W3_j[i,:] x) for every row i of
// every active job. CPL = 16-byte chunks per lane along d (d <= CPL * 512).
// Block 0 also publishes the job table and the partial count for the reduce.
// ---------------------------------------------------------------------------
template <int CPL>
__global__ __launch_bounds__(kBlock) void k_gate_up(FfnParams p)
{
    __shared__ JobLds t;
    build_jobs(p, t, false);
    const int njobs = p.k + 1;
    if (blockIdx.x == 0) {
        if (threadIdx.x < njobs) p.jobslot[threadIdx.x] = t.slot[threadIdx.x];
        if (threadIdx.x == 0) p.jobslot[kMetaParts] = t.part0[njobs];
    }

    const int lane = threadIdx.x & (kWave - 1);
    const int nwaves = gridDim.x * kWavesPerBlock;
    const int wid = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int total = t.row0[njobs];
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
        const int j = job_of(t.row0, njobs, it);
        const int i = it - t.row0[j];
        const uint4 *r1 = reinterpret_cast<const uint4 *>(t.slab[j] + (uint64_t)i * d * 2);
        const uint4 *r3 = reinterpret_cast<const uint4 *>(t.slab[j] + ((uint64_t)t.f[j] * d + (uint64_t)i * d) * 2);
        uint4 a[CPL], b[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int ch = c * kWave + lane;
            if (ch < nch) {
                a[c] = stream_load(r1 + ch);
                b[c] = stream_load(r3 + ch);
            } else {
                a[c] = make_uint4(0, 0, 0, 0);
                b[c] = make_uint4(0, 0, 0, 0);
            }
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

// True in the one work group of the grid that arrives last at this point. Every work
// group calls it once, with all its threads, after thread 0 alone wrote the group's
// partial results to global memory; those are visible to the last group after it
// returns (thread 0's device-scope release before the arrival counter, which the caller
// zeroed before the launch or the last group resets, and an acquire in every thread of
// the last group). One release per work group: each writes the XCD's L2 back.
__device__ __forceinline__ bool arrive_last(unsigned *ticket)
{
    __shared__ int last;
    if (threadIdx.x == 0) {
        __threadfence();
        last = atomicAdd(ticket, 1u) == gridDim.x - 1;
    }
    __syncthreads();
    if (!last) return false;
    __threadfence();
    return true;
}

// ---------------------------------------------------------------------------
// Down: partial[part0[j] + s][i] = w_j * sum over segment s of W2_j[i, c] h_j[c].
// The (segment, row) pairs of all active jobs, in (job, segment, row) order, are
// split into one contiguous, equal range per wave; the wave reloads its h segment
// (registers) only where its range crosses a segment, and streams two rows per step.
// ---------------------------------------------------------------------------
constexpr int kCplK = kSegMax / (8 * kWave);   // chunks per lane of one segment

__global__ __launch_bounds__(kBlock) void k_down(FfnParams p)
{
    __shared__ JobLds t;
    build_jobs(p, t, true);
    const int njobs = p.k + 1;
    const int d = p.d;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t nwaves = (int64_t)gridDim.x * kWavesPerBlock;
    const int64_t wid = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int64_t total = (int64_t)t.part0[njobs] * d;
    int64_t r = total * wid / nwaves;
    const int64_t r_end = total * (wid + 1) / nwaves;

    while (r < r_end) {
        const int q = (int)(r / d);                 // compact segment index
        const int j = job_of(t.part0, njobs, q);
        const int s = q - t.part0[j];
        const int i0 = (int)(r - (int64_t)q * d);
        const int64_t seg_end = (int64_t)(q + 1) * d;
        const int64_t run_end = r_end < seg_end ? r_end : seg_end;
        const int i1 = (int)(run_end - (int64_t)q * d);
        const int fj = t.f[j];
        const int seg = seg_len(fj);
        const int c0 = s * seg;
        const int len = min(seg, fj - c0);
        const int nch = len >> 3;
        const float wj = t.w[j];

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
        float *out = p.partial + (size_t)q * d;
        for (int i = i0; i < i1; i += 2) {
            const bool two = (i + 1 < i1);
            const uint4 *ra = reinterpret_cast<const uint4 *>(w2 + ((uint64_t)i * fj + c0) * 2);
            const uint4 *rb = reinterpret_cast<const uint4 *>(w2 + ((uint64_t)(two ? i + 1 : i) * fj + c0) * 2);
            uint4 a[kCplK], b[kCplK];
#pragma unroll
            for (int c = 0; c < kCplK; ++c) {
                const int ch = c * kWave + lane;
                if (ch < nch) {
                    a[c] = stream_load(ra + ch);
                    b[c] = two ? stream_load(rb + ch) : make_uint4(0, 0, 0, 0);
                } else {
                    a[c] = make_uint4(0, 0, 0, 0);
                    b[c] = make_uint4(0, 0, 0, 0);
                }
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
                out[i] = wj * ya;
                if (two) out[i + 1] = wj * yb;
            }
        }
        r = run_end;
    }
}

// out[i] = the compact partials summed in index order (+ y_extra[i]). The first kRedU
// partial rows (the workspace always holds kMaxJobs x smax of them) and y_extra are
// loaded together with the partial count, so the kernel waits for one round trip
// rather than for the count and then for the rows; the sum keeps the index order.
constexpr int kRedU = 8;
static_assert(kRedU <= kMaxJobs, "rows loaded ahead of the count lie in the partial region");

__global__ __launch_bounds__(kBlock) void k_reduce(FfnParams p, const float *y_extra, float *out)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= p.d) return;
    const float *src = p.partial + i;
    const size_t ld = (size_t)p.d;
    float v[kRedU];
#pragma unroll
    for (int q = 0; q < kRedU; ++q) v[q] = src[q * ld];
    const float ye = y_extra ? y_extra[i] : 0.f;
    const int nparts = p.jobslot[kMetaParts];
    float acc = 0.f;
#pragma unroll
    for (int q = 0; q < kRedU; ++q)
        if (q < nparts) acc += v[q];
    for (int q = kRedU; q < nparts; ++q) acc += src[q * ld];
    if (y_extra) acc += ye;
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
// Top-k of n fp64 logits held in LDS, by one wave: the k largest (ties to the lower
// id; NaN ranked as -inf so ids are always valid), ordered (logit desc, id asc), with
// weights w_r = exp(l_r - l_0) / sum_{s<k} exp(l_s - l_0), the softmax restricted to
// the selected set (equal to p_S / sum p_S). Lanes r < k write idx[r], w[r] (and the
// mailbox entries when mbox is set).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void select_topk(const double *logit, int n, int k, int lane, int32_t *idx, float *wout,
                                            RouteMailbox *mbox)
{
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
    // Lane r keeps the r-th selected (logit, id).
    double my_l = -INFINITY;
    int my_i = -1;
    for (int r = 0; r < k; ++r) {
        double bv = -INFINITY;
        int bi = 0x7fffffff;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int e = q * kWave + lane;
            if (!taken[q] && (v[q] > bv || (v[q] == bv && e < bi))) {
                bv = v[q];
                bi = e;
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const double ov = __shfl_xor(bv, o, kWave);
            const int oi = __shfl_xor(bi, o, kWave);
            if (ov > bv || (ov == bv && oi < bi)) {
                bv = ov;
                bi = oi;
            }
        }
        if (lane == r) {
            my_l = bv;
            my_i = bi;
        }
#pragma unroll
        for (int q = 0; q < kPer; ++q)
            if (q * kWave + lane == bi) taken[q] = true;
    }
    const double l0 = __shfl(my_l, 0, kWave);
    const double ex = (lane < k) ? exp(my_l - l0) : 0.0;
    const double z = wave_sum(ex);
    if (lane < k) {
        const float wr32 = (float)(ex / z);
        idx[lane] = my_i;
        wout[lane] = wr32;
        if (mbox) {
            mbox->idx[lane] = my_i;
            mbox->w[lane] = wr32;
        }
    }
}

// ---------------------------------------------------------------------------
// Router: one block per token. x is staged in LDS; each wave takes whole experts,
// issuing all CPR 16-byte loads of a router row at once, and accumulates the exact
// fp64 products of the fp32 inputs. Wave 0 then selects the top-k in fp64 (ties to
// the lower id; NaN ranked as -inf so ids are always valid) and forms the weights.
// CPR = float4 chunks per lane along d (d <= CPR * 256).
// ---------------------------------------------------------------------------
template <int CPR>
__global__ __launch_bounds__(kRouterBlock) void k_router(const float *X, const float *Wr, int d, int n, int k,
                                                         int32_t *idx, float *wout, RouteMailbox *mbox,
                                                         float *x_host, int32_t seq, const int32_t *row_src,
                                                         int32_t *row_dst)
{
    // Decode only: install the layer's expert->slot mirror row that the hit kernels after
    // this one read (the host's view of which slots hold landed experts).
    if (row_src)
        for (int i = threadIdx.x; i < n; i += kRouterBlock) row_dst[i] = row_src[i];
    constexpr int kWaves = kRouterBlock / kWave;
    __shared__ double logit[MOE_MAX_EXPERTS];
    __shared__ float4 xs[CPR * kWave];
    const int t = blockIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int nq = d >> 2;   // float4 chunks of a row
    const float4 *x4 = reinterpret_cast<const float4 *>(X + (size_t)t * d);
    for (int q = threadIdx.x; q < CPR * kWave; q += kRouterBlock) xs[q] = q < nq ? x4[q] : make_float4(0, 0, 0, 0);
    __syncthreads();
    for (int e = wv; e < n; e += kWaves) {
        const float4 *w4 = reinterpret_cast<const float4 *>(Wr + (size_t)e * d);
        double acc = 0.0;
        // Eight 16-byte loads in flight per lane per step keeps the registers bounded.
        constexpr int kStep = CPR < 8 ? CPR : 8;
#pragma unroll 1
        for (int mb = 0; mb < CPR; mb += kStep) {
            float4 wvv[kStep];
#pragma unroll
            for (int m = 0; m < kStep; ++m)   // unconditional (xs is zero past the row)
                wvv[m] = w4[min((mb + m) * kWave + lane, nq - 1)];
#pragma unroll
            for (int m = 0; m < kStep; ++m) {
                const float4 xv = xs[(mb + m) * kWave + lane];
                acc += (double)wvv[m].x * (double)xv.x;
                acc += (double)wvv[m].y * (double)xv.y;
                acc += (double)wvv[m].z * (double)xv.z;
                acc += (double)wvv[m].w * (double)xv.w;
            }
        }
        acc = wave_sum(acc);
        if (lane == 0) logit[e] = acc;
    }
    __syncthreads();
    if (wv == 0) {
        select_topk(logit, n, k, lane, idx + (size_t)t * k, wout + (size_t)t * k, mbox);
    } else if (x_host) {
        // The other waves hand the hidden state to the host for the miss path.
        float4 *xh = reinterpret_cast<float4 *>(x_host);
        for (int q = threadIdx.x - kWave; q < nq; q += kRouterBlock - kWave) xh[q] = xs[q];
    }
    if (mbox) {
        __threadfence_system();
        __syncthreads();
        if (threadIdx.x == 0) __hip_atomic_store(&mbox->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

// ---------------------------------------------------------------------------
// Single-token decode router over many work groups. Item (e, s) = expert e, segment s
// (kRouteSeg floats) of its router row; wave `item` of the grid streams that segment
// (four 16-byte loads per lane, all in flight at once) against the same slice of x and
// stores the fp64 partial logit part[e * nseg + s]. The work group that arrives last
// sums each expert's segments in order, selects the top-k, hands the routing and x to
// the host (mailbox, then the sequence number with a system-scope release) and resets
// the arrival counter. Work group 0 installs the layer's mirror row at its start.
// ---------------------------------------------------------------------------
constexpr int kRouteSeg = 1024;

__global__ __launch_bounds__(kBlock) void k_route1(const float *x, const float *Wr, int d, int n, int k,
                                                   int32_t *idx, float *wout, double *part, unsigned *ticket,
                                                   RouteMailbox *mbox, float *x_host, int32_t seq,
                                                   const int32_t *row_src, int32_t *row_dst)
{
    if (blockIdx.x == 0 && row_src)
        for (int i = threadIdx.x; i < n; i += kBlock) row_dst[i] = row_src[i];
    constexpr int kPerLane = kRouteSeg / (4 * kWave);   // float4 loads per lane
    const int lane = threadIdx.x & (kWave - 1);
    const int item = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int nseg = (d + kRouteSeg - 1) / kRouteSeg;
    const int nq = d >> 2;
    __shared__ double part_l[kWavesPerBlock];
    if (item < n * nseg) {
        const int e = item / nseg;
        const int q0 = (item - e * nseg) * (kRouteSeg / 4);
        const float4 *w4 = reinterpret_cast<const float4 *>(Wr + (size_t)e * d);
        const float4 *x4 = reinterpret_cast<const float4 *>(x);
        float4 wv[kPerLane], xv[kPerLane];
#pragma unroll
        for (int m = 0; m < kPerLane; ++m) {   // unconditional loads; past the row: zeroed x
            const int q = min(q0 + m * kWave + lane, nq - 1);
            wv[m] = w4[q];
            xv[m] = x4[q];
        }
#pragma unroll
        for (int m = 0; m < kPerLane; ++m)
            if (q0 + m * kWave + lane >= nq) xv[m] = make_float4(0, 0, 0, 0);
        double acc = 0.0;
#pragma unroll
        for (int m = 0; m < kPerLane; ++m) {
            acc += (double)wv[m].x * (double)xv[m].x;
            acc += (double)wv[m].y * (double)xv[m].y;
            acc += (double)wv[m].z * (double)xv[m].z;
            acc += (double)wv[m].w * (double)xv[m].w;
        }
        acc = wave_sum(acc);
        if (lane == 0) part_l[threadIdx.x >> 6] = acc;
    }
    __syncthreads();
    if (threadIdx.x == 0)   // the group's partials, written by the thread that releases them
        for (int w = 0; w < kWavesPerBlock; ++w) {
            const int it = blockIdx.x * kWavesPerBlock + w;
            if (it < n * nseg) part[it] = part_l[w];
        }
    if (!arrive_last(ticket)) return;
    __shared__ double logit[MOE_MAX_EXPERTS];
    for (int e = threadIdx.x; e < n; e += kBlock) {
        double l = 0.0;
        for (int sg = 0; sg < nseg; ++sg) l += part[e * nseg + sg];
        logit[e] = l;
    }
    if (threadIdx.x == 0) *ticket = 0u;
    __syncthreads();
    const int wv0 = threadIdx.x >> 6;
    if (wv0 == 0) {
        select_topk(logit, n, k, lane, idx, wout, mbox);
    } else if (x_host) {
        const float4 *x4 = reinterpret_cast<const float4 *>(x);
        float4 *xh = reinterpret_cast<float4 *>(x_host);
        for (int q = threadIdx.x - kWave; q < nq; q += kBlock - kWave) xh[q] = x4[q];
    }
    if (mbox) {
        __threadfence_system();
        __syncthreads();
        if (threadIdx.x == 0) __hip_atomic_store(&mbox->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

// ---------------------------------------------------------------------------
// Single-token decode router in one work group of 512 threads, for router matrices of
// at most kRouteBlkItems (expert, segment) items whose segment count divides 8: wave w
// takes items w, w + 8, ... (at most eight, all loads issued at once), which all lie in
// segment w mod nseg, so the wave loads that slice of x once. The fp64 partial logits go
// to LDS and wave 0 sums each expert's segments in order and selects the top-k. One work
// group needs no arrival counter or device-scope fence; the mailbox hand-off is that of
// k_router.
// ---------------------------------------------------------------------------
constexpr int kRouteBlkThreads = 512;
constexpr int kRouteBlkWaves = kRouteBlkThreads / kWave;
constexpr int kRouteBlkPerWave = 8;
constexpr int kRouteBlkItems = kRouteBlkWaves * kRouteBlkPerWave;

__global__ __launch_bounds__(kRouteBlkThreads) void k_router_blk(const float *x, const float *Wr, int d, int n, int k,
                                                                 int32_t *idx, float *wout, RouteMailbox *mbox,
                                                                 float *x_host, int32_t seq, const int32_t *row_src,
                                                                 int32_t *row_dst)
{
    if (row_src)
        for (int i = threadIdx.x; i < n; i += kRouteBlkThreads) row_dst[i] = row_src[i];
    constexpr int kPerLane = kRouteSeg / (4 * kWave);
    __shared__ double part[kRouteBlkItems];
    __shared__ double logit[MOE_MAX_EXPERTS];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int nseg = (d + kRouteSeg - 1) / kRouteSeg;   // divides kRouteBlkWaves
    const int items = n * nseg;
    const int nq = d >> 2;
    const int q0 = (wv % nseg) * (kRouteSeg / 4);        // this wave's slice of every row
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    float4 xq[kPerLane], wq[kRouteBlkPerWave][kPerLane];
    // Every load is unconditional (a branch per load would make each one wait for the
    // previous): positions past the row read its last chunk, items past the end the
    // last row, and those values are zeroed after the loads.
#pragma unroll
    for (int m = 0; m < kPerLane; ++m) xq[m] = x4[min(q0 + m * kWave + lane, nq - 1)];
#pragma unroll
    for (int u = 0; u < kRouteBlkPerWave; ++u) {
        const int item = wv + u * kRouteBlkWaves;
        const float4 *w4 = reinterpret_cast<const float4 *>(Wr + (size_t)min(item / nseg, n - 1) * d);
#pragma unroll
        for (int m = 0; m < kPerLane; ++m) wq[u][m] = w4[min(q0 + m * kWave + lane, nq - 1)];
    }
#pragma unroll
    for (int m = 0; m < kPerLane; ++m)
        if (q0 + m * kWave + lane >= nq) xq[m] = make_float4(0, 0, 0, 0);
    // x for the host: the first wave of each segment writes its slice as soon as it has
    // it, so the writes cross PCIe while the logits are computed (the system-scope fence
    // before the sequence number covers them)
    if (x_host && wv < nseg) {
        float4 *xh = reinterpret_cast<float4 *>(x_host);
#pragma unroll
        for (int m = 0; m < kPerLane; ++m) {
            const int q = q0 + m * kWave + lane;
            if (q < nq) xh[q] = xq[m];
        }
    }
#pragma unroll
    for (int u = 0; u < kRouteBlkPerWave; ++u) {
        // one item at a time: keeps the scheduler from widening every loaded value to
        // fp64 at once (which would not fit the registers)
        __builtin_amdgcn_sched_barrier(0);
        double acc = 0.0;
#pragma unroll
        for (int m = 0; m < kPerLane; ++m) {
            acc += (double)wq[u][m].x * (double)xq[m].x;
            acc += (double)wq[u][m].y * (double)xq[m].y;
            acc += (double)wq[u][m].z * (double)xq[m].z;
            acc += (double)wq[u][m].w * (double)xq[m].w;
        }
        acc = wave_sum(acc);
        const int item = wv + u * kRouteBlkWaves;
        if (lane == 0 && item < items) part[item] = acc;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < n; e += kRouteBlkThreads) {
        double l = 0.0;
        for (int sg = 0; sg < nseg; ++sg) l += part[e * nseg + sg];
        logit[e] = l;
    }
    __syncthreads();
    if (wv == 0) select_topk(logit, n, k, lane, idx, wout, mbox);
    if (mbox) {
        __threadfence_system();
        __syncthreads();
        if (threadIdx.x == 0) __hip_atomic_store(&mbox->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

// Resident blocks per CU of a kernel (cached by the caller; concurrent first calls
// store the same value). If the runtime cannot answer, the count is derived from the
// kernel's register use (512 VGPRs per SIMD lane, one wave per SIMD per 256-thread
// block), else 2.
template <typename K>
int blocks_per_cu(K kernel, int block, std::atomic<int> *cache)
{
    int c = cache->load(std::memory_order_relaxed);
    if (c <= 0) {
        int b = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, kernel, block, 0) != hipSuccess || b <= 0) {
            (void)hipGetLastError();
            hipFuncAttributes fa{};
            b = 2;
            if (hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(kernel)) == hipSuccess && fa.numRegs > 0) {
                const int regs = (fa.numRegs + 7) & ~7;
                b = 512 / regs;
                if (b > 8) b = 8;
                if (b < 1) b = 1;
            } else {
                (void)hipGetLastError();
            }
        }
        cache->store(b, std::memory_order_relaxed);
        c = b;
    }
    return c;
}

// Launch status: the runtime's last error is cleared before each launch (another
// library in the process may have left one) and read right after it.
inline void clear_launch_error() { (void)hipGetLastError(); }

template <int CPL>
hipError_t launch_gate_up_cpl(const FfnParams &p, int items, hipStream_t s, hipEvent_t e0, hipEvent_t e1)
{
    // Up to 4 x the resident work groups (more waves, each with a few row pairs, hide the
    // load latency better than fewer longer-lived ones), fewer while that would leave
    // under two row pairs per wave (each wave loads x before its first row).
    static std::atomic<int> occ{0};
    const int resident = blocks_per_cu(k_gate_up<CPL>, kBlock, &occ) * device_cu_count();
    int cap = resident * 4;
    while (cap > resident && (int64_t)cap * kWavesPerBlock * 2 > items) cap /= 2;
    int blocks = (items + kWavesPerBlock - 1) / kWavesPerBlock;
    blocks = blocks < 1 ? 1 : (blocks > cap ? cap : blocks);
    clear_launch_error();
    if (e0 || e1) hipExtLaunchKernelGGL(k_gate_up<CPL>, dim3(blocks), dim3(kBlock), 0, s, e0, e1, 0, p);
    else hipLaunchKernelGGL(k_gate_up<CPL>, dim3(blocks), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_gate_up(const FfnParams &p, int items, hipStream_t s, hipEvent_t e0, hipEvent_t e1)
{
    const int cpl = (p.d / 8 + kWave - 1) / kWave;
    switch (cpl) {
#define MOE_CPL_CASE(N) case N: return launch_gate_up_cpl<N>(p, items, s, e0, e1);
        MOE_CPL_CASE(1) MOE_CPL_CASE(2) MOE_CPL_CASE(3) MOE_CPL_CASE(4)
        MOE_CPL_CASE(5) MOE_CPL_CASE(6) MOE_CPL_CASE(7) MOE_CPL_CASE(8)
        MOE_CPL_CASE(9) MOE_CPL_CASE(10) MOE_CPL_CASE(11) MOE_CPL_CASE(12)
        MOE_CPL_CASE(13) MOE_CPL_CASE(14) MOE_CPL_CASE(15) MOE_CPL_CASE(16)
#undef MOE_CPL_CASE
    default: return hipErrorInvalidValue;
    }
}

template <int CPR>
hipError_t launch_router_cpr(const float *x, const float *wr, int T, int d, int n, int k, int32_t *idx, float *w,
                             hipStream_t s, RouteMailbox *mbox, float *x_host, int32_t seq, const int32_t *row_src,
                             int32_t *row_dst)
{
    clear_launch_error();
    hipLaunchKernelGGL(k_router<CPR>, dim3(T), dim3(kRouterBlock), 0, s, x, wr, d, n, k, idx, w, mbox, x_host, seq,
                       row_src, row_dst);
    return hipGetLastError();
}

}  // namespace

// Device scratch of the allocation-free hit FFN (moe_expert_ffn_hits_noalloc): the
// job-table header, h and the split-K partials of one call live here instead of in a
// caller workspace. One copy per device, held until the process ends; every call on a
// device shares it, so calls that overlap on one device race. Nothing in it needs to
// start at zero: the gate/up kernel writes the header and every h row it owns, the down
// kernel every partial the reduce reads.
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

hipError_t noalloc_scratch(void **ptr)
{
    // Host code may not pass `scratch` itself to a kernel (its host-side name is not a
    // device address): its address on the current device is looked up once per device.
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

int device_cu_count()
{
    static std::atomic<int> cached[64] = {};   // per device; concurrent first calls store the same value
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cached[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cached[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

size_t ffn_workspace_bytes(int max_jobs, int d, int f_max)
{
    (void)max_jobs;
    const size_t hstride = (size_t)((f_max + 63) & ~63);
    const size_t smax = (size_t)seg_count(f_max);
    return align256(sizeof(int32_t) * 64) + align256(sizeof(float) * kMaxJobs * hstride) +
           align256(sizeof(float) * kMaxJobs * smax * (size_t)d);
}

void ffn_bind_workspace(FfnParams &p, void *ws, int max_jobs, int d, int f_max)
{
    (void)max_jobs;
    const size_t hstride = (size_t)((f_max + 63) & ~63);
    uint8_t *b = static_cast<uint8_t *>(ws);
    p.jobslot = reinterpret_cast<int32_t *>(b);
    b += align256(sizeof(int32_t) * 64);
    p.h = reinterpret_cast<float *>(b);
    p.hstride = (int)hstride;
    b += align256(sizeof(float) * kMaxJobs * hstride);
    p.partial = reinterpret_cast<float *>(b);
    p.smax = seg_count(f_max);
}

hipError_t launch_router(const float *x, const float *wr, int T, int d, int n, int k, int32_t *idx,
                         float *w, hipStream_t s, RouteMailbox *mbox, float *x_host, int32_t seq,
                         const int32_t *row_src, int32_t *row_dst)
{
    if (T <= 0) return hipSuccess;
    if (T != 1) mbox = nullptr, x_host = nullptr, row_src = nullptr;
    if (!row_dst) row_src = nullptr;
    const int cpr = (d / 4 + kWave - 1) / kWave;
#define MOE_CPR_CASE(N) \
    if (cpr <= N) return launch_router_cpr<N>(x, wr, T, d, n, k, idx, w, s, mbox, x_host, seq, row_src, row_dst);
    MOE_CPR_CASE(1) MOE_CPR_CASE(2) MOE_CPR_CASE(4) MOE_CPR_CASE(8) MOE_CPR_CASE(16) MOE_CPR_CASE(32)
#undef MOE_CPR_CASE
    return hipErrorInvalidValue;
}

size_t route1_scratch_bytes(int n, int d)
{
    const size_t nseg = (size_t)((d + kRouteSeg - 1) / kRouteSeg);
    return align256(sizeof(double) * (size_t)n * nseg) + 256;   // partial logits, then the counter
}

hipError_t launch_route1(const float *x, const float *wr, int d, int n, int k, int32_t *idx, float *w,
                         void *scratch, hipStream_t s, RouteMailbox *mbox, float *x_host, int32_t seq,
                         const int32_t *row_src, int32_t *row_dst)
{
    const int nseg = (d + kRouteSeg - 1) / kRouteSeg;
    if (!row_dst) row_src = nullptr;
    if (n * nseg <= kRouteBlkItems && kRouteBlkWaves % nseg == 0) {   // one work group reads it all at once
        clear_launch_error();
        hipLaunchKernelGGL(k_router_blk, dim3(1), dim3(kRouteBlkThreads), 0, s, x, wr, d, n, k, idx, w, mbox, x_host,
                           seq, row_src, row_dst);
        return hipGetLastError();
    }
    const int blocks = (n * nseg + kWavesPerBlock - 1) / kWavesPerBlock;
    double *part = static_cast<double *>(scratch);
    unsigned *ticket = reinterpret_cast<unsigned *>(static_cast<uint8_t *>(scratch) +
                                                    align256(sizeof(double) * (size_t)n * nseg));
    clear_launch_error();
    hipLaunchKernelGGL(k_route1, dim3(blocks), dim3(kBlock), 0, s, x, wr, d, n, k, idx, w, part, ticket, mbox,
                       x_host, seq, row_src, row_dst);
    return hipGetLastError();
}

hipError_t launch_ffn_stream(const FfnParams &p, hipStream_t s, const FfnEvents *ev)
{
    // Upper bound of the gate/up rows (every routed job active); waves with no row exit.
    const int rows_max = p.k * p.f + (p.shared ? p.f_shared : 0);
    hipError_t e;
    if ((e = launch_gate_up(p, rows_max, s, ev ? ev->gu_start : nullptr, ev ? ev->gu_stop : nullptr)) != hipSuccess)
        return e;
    static std::atomic<int> occ_down{0};
    const int blocks = blocks_per_cu(k_down, kBlock, &occ_down) * device_cu_count();
    clear_launch_error();
    if (ev && (ev->dn_start || ev->dn_stop))
        hipExtLaunchKernelGGL(k_down, dim3(blocks), dim3(kBlock), 0, s, ev->dn_start, ev->dn_stop, 0, p);
    else
        hipLaunchKernelGGL(k_down, dim3(blocks), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_ffn_reduce(const FfnParams &p, const float *y_extra, float *out, hipStream_t s)
{
    clear_launch_error();
    hipLaunchKernelGGL(k_reduce, dim3((p.d + kBlock - 1) / kBlock), dim3(kBlock), 0, s, p, y_extra, out);
    return hipGetLastError();
}

hipError_t launch_combine(const float *a, const float *b, const float *c, int d, float *out, hipStream_t s)
{
    if (d <= 0) return hipSuccess;
    clear_launch_error();
    hipLaunchKernelGGL(k_combine, dim3((d + kBlock - 1) / kBlock), dim3(kBlock), 0, s, a, b, c, d, out);
    return hipGetLastError();
}

}  // namespace moe
