// Multi-token decode FFN for small batches (T <= 8 tokens, every selected expert resident):
//   y[t] = sum_j w[t][j] * FFN(slab at slots[t][j], x[t])  (SwiGLU, Section I's expert FFN)
//
// Between one-token decode (one GEMV per hit expert) and prefill (grouped MFMA GEMMs)
// lies the case of a few tokens per step. Run per token, the GEMV path reads an expert
// once for every token that selected it; the grouped GEMMs read it once but in the MFMA
// operand layout, whose weight stream runs well below HBM speed. These kernels keep the
// GEMV's streaming (each wave reads whole weight rows with 16-byte nontemporal loads) and
// read each selected slab once: the rows of a slab are dotted with the hidden states of
// all the tokens that selected it, which sit in LDS (x for gate/up, a segment of h for
// down). Three kernels on one stream: gate/up/SiLU -> down (split-K over segments of f,
// weighted partials) -> reduce (fixed order). Every block builds the same job table
// (distinct slots in order of first appearance; each job's (token, rank) pairs in order)
// from the T*k selections.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"
#include "moe_internal.h"
#include "stream_ops.h"

namespace moe {
namespace {

using namespace stream_ops;

constexpr int kTokThreads = 512;                         // 8 waves share the LDS copy
constexpr int kTokWaves = kTokThreads / kWave;
constexpr int kMaxPairs = MOE_MAX_TOKENS * MOE_MAX_TOPK_INTERNAL;   // 128
constexpr int kDownRows = 128;                           // W2 rows per down work group

static_assert(kMaxPairs <= kTokThreads, "one thread per (token, rank) pair");

struct TokJobs {
    int njobs;
    int slot[kMaxPairs];        // job -> slot
    int first[kMaxPairs + 1];   // job -> its range in `pair`
    int pair[kMaxPairs];        // pair ids t*k + r grouped by job, ascending within a job
    int lead[kMaxPairs];        // scratch: first pair with the same slot, -1 if skipped
};

// Every thread p < T*k takes one pair; all loops are over at most 128 entries.
__device__ void build_jobs(const int32_t *slots, int npairs, int nslots, TokJobs &J)
{
    const int p = threadIdx.x;
    int s = -1;
    if (p < npairs) {
        s = slots[p];
        if (s < 0 || s >= nslots) s = -1;
    }
    if (p < kMaxPairs) J.lead[p] = -1;
    __syncthreads();
    if (p < npairs && s >= 0) {
        int l = p;
        for (int q = 0; q < p; ++q)
            if (slots[q] == s) {   // the same valid slot (s is in range)
                l = q;
                break;
            }
        J.lead[p] = l;
    }
    __syncthreads();
    if (p < npairs && s >= 0) {
        const int l = J.lead[p];
        int start = 0, pos = 0, job = 0;
        for (int q = 0; q < npairs; ++q) {
            const int lq = J.lead[q];
            if (lq < 0) continue;
            start += lq < l;             // pairs of earlier jobs (jobs ordered by their lead)
            pos += (lq == l && q < p);   // earlier pairs of this job
            job += (lq == q && q < l);   // jobs led before this one
        }
        J.pair[start + pos] = p;
        if (l == p) {
            J.slot[job] = s;
            J.first[job] = start;
        }
    }
    if (p == 0) {
        int nj = 0, nv = 0;
        for (int q = 0; q < npairs; ++q) {
            nv += J.lead[q] >= 0;
            nj += J.lead[q] == q;
        }
        J.njobs = nj;
        J.first[nj] = nv;
    }
    __syncthreads();
}

struct TokParams {
    const float *x;          // [T][d]
    const uint8_t *pool;
    uint64_t slab_stride;
    const int32_t *slots;    // [T][k]
    const float *w;          // [T][k]
    int T, k, nslots, d, f;
    int nseg, seg;           // down: reduction segments of f and their length
    float *h;                // [T*k][f]
    float *partial;          // [T*k][nseg][d]
};

// h[p][i] = SiLU(W1_i x_t) * (W3_i x_t) for every pair p = (t, r) of every job, row i.
// CPL = 16-byte chunks per lane along d (d <= CPL * 512).
template <int CPL>
__global__ __launch_bounds__(kTokThreads) void k_tok_gate_up(TokParams p)
{
    __shared__ TokJobs J;
    extern __shared__ float4 xs4[];   // [T][d] fp32, 16-byte aligned
    float *xs = reinterpret_cast<float *>(xs4);
    build_jobs(p.slots, p.T * p.k, p.nslots, J);
    const int d = p.d, nch = d >> 3;
    for (int i = threadIdx.x; i < p.T * d / 4; i += kTokThreads) xs4[i] = reinterpret_cast<const float4 *>(p.x)[i];
    __syncthreads();

    const int lane = threadIdx.x & (kWave - 1);
    const int nwaves = gridDim.x * kTokWaves;
    const int total = J.njobs * p.f;
    // Two register sets: the next row pair is in flight while this one is dotted with
    // the tokens. Loads are unconditional (past the end they re-read the last row pair)
    // so that each wait covers only the older set.
    uint4 a[2][CPL], b[2][CPL];
#define MOE_TOK_LOAD(set, item)                                                                        \
    do {                                                                                               \
        const int it_ = min((item), total - 1);                                                        \
        const int job_ = it_ / p.f, i_ = it_ - job_ * p.f;                                              \
        const uint8_t *slab_ = p.pool + (uint64_t)J.slot[job_] * p.slab_stride;                        \
        const uint4 *r1_ = reinterpret_cast<const uint4 *>(slab_ + (uint64_t)i_ * d * 2);              \
        const uint4 *r3_ = reinterpret_cast<const uint4 *>(slab_ + ((uint64_t)p.f * d + (uint64_t)i_ * d) * 2); \
        _Pragma("unroll") for (int c = 0; c < CPL; ++c) {                                              \
            const int ch = min(c * kWave + lane, nch - 1);                                             \
            a[set][c] = stream_load(r1_ + ch);                                                         \
            b[set][c] = stream_load(r3_ + ch);                                                         \
        }                                                                                              \
    } while (0)
#define MOE_TOK_DOT(set, item)                                                                         \
    do {                                                                                               \
        const int job_ = (item) / p.f, i_ = (item) - job_ * p.f;                                        \
        for (int q = J.first[job_]; q < J.first[job_ + 1]; ++q) {                                      \
            const int pr = J.pair[q];                                                                  \
            const float *xt = xs + (pr / p.k) * d;                                                     \
            float g = 0.f, u = 0.f;                                                                    \
            _Pragma("unroll") for (int c = 0; c < CPL; ++c) {                                          \
                const int ch = c * kWave + lane;                                                       \
                if (ch < nch) {                                                                        \
                    float xv[8];                                                                       \
                    load8(xt + ch * 8, xv);                                                            \
                    g = dot8(a[set][c], xv, g);                                                        \
                    u = dot8(b[set][c], xv, u);                                                        \
                }                                                                                      \
            }                                                                                          \
            g = wave_sum(g);                                                                           \
            u = wave_sum(u);                                                                           \
            if (lane == 0) p.h[(size_t)pr * p.f + i_] = g / (1.0f + expf(-g)) * u;                      \
        }                                                                                              \
    } while (0)

    int it = blockIdx.x * kTokWaves + (threadIdx.x >> 6);
    if (it < total) MOE_TOK_LOAD(0, it);
    for (; it < total; it += 2 * nwaves) {
        MOE_TOK_LOAD(1, it + nwaves);
        MOE_TOK_DOT(0, it);
        if (it + nwaves >= total) break;
        MOE_TOK_LOAD(0, it + 2 * nwaves);
        MOE_TOK_DOT(1, it + nwaves);
    }
#undef MOE_TOK_LOAD
#undef MOE_TOK_DOT
}

// partial[p][s][r] = w_p * sum over segment s of W2_r h_p, for every pair p of a job.
// Work group b: job b / (nseg * nchunk), segment, and kDownRows consecutive rows r; the
// h segments of the job's pairs are staged in LDS. CPK = 16-byte chunks per lane of a
// segment (seg <= CPK * 512).
template <int CPK>
__global__ __launch_bounds__(kTokThreads) void k_tok_down(TokParams p)
{
    __shared__ TokJobs J;
    extern __shared__ float4 hs4[];   // [pairs of the job][seg] fp32, 16-byte aligned
    float *hs = reinterpret_cast<float *>(hs4);
    build_jobs(p.slots, p.T * p.k, p.nslots, J);
    const int nchunk = (p.d + kDownRows - 1) / kDownRows;
    const int job = blockIdx.x / (p.nseg * nchunk);
    if (job >= J.njobs) return;
    const int sgi = (blockIdx.x / nchunk) % p.nseg;
    const int r0 = (blockIdx.x % nchunk) * kDownRows;
    const int c0 = sgi * p.seg;
    const int len = min(p.seg, p.f - c0);
    const int nch = len >> 3;
    const int q0 = J.first[job], np = J.first[job + 1] - q0;
    const int lane = threadIdx.x & (kWave - 1);
    const uint8_t *w2 = p.pool + (uint64_t)J.slot[job] * p.slab_stride + (uint64_t)2 * p.f * p.d * 2;
    const int r1 = min(r0 + kDownRows, p.d);
    // LDS holds the h segments of T pairs; a job has at most T (one per token) unless a
    // token listed a slot twice, and then its pairs go through in groups of T.
    for (int qc = 0; qc < np; qc += p.T) {
        const int nq = min(p.T, np - qc);
        if (qc) __syncthreads();   // the previous group's segments are no longer read
        for (int i = threadIdx.x; i < nq * (len / 4); i += kTokThreads) {
            const int q = i / (len / 4), e = i - q * (len / 4);
            hs4[(q * p.seg) / 4 + e] = reinterpret_cast<const float4 *>(p.h + (size_t)J.pair[q0 + qc + q] * p.f + c0)[e];
        }
        __syncthreads();
        // rows r, r + 8, ... of this group, two register sets (the next row's segment in
        // flight while this one is dotted); loads past the last row re-read it
        uint4 a[2][CPK];
#define MOE_TOK_LOAD_ROW(set, rr)                                                                      \
        do {                                                                                           \
            const uint4 *row_ = reinterpret_cast<const uint4 *>(w2 + ((uint64_t)min((rr), r1 - 1) * p.f + c0) * 2); \
            _Pragma("unroll") for (int c = 0; c < CPK; ++c) a[set][c] = stream_load(row_ + min(c * kWave + lane, nch - 1)); \
        } while (0)
#define MOE_TOK_DOT_ROW(set, rr)                                                                       \
        do {                                                                                           \
            for (int q = 0; q < nq; ++q) {                                                             \
                const float *ht = hs + q * p.seg;                                                      \
                float acc = 0.f;                                                                       \
                _Pragma("unroll") for (int c = 0; c < CPK; ++c) {                                      \
                    const int ch = c * kWave + lane;                                                   \
                    if (ch < nch) {                                                                    \
                        float hv[8];                                                                   \
                        load8(ht + ch * 8, hv);                                                        \
                        acc = dot8(a[set][c], hv, acc);                                                \
                    }                                                                                  \
                }                                                                                      \
                acc = wave_sum(acc);                                                                   \
                if (lane == 0) {                                                                       \
                    const int pr = J.pair[q0 + qc + q];                                                \
                    p.partial[((size_t)pr * p.nseg + sgi) * p.d + (rr)] = p.w[pr] * acc;               \
                }                                                                                      \
            }                                                                                          \
        } while (0)
        int r = r0 + (threadIdx.x >> 6);
        if (r < r1) MOE_TOK_LOAD_ROW(0, r);
        for (; r < r1; r += 2 * kTokWaves) {
            MOE_TOK_LOAD_ROW(1, r + kTokWaves);
            MOE_TOK_DOT_ROW(0, r);
            if (r + kTokWaves >= r1) break;
            MOE_TOK_LOAD_ROW(0, r + 2 * kTokWaves);
            MOE_TOK_DOT_ROW(1, r + kTokWaves);
        }
#undef MOE_TOK_LOAD_ROW
#undef MOE_TOK_DOT_ROW
    }
}

// y[t][i] = sum over ranks r (ascending) of valid pairs, over segments (ascending), of the
// partials; zero for a token with no valid pair.
__global__ __launch_bounds__(256) void k_tok_reduce(TokParams p, float *y)
{
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int t = blockIdx.y;
    if (i >= p.d) return;
    float acc = 0.f;
    for (int r = 0; r < p.k; ++r) {
        const int s = p.slots[t * p.k + r];
        if (s < 0 || s >= p.nslots) continue;
        const float *src = p.partial + (size_t)(t * p.k + r) * p.nseg * p.d + i;
        for (int g = 0; g < p.nseg; ++g) acc += src[(size_t)g * p.d];
    }
    y[(size_t)t * p.d + i] = acc;
}

size_t a256(size_t v) { return (v + 255) & ~(size_t)255; }
int seg_count_tok(int f) { return (f + kSegMax - 1) / kSegMax; }
int seg_len_tok(int f)
{
    const int s = seg_count_tok(f);
    return (((f + s - 1) / s) + 7) & ~7;
}

// Allows `lds` bytes of dynamic LDS (beyond 64 KiB it has to be allowed per kernel;
// gfx950 has 160 KiB per CU) and launches; grid <= 0: as many work groups as fit on the
// device at once.
template <typename K>
hipError_t launch_dyn(K kernel, int grid, size_t lds, hipStream_t s, const TokParams &p)
{
    (void)hipFuncSetAttribute(reinterpret_cast<const void *>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds);
    (void)hipGetLastError();
    if (grid <= 0) {
        int occ = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, kTokThreads, lds) != hipSuccess || occ < 1) {
            (void)hipGetLastError();
            occ = 1;
        }
        grid = occ * device_cu_count();
    }
    hipLaunchKernelGGL(kernel, dim3(grid), dim3(kTokThreads), lds, s, p);
    return hipGetLastError();
}

}  // namespace

size_t tok_workspace_bytes(int T, int k, int d, int f)
{
    const size_t pairs = (size_t)T * k;
    return a256(pairs * f * sizeof(float)) + a256(pairs * seg_count_tok(f) * (size_t)d * sizeof(float));
}

hipError_t launch_tokens(const float *x, const uint8_t *pool, uint64_t stride, int nslots, const int32_t *slots,
                         const float *w, int T, int k, int d, int f, float *y, void *ws, hipStream_t s)
{
    TokParams p{};
    p.x = x;
    p.pool = pool;
    p.slab_stride = stride;
    p.slots = slots;
    p.w = w;
    p.T = T;
    p.k = k;
    p.nslots = nslots;
    p.d = d;
    p.f = f;
    p.nseg = seg_count_tok(f);
    p.seg = seg_len_tok(f);
    p.h = static_cast<float *>(ws);
    p.partial = reinterpret_cast<float *>(static_cast<uint8_t *>(ws) + a256((size_t)T * k * f * sizeof(float)));
    const int max_jobs = T * k < nslots ? T * k : nslots;
    hipError_t e;
    // gate/up: grid-stride over (job, row), one round of resident work groups
    const int cpl = (d / 8 + kWave - 1) / kWave;
    const size_t lds_x = (size_t)T * d * sizeof(float);
    const int gu_grid = 0;
    switch (cpl) {
#define MOE_TOK_CPL(N) \
    case N: e = launch_dyn(k_tok_gate_up<N>, gu_grid, lds_x, s, p); break;
        MOE_TOK_CPL(1) MOE_TOK_CPL(2) MOE_TOK_CPL(3) MOE_TOK_CPL(4) MOE_TOK_CPL(5) MOE_TOK_CPL(6)
        MOE_TOK_CPL(7) MOE_TOK_CPL(8) MOE_TOK_CPL(9) MOE_TOK_CPL(10) MOE_TOK_CPL(11) MOE_TOK_CPL(12)
        MOE_TOK_CPL(13) MOE_TOK_CPL(14) MOE_TOK_CPL(15) MOE_TOK_CPL(16)
#undef MOE_TOK_CPL
    default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    // down: one work group per (job, segment, kDownRows rows); groups past the job count exit
    const int nchunk = (d + kDownRows - 1) / kDownRows;
    const int dn_grid = max_jobs * p.nseg * nchunk;
    const size_t lds_h = (size_t)T * p.seg * sizeof(float);
    const int cpk = (p.seg / 8 + kWave - 1) / kWave;
    if (dn_grid > 0) {
        switch (cpk) {
#define MOE_TOK_CPK(N) \
    case N: e = launch_dyn(k_tok_down<N>, dn_grid, lds_h, s, p); break;
            MOE_TOK_CPK(1) MOE_TOK_CPK(2) MOE_TOK_CPK(3) MOE_TOK_CPK(4) MOE_TOK_CPK(5) MOE_TOK_CPK(6)
            MOE_TOK_CPK(7) MOE_TOK_CPK(8)
#undef MOE_TOK_CPK
        default: return hipErrorInvalidValue;
        }
        if (e != hipSuccess) return e;
    }
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_tok_reduce, dim3((d + 255) / 256, T), dim3(256), 0, s, p, y);
    return hipGetLastError();
}

}  // namespace moe

extern "C" {

size_t moe_ffn_tokens_workspace_bytes(int T, int k, int d, int f)
{
    if (T < 1 || k < 1 || d <= 0 || f <= 0) return 0;
    return moe::tok_workspace_bytes(T, k, d, f);
}

int moe_expert_ffn_tokens(const float *x, const void *slot_pool, int n_slots, const int32_t *slots, const float *w,
                          int T, int k, int d, int f, float *y, void *workspace, size_t workspace_bytes, void *stream)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(T >= 1 && T <= MOE_MAX_TOKENS, "moe_expert_ffn_tokens: T=%d out of [1,%d]", T, MOE_MAX_TOKENS);
    MOE_REQUIRE(k >= 1 && k <= MOE_MAX_TOPK, "moe_expert_ffn_tokens: k=%d out of [1,%d]", k, MOE_MAX_TOPK);
    MOE_REQUIRE(d > 0 && d % 8 == 0 && d <= MOE_MAX_D, "moe_expert_ffn_tokens: d=%d must be a multiple of 8 in [8,%d]",
                d, MOE_MAX_D);
    MOE_REQUIRE(f > 0 && f % 8 == 0, "moe_expert_ffn_tokens: f=%d must be a positive multiple of 8", f);
    MOE_REQUIRE((size_t)T * d * sizeof(float) <= (size_t)MOE_TOKENS_LDS_BYTES,
                "moe_expert_ffn_tokens: T*d=%d floats exceed the %d-byte staging of the hidden states", T * d,
                MOE_TOKENS_LDS_BYTES);
    MOE_REQUIRE(n_slots >= 0, "moe_expert_ffn_tokens: n_slots=%d < 0", n_slots);
    MOE_REQUIRE(x && slots && w && y && workspace && (slot_pool || n_slots == 0),
                "moe_expert_ffn_tokens: null pointer");
    MOE_REQUIRE(moe::aligned16(x) && moe::aligned16(y) && (!slot_pool || moe::aligned16(slot_pool)),
                "moe_expert_ffn_tokens: x, y and slot_pool must be 16-byte aligned");
    MOE_REQUIRE(((uintptr_t)workspace & 255u) == 0, "moe_expert_ffn_tokens: workspace not 256-byte aligned");
    const size_t need = moe::tok_workspace_bytes(T, k, d, f);
    MOE_REQUIRE(workspace_bytes >= need, "moe_expert_ffn_tokens: workspace %zu < %zu bytes", workspace_bytes, need);
    MOE_HIP(moe::launch_tokens(x, static_cast<const uint8_t *>(slot_pool), moe_slab_bytes(d, f), n_slots, slots, w,
                               T, k, d, f, y, workspace, (hipStream_t)stream));
    return MOE_OK;
    MOE_GUARD_END
}

}  // extern "C"
