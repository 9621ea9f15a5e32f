// Prefill MoE layer: T tokens through one layer with every expert resident.
//
// Steps (each a kernel on one stream):
//   1. router for all T tokens (the decode router kernel, one block per token);
//   2. grouping: a stable counting sort of the T*k (token, rank) pairs by expert,
//      giving per-expert offsets, the sorted pair list and its inverse;
//   3. hidden states rounded to bf16 for the matrix cores;
//   4. grouped GEMM gate/up: for each expert e, H_e = SiLU(X_e W1_e^T) * (X_e W3_e^T),
//      bf16 MFMA (v_mfma_f32_32x32x16_bf16) with fp32 accumulation, H_e stored bf16;
//   5. grouped GEMM down: Y_e = H_e W2_e^T, split in two along f, fp32 partials;
//   6. combine: OUT[t] = sum_r w[t][r] * Y[pair(t, r)], in a fixed order.
//
// Both GEMM operands are K-contiguous rows (token rows of X or H, weight rows of W), so
// every lane's MFMA operand is one 16-byte run of a row. Tiles are staged through LDS
// with a register prefetch of the next K step. Work items (expert, M tile, N tile,
// K split) are laid out so that every item of one expert lands on the same XCD (work
// group b runs on XCD b mod 8) and the M tiles sharing a weight tile run back to back,
// so a weight tile is fetched from HBM once and re-read from that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kBM = 128;        // tokens per tile
constexpr int kBK = 64;         // K per stage
constexpr int kBRows = 128;     // weight rows per tile (gate/up: 64 of W1 + 64 of W3)
constexpr int kLdsStride = kBK + 8;   // bf16 per LDS row (16-byte pad against bank conflicts)
constexpr int kXcds = 8;
constexpr int kDownSplits = 2;

__device__ __forceinline__ uint16_t f2bf(float f)
{
    // round to nearest even (inputs are finite)
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__global__ __launch_bounds__(kThreads) void k_cast_bf16(const float *x, uint16_t *y, int64_t n8)
{
    for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < n8; i += (int64_t)gridDim.x * kThreads) {
        const float4 a = reinterpret_cast<const float4 *>(x)[2 * i];
        const float4 b = reinterpret_cast<const float4 *>(x)[2 * i + 1];
        uint4 o;
        o.x = f2bf(a.x) | ((uint32_t)f2bf(a.y) << 16);
        o.y = f2bf(a.z) | ((uint32_t)f2bf(a.w) << 16);
        o.z = f2bf(b.x) | ((uint32_t)f2bf(b.y) << 16);
        o.w = f2bf(b.z) | ((uint32_t)f2bf(b.w) << 16);
        reinterpret_cast<uint4 *>(y)[i] = o;
    }
}

// Stable counting sort of the pairs p = t*k + r by expert idx[p] (one block).
// off[e] .. off[e+1] is expert e's range in `perm` (pair ids in increasing order);
// pos[p] is the place of pair p in that order.
constexpr int kGroupChunk = 8192;
__global__ __launch_bounds__(kThreads) void k_group(const int32_t *idx, int npairs, int n, int32_t *off,
                                                    int32_t *perm, int32_t *pos)
{
    __shared__ uint8_t ids[kGroupChunk];
    __shared__ int32_t cnt[kThreads + 1];
    const int e = threadIdx.x;
    int c = 0;
    for (int base = 0; base < npairs; base += kGroupChunk) {
        const int m = min(kGroupChunk, npairs - base);
        __syncthreads();
        for (int i = threadIdx.x; i < m; i += kThreads) ids[i] = (uint8_t)idx[base + i];
        __syncthreads();
        if (e < n)
            for (int i = 0; i < m; ++i) c += (ids[i] == e);
    }
    cnt[e] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        int acc = 0;
        for (int q = 0; q < n; ++q) {
            const int v = cnt[q];
            cnt[q] = acc;
            off[q] = acc;
            acc += v;
        }
        off[n] = acc;
    }
    __syncthreads();
    int w = cnt[e];
    for (int base = 0; base < npairs; base += kGroupChunk) {
        const int m = min(kGroupChunk, npairs - base);
        __syncthreads();
        for (int i = threadIdx.x; i < m; i += kThreads) ids[i] = (uint8_t)idx[base + i];
        __syncthreads();
        if (e < n)
            for (int i = 0; i < m; ++i)
                if (ids[i] == e) {
                    perm[w] = base + i;
                    pos[base + i] = w;
                    ++w;
                }
    }
}

struct GemmArgs {
    const uint16_t *a;        // gate/up: X bf16 [T][d] (rows gathered by token); down: H bf16 [P][f]
    const uint8_t *pool;      // expert slabs
    uint64_t slab_stride;
    const int32_t *off;       // [n+1]
    const int32_t *perm;      // [P] pair ids sorted by expert
    int n, k, d, f;
    int mtiles;               // M tiles per expert (upper bound)
    int ntiles;               // N tiles per matrix
    int ksplit;               // K splits
    int per_xcd;              // work items per XCD
    uint16_t *h;              // gate/up output, bf16 [P][f]
    float *yp;                // down output, fp32 [ksplit][P][d]
};

// Grouped GEMM, one 128 x 128 output tile per work group (gate/up: 128 tokens x
// (64 gate + 64 up) rows; down: 128 tokens x 128 output rows), 4 waves as 2 x 2.
template <bool kGateUp>
__global__ __launch_bounds__(kThreads) void k_group_gemm(GemmArgs g)
{
    __shared__ uint16_t lds_a[2][kBM * kLdsStride];
    __shared__ uint16_t lds_b[2][kBRows * kLdsStride];

    // work item -> (expert, m tile, n tile, k split); all items of an expert on one XCD
    const int xcd = blockIdx.x % kXcds;
    int q = blockIdx.x / kXcds;
    if (q >= g.per_xcd) return;
    const int per_expert = g.mtiles * g.ntiles * g.ksplit;
    const int e = xcd + kXcds * (q / per_expert);
    if (e >= g.n) return;
    q %= per_expert;
    const int ks = q % g.ksplit;
    q /= g.ksplit;
    const int mt = q % g.mtiles;
    const int nt = q / g.mtiles;
    const int row0 = g.off[e] + mt * kBM;          // first pair row of this tile
    const int rows = min(kBM, g.off[e + 1] - row0);
    if (rows <= 0) return;

    const int K = kGateUp ? g.d : g.f;
    const int kspan = K / g.ksplit;
    const int k0 = ks * kspan;
    const int nsteps = kspan / kBK;
    const uint8_t *slab = g.pool + (uint64_t)e * g.slab_stride;
    const int tid = threadIdx.x;

    // Global sources of the 4 A chunks and 4 B chunks this thread stages per step
    // (chunk c = tid + 256 i: row c / 8, 16-byte column c % 8).
    const uint16_t *asrc[4];
    const uint16_t *bsrc[4];
    bool avalid[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int c = tid + kThreads * i;
        const int r = c >> 3, col = (c & 7) * 8;
        avalid[i] = r < rows;
        const int rr = avalid[i] ? r : 0;
        if (kGateUp) {
            const int token = g.perm[row0 + rr] / g.k;
            asrc[i] = g.a + (size_t)token * g.d + k0 + col;
            const uint16_t *w = reinterpret_cast<const uint16_t *>(slab);
            const int wrow = nt * 64 + (r & 63);
            bsrc[i] = (r < 64) ? w + (size_t)wrow * g.d + k0 + col
                               : w + (size_t)g.f * g.d + (size_t)wrow * g.d + k0 + col;
        } else {
            asrc[i] = g.a + (size_t)(row0 + rr) * g.f + k0 + col;
            const uint16_t *w2 = reinterpret_cast<const uint16_t *>(slab) + (size_t)2 * g.f * g.d;
            bsrc[i] = w2 + (size_t)(nt * kBRows + r) * g.f + k0 + col;
        }
    }

    u32x4_t ra[4], rb[4];
#define MOE_FETCH1(i, ko)                                                                                 \
    ra[i] = avalid[i] ? *reinterpret_cast<const u32x4_t *>(asrc[i] + (ko)) : u32x4_t{0, 0, 0, 0};       \
    rb[i] = *reinterpret_cast<const u32x4_t *>(bsrc[i] + (ko));
#define MOE_FETCH(step)                                                                                   \
    do {                                                                                                  \
        const int ko_ = (step) * kBK;                                                                     \
        MOE_FETCH1(0, ko_) MOE_FETCH1(1, ko_) MOE_FETCH1(2, ko_) MOE_FETCH1(3, ko_)                       \
    } while (0)
#define MOE_STASH1(i, buf)                                                                                \
    {                                                                                                     \
        const int c_ = tid + kThreads * (i);                                                              \
        const int o_ = (c_ >> 3) * kLdsStride + (c_ & 7) * 8;                                             \
        *reinterpret_cast<u32x4_t *>(&lds_a[(buf)][o_]) = ra[i];                                          \
        *reinterpret_cast<u32x4_t *>(&lds_b[(buf)][o_]) = rb[i];                                          \
    }
#define MOE_STASH(buf)                                                                                    \
    do {                                                                                                  \
        MOE_STASH1(0, buf) MOE_STASH1(1, buf) MOE_STASH1(2, buf) MOE_STASH1(3, buf)                       \
    } while (0)

    const int lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    // B rows of this wave: gate/up -> gate rows wn*32.. and up rows 64+wn*32..;
    // down -> rows wn*64 .. +64 (two 32-row blocks).
    const int brow0 = kGateUp ? wn * 32 : wn * 64;
    const int brow1 = kGateUp ? 64 + wn * 32 : wn * 64 + 32;
    floatx16_t acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    MOE_FETCH(0);
    MOE_STASH(0);
    __syncthreads();
    for (int s = 0; s < nsteps; ++s) {
        const int buf = s & 1;
        if (s + 1 < nsteps) MOE_FETCH(s + 1);
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int kc = kk * 16 + 8 * (lane >> 5);
            bf16x8_t af[2], bfr[2];
#pragma unroll
            for (int a = 0; a < 2; ++a)
                af[a] = *reinterpret_cast<const bf16x8_t *>(&lds_a[buf][(wm * 64 + a * 32 + (lane & 31)) * kLdsStride + kc]);
            bfr[0] = *reinterpret_cast<const bf16x8_t *>(&lds_b[buf][(brow0 + (lane & 31)) * kLdsStride + kc]);
            bfr[1] = *reinterpret_cast<const bf16x8_t *>(&lds_b[buf][(brow1 + (lane & 31)) * kLdsStride + kc]);
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
        }
        if (s + 1 < nsteps) {
            MOE_STASH(buf ^ 1);
            __syncthreads();
        }
    }
#undef MOE_FETCH
#undef MOE_FETCH1
#undef MOE_STASH
#undef MOE_STASH1

    // Epilogue. Output element r of a 32x32 block sits at row 8*(r/4) + 4*(lane/32) + r%4,
    // column lane%32.
#pragma unroll
    for (int a = 0; a < 2; ++a) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int tr = wm * 64 + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (tr >= rows) continue;
            const size_t prow = (size_t)(row0 + tr);
            if (kGateUp) {
                const float gv = acc[a][0][r], uv = acc[a][1][r];
                const float hv = gv / (1.0f + expf(-gv)) * uv;
                g.h[prow * g.f + nt * 64 + wn * 32 + (lane & 31)] = f2bf(hv);
            } else {
                const int P = g.off[g.n];
                float *dst = g.yp + ((size_t)ks * P + prow) * g.d + nt * kBRows;
                dst[wn * 64 + (lane & 31)] = acc[a][0][r];
                dst[wn * 64 + 32 + (lane & 31)] = acc[a][1][r];
            }
        }
    }
}

// OUT[t][i] = sum_r w[t][r] * sum_s Yp[s][pos[t*k+r]][i]
__global__ __launch_bounds__(kThreads) void k_prefill_combine(const float *yp, const int32_t *pos, const float *w,
                                                              int k, int d, int P, int ksplit, float *out)
{
    const int t = blockIdx.x;
    for (int i = threadIdx.x; i < d; i += kThreads) {
        float acc = 0.f;
        for (int r = 0; r < k; ++r) {
            const int pr = pos[t * k + r];
            float s = 0.f;
            for (int q = 0; q < ksplit; ++q) s += yp[((size_t)q * P + pr) * d + i];
            acc = fmaf(w[t * k + r], s, acc);
        }
        out[(size_t)t * d + i] = acc;
    }
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

struct PrefillWs {
    uint16_t *xb;
    int32_t *idx, *off, *perm, *pos;
    float *w;
    uint16_t *h;
    float *yp;
};

size_t layout(int d, int f, int n, int k, int T, uint8_t *base, PrefillWs *ws)
{
    const size_t P = (size_t)T * k;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align256(bytes);
        return base ? base + at : nullptr;
    };
    uint8_t *xb = take((size_t)T * d * 2);
    uint8_t *idx = take(P * 4);
    uint8_t *w = take(P * 4);
    uint8_t *off = take((size_t)(n + 1) * 4);
    uint8_t *perm = take(P * 4);
    uint8_t *pos = take(P * 4);
    uint8_t *h = take(P * f * 2);
    uint8_t *yp = take((size_t)kDownSplits * P * d * 4);
    if (ws) {
        ws->xb = reinterpret_cast<uint16_t *>(xb);
        ws->idx = reinterpret_cast<int32_t *>(idx);
        ws->w = reinterpret_cast<float *>(w);
        ws->off = reinterpret_cast<int32_t *>(off);
        ws->perm = reinterpret_cast<int32_t *>(perm);
        ws->pos = reinterpret_cast<int32_t *>(pos);
        ws->h = reinterpret_cast<uint16_t *>(h);
        ws->yp = reinterpret_cast<float *>(yp);
    }
    return o;
}

}  // namespace

size_t prefill_workspace_bytes(int d, int f, int n, int k, int T) { return layout(d, f, n, k, T, nullptr, nullptr); }

hipError_t launch_prefill(const PrefillPlan &P, const float *X, float *OUT, int32_t *idx, float *w, void *wsp,
                          hipStream_t s)
{
    PrefillWs ws{};
    layout(P.d, P.f, P.n, P.k, P.T, static_cast<uint8_t *>(wsp), &ws);
    int32_t *idx_d = idx ? idx : ws.idx;
    float *w_d = w ? w : ws.w;
    hipError_t e;
    if ((e = launch_router(X, P.wr, P.T, P.d, P.n, P.k, idx_d, w_d, s)) != hipSuccess) return e;
    const int npairs = P.T * P.k;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_group, dim3(1), dim3(kThreads), 0, s, idx_d, npairs, P.n, ws.off, ws.perm, ws.pos);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t n8 = (int64_t)P.T * P.d / 8;
    const int cast_blocks = (int)std::min<int64_t>((n8 + kThreads - 1) / kThreads, 4096);
    hipLaunchKernelGGL(k_cast_bf16, dim3(cast_blocks), dim3(kThreads), 0, s, X, ws.xb, n8);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    GemmArgs g{};
    g.pool = P.pool;
    g.slab_stride = P.slab_stride;
    g.off = ws.off;
    g.perm = ws.perm;
    g.n = P.n;
    g.k = P.k;
    g.d = P.d;
    g.f = P.f;
    g.mtiles = (P.T + kBM - 1) / kBM;
    g.h = ws.h;
    g.yp = ws.yp;
    const int groups = (P.n + kXcds - 1) / kXcds;

    // gate/up: N tiles of 64 rows per matrix over f, K = d
    g.a = ws.xb;
    g.ntiles = P.f / 64;
    g.ksplit = 1;
    g.per_xcd = groups * g.mtiles * g.ntiles * g.ksplit;
    hipLaunchKernelGGL(k_group_gemm<true>, dim3(kXcds * g.per_xcd), dim3(kThreads), 0, s, g);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    // down: N tiles of 128 output rows over d, K = f split in two
    g.a = ws.h;
    g.ntiles = P.d / kBRows;
    g.ksplit = kDownSplits;
    g.per_xcd = groups * g.mtiles * g.ntiles * g.ksplit;
    hipLaunchKernelGGL(k_group_gemm<false>, dim3(kXcds * g.per_xcd), dim3(kThreads), 0, s, g);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    hipLaunchKernelGGL(k_prefill_combine, dim3(P.T), dim3(kThreads), 0, s, ws.yp, ws.pos, w_d, P.k, P.d, npairs,
                       kDownSplits, OUT);
    return hipGetLastError();
}

}  // namespace moe

extern "C" {

size_t moe_prefill_workspace_bytes(const moe_prefill_desc *P, int T)
{
    if (!P || T < 0 || P->d <= 0 || P->f <= 0 || P->n <= 0 || P->k <= 0) return 0;
    return moe::prefill_workspace_bytes(P->d, P->f, P->n, P->k, T);
}

int moe_prefill_forward(const moe_prefill_desc *P, const float *X_dev, int T, float *OUT_dev, int32_t *idx_dev,
                        float *w_dev, void *workspace, size_t workspace_bytes, void *stream)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(P, "moe_prefill_forward: null descriptor");
    MOE_REQUIRE(T >= 0, "moe_prefill_forward: T=%d < 0", T);
    MOE_REQUIRE(P->d > 0 && P->d % 128 == 0 && P->d <= MOE_MAX_D,
                "moe_prefill_forward: d=%d must be a multiple of 128 in [128,%d]", P->d, MOE_MAX_D);
    MOE_REQUIRE(P->f > 0 && P->f % 128 == 0, "moe_prefill_forward: f=%d must be a positive multiple of 128", P->f);
    MOE_REQUIRE(P->n >= 1 && P->n <= MOE_MAX_EXPERTS, "moe_prefill_forward: n=%d out of range", P->n);
    MOE_REQUIRE(P->k >= 1 && P->k <= P->n && P->k <= MOE_MAX_TOPK, "moe_prefill_forward: k=%d out of range", P->k);
    if (T == 0) return MOE_OK;
    MOE_REQUIRE(X_dev && OUT_dev && workspace && P->w_router && P->expert_pool, "moe_prefill_forward: null pointer");
    MOE_REQUIRE(moe::aligned16(X_dev) && moe::aligned16(OUT_dev) && moe::aligned16(P->w_router) &&
                    moe::aligned16(P->expert_pool),
                "moe_prefill_forward: device pointers must be 16-byte aligned");
    MOE_REQUIRE(((uintptr_t)workspace & 255u) == 0, "moe_prefill_forward: workspace not 256-byte aligned");
    const size_t need = moe::prefill_workspace_bytes(P->d, P->f, P->n, P->k, T);
    MOE_REQUIRE(workspace_bytes >= need, "moe_prefill_forward: workspace %zu < %zu bytes", workspace_bytes, need);
    moe::PrefillPlan plan{};
    plan.d = P->d;
    plan.f = P->f;
    plan.n = P->n;
    plan.k = P->k;
    plan.T = T;
    plan.wr = P->w_router;
    plan.pool = static_cast<const uint8_t *>(P->expert_pool);
    plan.slab_stride = moe_slab_bytes(P->d, P->f);
    MOE_HIP(moe::launch_prefill(plan, X_dev, OUT_dev, idx_dev, w_dev, workspace, (hipStream_t)stream));
    return MOE_OK;
    MOE_GUARD_END
}

}  // extern "C"
