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
//
// Each wave dots one weight row with several tokens, so the arithmetic per byte grows
// with the tokens per slab. The hidden states are staged as two bf16 parts, hi = bf16(v)
// and lo = bf16(v - hi) (|v - hi - lo| <= 2^-18 |v|), so that a 16-byte chunk of bf16
// weights meets them through v_dot2_f32_bf16 (exact bf16 products, fp32 sums) without
// widening the weights to fp32 once per token.
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
static_assert(kMaxPairs <= 2 * kWave, "a wave keeps a job's pair results in two registers");

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// c + a[0] b[0] + a[1] b[1] over two packed bf16 pairs (element 0 in the low half)
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c, false);
}

// acc + dot(8 bf16 weights, 8 bf16 activation parts)
__device__ __forceinline__ float dot8_bf(const uint4 w, const uint4 v, float acc)
{
    acc = dot2(w.x, v.x, acc);
    acc = dot2(w.y, v.y, acc);
    acc = dot2(w.z, v.z, acc);
    return dot2(w.w, v.w, acc);
}

// Sum over the 64 lanes of a wave, returned to every lane. Cross-lane moves use DPP
// (quad permutes, row mirrors, then row broadcasts of lanes 15 and 31, leaving the total
// in lane 63): VALU operations, where a shuffle butterfly would make six dependent
// round trips through the LDS crossbar per sum. Fixed order, so deterministic.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float add_dpp(float v)
{
    // lanes of rows outside kRowMask add the `old` operand, 0
    const int t = __builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, kRowMask, 0xF, false);
    return v + __int_as_float(t);
}

__device__ __forceinline__ float wave_total(float v)
{
    v = add_dpp<0xB1, 0xF>(v);    // quad_perm [1,0,3,2]: pairs
    v = add_dpp<0x4E, 0xF>(v);    // quad_perm [2,3,0,1]: quads
    v = add_dpp<0x141, 0xF>(v);   // row_half_mirror: 8 lanes
    v = add_dpp<0x140, 0xF>(v);   // row_mirror: the 16 lanes of a row
    v = add_dpp<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3: rows 0+1, 2+3
    v = add_dpp<0x143, 0xC>(v);   // row_bcast:31 into rows 2 and 3: lane 63 holds the total
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ uint32_t bf_bits(__bf16 v) { return __builtin_bit_cast(uint16_t, v); }

// (a, b) -> packed hi parts and packed lo parts, both rounded to nearest even
__device__ __forceinline__ void split2(float a, float b, uint32_t &hi, uint32_t &lo)
{
    const __bf16 ah = static_cast<__bf16>(a), bh = static_cast<__bf16>(b);
    const __bf16 al = static_cast<__bf16>(a - static_cast<float>(ah));
    const __bf16 bl = static_cast<__bf16>(b - static_cast<float>(bh));
    hi = bf_bits(ah) | (bf_bits(bh) << 16);
    lo = bf_bits(al) | (bf_bits(bl) << 16);
}

// 8 consecutive fp32 values -> one chunk of hi parts and one of lo parts
__device__ __forceinline__ void split8(const float *src, uint4 *hi, uint4 *lo)
{
    const float4 v0 = reinterpret_cast<const float4 *>(src)[0];
    const float4 v1 = reinterpret_cast<const float4 *>(src)[1];
    uint4 h, l;
    split2(v0.x, v0.y, h.x, l.x);
    split2(v0.z, v0.w, h.y, l.y);
    split2(v1.x, v1.y, h.z, l.z);
    split2(v1.z, v1.w, h.w, l.w);
    *hi = h;
    *lo = l;
}

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
    constexpr int kPitch = CPL * kWave;   // chunks per token row in LDS
    __shared__ TokJobs J;
    extern __shared__ uint4 xs4[];        // hi parts [T][kPitch], then lo parts [T][kPitch]
    build_jobs(p.slots, p.T * p.k, p.nslots, J);
    const int d = p.d, nch = d >> 3, lo_off = p.T * kPitch;
    // chunks past d/8 hold zeros: a lane's last chunk, whose weights are re-read from the
    // row's last chunk, then adds nothing, and every chunk is dotted without a branch
    for (int i = threadIdx.x; i < lo_off; i += kTokThreads) {
        const int t = i / kPitch, e = i - t * kPitch;
        if (e < nch) split8(p.x + (size_t)t * d + e * 8, xs4 + i, xs4 + lo_off + i);
        else xs4[i] = xs4[lo_off + i] = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();

    const int lane = threadIdx.x & (kWave - 1);
    const int nwaves = gridDim.x * kTokWaves;
    const int total = J.njobs * p.f;
    // Two register sets: the next row pair is in flight while this one is dotted with
    // the tokens. Loads are unconditional (past the end they re-read the last row pair)
    // so that each wait covers only the older set. Every path through the dot reads every
    // register of its set (a do-while over the pairs, no per-chunk branch): a register left
    // unread on some path, or a loop that stores to global memory while reading registers
    // still being loaded, makes the compiler wait for every outstanding load, the
    // prefetched set included. Lane j keeps the result of the job's pair j (j + 64 in h1_)
    // and the stores follow the pair loop.
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
        const bool live_ = (item) < total;                                                             \
        const int it_ = min((item), total - 1);                                                        \
        const int job_ = it_ / p.f, i_ = it_ - job_ * p.f;                                              \
        const int q0_ = J.first[job_], nq_ = live_ ? J.first[job_ + 1] - q0_ : 1;                      \
        float h0_ = 0.f, h1_ = 0.f;                                                                    \
        int q = 0;                                                                                     \
        do {                                                                                           \
            const uint4 *xt = xs4 + (J.pair[q0_ + q] / p.k) * kPitch + lane;                           \
            float gh = 0.f, gl = 0.f, uh = 0.f, ul = 0.f;                                              \
            _Pragma("unroll") for (int c = 0; c < CPL; ++c) {                                          \
                const uint4 xh = xt[c * kWave], xl = xt[lo_off + c * kWave];                           \
                gh = dot8_bf(a[set][c], xh, gh);                                                       \
                gl = dot8_bf(a[set][c], xl, gl);                                                       \
                uh = dot8_bf(b[set][c], xh, uh);                                                       \
                ul = dot8_bf(b[set][c], xl, ul);                                                       \
            }                                                                                          \
            const float g = wave_total(gh + gl);                                                         \
            const float u = wave_total(uh + ul);                                                         \
            const float hv = g / (1.0f + expf(-g)) * u;                                                \
            if (lane == (q & (kWave - 1))) {                                                           \
                if (q < kWave) h0_ = hv;                                                               \
                else h1_ = hv;                                                                         \
            }                                                                                          \
        } while (++q < nq_);   /* a job has at least one pair */                                       \
        const int ns_ = live_ ? nq_ : 0;                                                               \
        if (lane < ns_) p.h[(size_t)J.pair[q0_ + lane] * p.f + i_] = h0_;                              \
        if (lane + kWave < ns_) p.h[(size_t)J.pair[q0_ + kWave + lane] * p.f + i_] = h1_;              \
    } while (0)

    // The loop control is uniform (the wave index through readfirstlane) and has no exit
    // between the halves: an item past the end in the second half is dotted (one pair,
    // the loaded last row) but not stored. A mid-loop exit, or a divergent one, is a path
    // to the loop head that skips the second dot, and the compiler would again wait for
    // both sets there.
    int it = blockIdx.x * kTokWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (it < total) MOE_TOK_LOAD(0, it);
    for (; it < total; it += 2 * nwaves) {
        MOE_TOK_LOAD(1, it + nwaves);
        MOE_TOK_DOT(0, it);
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
    constexpr int kPitch = CPK * kWave;   // chunks per staged pair row in LDS
    __shared__ TokJobs J;
    extern __shared__ uint4 hs4[];        // hi parts [T][kPitch], then lo parts [T][kPitch]
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
    const int lo_off = p.T * kPitch;
    const int lane = threadIdx.x & (kWave - 1);
    const uint8_t *w2 = p.pool + (uint64_t)J.slot[job] * p.slab_stride + (uint64_t)2 * p.f * p.d * 2;
    const int r1 = min(r0 + kDownRows, p.d);
    // LDS holds the h segments of T pairs; a job has at most T (one per token) unless a
    // token listed a slot twice, and then its pairs go through in groups of T.
    for (int qc = 0; qc < np; qc += p.T) {
        const int nq = min(p.T, np - qc);
        if (qc) __syncthreads();   // the previous group's segments are no longer read
        // chunks past the segment's end hold zeros (see k_tok_gate_up)
        for (int i = threadIdx.x; i < nq * kPitch; i += kTokThreads) {
            const int q = i / kPitch, e = i - q * kPitch;
            if (e < nch) split8(p.h + (size_t)J.pair[q0 + qc + q] * p.f + c0 + e * 8, hs4 + i, hs4 + lo_off + i);
            else hs4[i] = hs4[lo_off + i] = make_uint4(0, 0, 0, 0);
        }
        __syncthreads();
        // lane q < nq holds pair q's id and combine weight, and keeps its dot product;
        // the stores follow the pair loop (see k_tok_gate_up)
        const int pr_l = lane < nq ? J.pair[q0 + qc + lane] : 0;
        const float w_l = lane < nq ? p.w[pr_l] : 0.f;
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
            const bool live_ = (rr) < r1;                                                              \
            const int nl_ = live_ ? nq : 1;                                                            \
            float o_ = 0.f;                                                                            \
            int q = 0;                                                                                 \
            do {                                                                                       \
                const uint4 *ht = hs4 + q * kPitch + lane;                                             \
                float ah = 0.f, al = 0.f;                                                              \
                _Pragma("unroll") for (int c = 0; c < CPK; ++c) {                                      \
                    ah = dot8_bf(a[set][c], ht[c * kWave], ah);                                        \
                    al = dot8_bf(a[set][c], ht[lo_off + c * kWave], al);                               \
                }                                                                                      \
                const float acc = wave_total(ah + al);                                                   \
                if (lane == q) o_ = acc;                                                               \
            } while (++q < nl_);                                                                       \
            if (live_ && lane < nq) p.partial[((size_t)pr_l * p.nseg + sgi) * p.d + (rr)] = w_l * o_;  \
        } while (0)
        // uniform loop control without a mid-loop exit; a row past the end is dotted with
        // one pair and not stored (see k_tok_gate_up)
        int r = r0 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        if (r < r1) MOE_TOK_LOAD_ROW(0, r);
        for (; r < r1; r += 2 * kTokWaves) {
            MOE_TOK_LOAD_ROW(1, r + kTokWaves);
            MOE_TOK_DOT_ROW(0, r);
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
    // T rows of cpl * 64 chunks, each chunk 16 bytes of hi parts and 16 of lo parts
    const size_t lds_x = (size_t)T * cpl * kWave * 32;
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
    const int cpk = (p.seg / 8 + kWave - 1) / kWave;
    const size_t lds_h = (size_t)T * cpk * kWave * 32;
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
