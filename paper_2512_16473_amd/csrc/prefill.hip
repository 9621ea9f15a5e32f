// Prefill MoE layer: T tokens through one layer with every expert resident.
//
// Steps (each a kernel on one stream):
//   1. router for all T tokens (the decode router kernel, one block per token);
//   2. grouping: a stable counting sort of the T*k (token, rank) pairs by expert,
//      giving per-expert offsets, the sorted pair list and its inverse;
//   3. hidden states rounded to bf16 for the matrix cores (other blocks of the grouping
//      launch: it does not depend on the routing);
//   4. grouped GEMM gate/up: for each expert e, H_e = SiLU(X_e W1_e^T) * (X_e W3_e^T),
//      bf16 MFMA (v_mfma_f32_16x16x32_bf16) with fp32 accumulation, H_e stored bf16; the
//      tiles of a last, partial round of work groups are split over K, and
//   4b. a small kernel adds their parts and applies SiLU * up;
//   5. grouped GEMM down: Y_e = H_e W2_e^T, K split in four (or two), fp32 partials;
//   6. combine: OUT[t] = sum_r w[t][r] * Y[pair(t, r)], in a fixed order.
//
// With about T k / n tokens per expert (128 for a 512-token prompt on 8 experts, top-2)
// the GEMMs are bound by reading the expert weights from HBM, so the kernel is built to
// keep many weight bytes in flight: each wave loads its own weight rows into registers,
// several K steps ahead, with whole cache lines per load instruction, and only the token
// tile is shared through LDS.
// Work items (expert, M tile, N tile, K split) are laid out so that every item of one
// expert lands on the same XCD (work group b runs on XCD b mod 8), where its token rows
// stay in that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>

#include "common.h"
#include "moe_internal.h"

namespace moe {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kBK = 64;         // K per stage
constexpr int kLdsStride = kBK + 8;   // bf16 per LDS row (16-byte pad against bank conflicts)
constexpr int kRowChunks = kBK / 8;  // 16-byte chunks of a token row per step
constexpr int kXcds = 8;
constexpr int kSpreadTokens = 64;   // below this many (token, expert) pairs per expert, spread items over XCDs
constexpr int kMaxDownSplits = 4;
constexpr int kMaxTailSlots = 32;   // gate/up tail: work groups per XCD the split tiles may use
constexpr int kMaxTailSplit = 16;   // gate/up tail: K parts per split tile

__device__ __forceinline__ uint16_t f2bf(float f)
{
    // round to nearest even (inputs are finite)
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// y = bf16(x) over n8 groups of 8 values; `first`, `stride`: this thread's first group
// and the step between its groups.
__device__ __forceinline__ void cast_bf16(const float *x, uint16_t *y, int64_t n8, int64_t first, int64_t stride)
{
    for (int64_t i = first; i < n8; i += stride) {
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

// Block 0: the grouping below. Blocks 1 ..: the hidden states rounded to bf16 for the
// matrix cores (independent of the routing, so the two share one launch).
// Stable counting sort of the pairs p = t*k + r by expert idx[p] (one block).
// off[e] .. off[e+1] is expert e's range in `perm` (pair ids in increasing order);
// pos[p] is the place of pair p in that order. The per-expert counts come from LDS
// atomics; the place of a pair within its expert is the number of earlier pairs with
// the same expert, counted over the chunk's ids in LDS four at a time.
constexpr int kGroupThreads = 1024;
__global__ __launch_bounds__(kGroupThreads) void k_group(const int32_t *idx, int npairs, int n, int32_t *off,
                                                         int32_t *perm, int32_t *pos, const float *x, uint16_t *xb,
                                                         int64_t n8)
{
    if (blockIdx.x > 0) {
        cast_bf16(x, xb, n8, (int64_t)(blockIdx.x - 1) * kGroupThreads + threadIdx.x,
                  (int64_t)(gridDim.x - 1) * kGroupThreads);
        return;
    }
    __shared__ int32_t base[MOE_MAX_EXPERTS];    // counts, then the next free place of each expert
    __shared__ int32_t hist[MOE_MAX_EXPERTS];
    __shared__ uint32_t ids32[kGroupThreads / 4];
    uint8_t *ids = reinterpret_cast<uint8_t *>(ids32);
    const int t = threadIdx.x;
    for (int e = t; e < n; e += kGroupThreads) base[e] = 0;
    __syncthreads();
    for (int p = t; p < npairs; p += kGroupThreads) atomicAdd(&base[idx[p]], 1);
    __syncthreads();
    if (t == 0) {
        int acc = 0;
        for (int e = 0; e < n; ++e) {
            const int c = base[e];
            base[e] = acc;
            off[e] = acc;
            acc += c;
        }
        off[n] = acc;
    }
    for (int c0 = 0; c0 < npairs; c0 += kGroupThreads) {
        const int m = min(kGroupThreads, npairs - c0);
        const int my = t < m ? idx[c0 + t] : 0;
        __syncthreads();
        if (t < m) ids[t] = (uint8_t)my;
        for (int e = t; e < n; e += kGroupThreads) hist[e] = 0;
        __syncthreads();
        if (t < m) {
            // rank = number of j < t with ids[j] == my (a zero byte of ids ^ my marks a match)
            const uint32_t pat = 0x01010101u * (uint32_t)my;
            int rank = 0;
            for (int j = 0; j < (t >> 2); ++j) {
                const uint32_t x = ids32[j] ^ pat;
                const uint32_t z = ~(((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x | 0x7F7F7F7Fu);
                rank += __popc(z);
            }
            for (int j = t & ~3; j < t; ++j) rank += ids[j] == (uint8_t)my;
            const int w = base[my] + rank;
            perm[w] = c0 + t;
            pos[c0 + t] = w;
            atomicAdd(&hist[my], 1);
        }
        __syncthreads();
        for (int e = t; e < n; e += kGroupThreads) base[e] += hist[e];
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
    int per_xcd;              // work items per XCD (expert-per-XCD layout)
    int spread;               // 1: item b is simply the b-th (expert, m, n, k) item
    int tail;                 // gate/up, expert-per-XCD layout: split the last partial round over K
    int slots;                // tail: work groups resident per XCD (<= kMaxTailSlots)
    float *part;              // tail: fp32 (g, u) partial sums [8][slots][kTileM][2 kGuCols]
    uint16_t *h;              // gate/up output, bf16 [P][f]
    float *yp;                // down output, fp32 [ksplit][P][d]
};

// Grouped GEMM with the weight operand fed from HBM into MFMA registers without a shared
// staging buffer: each wave loads its own weight rows and passes them through its own
// LDS region into the operand layout (see gemm_k_loop).
//
// A work group (kGWaves waves) owns up to 192 tokens of one expert and a tile of weight
// rows: for gate/up kGuCols columns of H (that many W1 rows and the same W3 rows), for
// down 256 (or 128) rows of W2. Each wave owns kNB 16-row MFMA column blocks of them (for
// gate/up the first kNB/2 are W1 blocks and the rest the matching W3 blocks, so the gate
// and up values of an output sit in the same lane) and all the tokens (twelve 16-row
// blocks). In v_mfma_f32_16x16x32_bf16 the B operand of lane l is 8 consecutive K values
// of column l mod 16, the four lanes l mod 16 + 16 i covering 32 consecutive K values;
// each weight byte is loaded once per work group. The token tile (shared by the waves) is
// staged in LDS, double-buffered.
//
// Weight loads run kS - 1 K steps ahead in a ring of kS register sets (kS = 3 below), the
// token loads one step ahead in a ring of two; the K loop is unrolled so that every set is
// a fixed group of registers. All loads are unconditional: token rows past the tile
// re-read row 0 (their outputs are dropped) and steps past the end re-read the last step.
// K = f of the down projection is split in ksplit parts that write separate fp32 partial
// sums.
//
// Eight waves of 32 weight rows each (kNB = 2) and four waves of 64 rows (kNB = 4, one
// wave per SIMD, accumulators in AGPRs, half the LDS reads of token operands per MFMA)
// ran within 2 % of each other on the Mixtral-shaped layer; a per-wave clock trace shows
// the K step bound by the LDS reads of the token operands and the MFMAs that wait for
// them, not by the weight stream (the step takes as long with the weight loads removed).
typedef float floatx4_t __attribute__((ext_vector_type(4)));
constexpr int kGWaves = 8;                             // waves per work group of the launches below
constexpr int kGuCols = 128;                           // H columns per gate/up work group
constexpr int kGuNB = 2 * kGuCols / (16 * kGWaves);    // gate/up column blocks per wave (W1 and W3 halves)
constexpr int kDnNB = 256 / (16 * kGWaves);            // down column blocks per wave (256-row tiles)
constexpr int kMBlocks = 12;                           // 16-token blocks per tile
constexpr int kTileM = kMBlocks * 16;                  // 192 tokens
constexpr int kKBlocks = kBK / 32;                     // MFMA K blocks per step

// Weight rows of one wave staged for the row-contiguous path: 16 kNB rows of one K step
// (128 bytes each), padded by 16 bytes per row.
constexpr int kWStride = kBK + 8;

// The K loop of k_moe_gemm for a tile of NMB 16-token blocks. NMB is a compile-time
// constant so the MFMA sequence of a step has no branches, and the LDS reads of the
// token blocks are issued kAP MFMA items ahead of their use (with a run-time block count
// every block was its own branch, and each MFMA pair waited for its own LDS read; with a
// constant count but no pinned order, the compiler still read each block just before its
// MFMAs: 632 against 601 us per Mixtral-shaped layer with the lookahead). Blocks past the
// tile's last token are not computed.
//
// Weights reach the MFMA operand registers row-contiguously: load instruction i reads the
// wave's rows 8i .. 8i+7, 128 bytes (one K step) of each, with the nontemporal hint, and
// the wave passes them through its own LDS region (written, then read back in the
// operand layout; no other wave touches it, so no barrier). Each instruction touches 8
// whole cache lines, where loading each lane's operand pieces directly touches halves of
// 16: half the L1 requests per weight byte, and whole lines for the nontemporal hint (with
// half lines it fetched each line twice). The down projection ran 13 % faster this way
// (223 -> 194 us per Mixtral-shaped layer); gate/up needs it together with kStagger.
//
// kStagger (gate/up): each work group starts its K walk at its own step (block id x 7
// mod the step count) and wraps around, so work groups running at the same time read
// different 128-byte columns of rows 8 KiB apart instead of the same one. Together with the
// row-contiguous loads this took gate/up from 414 to 400 us per Mixtral-shaped layer in a
// same-box A/B; either alone was neutral or slower, and the stagger slowed down (205 ->
// 208 us), which keeps its fixed K order.
template <int kS, int kAP, int kNB, int kAN, int kThr, int NMB, bool kStagger>
__device__ __forceinline__ void gemm_k_loop(uint16_t (*lds_a)[kTileM * kLdsStride], const uint16_t *const (&asrc)[kAN],
                                            const uint16_t *const (&bsrc)[2 * kNB], uint16_t *lds_w, int nsteps,
                                            floatx4_t (&acc)[kMBlocks][kNB])
{
    const int kstag = kStagger ? (int)(blockIdx.x * 7u % (unsigned)nsteps) : 0;
    static_assert(kBK == 64, "row-contiguous weight loads cover 128 bytes of a row per step");
    constexpr int kLB = 2 * kNB;   // weight loads per lane per step
    constexpr int kSA = 2;         // token register sets: one step ahead
    constexpr int kU = kS % kSA == 0 ? kS : kS * kSA;   // unroll: both rings at fixed registers
    // only the NMB token blocks that hold tokens are staged (the first kAL of the thread's
    // kAN chunks): a tile of 128 tokens stages 128 rows per step, not 192
    constexpr int kChunks = NMB * 16 * kRowChunks;
    constexpr int kAL = (kChunks + kThr - 1) / kThr;
    static_assert(kAL <= kAN, "staged chunks within the tile's");
    const int tid = threadIdx.x, lane = tid & 63;
    u32x4_t ra[kSA][kAL], rb[kS][kLB];
    u32x4_t rt[kNB * kKBlocks];                                  // operand pieces after the LDS pass
#define MOE_KOFF(step) (((min((step), nsteps - 1) + kstag) % nsteps) * kBK)
#define MOE_LOAD_A(set, step)                                                                         \
    do {                                                                                              \
        const int ko_ = MOE_KOFF(step);                                                               \
        _Pragma("unroll") for (int i = 0; i < kAL; ++i) ra[set][i] =                                  \
            *reinterpret_cast<const u32x4_t *>(asrc[i] + ko_);                                        \
    } while (0)
#define MOE_LOAD_W(set, step)                                                                         \
    do {                                                                                              \
        const int ko_ = MOE_KOFF(step);                                                               \
        _Pragma("unroll") for (int i = 0; i < kLB; ++i) rb[set][i] =                                  \
            __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(bsrc[i] + ko_));             \
    } while (0)
#define MOE_STASH(set, buf)                                                                           \
    do {                                                                                              \
        _Pragma("unroll") for (int i = 0; i < kAL; ++i) {                                             \
            const int c_ = tid + kThr * i;                                                            \
            if (kChunks % kThr == 0 || c_ < kChunks)                                                  \
                *reinterpret_cast<u32x4_t *>(&lds_a[buf][(c_ / kRowChunks) * kLdsStride + (c_ % kRowChunks) * 8]) = ra[set][i]; \
        }                                                                                             \
    } while (0)
    // rows 8i + lane/8 in, operand pieces (row 16 nb + lane mod 16, K 32 kb + 8 (lane / 16)) out
#define MOE_TRANSPOSE(set)                                                                            \
    do {                                                                                              \
        _Pragma("unroll") for (int i = 0; i < kLB; ++i)                                               \
            *reinterpret_cast<u32x4_t *>(&lds_w[(8 * i + (lane >> 3)) * kWStride + (lane & 7) * 8]) = rb[set][i]; \
        _Pragma("unroll") for (int nb = 0; nb < kNB; ++nb)                                            \
        _Pragma("unroll") for (int kb = 0; kb < kKBlocks; ++kb) rt[nb * kKBlocks + kb] =              \
            *reinterpret_cast<const u32x4_t *>(&lds_w[(16 * nb + (lane & 15)) * kWStride + kb * 32 + 8 * (lane >> 4)]); \
    } while (0)
    // token operand of MFMA item j (K block j / NMB, token block j mod NMB)
#define MOE_AREAD(j, buf)                                                                             \
    (*reinterpret_cast<const bf16x8_t *>(                                                             \
        &lds_a[buf][(((j) % NMB) * 16 + (lane & 15)) * kLdsStride + ((j) / NMB) * 32 + 8 * (lane >> 4)]))
    // The token operands are read kAP items ahead of their MFMAs, in a ring of kAP registers,
    // and the order is pinned (left to itself the compiler read each operand just before its
    // MFMA pair and waited for it, so the LDS latency was paid once per token block).
#define MOE_MMA(buf)                                                                                  \
    do {                                                                                              \
        constexpr int kJ_ = kKBlocks * NMB;                                                           \
        bf16x8_t aq_[kAP];                                                                            \
        _Pragma("unroll") for (int j = 0; j < kAP; ++j) if (j < kJ_) aq_[j] = MOE_AREAD(j, buf);      \
        _Pragma("unroll") for (int j = 0; j < kJ_; ++j) {                                             \
            const bf16x8_t a_ = aq_[j % kAP];                                                         \
            if (j + kAP < kJ_) aq_[j % kAP] = MOE_AREAD(j + kAP, buf);                                \
            _Pragma("unroll") for (int nb = 0; nb < kNB; ++nb) acc[j % NMB][nb] =                     \
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(                                              \
                    a_, __builtin_bit_cast(bf16x8_t, rt[nb * kKBlocks + j / NMB]),                    \
                    acc[j % NMB][nb], 0, 0, 0);                                                       \
            __builtin_amdgcn_sched_barrier(0);                                                        \
        }                                                                                             \
    } while (0)

    // Step t: the tokens of step t + 1 are loaded first, then the weights of step
    // t + kS - 1; the token stash at the end of the step waits for the former, and since
    // loads complete in issue order that also covers every weight set issued before it.
    MOE_LOAD_A(0, 0);
#pragma unroll
    for (int p = 0; p < kS - 1; ++p) MOE_LOAD_W(p, p);
    MOE_STASH(0, 0);
    __syncthreads();
    for (int s = 0; s < nsteps; s += kU) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            if (s + u >= nsteps) break;
            MOE_TRANSPOSE(u % kS);
            MOE_LOAD_A((u + 1) % kSA, s + u + 1);
            MOE_LOAD_W((u + kS - 1) % kS, s + u + kS - 1);
            MOE_MMA((s + u) & 1);
            MOE_STASH((u + 1) % kSA, (s + u + 1) & 1);
            __syncthreads();
        }
    }
#undef MOE_KOFF
#undef MOE_LOAD_A
#undef MOE_LOAD_W
#undef MOE_STASH
#undef MOE_TRANSPOSE
#undef MOE_MMA
#undef MOE_AREAD
}

// Gate/up tail split (expert-per-XCD layout). The live tiles of XCD x (its experts x,
// x + 8, ... times their occupied M tiles and the N tiles) run in rounds of g.slots work
// groups; the r tiles of a last, partial round are split over K into s parts, as many as
// the idle work groups allow (s r <= slots), and a second kernel adds the parts.
struct TailPlan {
    int U, R, r, s;   // live tiles, full rounds, tiles of the partial round, K parts per tile
};

__device__ __forceinline__ TailPlan tail_plan(const GemmArgs &g, int xcd)
{
    TailPlan p;
    p.U = 0;
    for (int e = xcd; e < g.n; e += kXcds) p.U += (g.off[e + 1] - g.off[e] + kTileM - 1) / kTileM * g.ntiles;
    p.R = p.U / g.slots;
    p.r = p.U - p.R * g.slots;
    p.s = 1;
    while (p.r > 0 && 2 * p.s * p.r <= g.slots && 2 * p.s <= kMaxTailSplit && (g.d / kBK) % (2 * p.s) == 0) p.s *= 2;
    return p;
}

// live tile t (< U) of XCD xcd -> expert, M tile, N tile (N-major within an expert)
__device__ __forceinline__ void tail_tile(const GemmArgs &g, int xcd, int t, int &e, int &mt, int &nt)
{
    for (e = xcd;; e += kXcds) {
        const int m_e = (g.off[e + 1] - g.off[e] + kTileM - 1) / kTileM;
        if (t < m_e * g.ntiles) {
            mt = t % m_e;
            nt = t / m_e;
            return;
        }
        t -= m_e * g.ntiles;
    }
}

template <bool kGateUp, int kS, int kNB, int kWaves>
__global__ __launch_bounds__(kWaves * 64) void k_moe_gemm(GemmArgs g)
{
    constexpr int kThr = kWaves * 64;
    constexpr int kAN = (kTileM * kRowChunks + kThr - 1) / kThr;   // token-tile 16-byte chunks per thread per step
    __shared__ uint16_t lds_a[2][kTileM * kLdsStride];
    __shared__ uint16_t lds_w[kWaves][16 * kNB * kWStride];

    const int K = kGateUp ? g.d : g.f;
    int e, mt, nt, ks = 0, kparts = g.ksplit;
    int xcd = 0, tail_v = -1, tail_s = 1;   // tail: unit v of a tile split in tail_s K parts
    if (kGateUp && g.tail) {
        // units: the full tiles (whole K) first, then the K parts of the partial round's tiles
        xcd = blockIdx.x % kXcds;
        const int u = blockIdx.x / kXcds;
        const TailPlan tp = tail_plan(g, xcd);
        tail_s = tp.s;
        int t;
        if (u < tp.R * g.slots || tail_s == 1) {
            if (u >= tp.U) return;
            t = u;
        } else {
            const int v = u - tp.R * g.slots;
            if (v >= tp.r * tail_s) return;
            t = tp.R * g.slots + v / tail_s;
            ks = v % tail_s;
            kparts = tail_s;
            tail_v = v;
        }
        tail_tile(g, xcd, t, e, mt, nt);
    } else {
        const int per_expert = g.mtiles * g.ntiles * g.ksplit;
        int q;
        if (g.spread) {   // few tokens per expert: an expert's items go round all XCDs
            q = blockIdx.x;
            e = q / per_expert;
        } else {          // an expert's items stay on XCD e mod 8, sharing its token rows in L2
            q = blockIdx.x / kXcds;
            if (q >= g.per_xcd) return;
            e = blockIdx.x % kXcds + kXcds * (q / per_expert);
        }
        if (e >= g.n) return;
        q %= per_expert;
        ks = q % g.ksplit;
        q /= g.ksplit;
        mt = q % g.mtiles;
        nt = q / g.mtiles;
    }
    const int row0 = g.off[e] + mt * kTileM;
    const int rows = min(kTileM, g.off[e + 1] - row0);
    if (rows <= 0) return;

    const int kspan = K / kparts;
    const int k0 = ks * kspan;
    const int nsteps = kspan / kBK;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int nmb = (rows + 15) >> 4;                  // token blocks holding tokens of this tile
    const uint16_t *w = reinterpret_cast<const uint16_t *>(g.pool + (uint64_t)e * g.slab_stride);

    static_assert(!kGateUp || (kNB % 2 == 0 && kWaves * 8 * kNB == kGuCols),
                  "gate/up pairs each W1 block with a W3 block over kGuCols columns");
    // this lane's weight row and K offset for the row-contiguous loads: row 8i + lane / 8 of
    // the wave's rows, 8 (lane mod 8) elements into the K step
    const uint16_t *bsrc[2 * kNB];
    if constexpr (kGateUp) {   // the wave's 8 kNB W1 rows (loads 0 .. kNB-1), then the same W3 rows
#pragma unroll
        for (int i = 0; i < 2 * kNB; ++i) {
            const size_t wrow = (size_t)nt * kGuCols + wv * 8 * kNB + 8 * (i % kNB) + (lane >> 3);
            bsrc[i] = w + (i >= kNB ? (size_t)g.f * g.d : 0) + wrow * g.d + k0 + 8 * (lane & 7);
        }
    } else {
#pragma unroll
        for (int i = 0; i < 2 * kNB; ++i) {
            const size_t wrow = (size_t)nt * (kWaves * 16 * kNB) + wv * 16 * kNB + 8 * i + (lane >> 3);
            bsrc[i] = w + (size_t)2 * g.f * g.d + wrow * g.f + k0 + 8 * (lane & 7);
        }
    }
    // token-tile chunks staged by this thread: chunk c = tid + kThr i is row c / kRowChunks, column
    // c % kRowChunks (chunks past the tile, when the threads do not divide it, load row 0 and are not stored)
    const uint16_t *asrc[kAN];
#pragma unroll
    for (int i = 0; i < kAN; ++i) {
        const int c = tid + kThr * i;
        const int r = c / kRowChunks, col = (c % kRowChunks) * 8;
        const int rr = r < rows ? r : 0;
        if (kGateUp) asrc[i] = g.a + (size_t)(g.perm[row0 + rr] / g.k) * g.d + k0 + col;
        else asrc[i] = g.a + (size_t)(row0 + rr) * g.f + k0 + col;
    }

    floatx4_t acc[kMBlocks][kNB];
#pragma unroll
    for (int m = 0; m < kMBlocks; ++m)
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) acc[m][nb] = floatx4_t{0.f, 0.f, 0.f, 0.f};

    // One copy of the K loop per token-block count, chosen once per work group.
    constexpr int kTokAhead = 6;   // token operand reads kept ahead of the MFMAs
    switch (nmb) {
#define MOE_NMB_CASE(N) \
    case N: gemm_k_loop<kS, kTokAhead, kNB, kAN, kThr, N, kGateUp>(lds_a, asrc, bsrc, lds_w[wv], nsteps, acc); \
        break;
        MOE_NMB_CASE(1) MOE_NMB_CASE(2) MOE_NMB_CASE(3) MOE_NMB_CASE(4) MOE_NMB_CASE(5) MOE_NMB_CASE(6)
        MOE_NMB_CASE(7) MOE_NMB_CASE(8) MOE_NMB_CASE(9) MOE_NMB_CASE(10) MOE_NMB_CASE(11) MOE_NMB_CASE(12)
#undef MOE_NMB_CASE
    default: break;
    }

    // Output element r of a 16x16 block sits at row 4*(lane/16) + r, column lane%16.
    if constexpr (kGateUp) {
        if (tail_v >= 0) {   // a K part of a split tile: its fp32 (g, u) sums, added by k_tail_combine
            constexpr int kCols = 2 * kGuCols;   // g columns, then u columns
            float *mine = g.part + ((size_t)xcd * g.slots + tail_v) * kTileM * kCols;
#pragma unroll
            for (int m = 0; m < kMBlocks; ++m)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int tr = m * 16 + 4 * (lane >> 4) + r;
                    if (tr >= rows) continue;
#pragma unroll
                    for (int nb = 0; nb < kNB / 2; ++nb) {
                        const int c = wv * 8 * kNB + 16 * nb + (lane & 15);
                        mine[tr * kCols + c] = acc[m][nb][r];
                        mine[tr * kCols + kGuCols + c] = acc[m][nb + kNB / 2][r];
                    }
                }
            return;
        }
    }
    const int P = g.off[g.n];
#pragma unroll
    for (int m = 0; m < kMBlocks; ++m) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int tr = m * 16 + 4 * (lane >> 4) + r;
            if (tr >= rows) continue;
            if constexpr (kGateUp) {
#pragma unroll
                for (int nb = 0; nb < kNB / 2; ++nb) {
                    const float gv = acc[m][nb][r], uv = acc[m][nb + kNB / 2][r];
                    const float hv = gv / (1.0f + expf(-gv)) * uv;
                    g.h[(size_t)(row0 + tr) * g.f + nt * kGuCols + wv * 8 * kNB + 16 * nb + (lane & 15)] = f2bf(hv);
                }
            } else {
                float *dst = g.yp + ((size_t)ks * P + row0 + tr) * g.d + nt * (kWaves * 16 * kNB) + wv * 16 * kNB +
                             (lane & 15);
#pragma unroll
                for (int nb = 0; nb < kNB; ++nb) dst[16 * nb] = acc[m][nb][r];
            }
        }
    }
}

// H of the gate/up tiles split over K: h = SiLU(sum of the g parts) * (sum of the u parts),
// the parts added in order. Work group b: XCD b mod 8, then tile i of that XCD's partial
// round and a block of 16 of its rows (the plan is recomputed from the expert offsets
// exactly as the GEMM did); each thread takes 4 consecutive columns of 2 rows.
constexpr int kTailRows = 16;
__global__ __launch_bounds__(kThreads) void k_tail_combine(GemmArgs g)
{
    constexpr int kCols = 2 * kGuCols;   // g columns, then u columns
    constexpr int kQuads = kGuCols / 4;  // 4-column groups of the tile's columns
    const int xcd = blockIdx.x % kXcds;
    const int i = (blockIdx.x / kXcds) % g.slots;
    const int rb = blockIdx.x / kXcds / g.slots;
    const TailPlan tp = tail_plan(g, xcd);
    if (tp.s == 1 || i >= tp.r) return;
    int e, mt, nt;
    tail_tile(g, xcd, tp.R * g.slots + i, e, mt, nt);
    const int row0 = g.off[e] + mt * kTileM;
    const int rows = min(kTileM, g.off[e + 1] - row0);
    const float *p0 = g.part + ((size_t)xcd * g.slots + (size_t)i * tp.s) * kTileM * kCols;
    for (int c = threadIdx.x; c < kTailRows * kQuads; c += kThreads) {
        const int tr = rb * kTailRows + c / kQuads, col = (c % kQuads) * 4;
        if (tr >= rows) continue;
        float4 gv = make_float4(0.f, 0.f, 0.f, 0.f), uv = gv;
        for (int j = 0; j < tp.s; ++j) {
            const float *pj = p0 + (size_t)j * kTileM * kCols + tr * kCols + col;
            const float4 a = *reinterpret_cast<const float4 *>(pj);
            const float4 b = *reinterpret_cast<const float4 *>(pj + kCols / 2);
            gv.x += a.x; gv.y += a.y; gv.z += a.z; gv.w += a.w;
            uv.x += b.x; uv.y += b.y; uv.z += b.z; uv.w += b.w;
        }
        uint2 o;
        o.x = f2bf(gv.x / (1.0f + expf(-gv.x)) * uv.x) | ((uint32_t)f2bf(gv.y / (1.0f + expf(-gv.y)) * uv.y) << 16);
        o.y = f2bf(gv.z / (1.0f + expf(-gv.z)) * uv.z) | ((uint32_t)f2bf(gv.w / (1.0f + expf(-gv.w)) * uv.w) << 16);
        *reinterpret_cast<uint2 *>(g.h + (size_t)(row0 + tr) * g.f + nt * kGuCols + col) = o;
    }
}

// OUT[t][i] = sum_r w[t][r] * sum_s Yp[s][pos[t*k+r]][i], four consecutive i per thread;
// work group b covers token b / nparts, columns (b mod nparts) * 1024 ...
__global__ __launch_bounds__(kThreads) void k_prefill_combine(const float *yp, const int32_t *pos, const float *w,
                                                              int k, int d, int P, int ksplit, int nparts, float *out)
{
    const int t = blockIdx.x / nparts;
    const int i = ((blockIdx.x % nparts) * kThreads + threadIdx.x) * 4;
    if (i >= d) return;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int r = 0; r < k; ++r) {
        const int pr = pos[t * k + r];
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int q = 0; q < ksplit; ++q) {
            const float4 v = *reinterpret_cast<const float4 *>(yp + ((size_t)q * P + pr) * d + i);
            s.x += v.x;
            s.y += v.y;
            s.z += v.z;
            s.w += v.w;
        }
        const float wr = w[t * k + r];
        acc.x = fmaf(wr, s.x, acc.x);
        acc.y = fmaf(wr, s.y, acc.y);
        acc.z = fmaf(wr, s.z, acc.z);
        acc.w = fmaf(wr, s.w, acc.w);
    }
    *reinterpret_cast<float4 *>(out + (size_t)t * d + i) = acc;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// K splits of the down GEMM: four when each part is still a whole number of K steps.
int down_splits(int f) { return f % (kMaxDownSplits * kBK) == 0 ? kMaxDownSplits : 2; }

struct PrefillWs {
    uint16_t *xb;
    int32_t *idx, *off, *perm, *pos;
    float *w;
    uint16_t *h;
    float *yp;
    float *part;   // gate/up tail partial sums (expert-per-XCD layout only)
};

// Few (token, expert) pairs per expert: every expert's items are spread over all XCDs.
bool spread_layout(int n, int k, int T) { return (int64_t)T * k < (int64_t)kSpreadTokens * n; }

// fp32 (g, u) partial sums of the gate/up tiles split over K: [8][kMaxTailSlots][kTileM][2 * 128]
constexpr size_t kPartBytes = (size_t)kXcds * kMaxTailSlots * kTileM * 2 * kGuCols * sizeof(float);

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
    uint8_t *yp = take((size_t)kMaxDownSplits * P * d * 4);
    uint8_t *part = take(spread_layout(n, k, T) ? 0 : kPartBytes);
    if (ws) {
        ws->xb = reinterpret_cast<uint16_t *>(xb);
        ws->idx = reinterpret_cast<int32_t *>(idx);
        ws->w = reinterpret_cast<float *>(w);
        ws->off = reinterpret_cast<int32_t *>(off);
        ws->perm = reinterpret_cast<int32_t *>(perm);
        ws->pos = reinterpret_cast<int32_t *>(pos);
        ws->h = reinterpret_cast<uint16_t *>(h);
        ws->yp = reinterpret_cast<float *>(yp);
        ws->part = reinterpret_cast<float *>(part);
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
    const int64_t n8 = (int64_t)P.T * P.d / 8;
    const int cast_blocks = (int)std::min<int64_t>((n8 + kGroupThreads - 1) / kGroupThreads, 1024);
    hipLaunchKernelGGL(k_group, dim3(1 + cast_blocks), dim3(kGroupThreads), 0, s, idx_d, npairs, P.n, ws.off, ws.perm,
                       ws.pos, X, ws.xb, n8);
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
    g.mtiles = (P.T + kTileM - 1) / kTileM;
    g.h = ws.h;
    g.yp = ws.yp;
    const int groups = (P.n + kXcds - 1) / kXcds;
    // With few tokens per expert most experts are idle or nearly so, and keeping an
    // expert on one XCD would leave the others without work; spread its tiles instead.
    g.spread = spread_layout(P.n, P.k, P.T);
    auto grid_of = [&](const GemmArgs &a) {
        return g.spread ? P.n * a.mtiles * a.ntiles * a.ksplit : kXcds * a.per_xcd;
    };

    // gate/up: each work group covers 128 columns of H (128 W1 rows + the same 128 W3 rows), K = d
    g.a = ws.xb;
    g.ntiles = P.f / kGuCols;
    g.ksplit = 1;
    g.per_xcd = groups * g.mtiles * g.ntiles * g.ksplit;
    // Tail splitting (expert-per-XCD layout): the rounds of resident work groups per XCD
    // decide which tiles are split.
    static std::atomic<int> gu_occ_cache{-1};   // concurrent first calls store the same value
    int gu_occ = gu_occ_cache.load(std::memory_order_relaxed);
    if (gu_occ < 0) {
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&gu_occ, k_moe_gemm<true, 3, kGuNB, kGWaves>, kGWaves * 64,
                                                         0) != hipSuccess ||
            gu_occ < 1) {
            (void)hipGetLastError();
            gu_occ = 0;
        }
        gu_occ_cache.store(gu_occ, std::memory_order_relaxed);
    }
    const int slots = std::min(kMaxTailSlots, gu_occ * device_cu_count() / kXcds);
    g.tail = !g.spread && slots >= 2;
    g.slots = g.tail ? slots : 0;
    g.part = ws.part;
    // with tail splitting a work group takes a live tile or a K part of one: at most the
    // live tiles plus one round of parts
    const int gu_per_xcd = g.tail ? g.per_xcd + g.slots : g.per_xcd;
    const int gu_grid = g.spread ? grid_of(g) : kXcds * gu_per_xcd;
    hipLaunchKernelGGL((k_moe_gemm<true, 3, kGuNB, kGWaves>), dim3(gu_grid), dim3(kGWaves * 64), 0, s, g);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (g.tail) {
        hipLaunchKernelGGL(k_tail_combine, dim3(kXcds * g.slots * (kTileM / kTailRows)), dim3(kThreads), 0, s, g);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }

    // down: 256 (or 128) output rows per work group, K = f split in 4 (or 2) parts
    g.tail = 0;
    g.a = ws.h;
    g.ksplit = down_splits(P.f);
    const bool wide = P.d % 256 == 0;
    g.ntiles = P.d / (wide ? 256 : 128);
    g.per_xcd = groups * g.mtiles * g.ntiles * g.ksplit;
    if (wide) hipLaunchKernelGGL((k_moe_gemm<false, 3, kDnNB, kGWaves>), dim3(grid_of(g)), dim3(kGWaves * 64), 0, s, g);
    else hipLaunchKernelGGL((k_moe_gemm<false, 3, kDnNB / 2, kGWaves>), dim3(grid_of(g)), dim3(kGWaves * 64), 0, s, g);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    const int nparts = (P.d + 4 * kThreads - 1) / (4 * kThreads);
    hipLaunchKernelGGL(k_prefill_combine, dim3(P.T * nparts), dim3(kThreads), 0, s, ws.yp, ws.pos, w_d, P.k, P.d,
                       npairs, g.ksplit, nparts, OUT);
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
