// Host expert path for cache misses (Section III-A step 2(b)): the hidden state is
// brought to the host and the missed experts run on CPU threads, the number of
// threads being the knob the paper studies through OMP_NUM_THREADS (Section I,
// Table III). Each output row is one thread's fixed-order sum, so the result does
// not depend on the thread count.
//
// Two forms of the row dot product: (fp32) the bf16 weights widened to fp32 by a
// 16-bit shift and multiplied with fp32 FMAs; (bf16) the AVX512_BF16 pair-dot
// instruction, which multiplies bf16 by bf16 exactly and sums in fp32, with the fp32
// activation split into two bf16 parts, hi = bf16(v) and lo = bf16(v - hi), so that
// |v - hi - lo| <= 2^-18 |v| and each weight meets both parts.
#include <immintrin.h>

#include <cmath>
#include <cstdlib>
#include <cstring>

#include "common.h"
#include "hostpath.h"

namespace moe {

namespace {

inline float widen(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// dot(bf16 row, fp32 vector) over len elements (len a multiple of 8).
float dot_generic(const uint16_t *w, const float *x, int len)
{
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int j = 0; j < len; j += 8)
        for (int e = 0; e < 8; ++e) acc[e] += widen(w[j + e]) * x[j + e];
    return ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
}

__attribute__((target("avx512f,avx512bw,avx512vl"))) float dot_avx512(const uint16_t *w, const float *x, int len)
{
    __m512 a0 = _mm512_setzero_ps(), a1 = _mm512_setzero_ps(), a2 = _mm512_setzero_ps(),
           a3 = _mm512_setzero_ps();
    int j = 0;
    for (; j + 64 <= len; j += 64) {
        const __m512i w0 = _mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i *)(w + j)));
        const __m512i w1 = _mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i *)(w + j + 16)));
        const __m512i w2 = _mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i *)(w + j + 32)));
        const __m512i w3 = _mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i *)(w + j + 48)));
        a0 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(w0, 16)), _mm512_loadu_ps(x + j), a0);
        a1 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(w1, 16)), _mm512_loadu_ps(x + j + 16), a1);
        a2 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(w2, 16)), _mm512_loadu_ps(x + j + 32), a2);
        a3 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(w3, 16)), _mm512_loadu_ps(x + j + 48), a3);
    }
    for (; j + 16 <= len; j += 16) {
        const __m512i w0 = _mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i *)(w + j)));
        a0 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(w0, 16)), _mm512_loadu_ps(x + j), a0);
    }
    float acc = _mm512_reduce_add_ps(_mm512_add_ps(_mm512_add_ps(a0, a1), _mm512_add_ps(a2, a3)));
    for (; j < len; ++j) acc += widen(w[j]) * x[j];
    return acc;
}

// Round-to-nearest-even fp32 -> bf16 (finite inputs; the activations are finite).
inline uint16_t to_bf16(float v)
{
    uint32_t u;
    std::memcpy(&u, &v, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// hi[i] = bf16(v[i]), lo[i] = bf16(v[i] - hi[i]) for i < len.
void split_bf16(const float *v, int len, uint16_t *hi, uint16_t *lo)
{
    for (int i = 0; i < len; ++i) {
        hi[i] = to_bf16(v[i]);
        lo[i] = to_bf16(v[i] - widen(hi[i]));
    }
}

// dot(bf16 row, hi + lo) over len elements with the pair-dot instruction: each 64-byte
// load holds 32 weights; the tail (len a multiple of 8) is a masked load, zero-filled.
__attribute__((target("avx512f,avx512bw,avx512vl,avx512bf16"))) float dot_bf16x2(const uint16_t *w,
                                                                                   const uint16_t *hi,
                                                                                   const uint16_t *lo, int len)
{
    __m512 a0 = _mm512_setzero_ps(), a1 = _mm512_setzero_ps();
    int j = 0;
    for (; j + 64 <= len; j += 64) {
        const __m512i w0 = _mm512_loadu_si512(w + j), w1 = _mm512_loadu_si512(w + j + 32);
        a0 = _mm512_dpbf16_ps(a0, (__m512bh)w0, (__m512bh)_mm512_loadu_si512(hi + j));
        a1 = _mm512_dpbf16_ps(a1, (__m512bh)w1, (__m512bh)_mm512_loadu_si512(hi + j + 32));
        a0 = _mm512_dpbf16_ps(a0, (__m512bh)w0, (__m512bh)_mm512_loadu_si512(lo + j));
        a1 = _mm512_dpbf16_ps(a1, (__m512bh)w1, (__m512bh)_mm512_loadu_si512(lo + j + 32));
    }
    for (; j < len; j += 32) {
        const int rem = len - j;
        const __mmask32 m = rem >= 32 ? 0xffffffffu : ((1u << rem) - 1u);
        const __m512i w0 = _mm512_maskz_loadu_epi16(m, w + j);
        a0 = _mm512_dpbf16_ps(a0, (__m512bh)w0, (__m512bh)_mm512_maskz_loadu_epi16(m, hi + j));
        a0 = _mm512_dpbf16_ps(a0, (__m512bh)w0, (__m512bh)_mm512_maskz_loadu_epi16(m, lo + j));
    }
    return _mm512_reduce_add_ps(_mm512_add_ps(a0, a1));
}

bool cpu_has_avx512_bf16()
{
    __builtin_cpu_init();
    return __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") &&
           __builtin_cpu_supports("avx512vl") && __builtin_cpu_supports("avx512bf16");
}

using DotFn = float (*)(const uint16_t *, const float *, int);

DotFn pick_dot()
{
    __builtin_cpu_init();
    if (__builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") &&
        __builtin_cpu_supports("avx512vl"))
        return dot_avx512;
    return dot_generic;
}

const DotFn g_dot = pick_dot();

int default_threads()
{
    if (const char *s = std::getenv("OMP_NUM_THREADS")) {
        const int v = std::atoi(s);
        if (v > 0) return v;
    }
    const unsigned hc = std::thread::hardware_concurrency();
    return hc > 0 ? (int)hc : 1;
}

}  // namespace

HostPool::HostPool(int n_threads) : n_(n_threads > 0 ? n_threads : default_threads())
{
    for (int t = 1; t < n_; ++t) th_.emplace_back(&HostPool::worker, this, t);
}

HostPool::~HostPool()
{
    {
        std::lock_guard<std::mutex> lk(mu_);
        stop_ = true;
        ++gen_;
    }
    cv_go_.notify_all();
    for (auto &t : th_) t.join();
}

static inline void range_of(int64_t total, int n, int tid, int64_t &b, int64_t &e)
{
    b = total * tid / n;
    e = total * (tid + 1) / n;
}

void HostPool::worker(int tid)
{
    uint64_t seen = 0;
    for (;;) {
        const std::function<void(int, int64_t, int64_t)> *fn;
        int64_t total;
        {
            std::unique_lock<std::mutex> lk(mu_);
            cv_go_.wait(lk, [&] { return gen_ != seen; });
            seen = gen_;
            if (stop_) return;
            fn = fn_;
            total = total_;
        }
        int64_t b, e;
        range_of(total, n_, tid, b, e);
        if (b < e) (*fn)(tid, b, e);
        {
            std::lock_guard<std::mutex> lk(mu_);
            if (--pending_ == 0) cv_done_.notify_one();
        }
    }
}

bool HostPool::dot_supported(HostDot k)
{
    if (k == HostDot::kFp32) return true;
    if (k == HostDot::kBf16) return cpu_has_avx512_bf16();
    return false;
}

void HostPool::set_dot(HostDot k)
{
    std::lock_guard<std::mutex> call(call_mu_);
    dot_ = k;
}

void HostPool::parallel_for(int64_t total, const std::function<void(int, int64_t, int64_t)> &fn)
{
    std::lock_guard<std::mutex> call(call_mu_);
    run(total, fn);
}

void HostPool::run(int64_t total, const std::function<void(int, int64_t, int64_t)> &fn)
{
    if (n_ == 1 || total <= 1) {
        if (total > 0) fn(0, 0, total);
        return;
    }
    {
        std::lock_guard<std::mutex> lk(mu_);
        fn_ = &fn;
        total_ = total;
        pending_ = n_ - 1;
        ++gen_;
    }
    cv_go_.notify_all();
    int64_t b, e;
    range_of(total, n_, 0, b, e);
    if (b < e) fn(0, b, e);
    std::unique_lock<std::mutex> lk(mu_);
    cv_done_.wait(lk, [&] { return pending_ == 0; });
}

void HostPool::expert_ffn(const float *x, const void *const *slabs, const float *w, int ne, int d, int f, float *y)
{
    std::lock_guard<std::mutex> call(call_mu_);
    if (ne == 0) {
        std::memset(y, 0, sizeof(float) * (size_t)d);
        return;
    }
    const size_t nh = (size_t)ne * f;
    if (h_.size() < nh) h_.resize(nh);
    float *h = h_.data();
    if (dot_ == HostDot::kBf16) {
        if (xh_.size() < (size_t)d) xh_.resize(d), xl_.resize(d);
        if (hh_.size() < nh) hh_.resize(nh), hl_.resize(nh);
        uint16_t *xh = xh_.data(), *xl = xl_.data(), *hh = hh_.data(), *hl = hl_.data();
        split_bf16(x, d, xh, xl);
        run((int64_t)nh, [&](int, int64_t b, int64_t e) {
            for (int64_t r = b; r < e; ++r) {
                const int j = (int)(r / f);
                const int i = (int)(r - (int64_t)j * f);
                const uint16_t *s = static_cast<const uint16_t *>(slabs[j]);
                const float g = dot_bf16x2(s + (size_t)i * d, xh, xl, d);
                const float u = dot_bf16x2(s + (size_t)f * d + (size_t)i * d, xh, xl, d);
                const float v = g / (1.0f + std::exp(-g)) * u;
                h[r] = v;
                hh[r] = to_bf16(v);
                hl[r] = to_bf16(v - widen(hh[r]));
            }
        });
        run(d, [&](int, int64_t b, int64_t e) {
            for (int64_t i = b; i < e; ++i) {
                float acc = 0.f;
                for (int j = 0; j < ne; ++j) {
                    const uint16_t *s = static_cast<const uint16_t *>(slabs[j]) + (size_t)2 * f * d;
                    acc += w[j] * dot_bf16x2(s + (size_t)i * f, hh + (size_t)j * f, hl + (size_t)j * f, f);
                }
                y[i] = acc;
            }
        });
        return;
    }
    const DotFn dot = g_dot;
    // gate/up/SiLU over all (expert, row) pairs
    run((int64_t)nh, [&](int, int64_t b, int64_t e) {
        for (int64_t r = b; r < e; ++r) {
            const int j = (int)(r / f);
            const int i = (int)(r - (int64_t)j * f);
            const uint16_t *s = static_cast<const uint16_t *>(slabs[j]);
            const float g = dot(s + (size_t)i * d, x, d);
            const float u = dot(s + (size_t)f * d + (size_t)i * d, x, d);
            h[r] = g / (1.0f + std::exp(-g)) * u;
        }
    });
    // down + weighted sum over the experts, in expert order
    run(d, [&](int, int64_t b, int64_t e) {
        for (int64_t i = b; i < e; ++i) {
            float acc = 0.f;
            for (int j = 0; j < ne; ++j) {
                const uint16_t *s = static_cast<const uint16_t *>(slabs[j]) + (size_t)2 * f * d;
                acc += w[j] * dot(s + (size_t)i * f, h + (size_t)j * f, f);
            }
            y[i] = acc;
        }
    });
}

}  // namespace moe

extern "C" {

int moe_host_alloc(size_t bytes, void **out)
{
    MOE_REQUIRE(out && bytes > 0, "moe_host_alloc: need bytes > 0 and an output pointer");
    *out = nullptr;
    const hipError_t e = hipHostMalloc(out, bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        *out = nullptr;
        moe::set_error("moe_host_alloc: hipHostMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
        return e == hipErrorOutOfMemory ? MOE_ENOMEM : MOE_EHIP;
    }
    return MOE_OK;
}

int moe_host_free(void *ptr)
{
    if (ptr) MOE_HIP(hipHostFree(ptr));
    return MOE_OK;
}

int moe_host_pool_create(int n_threads, moe_host_pool **out)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(out, "moe_host_pool_create: null output handle");
    MOE_REQUIRE(n_threads <= 4096, "moe_host_pool_create: n_threads=%d too large", n_threads);
    *out = reinterpret_cast<moe_host_pool *>(new moe::HostPool(n_threads));
    return MOE_OK;
    MOE_GUARD_END
}

void moe_host_pool_destroy(moe_host_pool *p) { delete reinterpret_cast<moe::HostPool *>(p); }

int moe_host_pool_threads(const moe_host_pool *p)
{
    MOE_REQUIRE(p, "moe_host_pool_threads: null handle");
    return reinterpret_cast<const moe::HostPool *>(p)->threads();
}

int moe_host_pool_set_dot(moe_host_pool *p, int kind)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(p, "moe_host_pool_set_dot: null handle");
    MOE_REQUIRE(kind == MOE_HOST_DOT_AUTO || kind == MOE_HOST_DOT_FP32 || kind == MOE_HOST_DOT_BF16,
                "moe_host_pool_set_dot: unknown kind %d", kind);
    const moe::HostDot k = kind == MOE_HOST_DOT_BF16 ? moe::HostDot::kBf16 : moe::HostDot::kFp32;
    MOE_REQUIRE(moe::HostPool::dot_supported(k), "moe_host_pool_set_dot: this CPU has no AVX512_BF16");
    reinterpret_cast<moe::HostPool *>(p)->set_dot(k);
    return MOE_OK;
    MOE_GUARD_END
}

int moe_host_pool_get_dot(const moe_host_pool *p)
{
    MOE_REQUIRE(p, "moe_host_pool_get_dot: null handle");
    return reinterpret_cast<const moe::HostPool *>(p)->dot() == moe::HostDot::kBf16 ? MOE_HOST_DOT_BF16
                                                                                     : MOE_HOST_DOT_FP32;
}

int moe_host_expert_ffn(moe_host_pool *p, const float *x, const void *const *slabs, const float *w, int n_experts,
                        int d, int f, float *y)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(p && x && y, "moe_host_expert_ffn: null pointer");
    MOE_REQUIRE(n_experts >= 0 && n_experts <= MOE_MAX_TOPK, "moe_host_expert_ffn: n_experts=%d out of [0,%d]",
                n_experts, MOE_MAX_TOPK);
    MOE_REQUIRE(n_experts == 0 || (slabs && w), "moe_host_expert_ffn: null slabs/w");
    MOE_REQUIRE(d > 0 && d % 8 == 0 && f > 0 && f % 8 == 0,
                "moe_host_expert_ffn: d=%d f=%d must be positive multiples of 8", d, f);
    for (int j = 0; j < n_experts; ++j) MOE_REQUIRE(slabs[j], "moe_host_expert_ffn: slabs[%d] is null", j);
    reinterpret_cast<moe::HostPool *>(p)->expert_ffn(x, slabs, w, n_experts, d, f, y);
    return MOE_OK;
    MOE_GUARD_END
}

}  // extern "C"
