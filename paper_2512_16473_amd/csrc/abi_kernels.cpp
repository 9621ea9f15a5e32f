// C-ABI entry points of the device kernels: router, hit-expert FFN, combine.
#include <cstring>

#include "common.h"
#include "moe_internal.h"

namespace moe {

static thread_local char g_err[512];

void set_error(const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
}

void clear_error() { g_err[0] = 0; }

}  // namespace moe

extern "C" {

const char *moe_last_error(void) { return moe::g_err; }

int moe_version(void) { return 100; }

size_t moe_slab_bytes(int d, int f)
{
    if (d <= 0 || f <= 0) return 0;
    const size_t b = (size_t)3 * (size_t)d * (size_t)f * 2;
    return (b + 255) & ~(size_t)255;
}

int moe_router_topk(const float *x, const float *w_router, int T, int d, int n, int k,
                    int32_t *idx_out, float *w_out, void *stream)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(T >= 0, "moe_router_topk: T=%d < 0", T);
    MOE_REQUIRE(d > 0 && d % 8 == 0, "moe_router_topk: d=%d must be a positive multiple of 8", d);
    MOE_REQUIRE(n >= 1 && n <= MOE_MAX_EXPERTS, "moe_router_topk: n=%d out of [1,%d]", n, MOE_MAX_EXPERTS);
    MOE_REQUIRE(k >= 1 && k <= n && k <= MOE_MAX_TOPK, "moe_router_topk: k=%d out of [1,min(n,%d)]", k,
                MOE_MAX_TOPK);
    if (T == 0) return MOE_OK;
    MOE_REQUIRE(x && w_router && idx_out && w_out, "moe_router_topk: null pointer");
    MOE_REQUIRE(moe::aligned16(x) && moe::aligned16(w_router), "moe_router_topk: x/w_router not 16-byte aligned");
    MOE_HIP(moe::launch_router(x, w_router, T, d, n, k, idx_out, w_out, (hipStream_t)stream));
    return MOE_OK;
    MOE_GUARD_END
}

size_t moe_ffn_workspace_bytes(int max_jobs, int d, int f_max)
{
    if (max_jobs < 0 || d <= 0 || f_max <= 0) return 0;
    return moe::ffn_workspace_bytes(max_jobs, d, f_max);
}

}  // extern "C"

namespace {

// Argument checks shared by the two hit-FFN entry points (workspace aside).
int check_ffn_hits(const char *fn, const float *x, const void *slot_pool, int n_slots, const int32_t *hit_slots,
                   const float *hit_w, int n_hits, int d, int f, float *y)
{
    MOE_REQUIRE(n_hits >= 0 && n_hits <= MOE_MAX_TOPK, "%s: n_hits=%d out of [0,%d]", fn, n_hits, MOE_MAX_TOPK);
    MOE_REQUIRE(d > 0 && d % 8 == 0 && d <= MOE_MAX_D, "%s: d=%d must be a multiple of 8 in [8,%d]", fn, d,
                MOE_MAX_D);
    MOE_REQUIRE(f > 0 && f % 8 == 0, "%s: f=%d must be a positive multiple of 8", fn, f);
    MOE_REQUIRE(x && y, "%s: null pointer", fn);
    MOE_REQUIRE(n_slots >= 0, "%s: n_slots=%d < 0", fn, n_slots);
    MOE_REQUIRE(n_hits == 0 || (slot_pool && hit_slots && hit_w), "%s: null pointer", fn);
    MOE_REQUIRE(moe::aligned16(x) && moe::aligned16(y) && moe::aligned16(slot_pool),
                "%s: x/y/slot_pool not 16-byte aligned", fn);
    return MOE_OK;
}

// gate/up, down and reduce of the hit experts over a bound workspace.
int run_ffn_hits(const float *x, const void *slot_pool, int n_slots, const int32_t *hit_slots, const float *hit_w,
                 int n_hits, int d, int f, float *y, void *workspace, void *stream)
{
    moe::FfnParams p{};
    p.x = x;
    p.pool = static_cast<const uint8_t *>(slot_pool);
    p.slab_stride = moe_slab_bytes(d, f);
    p.sel = hit_slots;
    p.slotmap = nullptr;
    p.w = hit_w;
    p.k = n_hits;
    p.n = 0;
    p.nslots = n_slots;
    p.shared = nullptr;
    p.f_shared = 0;
    p.d = d;
    p.f = f;
    moe::ffn_bind_workspace(p, workspace, n_hits, d, f);
    hipStream_t s = (hipStream_t)stream;
    MOE_HIP(moe::launch_ffn_stream(p, s, nullptr));
    MOE_HIP(moe::launch_ffn_reduce(p, nullptr, y, s));
    return MOE_OK;
}

}  // namespace

extern "C" {

int moe_expert_ffn_hits(const float *x, const void *slot_pool, int n_slots, const int32_t *hit_slots,
                        const float *hit_w, int n_hits, int d, int f, float *y, void *workspace,
                        size_t workspace_bytes, void *stream)
{
    MOE_GUARD_BEGIN
    int rc = check_ffn_hits("moe_expert_ffn_hits", x, slot_pool, n_slots, hit_slots, hit_w, n_hits, d, f, y);
    if (rc != MOE_OK) return rc;
    MOE_REQUIRE(workspace, "moe_expert_ffn_hits: null workspace");
    MOE_REQUIRE(((uintptr_t)workspace & 255u) == 0, "moe_expert_ffn_hits: workspace not 256-byte aligned");
    const size_t need = moe::ffn_workspace_bytes(n_hits, d, f);
    MOE_REQUIRE(workspace_bytes >= need, "moe_expert_ffn_hits: workspace %zu < %zu bytes", workspace_bytes, need);
    return run_ffn_hits(x, slot_pool, n_slots, hit_slots, hit_w, n_hits, d, f, y, workspace, stream);
    MOE_GUARD_END
}

size_t moe_ffn_noalloc_max_bytes(void) { return moe::kNoAllocScratchBytes; }

int moe_expert_ffn_hits_noalloc(const float *x, const void *slot_pool, int n_slots, const int32_t *hit_slots,
                                const float *hit_w, int n_hits, int d, int f, float *y, void *stream)
{
    MOE_GUARD_BEGIN
    int rc = check_ffn_hits("moe_expert_ffn_hits_noalloc", x, slot_pool, n_slots, hit_slots, hit_w, n_hits, d, f, y);
    if (rc != MOE_OK) return rc;
    const size_t need = moe::ffn_workspace_bytes(n_hits, d, f);
    MOE_REQUIRE(need <= moe::kNoAllocScratchBytes,
                "moe_expert_ffn_hits_noalloc: d=%d f=%d need %zu bytes of scratch, more than its %zu", d, f, need,
                moe::kNoAllocScratchBytes);
    void *scratch = nullptr;
    MOE_HIP(moe::noalloc_scratch(&scratch));
    return run_ffn_hits(x, slot_pool, n_slots, hit_slots, hit_w, n_hits, d, f, y, scratch, stream);
    MOE_GUARD_END
}

int moe_combine(const float *y_gpu, const float *y_host, const float *y_shared, int d, float *out, void *stream)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(d > 0, "moe_combine: d=%d must be positive", d);
    MOE_REQUIRE(out, "moe_combine: null output");
    MOE_HIP(moe::launch_combine(y_gpu, y_host, y_shared, d, out, (hipStream_t)stream));
    return MOE_OK;
    MOE_GUARD_END
}

}  // extern "C"
