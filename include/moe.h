/*
 * moe.h -- C ABI of the MI355X (gfx950) MoE expert-stage library (libmoe.so).
 *
 * The library implements the per-layer MoE expert stage of single-request decode
 * from Huang, Lin, Lee, "Efficient CPU-GPU Collaborative Inference for MoE-based
 * LLMs on Memory-Limited Systems" (ASP-DAC 2026): router gating, lookup of the
 * selected experts in a per-layer set-associative GPU expert cache with LRU
 * eviction, the SwiGLU FFN of cache-hit experts on the GPU, the FFN of missed
 * experts on a host thread pool, asynchronous post-fetch of missed experts into
 * the cache for later tokens, and the weighted combine (Section III-A steps 1-3,
 * Section III-B cache design, Section III-C copy streams). A batched prefill path
 * (all experts resident, grouped by expert, MFMA GEMMs) is also exported.
 *
 * Conventions
 *   - Every function returning int returns MOE_OK (0) or a negative MOE_E* code;
 *     moe_last_error() then holds a message (thread-local). No call aborts and no
 *     C++ exception crosses the ABI. On an argument error nothing is written.
 *   - The caller owns every buffer it passes (device memory, pinned host memory,
 *     streams). The library owns only its opaque handles and what they allocate
 *     at creation; nothing is allocated on the per-token path.
 *   - "device" pointers are HIP device addresses on the current device; "host"
 *     pointers are CPU addresses. Streams are hipStream_t passed as void*; NULL is
 *     the null stream. Device outputs are valid in stream order; host outputs are
 *     valid when the call returns.
 *   - Device pointers must be 16-byte aligned; d and f must be multiples of 8.
 *   - Expert slab layout (one contiguous block per expert, bf16, row-major
 *     [out, in]): W1 [f][d] | W3 [f][d] | W2 [d][f]. A slot pool is an array of
 *     slabs with stride moe_slab_bytes(d, f).
 *   - Expert FFN (Table II sizes read as three d x f matrices): SwiGLU,
 *     y = W2 (SiLU(W1 x) * (W3 x)), bf16 weights, fp32 activations and
 *     accumulation.
 *   - Router (Section I; Table II top-K): logits l = W_r x, p = softmax(l), the k
 *     largest logits with ties to the lower expert id, ordered by (logit desc, id
 *     asc), gate weights w = p_S / sum(p_S).
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_OK        0
#define MOE_EINVAL   -1   /* bad argument (null pointer, size, alignment) */
#define MOE_EHIP     -2   /* a HIP runtime call or kernel launch failed */
#define MOE_ESTATE   -3   /* handle in the wrong state for this call */
#define MOE_ENOMEM   -4   /* allocation at handle creation failed */

#define MOE_MAX_EXPERTS 256   /* n (experts per layer) upper bound */
#define MOE_MAX_TOPK     16   /* k upper bound */
#define MOE_MAX_D      8192   /* d_model upper bound of the GEMV kernels */
#define MOE_MAX_TOKENS    8   /* tokens per call of moe_expert_ffn_tokens */
#define MOE_TOKENS_LDS_BYTES 131072   /* moe_expert_ffn_tokens: T * d * 4 bytes at most */

/* Message of the last failing call on the calling thread ("" if none). */
const char *moe_last_error(void);

/* ABI version (major*100 + minor). */
int moe_version(void);

/* Bytes of one expert slab: 3*d*f*2 rounded up to 256. 0 on bad sizes. */
size_t moe_slab_bytes(int d, int f);

/* ------------------------------------------------------------------------- */
/* Router gating (Section I MoE layer; Table II top-K).                       */
/* ------------------------------------------------------------------------- */
/*
 * x         device fp32 [T][d] hidden states
 * w_router  device fp32 [n][d] router weights (row-major)
 * idx_out   device int32 [T][k] selected experts, ordered (logit desc, id asc)
 * w_out     device fp32  [T][k] gate weights in the same order (sum to 1)
 * 1 <= k <= min(n, MOE_MAX_TOPK), n <= MOE_MAX_EXPERTS, T >= 0 (T == 0 is a no-op).
 * Logits are accumulated in fp64 from the fp32 inputs.
 */
int moe_router_topk(const float *x, const float *w_router, int T, int d, int n, int k,
                    int32_t *idx_out, float *w_out, void *stream);

/* ------------------------------------------------------------------------- */
/* Expert cache: N-index (one per layer), M-way (Section III-B).             */
/* ------------------------------------------------------------------------- */
/*
 * Host-side slot table. Each layer owns one set of `ways` slots, initially empty.
 * Policy (readings of points the paper leaves open): hits are decided for all
 * selected experts against the state before the token; the set is then updated in
 * ascending expert-id order, a hit refreshing its slot's recency and a miss taking
 * the lowest-index empty slot, else the least recently used slot whose expert is
 * not selected by the current token. Every miss is inserted (step 3, post-fetch),
 * so ways >= top_k is required.
 */
typedef struct moe_cache moe_cache;

/* LRU cache. EINVAL unless 1 <= top_k <= ways <= n_experts <= MOE_MAX_EXPERTS, n_layers >= 1. */
int moe_cache_create(int n_layers, int n_experts, int ways, int top_k, moe_cache **out);

/*
 * Replacement policies compared in Section IV-D:
 *   MOE_POLICY_LRU    the paper's policy (above);
 *   MOE_POLICY_FIFO   as LRU, except that a hit does not refresh its slot, so the victim
 *                     is the earliest-inserted slot whose expert is not selected;
 *   MOE_POLICY_STATIC the paper's "random" policy: each set holds a fixed content of
 *                     `ways` experts for ever; misses are never inserted (no post-fetch).
 */
#define MOE_POLICY_LRU 0
#define MOE_POLICY_FIFO 1
#define MOE_POLICY_STATIC 2
/*
 * Cache with a policy. n_layers >= 0 sets (the covered layers; a runtime with more
 * layers runs the others entirely on the host). static_content: host int32
 * [n_layers][ways], distinct expert ids per layer, required for MOE_POLICY_STATIC
 * (the caller draws it, e.g. uniformly at random) and ignored otherwise; it is
 * copied. LRU/FIFO need top_k <= ways <= n_experts; STATIC needs 1 <= ways <= n_experts.
 */
int moe_cache_create_policy(int n_layers, int n_experts, int ways, int top_k, int policy,
                            const int32_t *static_content, moe_cache **out);
void moe_cache_destroy(moe_cache *c);
/* Back to the initial state: every set empty (LRU, FIFO) or the static content. */
int moe_cache_reset(moe_cache *c);
/*
 * Cache geometry from a memory budget (Section III-B): slots S = floor(budget_bytes /
 * expert_bytes), indexes N = floor(S / ways); covered_out = min(N, n_layers), the
 * layers 0..covered-1 that own a set. Either output may be NULL.
 */
int moe_cache_geometry(size_t budget_bytes, size_t expert_bytes, int ways, int n_layers,
                       int *slots_out, int *covered_out);
/*
 * Step 1 (cache check), pure. experts: host [k] distinct ids in [0, n).
 * slot_out: host [k] slot holding each expert, -1 on a miss; hit_out: host [k] 0/1.
 */
int moe_cache_lookup(const moe_cache *c, int layer, const int32_t *experts, int k,
                     int32_t *slot_out, uint8_t *hit_out);
/*
 * Check and update for one token at one layer (LRU step). Outputs aligned with
 * `experts`: fill_slot_out[j] = slot the missed expert j is inserted into (-1 on a
 * hit); evicted_out[j] = expert removed from that slot (-1 if it was empty or on a
 * hit). Either output may be NULL.
 */
int moe_cache_update(moe_cache *c, int layer, const int32_t *experts, int k,
                     int32_t *fill_slot_out, int32_t *evicted_out);
/*
 * moe_cache_update where insert (host uint8 [k], aligned with `experts`, NULL = all 1)
 * marks which misses may be inserted: a miss with insert[j] = 0 (its post-fetch was not
 * issued) takes no slot and evicts nothing (fill_slot_out[j] = evicted_out[j] = -1),
 * though it still advances the set's clock. Hits ignore the mask.
 */
int moe_cache_update_masked(moe_cache *c, int layer, const int32_t *experts, int k,
                            const uint8_t *insert, int32_t *fill_slot_out, int32_t *evicted_out);
/*
 * Expert -> slot table of one layer: host [n], -1 for experts not cached. (The device
 * [L][n] mirror that the hit kernels read belongs to the runtime, which installs a row
 * only once its post-fetch copies have landed; moe_runtime_device_slotmap reads it.)
 */
int moe_cache_slotmap(const moe_cache *c, int layer, int32_t *slotmap_out);
/*
 * Checkpoint and resume of the cache state (every set's slot contents, their recency
 * stamps and the set clocks), so a stopped decode can continue with the same hit/miss
 * sequence. moe_cache_state_bytes gives the size of a state (0 for NULL). moe_cache_save
 * writes it into host memory `buf` of `bytes` >= that size. moe_cache_restore loads a
 * saved state into a cache created with the same geometry, policy and static content;
 * `bytes` must equal the state size. It returns MOE_EINVAL, leaving the cache unchanged,
 * for another geometry or policy, or an inconsistent state: an expert id out of range or
 * in two slots of a set, a resident slot stamped 0, after its set's clock or with
 * another slot's stamp, a static set that differs from its content. A runtime created
 * over the restored cache fills the slots it holds (moe_runtime_create).
 */
size_t moe_cache_state_bytes(const moe_cache *c);
int moe_cache_save(const moe_cache *c, void *buf, size_t bytes);
int moe_cache_restore(moe_cache *c, const void *buf, size_t bytes);

/* ------------------------------------------------------------------------- */
/* Cache-hit expert FFN on the GPU (Section III-A step 2(a)).                 */
/* ------------------------------------------------------------------------- */
/* Device workspace bytes for up to max_jobs experts of d_ffn <= f_max. */
size_t moe_ffn_workspace_bytes(int max_jobs, int d, int f_max);
/*
 * y = sum_j hit_w[j] * FFN(slab at slot_pool + hit_slots[j]*moe_slab_bytes(d,f), x)
 * x          device fp32 [d]
 * slot_pool  device bf16 slabs, n_slots of them
 * hit_slots  device int32 [n_hits]; entries outside [0, n_slots) are skipped
 * hit_w      device fp32 [n_hits]
 * y          device fp32 [d] (overwritten)
 * workspace  device, >= moe_ffn_workspace_bytes(n_hits, d, f)
 * 0 <= n_hits <= MOE_MAX_TOPK; d <= MOE_MAX_D.
 */
int moe_expert_ffn_hits(const float *x, const void *slot_pool, int n_slots, const int32_t *hit_slots,
                        const float *hit_w, int n_hits, int d, int f, float *y,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * moe_expert_ffn_hits without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc). Same arguments, kernels and results as moe_expert_ffn_hits; the
 * job header, h and the split-K partials live in a library-owned static device array
 * of moe_ffn_noalloc_max_bytes() bytes (8 MiB), one per device, held until the process
 * ends. The call allocates nothing (no hipMalloc, hipFree or allocating library call).
 * MOE_EINVAL when moe_ffn_workspace_bytes(n_hits, d, f) exceeds that size (d = 4096
 * allows f up to about 40k), besides the argument errors of moe_expert_ffn_hits. Every
 * call on a device shares that device's array: calls that overlap on one device (two
 * streams, two threads) race and must be ordered by the caller.
 */
size_t moe_ffn_noalloc_max_bytes(void);
int moe_expert_ffn_hits_noalloc(const float *x, const void *slot_pool, int n_slots, const int32_t *hit_slots,
                                const float *hit_w, int n_hits, int d, int f, float *y, void *stream);

/*
 * Several decode tokens at once (a small batch), every selected expert resident:
 *   y[t] = sum_j w[t][j] * FFN(slab at slot_pool + slots[t][j]*moe_slab_bytes(d,f), x[t])
 * for t < T. Each slab is read from HBM once for all the tokens that selected it (the
 * one-token path run per token would read it once per token). Not in the paper: the
 * bridge between single-token decode and prefill. The fp32 activations meet the bf16
 * weights as two bf16 parts (hi + lo, within 2^-18 relative of the fp32 value) with
 * exact products and fp32 sums, so results agree with the one-token path to fp32
 * accumulation order.
 * x          device fp32 [T][d]
 * slot_pool  device bf16 slabs, n_slots of them
 * slots      device int32 [T][k]; entries outside [0, n_slots) are skipped; a slot listed
 *            more than once (by one token or several) contributes once per listing, each
 *            with its own weight (routing gives distinct experts per token)
 * w          device fp32 [T][k] gate weights
 * y          device fp32 [T][d] (overwritten; zero for a token with no valid slot)
 * workspace  device, 256-byte aligned, >= moe_ffn_tokens_workspace_bytes(T, k, d, f)
 * 1 <= T <= MOE_MAX_TOKENS, 1 <= k <= MOE_MAX_TOPK, d % 8 == 0, d <= MOE_MAX_D,
 * f % 8 == 0, T*d*4 <= MOE_TOKENS_LDS_BYTES; MOE_EINVAL otherwise.
 */
size_t moe_ffn_tokens_workspace_bytes(int T, int k, int d, int f);
int moe_expert_ffn_tokens(const float *x, const void *slot_pool, int n_slots, const int32_t *slots,
                          const float *w, int T, int k, int d, int f, float *y,
                          void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------- */
/* Weighted combine (Section I layer output; Section III-A hit/miss split).   */
/* ------------------------------------------------------------------------- */
/*
 * out = y_gpu + y_host + y_shared over d elements, where y_gpu is the gate-weighted
 * sum of the cache-hit experts, y_host that of the missed experts (computed on the
 * host and copied in), y_shared an always-active expert with weight 1. Each input
 * is device fp32 [d] and may be NULL (treated as zero). out: device fp32 [d].
 */
int moe_combine(const float *y_gpu, const float *y_host, const float *y_shared, int d,
                float *out, void *stream);

/* ------------------------------------------------------------------------- */
/* Host expert path for cache misses (Section III-A step 2(b); Section I       */
/* OMP_NUM_THREADS study).                                                    */
/* ------------------------------------------------------------------------- */
typedef struct moe_host_pool moe_host_pool;

/* n_threads <= 0: OMP_NUM_THREADS if set, else the hardware thread count. */
int moe_host_pool_create(int n_threads, moe_host_pool **out);
void moe_host_pool_destroy(moe_host_pool *p);
int moe_host_pool_threads(const moe_host_pool *p);
/*
 * Form of the host path's row dot products (the Table III CPU study on this host):
 *   MOE_HOST_DOT_FP32  bf16 weights widened to fp32, fp32 FMAs (AVX-512F when the CPU
 *                      has it, else scalar). The default.
 *   MOE_HOST_DOT_BF16  the AVX512_BF16 pair-dot instruction (exact bf16 x bf16 products,
 *                      fp32 sums); x and h are each split into two bf16 parts hi + lo with
 *                      |v - hi - lo| <= 2^-18 |v|, so results stay at fp32-accumulation
 *                      error. MOE_EINVAL on a CPU without AVX512_BF16.
 *   MOE_HOST_DOT_AUTO  the default form.
 * Either way each output row is one thread's fixed-order sum. moe_host_pool_get_dot
 * returns the form in use (FP32 or BF16), or MOE_EINVAL for a null handle.
 */
#define MOE_HOST_DOT_AUTO 0
#define MOE_HOST_DOT_FP32 1
#define MOE_HOST_DOT_BF16 2
int moe_host_pool_set_dot(moe_host_pool *p, int kind);
int moe_host_pool_get_dot(const moe_host_pool *p);
/*
 * y = sum_j w[j] * FFN(slabs[j], x), all host memory: x fp32 [d], slabs[j] bf16
 * slab pointers, w fp32 [n_experts], y fp32 [d] (overwritten). Rows are split
 * across the pool's threads; each row is one thread's fixed-order sum, so the
 * result does not depend on the thread count. 0 <= n_experts <= MOE_MAX_TOPK.
 * A pool serves one call at a time: calls that overlap (from several threads, or
 * several runtimes sharing the pool) are serialised.
 */
int moe_host_expert_ffn(moe_host_pool *p, const float *x, const void *const *slabs,
                        const float *w, int n_experts, int d, int f, float *y);

/*
 * Pinned (page-locked) host memory for expert slabs and staging, so post-fetch
 * copies run as asynchronous DMA. moe_host_alloc returns EINVAL for bytes == 0,
 * ENOMEM if the allocation fails; moe_host_free(NULL) is a no-op.
 */
int moe_host_alloc(size_t bytes, void **out);
int moe_host_free(void *ptr);

/* ------------------------------------------------------------------------- */
/* One MoE layer for one decode token: steps 1-3 of Section III-A.            */
/* ------------------------------------------------------------------------- */
typedef struct moe_layer_desc {
    int d, f;            /* d_model, d_ffn of a routed expert */
    int n, k;            /* experts per layer, experts per token */
    int ways;            /* cache slots per layer (M) */
    int n_layers;        /* layers; the first cache->n_layers own a cache set, the rest
                            (uncovered, Section III-B) run every expert on the host */
    int f_shared;        /* d_ffn of an always-active shared expert, 0 = none */
    const float *w_router;       /* device fp32 [n_layers][n][d] */
    void *slot_pool;             /* device, covered*ways slabs (layer-major), stride moe_slab_bytes(d,f);
                                    may be NULL when no layer is covered */
    const void *shared_pool;     /* device, n_layers slabs of moe_slab_bytes(d,f_shared), or NULL */
    const void *const *host_slabs; /* host array of n_layers*n pointers to pinned host slabs (copied at create) */
    moe_cache *cache;            /* covered <= n_layers sets, `ways` ways, top_k == k (borrowed) */
    moe_host_pool *pool;         /* host thread pool (borrowed) */
} moe_layer_desc;

typedef struct moe_runtime moe_runtime;

/*
 * Allocates at creation (never per token): device workspace, device expert->slot
 * mirror [n_layers][n], pinned staging, events. Slots the cache already holds at
 * creation (a static content, a warm cache) are filled from the host slabs then,
 * synchronously, so the pool is consistent with the cache.
 */
int moe_runtime_create(const moe_layer_desc *desc, moe_runtime **out);
void moe_runtime_destroy(moe_runtime *rt);

/*
 * One token through one layer.
 * x_dev    device fp32 [d] hidden state; out_dev device fp32 [d] routed-expert output
 *          (+ shared expert).
 * idx_host host int32 [k], w_host host fp32 [k]: routing in rank order (nullable).
 * hit_host host uint8 [k]: 1 if the expert ran on the GPU as a cache hit (nullable); in
 *          parity mode exactly the cache hits.
 * compute_stream runs the router, hit FFN and combine; copy_stream the post-fetch of
 * missed experts. act_stream is accepted for ABI stability and may be NULL: the
 * router kernel itself writes the routing and the hidden state into coherent pinned
 * memory that the host polls, so activations never queue behind weight copies
 * (Section III-C keeps them apart). The call returns after the host part (cache
 * update, miss FFN) is done and the device work is enqueued. Post-fetched experts
 * become usable from the next token at this layer; that next use waits for the copy.
 * Calls on one runtime must not overlap (one calling thread at a time).
 * Errors: MOE_EINVAL for bad arguments, with nothing changed. MOE_EHIP (a HIP failure,
 * or routing not published within 60 s) can come after this call's cache update and
 * copies were applied in part; the runtime is then unusable and must be destroyed.
 */
int moe_layer_forward(moe_runtime *rt, int layer, const float *x_dev, float *out_dev,
                      int32_t *idx_host, float *w_host, uint8_t *hit_host,
                      void *compute_stream, void *act_stream, void *copy_stream);

/*
 * One decode token through layers 0..n_layers-1 (moe_layer_forward in order).
 * x_dev, out_dev: device fp32 [n_layers][d]; idx_host/w_host/hit_host: host
 * [n_layers][k] (nullable).
 */
int moe_decode_step(moe_runtime *rt, const float *x_dev, float *out_dev, int32_t *idx_host,
                    float *w_host, uint8_t *hit_host, void *compute_stream, void *act_stream,
                    void *copy_stream);

/*
 * Bounded post-fetch. With max_slabs_in_flight = Q > 0, a missed expert is post-fetched
 * (and inserted into the cache) only while fewer than Q slabs are still being copied on
 * the copy stream; the other misses run on the host as usual but are not inserted
 * (moe_cache_update_masked semantics), so tokens never queue behind a backlog of
 * weight copies. The budget goes to the misses in ascending expert id. Which misses are
 * inserted then depends on copy timing; the cache table records it. Q = 0 (the
 * default) inserts every miss, as Section III-A step 3 describes.
 */
int moe_runtime_set_fill_limit(moe_runtime *rt, int max_slabs_in_flight);

/*
 * Non-blocking post-fetch (enable != 0). By default (parity mode) a layer call whose set
 * still has a post-fetch in flight makes the compute stream wait for it, so a fetched
 * expert is used from the next token on and the hit/miss sequence does not depend on
 * timing. In non-blocking mode the call does not wait: experts whose copy has not
 * landed are run on the host for that call ("in flight => miss"); the cache table
 * (moe_cache_*) evolves exactly as in parity mode, only where experts run differs.
 * hit_host reports where each expert ran (1 = GPU).
 */
int moe_runtime_set_nonblocking(moe_runtime *rt, int enable);

/*
 * Blocks until every copy the runtime enqueued has finished and the device mirror holds
 * every landed post-fetch (synchronises the device).
 */
int moe_runtime_sync(moe_runtime *rt);

/* Device expert->slot mirror of one layer copied to host [n] (synchronous). */
int moe_runtime_device_slotmap(moe_runtime *rt, int layer, int32_t *slotmap_out);

/* Counters of the work done so far. */
typedef struct moe_runtime_stats {
    int64_t layer_calls;      /* moe_layer_forward calls */
    int64_t expert_hits;      /* selected experts found in the cache */
    int64_t expert_misses;    /* selected experts computed on the host */
    int64_t fills;            /* slabs post-fetched into the cache */
    double host_ffn_ms;       /* wall time of the host expert path */
    double route_wait_ms;     /* host time blocked on the routing read-back */
    /* kernel timing (only while timing is enabled, see moe_runtime_set_timing) */
    int64_t gate_up_launches;
    double gate_up_ms;        /* summed event time of the gate/up/SiLU kernel */
    double gate_up_bytes;     /* algorithmic bytes those launches read and wrote */
    int64_t down_launches;
    double down_ms;
    double down_bytes;
    int64_t fills_skipped;    /* misses not post-fetched because of the fill limit */
    int64_t inflight_misses;  /* cache hits run on the host because their post-fetch had
                                 not landed (non-blocking mode) */
} moe_runtime_stats;

/*
 * enable != 0: record HIP events around the hit-FFN kernels on the compute stream.
 * Turning timing off (or calling moe_runtime_stats) resolves pending events; the
 * caller must have synchronised the compute stream first.
 */
int moe_runtime_set_timing(moe_runtime *rt, int enable);
int moe_runtime_get_stats(moe_runtime *rt, moe_runtime_stats *out);
int moe_runtime_reset_stats(moe_runtime *rt);

/* ------------------------------------------------------------------------- */
/* Prefill: T tokens, all experts resident (no cache), grouped by expert.     */
/* ------------------------------------------------------------------------- */
typedef struct moe_prefill_desc {
    int d, f, n, k;
    const float *w_router;    /* device fp32 [n][d] */
    const void *expert_pool;  /* device, n slabs, stride moe_slab_bytes(d,f) */
} moe_prefill_desc;

size_t moe_prefill_workspace_bytes(const moe_prefill_desc *P, int T);
/*
 * OUT[t] = sum_j w[t][j] FFN_{idx[t][j]}(X[t]) for t < T.
 * X_dev device fp32 [T][d]; OUT_dev device fp32 [T][d]; idx_dev/w_dev device
 * [T][k] routing outputs (nullable). Activations are rounded to bf16 for the
 * matrix cores; accumulation is fp32. The workspace (device, 256-byte aligned,
 * >= moe_prefill_workspace_bytes(P, T)) holds the grouping and the intermediate
 * activations, so the call allocates nothing. d and f must be multiples of 128
 * (d <= MOE_MAX_D); MOE_EINVAL otherwise; T == 0 is a no-op.
 */
int moe_prefill_forward(const moe_prefill_desc *P, const float *X_dev, int T, float *OUT_dev,
                        int32_t *idx_dev, float *w_dev, void *workspace, size_t workspace_bytes,
                        void *stream);

/* ------------------------------------------------------------------------- */
/* Measurement yardstick (not part of the method).                           */
/* ------------------------------------------------------------------------- */
/*
 * Reads `bytes` bytes at `buf` (device, 16-byte aligned; bytes a multiple of 16) with
 * 16-byte nontemporal loads, 64 lanes covering 1 KiB per load (the access pattern of
 * the decode weight kernels). The rate at which it runs is the practical HBM read
 * ceiling that the weight-streaming kernels are compared with. `sink` (device, 4 bytes,
 * caller-owned) receives a word only if a lane's XOR fold of what it read equals a
 * fixed constant, which keeps the loads from being removed. grid = work groups of 256
 * threads (0: eight per compute unit). Launched on `stream`; the caller times it.
 * MOE_EINVAL on a null or misaligned pointer, bytes % 16 != 0 or grid < 0; bytes == 0
 * launches nothing.
 */
int moe_read_stream(const void *buf, size_t bytes, uint32_t *sink, int grid, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* MOE_H */
