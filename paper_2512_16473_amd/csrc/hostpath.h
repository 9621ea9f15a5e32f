// Host expert path: a persistent thread pool evaluating SwiGLU experts from
// bf16 weights held in host memory (the cache-miss path).
#pragma once

#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace moe {

// How a host row dot product meets the bf16 weights.
enum class HostDot { kFp32 = 1, kBf16 = 2 };

class HostPool {
public:
    explicit HostPool(int n_threads);
    ~HostPool();
    int threads() const { return n_; }
    // Calls fn(tid, begin, end) on contiguous, near-equal ranges of [0, total),
    // one per thread (the caller is thread 0); returns when all are done. Calls from
    // several threads are serialised.
    void parallel_for(int64_t total, const std::function<void(int, int64_t, int64_t)> &fn);
    // y = sum_j w[j] * FFN(slabs[j], x). Calls from several threads are serialised (the
    // pool's threads and scratch serve one call at a time).
    void expert_ffn(const float *x, const void *const *slabs, const float *w, int ne, int d, int f, float *y);
    // Dot-product form used by expert_ffn; kBf16 needs the CPU's AVX512_BF16.
    static bool dot_supported(HostDot k);
    void set_dot(HostDot k);
    HostDot dot() const { return dot_; }

private:
    void worker(int tid);
    void run(int64_t total, const std::function<void(int, int64_t, int64_t)> &fn);
    int n_;
    std::vector<std::thread> th_;
    std::mutex call_mu_;   // one parallel_for / expert_ffn at a time
    std::mutex mu_;
    std::condition_variable cv_go_, cv_done_;
    uint64_t gen_ = 0;
    int pending_ = 0;
    bool stop_ = false;
    int64_t total_ = 0;
    const std::function<void(int, int64_t, int64_t)> *fn_ = nullptr;
    HostDot dot_ = HostDot::kFp32;
    // scratch of the current call, grown on demand
    std::vector<float> h_;                 // [ne][f] activations
    std::vector<uint16_t> xh_, xl_;        // [d] bf16 parts of x (kBf16)
    std::vector<uint16_t> hh_, hl_;        // [ne][f] bf16 parts of h (kBf16)
};

}  // namespace moe
