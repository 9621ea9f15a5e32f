// Error reporting shared by the C-ABI entry points.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <new>
#include <string>

#include "moe.h"

namespace moe {

void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace moe

#define MOE_REQUIRE(cond, ...)              \
    do {                                    \
        if (!(cond)) {                      \
            ::moe::set_error(__VA_ARGS__);  \
            return MOE_EINVAL;              \
        }                                   \
    } while (0)

#define MOE_HIP(call)                                                                   \
    do {                                                                                \
        hipError_t e_ = (call);                                                         \
        if (e_ != hipSuccess) {                                                         \
            ::moe::set_error("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_),     \
                             __FILE__, __LINE__);                                       \
            return MOE_EHIP;                                                            \
        }                                                                               \
    } while (0)

// Wraps an entry-point body so no C++ exception crosses the ABI.
#define MOE_GUARD_BEGIN try {
#define MOE_GUARD_END                                              \
    }                                                              \
    catch (const std::bad_alloc &) {                               \
        ::moe::set_error("out of host memory");                    \
        return MOE_ENOMEM;                                         \
    }                                                              \
    catch (const std::exception &ex) {                             \
        ::moe::set_error("internal error: %s", ex.what());         \
        return MOE_ESTATE;                                         \
    }                                                              \
    catch (...) {                                                  \
        ::moe::set_error("internal error");                        \
        return MOE_ESTATE;                                         \
    }
