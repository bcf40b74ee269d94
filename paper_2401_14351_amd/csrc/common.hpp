// Shared helpers of the loader library: status/error reporting, checked
// arithmetic and wall-clock time.  Host-only (no HIP).
#pragma once

#include <chrono>
#include <cstdarg>
#include <cstdint>
#include <exception>
#include <new>
#include <string>

#include "sllm.h"

namespace sllm {

// Record a message for sllm_last_error() on this thread and return `code`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// a + b with overflow detection.
inline bool add_ok(uint64_t a, uint64_t b, uint64_t* out) { return !__builtin_add_overflow(a, b, out); }
inline bool mul_ok(uint64_t a, uint64_t b, uint64_t* out) { return !__builtin_mul_overflow(a, b, out); }

inline bool is_pow2(uint64_t a) { return a != 0 && (a & (a - 1)) == 0; }

// Smallest multiple of the power of two `a` that is >= x (false on overflow).
inline bool align_up(uint64_t x, uint64_t a, uint64_t* out) {
    uint64_t t;
    if (!add_ok(x, a - 1, &t)) return false;
    *out = t & ~(a - 1);
    return true;
}

inline uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }

inline double now_s() {
    using namespace std::chrono;
    return duration<double>(steady_clock::now().time_since_epoch()).count();
}

// Log level from SLLM_LOG_LEVEL (0 quiet, 1 info, 2 debug).
int log_level();
void log_msg(int level, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Named host ranges for rocprofv3's marker trace (roctx), when SLLM_ROCTX=1
// and the ROCm roctx library can be loaded at run time; otherwise each call
// costs one check.  Ranges nest per thread.
void range_push(const char* name);
void range_pop();

class Range {
  public:
    explicit Range(const char* name) { range_push(name); }
    ~Range() { range_pop(); }
    Range(const Range&) = delete;
    Range& operator=(const Range&) = delete;
};

}  // namespace sllm

// Closes the function-try-block of an extern "C" entry point that returns a
// status: no C++ exception crosses the C ABI.
#define SLLM_CATCH_ALL                                                          \
    catch (const std::bad_alloc&) {                                             \
        return ::sllm::fail(SLLM_E_NOMEM, "out of host memory");                \
    }                                                                           \
    catch (const std::exception& sllm_exc_) {                                   \
        return ::sllm::fail(SLLM_E_INVAL, "unexpected error: %s", sllm_exc_.what()); \
    }                                                                           \
    catch (...) {                                                               \
        return ::sllm::fail(SLLM_E_INVAL, "unexpected error");                  \
    }

// Evaluate a status-returning expression and return its status on failure.
#define SLLM_TRY(expr)                      \
    do {                                    \
        int32_t _st = (expr);               \
        if (_st != SLLM_OK) return _st;     \
    } while (0)
