#include "common.hpp"

#include <dlfcn.h>

#include <cstdio>
#include <cstdlib>

namespace sllm {

namespace {
thread_local std::string t_last_error;
}

int32_t fail(int32_t code, const char* fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_last_error = buf;
    log_msg(1, "error %d: %s", code, buf);
    return code;
}

void clear_error() { t_last_error.clear(); }

int log_level() {
    static const int level = [] {
        const char* s = std::getenv("SLLM_LOG_LEVEL");
        return s ? std::atoi(s) : 0;
    }();
    return level;
}

void log_msg(int level, const char* fmt, ...) {
    if (log_level() < level) return;
    va_list ap;
    va_start(ap, fmt);
    std::fprintf(stderr, "[sllm] ");
    std::vfprintf(stderr, fmt, ap);
    std::fprintf(stderr, "\n");
    va_end(ap);
}

namespace {

struct Roctx {
    int (*push)(const char*) = nullptr;
    int (*pop)() = nullptr;
};

// resolved once: the roctx entry points, or none
const Roctx& roctx() {
    static const Roctx r = [] {
        Roctx x;
        const char* on = std::getenv("SLLM_ROCTX");
        if (!on || *on != '1') return x;
        for (const char* lib : {"librocprofiler-sdk-roctx.so.1", "librocprofiler-sdk-roctx.so", "libroctx64.so.4"}) {
            void* h = dlopen(lib, RTLD_NOW | RTLD_LOCAL);
            if (!h) continue;
            auto push = reinterpret_cast<int (*)(const char*)>(dlsym(h, "roctxRangePushA"));
            auto pop = reinterpret_cast<int (*)()>(dlsym(h, "roctxRangePop"));
            if (push && pop) {
                x.push = push;
                x.pop = pop;
                log_msg(1, "roctx ranges through %s", lib);
                return x;
            }
            dlclose(h);
        }
        log_msg(1, "SLLM_ROCTX=1 but no roctx library could be loaded");
        return x;
    }();
    return r;
}

}  // namespace

void range_push(const char* name) {
    const Roctx& r = roctx();
    if (r.push) r.push(name);
}

void range_pop() {
    const Roctx& r = roctx();
    if (r.pop) r.pop();
}

}  // namespace sllm

extern "C" const char* sllm_last_error(void) { return sllm::t_last_error.c_str(); }

extern "C" const char* sllm_strerror(int32_t code) {
    switch (code) {
        case SLLM_OK: return "SLLM_OK";
        case SLLM_E_INVAL: return "SLLM_E_INVAL";
        case SLLM_E_IO: return "SLLM_E_IO";
        case SLLM_E_FORMAT: return "SLLM_E_FORMAT";
        case SLLM_E_NOMEM: return "SLLM_E_NOMEM";
        case SLLM_E_HIP: return "SLLM_E_HIP";
        case SLLM_E_RANGE: return "SLLM_E_RANGE";
        case SLLM_E_BUSY: return "SLLM_E_BUSY";
        case SLLM_E_NOTFOUND: return "SLLM_E_NOTFOUND";
        default: return "SLLM_E_UNKNOWN";
    }
}
