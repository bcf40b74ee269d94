#include "workers.hpp"

#include <pthread.h>

#include <cstdlib>
#include <thread>
#include <utility>
#include <vector>

#include "common.hpp"

namespace sllm {

namespace {

// One thread and its mailbox.  A worker either runs a task or waits in the
// idle list; it ends when it finishes a task while the list is full.
struct Worker {
    std::mutex mu;
    std::condition_variable cv;
    std::function<void()> task;
    bool has_task = false;
};

// Never destroyed: idle threads wait on their workers until the process
// ends, and a static destructor must not pull the list from under them.
struct Registry {
    std::mutex mu;
    std::vector<Worker*> idle;
};
Registry& registry();

// A child of fork() has only the thread that forked: the idle threads of the
// list do not exist there, so the child forgets them (their Worker records
// leak) and starts new threads when it needs some.  The list's lock is held
// across fork so that the child never inherits it locked.
void before_fork() { registry().mu.lock(); }
void after_fork_parent() { registry().mu.unlock(); }
void after_fork_child() {
    Registry& r = registry();
    r.idle.clear();
    r.mu.unlock();
}

Registry& registry() {
    static Registry* r = [] {
        auto* reg = new Registry;
        (void)pthread_atfork(before_fork, after_fork_parent, after_fork_child);
        return reg;
    }();
    return *r;
}

// Idle threads kept (SLLM_IDLE_WORKERS, at most kMaxIdleWorkers; 0 starts
// every task on a new thread, for comparison), read as each task ends.
uint32_t max_idle() {
    const char* s = std::getenv("SLLM_IDLE_WORKERS");
    if (!s || !*s) return kMaxIdleWorkers;
    char* end = nullptr;
    const long v = std::strtol(s, &end, 10);
    if (!end || *end != '\0' || v < 0) return kMaxIdleWorkers;
    return v < (long)kMaxIdleWorkers ? (uint32_t)v : kMaxIdleWorkers;
}

void worker_main(Worker* w) {
    for (;;) {
        std::function<void()> task;
        {
            std::unique_lock<std::mutex> lk(w->mu);
            w->cv.wait(lk, [&] { return w->has_task; });
            task = std::move(w->task);
            w->task = nullptr;
            w->has_task = false;
        }
        task();
        task = nullptr;  // drop what the task holds before going idle
        Registry& r = registry();
        const uint32_t keep = max_idle();
        {
            std::lock_guard<std::mutex> g(r.mu);
            if (r.idle.size() < keep) {
                r.idle.push_back(w);
                continue;
            }
        }
        delete w;
        return;
    }
}

// Hand `task` to an idle thread, else to a new one.  False if no thread
// could be started (the task is not run).
bool dispatch(std::function<void()> task) {
    Registry& r = registry();
    Worker* w = nullptr;
    if (max_idle() > 0) {
        std::lock_guard<std::mutex> g(r.mu);
        if (!r.idle.empty()) {
            w = r.idle.back();
            r.idle.pop_back();
        }
    }
    if (w) {
        {
            std::lock_guard<std::mutex> g(w->mu);
            w->task = std::move(task);
            w->has_task = true;
        }
        w->cv.notify_one();
        return true;
    }
    w = new (std::nothrow) Worker;
    if (!w) return false;
    w->task = std::move(task);
    w->has_task = true;
    try {
        std::thread(worker_main, w).detach();
    } catch (...) {
        delete w;
        return false;
    }
    return true;
}

}  // namespace

TaskGroup::TaskGroup() : st_(std::make_shared<State>()) {}

TaskGroup::~TaskGroup() { wait(); }

int32_t TaskGroup::start(uint32_t n, std::function<void(uint32_t)> fn) {
    if (started_) return fail(SLLM_E_INVAL, "a task group is started once");
    st_->fn = std::move(fn);
    for (uint32_t i = 0; i < n; ++i) {
        {
            std::lock_guard<std::mutex> g(st_->mu);
            ++st_->running;
        }
        std::shared_ptr<State> st = st_;
        const bool ok = dispatch([st, i] {
            st->fn(i);
            std::lock_guard<std::mutex> g(st->mu);
            if (--st->running == 0) st->cv.notify_all();
        });
        if (!ok) {
            std::lock_guard<std::mutex> g(st_->mu);
            --st_->running;
            return fail(SLLM_E_NOMEM, "cannot start thread %u of %u", i + 1, n);
        }
        ++started_;
    }
    return SLLM_OK;
}

void TaskGroup::wait() {
    std::unique_lock<std::mutex> lk(st_->mu);
    st_->cv.wait(lk, [&] { return st_->running == 0; });
}

uint32_t idle_workers() {
    Registry& r = registry();
    std::lock_guard<std::mutex> g(r.mu);
    return (uint32_t)r.idle.size();
}

}  // namespace sllm
