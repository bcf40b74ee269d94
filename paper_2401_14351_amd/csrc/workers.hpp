// Threads that outlive the calls that use them.  A streamed load starts one
// reader per I/O thread and the DRAM-tier fill one worker per thread; a new
// OS thread costs tens of microseconds to start (eight of them 0.13-0.28 ms
// on an MI355X host), which is a visible share of a small checkpoint's load.
// Finished tasks leave their thread idle in a process-wide list (at most
// kMaxIdleWorkers of them) for the next task, so a load wakes threads instead
// of creating them, and a thread's per-thread read buffer stays warm.
#pragma once

#include <condition_variable>
#include <cstdint>
#include <functional>
#include <memory>
#include <mutex>

namespace sllm {

constexpr uint32_t kMaxIdleWorkers = 64;

// fn(0) .. fn(n - 1), each on a thread of its own, running concurrently with
// the caller until wait().  The destructor waits too.
class TaskGroup {
  public:
    TaskGroup();
    TaskGroup(const TaskGroup&) = delete;
    TaskGroup& operator=(const TaskGroup&) = delete;
    ~TaskGroup();

    // Start fn(i) for i in [0, n); once per group.  SLLM_E_NOMEM if a thread
    // could not be started; the tasks started before it keep running
    // (started() of them) and wait() still waits for them.
    int32_t start(uint32_t n, std::function<void(uint32_t)> fn);
    uint32_t started() const { return started_; }
    void wait();

  private:
    struct State {
        std::mutex mu;
        std::condition_variable cv;
        uint32_t running = 0;
        std::function<void(uint32_t)> fn;
    };
    std::shared_ptr<State> st_;
    uint32_t started_ = 0;
};

// Idle threads in the process-wide list (for tests).
uint32_t idle_workers();

}  // namespace sllm
