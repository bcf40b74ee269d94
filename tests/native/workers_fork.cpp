// Kept worker threads across fork(): the child of a process whose threads
// wait idle in the list must not hand tasks to them (they do not exist in
// the child).  The child runs a task group of its own on new threads, under
// an alarm so that a hang ends it; the parent's idle threads still serve
// afterwards.  Prints "ok" and exits 0.
#include <signal.h>
#include <sys/wait.h>
#include <unistd.h>

#include <atomic>
#include <cstdio>

#include "common.hpp"
#include "workers.hpp"

using namespace sllm;

namespace {

// Runs n tasks in one group, each waiting (bounded) until all have started,
// so that they run on n threads; true if each ran once and all met.
bool run_group(uint32_t n) {
    std::atomic<uint32_t> ran{0}, met{0};
    TaskGroup g;
    const int32_t st = g.start(n, [&](uint32_t) {
        ran.fetch_add(1);
        for (int i = 0; i < 20000 && ran.load() < n; ++i) usleep(100);
        if (ran.load() == n) met.fetch_add(1);
    });
    g.wait();
    return st == SLLM_OK && ran.load() == n && met.load() == n;
}

// Waits (bounded) until at least n threads are idle.
bool wait_idle(uint32_t n) {
    for (int i = 0; i < 2000 && idle_workers() < n; ++i) usleep(1000);
    return idle_workers() >= n;
}

}  // namespace

int main() {
    if (!run_group(4) || !wait_idle(4)) {
        std::printf("parent: threads did not go idle\n");
        return 1;
    }
    const pid_t pid = fork();
    if (pid < 0) {
        std::printf("fork failed\n");
        return 1;
    }
    if (pid == 0) {
        alarm(20);
        if (idle_workers() != 0) _exit(3);
        if (!run_group(4)) _exit(4);
        _exit(0);
    }
    int status = 0;
    if (waitpid(pid, &status, 0) != pid || !WIFEXITED(status) || WEXITSTATUS(status) != 0) {
        std::printf("child failed: status 0x%x\n", status);
        return 1;
    }
    const uint32_t idle = idle_workers();
    if (!run_group(4) || idle < 4) {
        std::printf("parent after fork: %u idle threads\n", idle);
        return 1;
    }
    std::printf("ok\n");
    return 0;
}
