// Host check of the stream fork / join ordering (fork_join.hpp) with
// stand-in stream operations: records every call, injects failures, and
// checks that the caller's stream always ends up waiting for the side
// stream once work was put there.  Built with g++; no device is used.
#include <cstdio>
#include <string>
#include <vector>

#include "fork_join.hpp"

using elsaa::StreamOps;

namespace {

std::vector<std::string> g_log;
int g_fail_at = -1;     // index of the stream operation that fails (-1: none)
int g_ops = 0;

hipStream_t kMain = reinterpret_cast<hipStream_t>(0x10);
hipStream_t kSide = reinterpret_cast<hipStream_t>(0x20);
hipEvent_t kFork = reinterpret_cast<hipEvent_t>(0x30);
hipEvent_t kJoin = reinterpret_cast<hipEvent_t>(0x40);

const char* sname(hipStream_t s) { return s == kMain ? "main" : s == kSide ? "side" : "?"; }
const char* ename(hipEvent_t e) { return e == kFork ? "fork" : e == kJoin ? "join" : "?"; }

hipError_t op_result() { return g_ops++ == g_fail_at ? hipErrorInvalidValue : hipSuccess; }

hipError_t fake_record(hipEvent_t e, hipStream_t s)
{
    g_log.push_back(std::string("record ") + ename(e) + " on " + sname(s));
    return op_result();
}
hipError_t fake_wait(hipStream_t s, hipEvent_t e, unsigned int)
{
    g_log.push_back(std::string("wait ") + sname(s) + " for " + ename(e));
    return op_result();
}
hipError_t fake_sync(hipStream_t s)
{
    g_log.push_back(std::string("sync ") + sname(s));
    return hipSuccess;
}
hipError_t fake_clear() { return hipSuccess; }

const StreamOps kOps = {fake_record, fake_wait, fake_sync, fake_clear};

int g_bad = 0;

void expect(const char* what, hipError_t got, hipError_t want, const std::vector<std::string>& log)
{
    if (got != want || g_log != log) {
        ++g_bad;
        std::printf("FAIL %s: status %d (want %d)\n", what, (int)got, (int)want);
        for (auto& l : g_log) std::printf("   got:  %s\n", l.c_str());
        for (auto& l : log) std::printf("   want: %s\n", l.c_str());
    } else {
        std::printf("ok   %s\n", what);
    }
}

hipError_t run(int fail_op, hipError_t first_rc, hipError_t second_rc)
{
    g_log.clear();
    g_ops = 0;
    g_fail_at = fail_op;
    auto first = [&](hipStream_t s) {
        g_log.push_back(std::string("first on ") + sname(s));
        return first_rc;
    };
    auto second = [&](hipStream_t s) {
        g_log.push_back(std::string("second on ") + sname(s));
        return second_rc;
    };
    return elsaa::fork_join(kOps, kMain, kSide, kFork, kJoin, first, second);
}

}  // namespace

int main()
{
    const hipError_t ok = hipSuccess, bad = hipErrorLaunchFailure, inval = hipErrorInvalidValue;
    const std::vector<std::string> full = {"record fork on main", "wait side for fork", "first on side",
                                           "second on main", "record join on side", "wait main for join"};
    expect("all succeed", run(-1, ok, ok), ok, full);
    expect("first part fails: join still recorded and waited", run(-1, bad, ok), bad, full);
    expect("second part fails: join still recorded and waited", run(-1, ok, bad), bad, full);
    expect("both fail: first error returned", run(-1, hipErrorOutOfMemory, bad), hipErrorOutOfMemory, full);
    expect("join record fails: side stream drained on the host", run(2, ok, ok), inval,
           {"record fork on main", "wait side for fork", "first on side", "second on main", "record join on side",
            "sync side"});
    expect("join wait fails: side stream drained on the host", run(3, ok, ok), inval,
           {"record fork on main", "wait side for fork", "first on side", "second on main", "record join on side",
            "wait main for join", "sync side"});
    expect("fork record fails: both parts on main in order", run(0, ok, ok), ok,
           {"record fork on main", "first on main", "second on main"});
    expect("fork wait fails: both parts on main in order", run(1, ok, ok), ok,
           {"record fork on main", "wait side for fork", "first on main", "second on main"});
    expect("fork fails and first part fails: second not run", run(0, bad, ok), bad,
           {"record fork on main", "first on main"});
    std::printf("%s\n", g_bad ? "FAILED" : "ALL OK");
    return g_bad ? 1 : 0;
}
