// fork_join.hpp -- run two independent parts of one call on two streams.
//
// first(side) runs on a second stream and second(main) on the caller's
// stream, both ordered after everything `main` already holds; `main` then
// waits for the second stream, so the call behaves as if both parts ran on
// `main`.  The stream and event calls go through StreamOps so the ordering
// logic can be exercised on the host with stand-ins (no device needed).
#pragma once
#include <hip/hip_runtime_api.h>

namespace elsaa {

struct StreamOps {
    hipError_t (*record)(hipEvent_t, hipStream_t);
    hipError_t (*wait)(hipStream_t, hipEvent_t, unsigned int);
    hipError_t (*sync)(hipStream_t);
    hipError_t (*clear)();                   // reset the thread's sticky error after a failed call
};

// If the fork cannot be recorded, both parts run on `main` in order.  Once
// anything has been enqueued on the side stream, the join is recorded and
// waited for on every path (when that fails, the side stream is drained on
// the host instead), so `main` is ordered after the side stream's work even
// when a launch failed.  Returns the first error: first's, second's, then
// the join's.
template <class A, class B>
hipError_t fork_join(const StreamOps& ops, hipStream_t main, hipStream_t side, hipEvent_t fork, hipEvent_t join,
                     A first, B second)
{
    if (ops.record(fork, main) != hipSuccess || ops.wait(side, fork, 0) != hipSuccess) {
        (void)ops.clear();
        const hipError_t e = first(main);
        return e != hipSuccess ? e : second(main);
    }
    const hipError_t e1 = first(side);
    const hipError_t e2 = second(main);
    hipError_t ej = ops.record(join, side);
    if (ej == hipSuccess) ej = ops.wait(main, join, 0);
    if (ej != hipSuccess) {
        const hipError_t es = ops.sync(side);
        (void)es;
    }
    if (e1 != hipSuccess) return e1;
    if (e2 != hipSuccess) return e2;
    return ej;
}

}  // namespace elsaa
