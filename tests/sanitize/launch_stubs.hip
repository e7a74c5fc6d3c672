// Launcher stubs for the sanitizer build of the C ABI's host code (test
// infrastructure): the host checks never launch a kernel, so every launcher
// aborts -- a check that reached one would fail loudly.
#include <stdio.h>
#include <stdlib.h>

#include "fma_kernels.hpp"

namespace fma_dev {

[[noreturn]] static void reached(const char *what)
{
    fprintf(stderr, "host check reached %s\n", what);
    abort();
}

hipError_t launch_coarsen(const CoarsenArgs &, bool, size_t, hipStream_t) { reached("launch_coarsen"); }
hipError_t launch_attend(const AttnArgs &, bool, int, hipStream_t) { reached("launch_attend"); }
hipError_t launch_attend_bf16(const AttnArgs &, int, hipStream_t) { reached("launch_attend_bf16"); }
hipError_t launch_lin_far(const AttnArgs &, int, hipStream_t) { reached("launch_lin_far"); }
hipError_t launch_lists(int, int, int, int, const Levels &, int32_t *, hipStream_t) { reached("launch_lists"); }
hipError_t launch_backward(const BwdArgs &, bool, bool, hipStream_t) { reached("launch_backward"); }
hipError_t launch_stream_ref(const void *, long long, void *, long long, int, hipStream_t)
{
    reached("launch_stream_ref");
}
long long stream_ref_dst_words(long long nwords, int write_every)
{
    // the bench export sizes its destination with this; same formula as the kernel file
    return (nwords + 2047) / 2048 * (2048 / write_every);
}

}  // namespace fma_dev
