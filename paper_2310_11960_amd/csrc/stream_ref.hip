// stream_ref.hip -- achievable-bandwidth reference for the HBM-bound
// coarsening pass (a bench export, not part of the method): stream a buffer
// once with 16-byte loads and write one 16-byte word per `write_every` words
// read.  The coarsening reads K and V once and writes their coarse rows and
// partial sums, 1/40 to 1/60 of what it reads at n >= 16K, so the same
// read-dominated mix measured here is the ceiling it is compared with.
#include "fma_device.hpp"
#include "fma_kernels.hpp"

namespace fma_dev {

namespace {

constexpr int kRefThreads = 256;
constexpr int kRefLoads = 8;                          // 16-byte loads in flight per thread
constexpr int kRefChunk = kRefThreads * kRefLoads;    // words per chunk (32 KB)

// Streaming (non-temporal) loads, as the coarsening's: they measured
// 6.0-6.2 TB/s against 5.5-5.6 with the default policy.
// Chunk c of the source is words [c * kRefChunk, (c + 1) * kRefChunk); the
// workgroups take chunks with a grid stride.  Thread t of a chunk XORs its
// eight words and, if t < kRefChunk / write_every, stores the result at word
// c * (kRefChunk / write_every) + t of the destination (checked against its
// size), so that no load can be dropped.
__global__ __launch_bounds__(kRefThreads) void stream_ref_kernel(const uint4 *src, long long nwords, uint4 *dst,
                                                                 long long ndst, int write_every)
{
    const int t = threadIdx.x;
    const int per = kRefChunk / write_every;
    const long long nchunk = (nwords + kRefChunk - 1) / kRefChunk;
    for (long long c = blockIdx.x; c < nchunk; c += gridDim.x) {
        const long long base = c * kRefChunk + t;
        uint4 x[kRefLoads];
#pragma unroll
        for (int i = 0; i < kRefLoads; ++i) {
            const long long w = base + (long long)i * kRefThreads;
            typedef uint32_t u4v __attribute__((ext_vector_type(4)));
            const u4v t = w < nwords ? __builtin_nontemporal_load(reinterpret_cast<const u4v *>(src) + w)
                                     : u4v{0, 0, 0, 0};
            x[i] = make_uint4(t[0], t[1], t[2], t[3]);
        }
        uint4 acc = x[0];
#pragma unroll
        for (int i = 1; i < kRefLoads; ++i) {
            acc.x ^= x[i].x;
            acc.y ^= x[i].y;
            acc.z ^= x[i].z;
            acc.w ^= x[i].w;
        }
        const long long o = c * per + t;
        if (t < per && o < ndst) dst[o] = acc;
    }
}

}  // namespace

hipError_t launch_stream_ref(const void *src, long long nwords, void *dst, long long ndst, int write_every,
                             hipStream_t st)
{
    if (nwords == 0) return hipSuccess;
    const int slots = resident_slots(reinterpret_cast<const void *>(&stream_ref_kernel), kRefThreads, 0);
    if (slots <= 0) return hipErrorInvalidDevice;
    const long long nchunk = (nwords + kRefChunk - 1) / kRefChunk;
    long long grid = slots;
    if (grid > nchunk) grid = nchunk;
    hipLaunchKernelGGL(stream_ref_kernel, dim3((unsigned)grid), dim3(kRefThreads), 0, st,
                       static_cast<const uint4 *>(src), nwords, static_cast<uint4 *>(dst), ndst, write_every);
    return hipGetLastError();
}

// Words of destination the kernel writes for nwords source words.
long long stream_ref_dst_words(long long nwords, int write_every)
{
    const long long nchunk = (nwords + kRefChunk - 1) / kRefChunk;
    return nchunk * (kRefChunk / write_every);
}

}  // namespace fma_dev
