// lists.hip -- device export of the interaction lists (the groups G_l(i) /
// squares Q_l(i) of Sec. 3) exactly as the fused kernel evaluates them, so
// that tests can compare them bit for bit with the set-builder definition.
#include "fma_device.hpp"
#include "fma_kernels.hpp"

namespace fma_dev {

namespace {

// One thread per (base block, level): entries in ascending order, then -1.
// `lv` is a table of levels (one set per level), not of rank-p sets.
__global__ void lists_kernel(int two_d, int nblocks, int nby, int causal, Levels lv, int32_t *out)
{
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= nblocks * lv.nlev) return;
    const int b = idx / lv.nlev, lev = idx - b * lv.nlev;
    const int K = two_d ? kSlots2D : kSlots1D;
    int32_t *o = out + (long long)idx * K;
    int cnt = 0;
    for (int j = 0; j < K; ++j) {
        const int g = two_d ? list2d_entry(b / nby, b % nby, lv.lvl[lev], j, lv.M[lev], lv.My[lev])
                            : list1d_entry(b, lv.lvl[lev], j, lv.M[lev], causal);
        if (g >= 0) o[cnt++] = g;
    }
    for (; cnt < K; ++cnt) o[cnt] = -1;
}

}  // namespace

hipError_t launch_lists(int two_d, int nblocks, int nby, int causal, const Levels &lv,
                        int32_t *out, hipStream_t st)
{
    const int total = nblocks * lv.nlev;
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(lists_kernel, dim3((total + 127) / 128), dim3(128), 0, st,
                       two_d, nblocks, nby, causal, lv, out);
    return hipGetLastError();
}

}  // namespace fma_dev
