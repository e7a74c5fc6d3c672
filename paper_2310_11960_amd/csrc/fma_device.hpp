// fma_device.hpp -- geometry and helpers shared by the FMA kernels (gfx950).
//
// The interaction lists of Sec. 3 (Fast Multipole Attention, 1D and 2D far
// fields) are evaluated in closed form here: a base block b (2D: cell
// (cx, cy)) at level l sits in level-l group q = b >> (l-1); its parent pair
// is p = q >> 1.  The level-l window of the far-field definition is the
// three level-(l+1) blocks around the parent, i.e. groups 2p-2 .. 2p+3, and
// the groups q-1 .. q+1 were already taken by the finer levels.  What is
// left -- three groups in 1D, 6x6 - 3x3 = 27 squares in 2D -- is the list.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fma_dev {

constexpr int kHeadDim = 64;      // d
constexpr int kMaxCoarse = 16;    // coarse levels (L - 1) a plan may have
constexpr int kMaxSets = 64;      // coarse sets (level, basis): (L - 1) * rank
constexpr int kPassSets = 16;     // sets one coarsening pass builds (fp32 1D and 2D kernels)
constexpr int kStreamSets = 32;   // sets one pass of the 1D bf16 streaming kernel builds
constexpr int kSlots1D = 3;       // list entries per level, 1D
constexpr int kSlots2D = 27;      // list entries per level, 2D

// The 1D bf16 streaming coarsening (coarsen1d_stream<D, NWD>): weight loads
// per ring slot for a pass of `sets` coarse sets, four sets per load, as the
// kernel is instantiated (1, 2, 3, 4, 6 or 8 loads); 0 beyond kStreamSets.
__host__ __device__ constexpr int stream_weight_loads(int sets)
{
    return sets <= 4 ? 1 : sets <= 8 ? 2 : sets <= 12 ? 3 : sets <= 16 ? 4 : sets <= 24 ? 6 : sets <= 32 ? 8 : 0;
}

// LDS bytes one wave of that kernel uses: D ring slots (16 bf16 rows, 2 KB,
// and their weights, 256 B per four sets), 64 zero bytes, the output staging
// (16 bf16 rows, 2 KB) and its 16 row indices.
__host__ __device__ constexpr int stream_wave_lds(int depth, int nwd)
{
    return depth * (2048 + 256 * nwd) + 64 + 2048 + 64;
}

// The 2D bf16 streaming coarsening (coarsen2d_stream<D, NWY, CG>) streams
// 32x32-pixel tiles; a set of square side s has 32 / s accumulator columns
// (square columns of the tile) when s <= 32, else one.  A pass holds at
// most 32 such columns.
__host__ __device__ constexpr int stream2d_cols(int s) { return s <= 32 ? 32 / s : 1; }

// Its y-weight loads per ring slot for a pass of `sets` sets, four sets per
// load, as instantiated (1, 2, 4 or 8); 0 beyond 32 sets.
__host__ __device__ constexpr int stream2d_weight_loads(int sets)
{
    return sets <= 4 ? 1 : sets <= 8 ? 2 : sets <= 16 ? 4 : sets <= 32 ? 8 : 0;
}

// LDS bytes one wave of it uses: D ring slots (16 bf16 pixel rows, 2 KB; the
// pixels' y weights, 256 B per four sets; the row's x weight of every set,
// 256 B), 64 zero bytes, the output staging (16 bf16 rows, 2 KB) and its 16
// row indices.
__host__ __device__ constexpr int stream2d_wave_lds(int depth, int nwy)
{
    return depth * (2048 + 256 * nwy + 256) + 64 + 2048 + 64;
}

// Threads of a workgroup of the 2D tile coarsening (coarsen2d_tiles) for
// cells of side r and head dim d: a 32x32 tile splits into NT / (d / 8) runs
// of pixel rows, each RX = 128 d / (NT r) rows of one cell; at least 256
// threads, and enough that RX <= r, so that a run never straddles a square.
__host__ __device__ constexpr int coarsen2d_threads(int r, int d)
{
    int nt = 256;
    while (nt < 128 * d / (r * r)) nt *= 2;
    return nt;
}

// Level-l list entry j (0..2) of 1D base block b, or -1 when it falls
// outside [0, M) or (causal) is not entirely in the past.
__host__ __device__ inline int list1d_entry(int b, int l, int j, int M, int causal)
{
    const int q = b >> (l - 1);
    const int p = q >> 1;
    int g;
    if ((q & 1) == 0)
        g = (j == 0) ? 2 * p - 2 : 2 * p + 1 + j;   // {2p-2, 2p+2, 2p+3}
    else
        g = (j == 2) ? 2 * p + 3 : 2 * p - 2 + j;   // {2p-2, 2p-1, 2p+3}
    if (g < 0 || g >= M) return -1;
    if (causal && g > q - 2) return -1;             // visible iff g <= q - 2
    return g;
}

// Slot j (0..26) of a 2D level list: the j-th square, row-major, of the 6x6
// window of level-l squares around the parent, skipping the 3x3 block at
// window offset (ox, oy) -- the squares the finer levels already cover.
// Rows above the hole hold 6 squares, the three rows beside it 3, rows below 6.
__host__ __device__ inline void window_slot(int j, int ox, int oy, int &au, int &av)
{
    if (j < 6 * ox) {
        au = j / 6;
        av = j - 6 * au;
    } else if (j < 6 * ox + 9) {
        const int t = j - 6 * ox;
        const int k = t % 3;
        au = ox + t / 3;
        av = k < oy ? k : k + 3;
    } else {
        const int t = j - 6 * ox - 9;
        au = ox + 3 + t / 6;
        av = t % 6;
    }
}

// Level-l list entry j (0..26) of 2D cell (cx, cy) (cx counts cell rows,
// cy cell columns): the 6x6 window of level-l squares around the parent,
// row-major, without the 3x3 block around (qx, qy), on a level of Mx rows
// by My columns of squares.  Returns u*My + v, or -1 when outside the map.
__host__ __device__ inline int list2d_entry(int cx, int cy, int l, int j, int Mx, int My)
{
    const int qx = cx >> (l - 1), qy = cy >> (l - 1);
    int au, av;
    window_slot(j, 1 + (qx & 1), 1 + (qy & 1), au, av);   // excluded block inside the window
    const int u = 2 * (qx >> 1) - 2 + au;
    const int v = 2 * (qy >> 1) - 2 + av;
    if (u < 0 || u >= Mx || v < 0 || v >= My) return -1;
    return u * My + v;
}

// Whether the bf16 fused attention walks a 2D map two horizontally adjacent
// cells per workgroup (cells (x, 2c) and (x, 2c + 1), four waves): their
// near fields share six of their nine cells, so the pair loads 12 near tiles
// where two single cells load 18, and twice the waves share the LDS stages.
// Used for 8 x 8 cells on maps with an even number of cell columns (nby),
// either normalisation, without query downsampling, and when both cells'
// interaction-list tables fit the paired kernel's slot table
// (kMaxPairSlotTable; the other kernels' table holds kMaxSlotTable slots).
constexpr int kMaxSlotTable = 448;
constexpr int kMaxPairSlotTable = 768;
__host__ __device__ constexpr bool pair_cells_2d(int r, int nby, int nslot, [[maybe_unused]] int norm_level, int linear,
                                                 int bf16)
{
    return bf16 && !linear && r == 8 && nby % 2 == 0 && nslot <= kMaxSlotTable &&
           2 * ((nslot + 63) / 64) * 64 <= kMaxPairSlotTable;
}

// Coarse-set tables every kernel receives by value.  With coarse level
// rank p (Sec. 3) every level has p basis vectors and every group p
// aggregated keys/values; the kernels see each (level, basis) pair as a set
// of its own, laid out like a level: set e = (l - 1) * p + basis, with its
// own weights and its own block of coarse rows, in that order.  With p = 1
// the sets are the levels.
struct Levels {
    int nlev;                  // coarse sets, (L - 1) * p
    int off[kMaxSets];         // first coarse row of each set (per slice)
    int M[kMaxSets];           // groups of the set's level (2D: rows of squares, ceil(H / s))
    int My[kMaxSets];          // 2D: columns of squares, ceil(W / s) (1D: 1)
    int size[kMaxSets];        // s_l = r * 2^(l-1) of the set's level
    int woff[kMaxSets];        // weight offset of the set (floats)
    int lvl[kMaxSets];         // the set's level l (1 .. L-1)
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// bf16 <-> fp32 by bit manipulation (bf16 is the upper half of an fp32).
__device__ inline float bf16lo_to_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16hi_to_f32(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 with round-to-nearest-even (NaN kept quiet).
__device__ inline uint32_t f32_to_bf16_bits(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ inline uint32_t pack_bf16x2(float lo, float hi)
{
    return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

}  // namespace fma_dev
