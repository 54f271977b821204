// Internal layout shared by the host planner and the gfx950 kernels.
//
// A step is planned on the host into a flat list of work items, one per
// workgroup.  Rows are first grouped by adapter (the per-token gather of
// Sections 2.3 C2 / 4.1), then every group's adapter is cut into pieces of a
// fixed number of bytes: shrink items stream one K-chunk of A_g (h_in rows),
// expand items stream one column tile of B_g.  Piece size in rows/columns is
// inversely proportional to the rank, so every item moves about the same
// number of bytes whatever its rank (padding-free, Section 5's Sum-of-ranks
// cost), and items of every rank run side by side in one grid.
#pragma once
#include <stdint.h>

namespace lora {

constexpr int kThreads = 256;            // workgroup size: 4 wave64
constexpr int kMaxRank = 256;
constexpr int kChunkElems = 16384;       // elements of A_g / B_g per item (32 KiB)
constexpr int kShrinkRowTile = 4;        // rows of x held per pass (shrink)
constexpr int kExpandRowTile = 4;        // rows of v held per pass (expand)

// Item kinds.
enum : int32_t {
    kItemShrink = 1,     // v(rows, 0:r) [+]= x(rows, k0:k0+klen) . A(k0:k0+klen, 0:r)
    kItemExpand = 2,     // y(rows, n0:n0+nlen) += s * v(rows, 0:r) . B(0:r, n0:n0+nlen)
};

// One registered adapter, as the kernels read it (32 bytes).
struct DevAdapter {
    const void* A;       // [h_in, rank] row-major
    const void* B;       // [rank, h_out] row-major
    int32_t rank;
    float scale;
    int32_t pad0, pad1;
};
static_assert(sizeof(DevAdapter) == 32, "DevAdapter layout");

// One work item = one workgroup (32 bytes).
struct DevItem {
    int32_t kind;        // kItemShrink / kItemExpand
    int32_t adapter;     // index into the adapter table
    int32_t p0;          // first position of the group's rows in perm
    int32_t nrows;       // rows in the group
    int32_t lo;          // k0 (shrink) or n0 (expand)
    int32_t len;         // klen (shrink) or nlen (expand), multiple of 8
    int32_t group;       // group id: index of its arrival counter (shrink)
    int32_t split;       // shrink: (chunk << 16) | nsplit ; expand: 0
};
static_assert(sizeof(DevItem) == 32, "DevItem layout");

struct DevGroupPartials {
    int64_t off;         // float offset of the group's partials
};

// Kernel arguments shared by the shrink and expand kernels.
struct KernelArgs {
    const DevItem* items;
    const DevAdapter* table;
    const int32_t* perm;       // grouped row list
    int32_t* counters;         // one per group, zero between launches
    float* partials;           // split-K partial sums
    const int64_t* part_off;   // per group float offset into partials
    const void* x;
    int64_t ldx;
    float* v;                  // float32 intermediate
    int64_t ldv;
    int32_t v_by_row;          // 1: v row = perm[p]; 0: v row = p (compact)
    int32_t h_in;
    void* y;
    int64_t ldy;
    int32_t h_out;
    int32_t n_items;
};

}  // namespace lora
