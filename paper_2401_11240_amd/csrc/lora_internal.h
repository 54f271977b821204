// Internal layout shared by the host planner and the gfx950 kernels.
//
// A step is planned on the host into flat lists of work items, one per
// workgroup.  Rows are first grouped by adapter (the per-token gather of
// Sections 2.3 C2 / 4.1) and each group is cut into row blocks of at most
// 64 rows.  Every row block's adapter is cut into pieces of about 32 KiB:
// shrink items stream a K range of A_g (rows k0..k0+len of the [h_in, r]
// matrix), expand items one column tile of B_g.  The piece's extent in rows or
// columns shrinks as the rank grows, so every item moves about the same number
// of bytes whatever its rank (padding-free: the cost follows the sum of ranks,
// Section 5), and items of every rank run side by side in one grid.
//
// The shrink writes one float32 partial block per (row block, K range); the
// expand adds a row block's partial blocks in a fixed order while it stages v,
// so results never depend on timing.  The two run either as two launches (the
// launch boundary orders them) or as one step launch whose grid holds every
// shrink item before every expand item: a shrink workgroup writes its block
// with device-coherent stores into a buffer armed with a sentinel pattern
// (two buffers, used by alternate launches); an expand workgroup requests its
// B tile and its y values, then loads the partial values, again while any
// still holds the sentinel.  It only ever
// waits for workgroups earlier in the grid, which never wait themselves, and
// the wait is bounded (it gives up and raises a status flag).
//
// A plan depends on the batch, the ranks and the shapes only.  The weight
// pointers and scales of the groups it references travel in the kernel
// arguments of each launch, so one plan serves every layer's adapter table of
// the same ranks (the batch of a step is the same for all of them).
//
// Both kernels run the contraction on MFMA: the shrink as v^T = A^T x^T
// (16x16x32, K = h_in), the expand as y^T = B^T v^T (16x16x16, K = rank).  The
// factor tile is staged in LDS transposed into words holding two consecutive
// K elements, so every MFMA operand fragment is one LDS vector read.
#pragma once
#include <stdint.h>

#ifdef __HIPCC__
#define LORA_HD __host__ __device__
#else
#define LORA_HD
#endif

namespace lora {

constexpr int kThreads = 256;            // workgroup size: 4 wave64
constexpr int kMaxRank = 256;
constexpr int kMSub = 4;                 // 16-row MFMA subtiles per item at most
constexpr int kInlineRows = 16;          // items this small carry their rows inline
constexpr int kKargGroups = 128;         // groups whose pointers travel in the kernel arguments
constexpr int kShrinkLds = 52 * 1024;    // LDS bytes of the shrink kernel
constexpr int kExpandLds = 68 * 1024;    // LDS bytes of the expand kernel
constexpr int kStepLds = kExpandLds > kShrinkLds ? kExpandLds : kShrinkLds;
constexpr int kSyncStride = 32;          // 32-bit words between row block counters (one 128-byte line each)

// Item kinds.
enum : int32_t {
    kItemNop = 0,
    kItemShrink = 1,     // part = x(rows, k0:k0+len) . A(k0:k0+len, 0:r)
    kItemExpand = 2,     // y(rows, n0:n0+len) += s * (sum of parts) . B(0:r, n0:n0+len)
    kItemReduce = 3,     // v(rows, 0:r) = sum of parts
};

// One registered adapter, as the device-resident registry holds it (32 B).
struct DevAdapter {
    const void* A;       // [h_in, rank] row-major
    const void* B;       // [rank, h_out] row-major
    int32_t rank;
    float scale;
    int32_t pad0, pad1;
};
static_assert(sizeof(DevAdapter) == 32, "DevAdapter layout");

// One work item = one workgroup (128 bytes, read with scalar loads).
struct DevItem {
    int64_t part;        // float offset: shrink -> its own partial block; expand/reduce -> the row block's first
    int32_t kind;
    int32_t group;       // group of the batch (index into the launch's pointer table)
    int32_t adapter;     // adapter index (registry fallback when group >= kKargGroups)
    int32_t rank;
    int32_t nrows;       // rows in this item (<= 64)
    int32_t lo;          // k0 (shrink) or n0 (expand)
    int32_t len;         // K range (shrink) or column tile (expand), multiple of 8
    int32_t sub;         // shrink: K sub-chunk staged per pass (multiple of 32)
    int32_t nsplit;      // expand / reduce: partial blocks to add
    int32_t p0;          // position of the first row in the grouped row order (perm)
    int32_t pstride;     // floats between consecutive partial blocks of the row block
    int32_t rb;          // row block index (its counter of finished expand items in the step launch)
    int32_t nexp;        // expand items of the row block
    int32_t row0;        // the first row when the item's rows are consecutive (a prompt segment), else -1
    int32_t rows[kInlineRows];   // the item's rows when nrows <= kInlineRows
};
static_assert(sizeof(DevItem) == 128, "DevItem layout");

struct KernelArgs {
    const DevItem* items;
    const int32_t* perm;        // grouped row order
    const DevAdapter* table;    // registry (fallback for groups beyond the argument table)
    float* partials;            // split-K partial blocks
    const void* x;
    int64_t ldx;
    void* y;
    int64_t ldy;
    float* v;                   // caller's float32 v (lora_expand input / lora_shrink output)
    int64_t ldv;
    int32_t h_in;
    int32_t h_out;
    int32_t n_items;
    int32_t n_groups;
    uint32_t* sync;             // step launch: per row block (every kSyncStride words), expand items finished (wraps at 2 nexp)
    int32_t* status;            // step launch: set to 1 when a wait gave up
    int64_t pbuf;               // step launch: floats from the first partial buffer to the second
    int32_t spin_limit;         // step launch: polling rounds before a wait gives up
    int32_t pad;
    const void* gfac[2 * kKargGroups];   // per group g: [2g] = A_g, [2g + 1] = B_g
    float gscale[kKargGroups];           // per group: s_g
};
static_assert(sizeof(KernelArgs) <= 4096, "kernel arguments");

// ---------------------------------------------------------------------------
// Tiling, shared by the planner (sizes the items) and the kernels (lays out
// LDS).  All extents are in elements unless named *_bytes.
// ---------------------------------------------------------------------------
LORA_HD inline int round_up_i(int v, int m) { return (v + m - 1) / m * m; }
LORA_HD inline int min_i(int a, int b) { return a < b ? a : b; }
LORA_HD inline int max_i(int a, int b) { return a > b ? a : b; }
LORA_HD inline int msub_of(int nrows) { return (nrows + 15) / 16; }
// MFMA subtiles the kernel body is compiled for: 1, 2 or 4
LORA_HD inline int msub_body(int nrows) { const int m = msub_of(nrows); return m <= 1 ? 1 : (m <= 2 ? 2 : 4); }

// Rows per row block: 64, or 32 when the rank pads past 128 (expand LDS).
LORA_HD inline int row_block(int rank) { return round_up_i(rank, 16) > 128 ? 32 : 64; }

// Shrink: ranks padded to 16 (MFMA N); the K sub-chunk staged per pass is a
// multiple of 32 (MFMA K) with an A^T tile of at most 32 KiB.
LORA_HD inline int shrink_sub(int rank, int nrows) {
    const int rp = round_up_i(rank, 16);
    const int k = min_i(16384 / rp, 512 / msub_body(nrows)) & ~31;
    return max_i(32, k);
}
LORA_HD inline int shrink_kp(int sub) { return sub / 2 + 4; }   // words per A^T row, 4 (mod 8)
LORA_HD inline int shrink_kx(int sub) { return sub + 8; }       // halves per x row
LORA_HD inline int shrink_wn(int rank) {
    const int nt = round_up_i(rank, 16) / 16;
    return nt >= 4 ? 4 : (nt >= 2 ? 2 : 1);
}
LORA_HD inline int shrink_tq(int rank) {    // rank tiles per wave: 1, 2 or 4
    const int nt = round_up_i(rank, 16) / 16;
    const int q = (nt + shrink_wn(rank) - 1) / shrink_wn(rank);
    return q <= 1 ? 1 : (q <= 2 ? 2 : 4);
}
LORA_HD inline int shrink_lds_bytes(int rank, int sub, int nrows) {
    const int rp = round_up_i(rank, 16);
    const int staged = rp * shrink_kp(sub) * 4 + msub_body(nrows) * 16 * shrink_kx(sub) * 2;
    const int wk = 4 / shrink_wn(rank);
    const int red = wk > 1 ? wk * msub_body(nrows) * 16 * rp * 4 : 0;
    return max_i(staged, red);
}

// Expand: ranks padded to 16 (MFMA K); a column tile of 64 * q columns, q in
// {1, 2, 4, 8} with q * msub <= 16 (register budget) and the B^T tile within
// LDS.
LORA_HD inline int expand_rp(int rank) { return round_up_i(rank, 16) / 2 + 2; }  // words per row, 2 (mod 4)
LORA_HD inline int expand_nlen(int rank, int nrows) {
    const int cap = 8704 / expand_rp(rank);
    int n = 512;
    while (n > 64 && (n > cap || (n / 64) * msub_body(nrows) > 16)) n >>= 1;
    return n;
}
// The partial blocks of a row block are added in P interleaved parts (part q
// takes blocks q, q+P, ...; the parts are then added in order q = 0..P-1), P
// fixed by the row block's shape so that every reader adds in the same order.
LORA_HD inline int partial_parts(int nrows, int rank, int nsplit) {
    const int slots = nrows * round_up_i(rank, 16) / 2;
    int p = 1;
    while (p < 16 && 2 * p * slots <= kThreads && 2 * p <= nsplit) p *= 2;
    return p;
}

LORA_HD inline int expand_lds_bytes(int rank, int len, int nrows) {
    const int rp = expand_rp(rank);
    return round_up_i(len, 16) * rp * 4 + 2 * msub_body(nrows) * 16 * rp * 4 + kThreads * 8;
}

}  // namespace lora
