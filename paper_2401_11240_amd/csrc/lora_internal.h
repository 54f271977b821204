// Internal layout shared by the host planner and the gfx950 kernels.
//
// A step is planned on the host into flat lists of work items, one per
// workgroup.  Rows are first grouped by adapter (the per-token gather of
// Sections 2.3 C2 / 4.1) and each group is cut into row blocks of at most
// 64 rows.  Each row block then becomes three kinds of items:
//
//   shrink  (row block, K range of A_g): a float32 partial block
//           P_c[row, 0:Rv] = sum over the K range of x[row, k] A_g[k, :];
//   reduce  (row block, slice of its v block): v = sum_c P_c over that slice,
//           the partial blocks added in a fixed order;
//   expand  (row block, column tile of B_g): y[row, tile] is rounded once
//           from y + s_g * v[row, :] . B_g[:, tile].
//
// A K range streams about the same number of bytes whatever the rank
// (padding-free: the cost follows the sum of ranks, Section 5), and items of
// every rank run side by side in one grid.  The reduce items cut the row
// block's v into slices so that no item adds up more than a few tens of KB of
// partial values, and every expand tile reads the finished v once (a few KB)
// instead of the partial blocks.
//
// The three kinds run either as separate launches (launch boundaries order
// them) or as one step launch whose grid holds every shrink item, then every
// reduce item, then every expand item.  In the step launch the partial and v
// blocks live in two buffers used by alternate launches and hold a sentinel
// pattern until written; a consumer loads the values it needs with
// device-coherent loads and loads again those that still hold the sentinel.
// Every wait is on items earlier in the grid, which never wait on later ones,
// and the wait is bounded (it gives up and raises a status flag).
//
// A plan depends on the batch, the ranks and the shapes only.  The weight
// pointers and scales of the groups it references travel in the kernel
// arguments of each launch, so one plan serves every layer's adapter table of
// the same ranks (the batch of a step is the same for all of them).
//
// Both contractions run on MFMA (v_mfma_f32_16x16x32).  Shrink: v^T = A^T x^T,
// K = h_in; A is transposed in registers (8 K rows x 8 ranks per lane) and
// staged in LDS as 16-byte chunks of 8 consecutive K of one rank.  Expand:
// y^T = B^T v^T with the 32 K slots holding 16 ranks twice, once with the
// high and once with the low 16-bit part of v (v is never rounded to a single
// 16-bit value); B is transposed in registers, no LDS.
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
constexpr int kInlineRows = 16;          // items this small carry their rows inline
constexpr int kKargGroups = 128;         // groups whose pointers travel in the kernel arguments
constexpr int kShrinkStages = 4;         // LDS buffers of the direct-to-LDS shrink
constexpr int kStageChunks = 1024;       // 16-byte chunks per buffer (one 16 KiB pass)
constexpr int kShrinkLds = kShrinkStages * kStageChunks * 16;   // LDS bytes of the shrink bodies
constexpr int kExpandYsOff = 32 * 1024;  // expand: v fragments below, the staged y tile from here
constexpr int kExpandLds = kExpandYsOff + 33 * 1024 + 256;   // LDS bytes of the expand body
constexpr int kExpandVmaxOff = kExpandLds - 16;   // expand: per-wave largest |v| (4 floats) after the y tile
constexpr int kExpandTiles = 2;          // column tiles of a prompt expand item
constexpr int kReduceLds = kThreads * 16;
constexpr int kStepLds = kShrinkLds > kExpandLds ? kShrinkLds : kExpandLds;
constexpr int kSyncStride = 32;          // 32-bit words between row block counters (one 128-byte line each)
constexpr int kReduceBytes = 32 * 1024;  // partial bytes one reduce item adds up at most
constexpr int kDirectBytes = 16 * 1024;  // partial bytes up to which expand items add them up themselves
constexpr int kMaxSplitLoads = 16;       // partial blocks one reduce thread adds up
constexpr int kDirectSplits = 16;        // partial blocks an expand item adds up itself, at most
constexpr uint32_t kMaxSpan = 0x7fff0000u;  // x, y, factor and partial spans stay below 2 GiB (buffer offsets)
// Every plan and workspace starts with a header at a fixed place, whatever
// the batch: word 0 the generation of the work list that follows (a launch
// whose arguments carry another generation was recorded before the plan was
// re-planned; it does nothing), word 1 the status (0 ok, 1 a step launch's
// wait gave up, 2 a launch of another generation ran and did nothing).
constexpr int kHeaderBytes = 256;
enum : int32_t { kStatusOk = 0, kStatusGaveUp = 1, kStatusStale = 2 };
static_assert(kExpandLds <= kStepLds && kReduceLds <= kStepLds, "step LDS");

// Item kinds (an item of any other kind does nothing).
enum : int32_t {
    kItemShrink = 1,     // part = x(rows, k0:k0+len) . A(k0:k0+len, 0:r)
    kItemExpand = 2,     // y(rows, n0:n0+len) += s * v . B(0:r, n0:n0+len)
    kItemReduce = 3,     // v slice = sum of the row block's partial blocks
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
//   shrink: part = its partial block; lo, len = K range; sub = K per pass
//   reduce: part = first partial block of the row block (the v block follows
//           the nsplit partial blocks); lo = first float of the slice, len =
//           its floats (multiple of 4); sub = split groups (see reduce_body)
//   expand: part = first partial block of the row block (the v block follows
//           the nsplit partial blocks); lo, len = column tile; sub = 1 when
//           the item adds up the partial blocks itself (no reduce items for
//           a row block whose partial blocks are small), else 0
struct DevItem {
    int64_t part;        // float offset into the partial buffer
    int32_t kind;
    int32_t group;       // group of the batch (index into the launch's pointer table)
    int32_t adapter;     // adapter index (registry fallback when group >= kKargGroups)
    int32_t rank;
    int32_t nrows;       // rows in this item (<= 64)
    int32_t lo;
    int32_t len;
    int32_t sub;
    int32_t nsplit;      // partial blocks of the row block
    int32_t p0;          // position of the first row in the grouped row order (perm)
    int32_t pstride;     // floats of one partial block (= nrows * rv)
    int32_t rb;          // row block index (its counter of finished expand items in the step launch)
    int32_t nexp;        // expand items of the row block
    int32_t row0;        // the first row when the item's rows are consecutive (a prompt segment), else -1
    int32_t rows[kInlineRows];   // the item's rows when nrows <= kInlineRows
};
static_assert(sizeof(DevItem) == 128, "DevItem layout");

constexpr int kMaxProj = 4;       // projections one launch may carry (q, k, v; gate, up)
constexpr int kProjShift = 8;     // DevItem::kind holds the projection above this bit

struct KernelArgs {
    const DevItem* items;
    const int32_t* perm;        // grouped row order
    const DevAdapter* table;    // registry (fallback for groups beyond the argument table)
    float* partials;            // partial and v blocks
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
    int32_t* status;            // header word 1 (see kHeaderBytes)
    int64_t pbuf;               // step launch: floats from the first partial buffer to the second
    int32_t spin_limit;         // step launch: polling rounds before a wait gives up
    uint32_t x_bytes;           // bytes from x to the end of its last row (< 2 GiB)
    uint32_t y_bytes;           // bytes from y to the end of its last row (< 2 GiB)
    uint32_t generation;        // the work list these arguments were made for (header word 0)
    int32_t n_proj;             // projections sharing x in this launch (items carry their projection)
    const void* gfac[2 * kKargGroups];   // per group g: [2g] = A_g, [2g + 1] = B_g
    float gscale[kKargGroups];           // per group: s_g
    // launches of several projections sharing x: per projection, its adapter
    // registry and its y (factor pointers are then read from the registry)
    const DevAdapter* ptable[kMaxProj];
    void* py[kMaxProj];
    int64_t pldy[kMaxProj];
    uint32_t py_bytes[kMaxProj];
    int32_t ph_out[kMaxProj];
};
static_assert(sizeof(KernelArgs) <= 4096, "kernel arguments");

// ---------------------------------------------------------------------------
// Fused base projection (Eq. 1 whole): y = x W + s_g (x A_g) B_g for every
// row, one MFMA GEMM over square tiles of kBaseBig or kBaseSmall rows x as
// many columns, the adapter delta added in the tile's epilogue from a float32
// v computed beforehand.  A stage holds the tile's x and W slices over
// kBaseStageBytes / (4 tile) of K: 64 along K for the big tile (one
// 128-byte line per row), 128 for the small one.
// ---------------------------------------------------------------------------
constexpr int kBaseBig = 256;            // tile edge while whole tiles fill the compute units
constexpr int kBaseSmall = 128;          // tile edge of launches with fewer big tiles than compute units
constexpr int kBaseThreads = 256;        // 4 wave64: 2 (rows) x 2 (columns), each a quarter of the tile
constexpr int kBaseStageBytes = 64 * 1024;   // x slice, then W slice
constexpr int kBaseMinSplitStages = 8;   // fewest K stages of a split range
constexpr int kBaseLoraRanks = 64;       // ranks of B_g staged in LDS at a time (one stage buffer)
constexpr int kBasePanel = 8;            // row tiles per panel of the tile order
LORA_HD constexpr int base_bk(int tile) { return kBaseStageBytes / (4 * tile); }

// One run of a tile's rows that share an adapter (g >= 0): rows [lo, hi).
struct BasePiece {
    int32_t lo, hi, adapter, pad;
};

struct BaseArgs {
    const void* x;                 // [M, ldx] 16-bit
    const void* wt;                // [N, ldw] 16-bit: the base weight transposed (row n = column n of W)
    void* y;                       // [M, ldy] 16-bit, written
    const float* v;                // [M, ldv] float32: v[t, 0:r_g] = x[t] . A_g
    const DevAdapter* table;       // registry: B_g, rank, scale
    const int32_t* piece_off;      // [n_mt + 1]: pieces of row tile mt are [piece_off[mt], piece_off[mt+1])
    const BasePiece* pieces;
    int64_t ldx, ldw, ldy, ldv;
    int32_t M, N, K;               // rows, h_out, h_in
    int32_t tile;                  // tile edge: kBaseBig or kBaseSmall
    int32_t n_mt, n_nt;            // row tiles, column tiles
    int32_t n_xcd, per_xcd;        // XCDs, whole tiles per XCD (rounded up): n_xcd per_xcd workgroups
    // Tiles [0, n_whole) run whole, one workgroup each.  Each tile of
    // [n_whole, n_mt n_nt) is split into `split` K ranges of `chunk` stages
    // (workgroup n_xcd per_xcd + (tile - n_whole) split + s takes range s), which
    // write float32 partial tiles to `part`; a second kernel adds them in the
    // order of s, rounds and stores.  Range 0 carries the adapter delta.
    int32_t n_whole, split, chunk;
    float* part;                   // [(n_mt n_nt - n_whole) split][tile tile] in accumulator order
    uint32_t x_bytes, w_bytes, y_bytes, v_bytes;
    int32_t b_span_ok;             // 1: every B_g spans < 2 GiB (checked on the host)
};

// ---------------------------------------------------------------------------
// Tiling, shared by the planner (sizes the items) and the kernels (lay out
// LDS).  All extents are in elements unless named *_bytes.
// ---------------------------------------------------------------------------
LORA_HD inline int round_up_i(int v, int m) { return (v + m - 1) / m * m; }
LORA_HD inline int min_i(int a, int b) { return a < b ? a : b; }
LORA_HD inline int max_i(int a, int b) { return a > b ? a : b; }
LORA_HD inline int msub_of(int nrows) { return (nrows + 15) / 16; }
// MFMA subtiles the kernel bodies are compiled for: 1, 2 or 4
LORA_HD inline int msub_body(int nrows) { const int m = msub_of(nrows); return m <= 1 ? 1 : (m <= 2 ? 2 : 4); }

// Row stride of partial and v blocks: the rank rounded up to 8 floats.
LORA_HD inline int rank_stride(int rank) { return round_up_i(rank, 8); }

// Rows per row block: 64, or 32 when the rank pads past 128.
LORA_HD inline int row_block(int rank) { return round_up_i(rank, 16) > 128 ? 32 : 64; }

// ---- shrink ----
// A pass stages `sub` K (a multiple of 32) of A^T and of the row block's x
// in LDS, each row as sub/8 + 1 chunks of 16 bytes (an odd chunk stride: 16-
// byte reads and writes of eight consecutive lanes hit distinct banks).
LORA_HD inline int shrink_chunks(int sub) { return sub / 8 + 1; }
// Waves side by side over rank tiles (1, 2 or 4); the others split K.  Items
// of one 16-row subtile (decode) never split K: their MFMA work is a few
// hundred cycles, less than adding wave sums through LDS would cost.
LORA_HD inline int shrink_wn(int rank, int nrows) {
    const int nt = round_up_i(rank, 16) / 16;
    if (msub_body(nrows) == 1) return 4;
    return nt >= 4 ? 4 : (nt >= 2 ? 2 : 1);
}
LORA_HD inline int shrink_tq(int rank, int nrows) {     // rank tiles per wave: 1, 2 or 4
    const int nt = round_up_i(rank, 16) / 16;
    const int wn = shrink_wn(rank, nrows);
    const int q = (nt + wn - 1) / wn;
    return q <= 1 ? 1 : (q <= 2 ? 2 : 4);
}
LORA_HD inline int shrink_lds_bytes(int rank, int sub, int nrows) {
    const int rp = round_up_i(rank, 16);
    const int staged = (rp + msub_body(nrows) * 16) * shrink_chunks(sub) * 16;
    const int wk = 4 / shrink_wn(rank, nrows);
    const int red = wk > 1 ? wk * msub_body(nrows) * 16 * (rp + 4) * 4 : 0;   // rows padded by 4 floats
    return max_i(staged, red);
}
// K per pass: a multiple of 32 with the A pass at most 32 KiB (sub * rank <=
// 16384), at most 4 x chunks per thread (msub * sub <= 512), eight-row units
// of the A transpose covering it (see shrink_body), and the staging within LDS.
LORA_HD inline int shrink_sub(int rank, int nrows) {
    const int ms = msub_body(nrows);
    int k = 512 / ms;
    if (rank % 8 == 0) {
        const int vpr = rank / 8;
        k = min_i(k, 64 * (32 / vpr));
    }
    k = min_i(k, 16384 / round_up_i(rank, 8));
    k &= ~31;
    while (k > 32 && shrink_lds_bytes(rank, k, nrows) > kShrinkLds) k -= 32;
    return max_i(32, k);
}

// K per pass of the direct-to-LDS shrink (ranks that are a multiple of 8):
// the largest multiple of 64 (else 32) up to 512 whose A rows (rounded to
// whole 1 KiB wave loads) and x rows fit one buffer; 0 when none does (the
// register-staged body then runs the item).
LORA_HD inline int shrink_stage_sub(int rank, int nrows) {
    if (rank % 8 != 0) return 0;
    const int ms = msub_body(nrows);
    for (int k = 512; k >= 32; k -= (k > 64 ? 64 : 32))
        if (round_up_i(k * (rank / 8), 64) + 2 * ms * k <= kStageChunks) return k;
    return 0;
}
// Only row blocks of more than one 16-row subtile stream through the LDS
// buffers; a decode block's pass is one memory round trip either way, and the
// register-staged body measured faster there.
LORA_HD inline bool shrink_uses_dma(int rank, int nrows) {
    return msub_body(nrows) > 1 && shrink_stage_sub(rank, nrows) >= 32;
}

// ---- expand ----
// Column tiles of 256 * q columns (q column blocks of 64 per wave) with
// q * msub <= 4 (registers) and a B tile of about 32 KiB.  Ranks are taken in
// groups of ksg steps of 16 (q * ksg = 4 or less): every B load of a group is
// in flight at once.
LORA_HD inline int expand_q(int rank, int nrows) {
    const int ms = msub_body(nrows);
    const int rk = round_up_i(rank, 16);
    int q = 32768 / (rk * 512);
    q = q >= 4 ? 4 : (q >= 2 ? 2 : 1);
    while (q * ms > 4) q >>= 1;
    return q;
}
LORA_HD inline int expand_ksg(int rank, int nrows) {
    const int ks = round_up_i(rank, 16) / 16;
    // items of four subtiles keep the next group's B in flight beside their
    // accumulators: groups of at most 2 steps
    const int cap = msub_body(nrows) >= 4 ? 2 : 4 / expand_q(rank, nrows);
    return ks >= cap ? cap : (ks >= 2 ? 2 : 1);
}
// Columns of an expand item: one tile of 256 q, or kExpandTiles tiles for
// items of four 16-row subtiles (they make their v fragments once).
LORA_HD inline int expand_tile(int rank, int nrows) { return 256 * expand_q(rank, nrows); }
LORA_HD inline int expand_nlen(int rank, int nrows) {
    return expand_tile(rank, nrows) * (msub_body(nrows) == 4 ? kExpandTiles : 1);
}
// The v fragments (below kExpandYsOff) and, for items of more than one
// 16-row subtile, the y tile staged through LDS ([rows][256 q / 8 + 1] chunks
// of 16 bytes, from kExpandYsOff) fit the expand's LDS.
LORA_HD inline bool expand_fits_lds(int rank, int nrows) {
    const int ms = msub_body(nrows);
    const int vf = ms * (round_up_i(rank, 16) / 16) * 64 * 16;
    const int yt = ms > 1 ? ms * 16 * (32 * expand_q(rank, nrows) + 1) * 16 : 0;
    return vf <= kExpandYsOff && kExpandYsOff + yt <= kExpandVmaxOff;
}

}  // namespace lora
