/*
 * lora.h - C ABI of the batched, heterogeneous-rank LoRA delta on MI355X (gfx950).
 *
 * What is computed.  The paper's Eq. 1 (Section 2.1, "LLM adaption") adapts a
 * weight W in R^{H1 x H2} by A in R^{H1 x r} and B in R^{r x H2}:
 * y' = xW + xAB, row vectors.  Section 2.2 keeps one base model and computes
 * xAB on the fly per request, adding it to the shared xW; Sections 2.3 (C2)
 * and 4.1 batch many requests of different adapters and ranks into one step,
 * each token gathering its own adapter.  This library computes, in place,
 *
 *     y[t, :] <- round( y[t, :] + s_g * (x[t, :] . A_g) . B_g )
 *
 * for every row t of a segment whose adapter is g >= 0, where y = xW is the
 * caller's base output, s_g a per-adapter float scale (1.0 recovers Eq. 1)
 * and "round" one round-to-nearest-even of the float32 sum to the storage
 * dtype.  The rank-r intermediate x.A_g is kept in float32.  Rows of
 * segments with adapter -1 are never read from x nor written in y.
 *
 * A step is described by segments: a decode token is a segment of length 1,
 * a prompt is one segment of its length (continuous batching, Section 2.2).
 *
 * Layout (paper's row-vector convention, Section 2.1):
 *   x  [n_rows, h_in]  row-major, leading dimension ldx (elements)
 *   y  [n_rows, h_out] row-major, leading dimension ldy (elements)
 *   A_g [h_in, r_g]    row-major (dense, leading dimension r_g)
 *   B_g [r_g, h_out]   row-major (dense, leading dimension h_out)
 *   v  [n_rows, ldv]   float32, v[t, 0:r_g] = x[t].A_g (shrink result)
 * 16-bit elements are IEEE binary16 (LORA_F16) or bfloat16 (LORA_BF16).
 *
 * Requirements, all checked on the host before anything is enqueued; a
 * violation returns a negative code, sets lora_last_error() and enqueues
 * nothing:
 *   - h_in, h_out, ldx, ldy: positive multiples of 8 (16-byte rows);
 *     ldx >= h_in, ldy >= h_out; ldv a multiple of 4 with ldv >= the largest
 *     rank used in the batch;
 *   - x, y, v, every A_g and B_g: 16-byte aligned device pointers;
 *   - ranks in [1, 256]; adapter indices in [-1, n_adapters);
 *   - seg_offset[0] = 0, nondecreasing, seg_offset[n_segments] = n_rows;
 *   - x and y do not overlap;
 *   - x and y each span less than 2 GiB from their first element to the end
 *     of their last row, and h_in, h_out are at most 4 Mi (the kernels
 *     address them with 32-bit buffer offsets).
 *
 * Asynchrony.  Every compute call is enqueued on the caller's HIP stream
 * (a hipStream_t passed as void*, NULL = the null stream) and returns
 * without waiting for the GPU.  No call except lora_register_adapters,
 * lora_plan_create(_reserved) and the destroy/release calls allocates device
 * memory.
 * Calls are deterministic: the same inputs give the same bits.
 *
 * Thread safety.  Distinct tables and plans may be used from any threads.
 * Calls sharing one workspace or one plan must be ordered (one stream).
 */
#ifndef LORA_H
#define LORA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LORA_ABI_VERSION 4

typedef enum { LORA_F16 = 0, LORA_BF16 = 1 } lora_dtype_t;

enum {
    LORA_OK = 0,
    LORA_E_ARG = -1,        /* null pointer, negative count, bad dtype/device   */
    LORA_E_SHAPE = -2,      /* h / ld not a multiple of 8, ld too small, segments malformed */
    LORA_E_RANK = -3,       /* rank outside [1, 256]                             */
    LORA_E_INDEX = -4,      /* adapter index outside [-1, n_adapters)            */
    LORA_E_ALIGN = -5,      /* pointer not 16-byte aligned                       */
    LORA_E_NOMEM = -6,      /* host or device allocation failed                  */
    LORA_E_HIP = -7,        /* a HIP runtime call or kernel launch failed        */
    LORA_E_WORKSPACE = -8,  /* workspace smaller than lora_workspace_bytes()     */
    LORA_E_OVERLAP = -9,    /* x and y overlap                                   */
    LORA_E_SYNC = -10,      /* a step launch gave up waiting (lora_plan_status)  */
    LORA_E_CAPTURE = -11,   /* the call cannot be recorded in a HIP graph        */
    LORA_E_STALE = -12      /* a launch recorded before lora_plan_update ran and did nothing */
};

/* A step's batch, in HOST memory; read during the call only. */
typedef struct {
    int32_t n_rows;             /* rows of x and y in this step                     */
    int32_t n_segments;
    const int32_t* seg_offset;  /* [n_segments + 1]                                 */
    const int32_t* seg_adapter; /* [n_segments], -1 = no adapter for that segment   */
} lora_batch_t;

typedef struct lora_table_s* lora_table_t; /* adapters of one projection, library-owned */
typedef struct lora_plan_s* lora_plan_t;   /* a batch planned against a table, library-owned */

/*
 * Register the adapters of one projection h_in -> h_out (the registry of
 * adapter ranks and weights of Section 4, kept resident on the device).
 * A_ptrs[i] / B_ptrs[i] are DEVICE pointers owned by the caller that must stay
 * valid until lora_release_adapters; ranks[i] in [1,256]; scales[i] is s_i.
 * The library copies the pointer / rank / scale table into device memory it
 * owns on `device` (synchronously on `stream`; the host arrays may be freed on
 * return).  All adapters of one table share dtype, h_in and h_out.
 * On success *out is a new table; on failure *out is left NULL.
 */
int lora_register_adapters(lora_table_t* out, int device, int h_in, int h_out, int dtype,
                           int n_adapters, const void* const* A_ptrs, const void* const* B_ptrs,
                           const int32_t* ranks, const float* scales, void* stream);

/* Free the table's device copy. The caller's A/B memory is not touched.
 * The caller must make sure no enqueued call still uses the table. */
int lora_release_adapters(lora_table_t t);

/* Bytes of device workspace that lora_shrink / lora_expand / lora_apply_fused
 * need for this batch (plan, float32 intermediate, split-K partials). */
int lora_workspace_bytes(lora_table_t t, const lora_batch_t* b, size_t* bytes);

/*
 * Shrink half of xAB (the gathered x.A_g of Section 4.1's batched operator):
 * v[t, 0:r_g] = x[t, :] . A_g in float32 for every row with adapter g >= 0.
 * Rows without an adapter and columns j >= r_g of v are not written.
 * ws: device workspace of ws_bytes >= lora_workspace_bytes(t, b), any
 * contents; it is overwritten.
 */
int lora_shrink(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, float* v,
                int64_t ldv, void* ws, size_t ws_bytes, void* stream);

/*
 * Expand half and the add into the base output (Eq. 1's xW + xAB):
 * y[t, :] <- round(y[t, :] + s_g * v[t, 0:r_g] . B_g) for every row with
 * adapter g >= 0, in place.  v is float32 [n_rows, ldv] on the device.
 */
int lora_expand(lora_table_t t, const lora_batch_t* b, const float* v, int64_t ldv, void* y,
                int64_t ldy, void* ws, size_t ws_bytes, void* stream);

/*
 * The whole delta in one call: y[t,:] <- round(y[t,:] + s_g (x[t,:].A_g).B_g).
 * The float32 intermediate lives only in ws.  Uploads the plan of this batch
 * into ws, then runs the kernels; no host synchronisation.
 *
 * lora_shrink, lora_expand and lora_apply_fused upload their work list from a
 * small ring of pinned host buffers that later calls reuse (the host waits on
 * a slot only when 16 uploads are still in flight).  A graph replay would copy
 * whatever the slot holds by then, so these three calls refuse a stream that
 * is being captured: LORA_E_CAPTURE, nothing enqueued.  Record the lora_plan_*
 * calls instead.
 */
int lora_apply_fused(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, void* y,
                     int64_t ldy, void* ws, size_t ws_bytes, void* stream);

/*
 * Eq. 1 whole (Section 2.1, y' = xW + xAB) for a step's rows, the base
 * projection fused with the adapter delta (Section 4.1 folds the adapter into
 * the base model's inference):
 *
 *     y[t, :] = round( x[t, :] . W  +  s_g (x[t, :] . A_g) . B_g )
 *
 * for every row t of the batch, g the adapter of its segment; rows of adapter
 * -1 get round(x[t, :] . W).  y is OUTPUT only (every row is written, nothing
 * is read from it).  The base weight is passed transposed: wt [h_out, ldw]
 * row-major, row n holding column n of W (the layout of a linear layer's
 * weight), ldw >= h_in and a multiple of 8, 16-byte aligned, spanning less
 * than 2 GiB; the adapters are table t's (A_g [h_in, r_g], B_g [r_g, h_out]).
 * The float32 x . A_g is computed first into ws (the shrink kernels), then one
 * MFMA GEMM over tiles of 256 rows x 256 columns adds the delta in each tile's
 * epilogue; results are rounded once.  The tiles of a last round that would
 * leave compute units idle are split along h_in: their float32 partial tiles
 * go to ws and a second kernel adds them in a fixed order (so results do not
 * depend on timing), then rounds.  Meant for prompt segments (rows of one
 * adapter run together); decode tokens work, each adapter run of a tile
 * costing one epilogue pass.  ws: device workspace of
 * lora_base_workspace_bytes(t, b) bytes, any contents.  Uploads its work list
 * through the same reused pinned ring as lora_apply_fused, so it refuses a
 * capturing stream (LORA_E_CAPTURE).  Errors as lora_apply_fused's, plus wt
 * and y must not overlap (LORA_E_OVERLAP).
 */
int lora_base_workspace_bytes(lora_table_t t, const lora_batch_t* b, size_t* bytes);
int lora_base_apply(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, const void* wt,
                    int64_t ldw, void* y, int64_t ldy, void* ws, size_t ws_bytes, void* stream);

/*
 * lora_base_apply planned once for a batch (the same batch runs every layer
 * of a prompt step, Section 2.2): lora_base_plan_create builds the work list
 * and the tile pieces, allocates the plan's device memory (work list, float32
 * v, partial tiles) and uploads them, synchronising `stream` once; it refuses
 * a capturing stream.  lora_base_plan_apply then enqueues kernels only (the
 * shrink, its reduction into v, the GEMM, and the reduction of split tiles)
 * and may be recorded in a HIP graph; it runs on any table whose shapes,
 * dtype and referenced ranks match the plan's (NULL: the plan's own table),
 * with the operand rules of lora_base_apply.  Launches on one plan use the
 * plan's memory: order them on one stream.  lora_base_plan_destroy frees it.
 */
typedef struct lora_base_plan_s* lora_base_plan_t;
int lora_base_plan_create(lora_base_plan_t* out, lora_table_t t, const lora_batch_t* b, void* stream);
int lora_base_plan_apply(lora_base_plan_t p, lora_table_t t, const void* x, int64_t ldx, const void* wt, int64_t ldw,
                         void* y, int64_t ldy, void* stream);
int lora_base_plan_destroy(lora_base_plan_t p);

/*
 * lora_apply_fused without a workspace argument and without allocating, for
 * callers that cannot allocate device memory (code that must not call
 * hipMalloc, harnesses that forbid it, tight serving loops).  The work list
 * and the float32 partial results live in a static device array of 16 MiB
 * (one per GPU the library runs on, held until the process ends); a batch
 * whose workspace (lora_workspace_bytes) exceeds it returns LORA_E_WORKSPACE
 * with nothing enqueued.  The first call on a device looks up the array's
 * device address.  The work list is copied from pageable host memory, which
 * HIP performs synchronously: the call returns once the copy is done, after
 * the stream's earlier work.  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other streams, other threads) race and must
 * be ordered by the caller.  A capturing stream is refused (LORA_E_CAPTURE).
 * Results are those of lora_apply_fused, bit for bit; arguments and errors as
 * there.
 */
int lora_apply_fused_static(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, void* y,
                            int64_t ldy, void* stream);

/*
 * Plan a batch once and apply it many times: the batch of a step is the same
 * for every adapted projection of every layer, so the grouping and the work
 * list are built once.  lora_plan_create validates the batch, builds the
 * rank-bucketed work list on the host from table t's ranks and shapes and
 * uploads it, with its own workspace, to device memory owned by the plan
 * (allocates; not for the hot loop).
 *
 * lora_plan_apply runs the whole delta (lora_apply_fused without the upload)
 * with the adapters of table t, or of the table the plan was made with when t
 * is NULL, as ONE kernel launch: its grid holds the shrink work items (float32
 * partial results over a K range of A_g), then the reduce work items (the sum
 * of a row block's partial results, its v), then the expand work items.  The
 * partial and v blocks of this launch live in plan memory armed with a
 * sentinel bit pattern (all ones, a NaN that no 16-bit input can produce);
 * two such buffers serve alternate launches, and each producer arms its block
 * in the other one.  Producers write with device-coherent stores; an expand
 * workgroup requests its B tile and its y values, then loads the values it
 * needs (v, or the partial results themselves for a row block small enough to
 * have no reduce items), again while any still holds the sentinel.  A
 * workgroup waits only for workgroups earlier in the grid, which never wait
 * for later ones, and the wait is bounded: past lora_plan_set_spin_limit polling rounds per
 * thread (default 2^18, about a quarter of a second) it gives up, raises the
 * plan's status flag and finishes with invalid results, which
 * lora_plan_status reports.  The partial blocks are added in a fixed order,
 * so the result is the same bits as lora_plan_shrink followed by
 * lora_plan_expand, whatever the timing.  Any table with the same h_in, h_out and
 * dtype whose adapters referenced by the batch have the same ranks may be
 * used (e.g. the same adapters' factors in another layer); the weight
 * pointers and scales travel in the launch arguments.  A mismatch returns
 * LORA_E_SHAPE / LORA_E_RANK / LORA_E_INDEX and enqueues nothing.
 *
 * lora_plan_shrink and lora_plan_expand are the two halves as separate
 * launches, for callers that schedule or time them apart: the shrink (a
 * shrink kernel, then a reduce kernel) writes the float32 results of x.A_g
 * into the plan's workspace, the expand adds s_g * v.B_g into y from there.  An expand must
 * follow a shrink of the same plan in stream order; the pair computes exactly
 * what lora_plan_apply computes.  Calls on one plan must be ordered (one
 * stream): they share its workspace.
 */
int lora_plan_create(lora_plan_t* out, lora_table_t t, const lora_batch_t* b, void* stream);

/*
 * Re-planning for continuous batching (Section 2.2: the batch changes every
 * iteration).  A plan owns a fixed amount of device memory and two pinned
 * host staging buffers of the same size, allocated at creation:
 * lora_plan_create sizes them for its batch, lora_plan_create_reserved for at
 * least min_bytes (lora_plan_bytes tells what one batch needs; take the
 * largest over the batches to come).  lora_plan_update plans batch b against
 * table t (NULL: the plan's table, which t then replaces) into that memory:
 * it validates b, builds the work list on the host, copies it into the next
 * staging buffer, enqueues one host-to-device copy and a small fill kernel
 * that arms the step buffers, and returns.  No device or host allocation, no
 * memset, no stream synchronisation (the host waits only when it is two
 * updates ahead of the stream's copies).  A batch that needs more than the
 * capacity returns LORA_E_WORKSPACE and leaves the plan as it was; errors of
 * b are those of lora_plan_create.  Updates and the plan's launches must be
 * ordered on one stream.  lora_plan_update also clears the plan's status.
 *
 * Graphs.  lora_plan_apply, _shrink and _expand may be recorded in a HIP graph:
 * the record holds the launch of the batch planned at that moment.  Every
 * upload stamps the work list with a new generation, and a launch carries the
 * generation it was made for: a replay after lora_plan_update finds another
 * generation in the plan's header, does nothing (y untouched), and leaves
 * LORA_E_STALE for lora_plan_status.  Record again after re-planning.
 * lora_plan_create(_reserved) and lora_plan_update refuse a capturing stream
 * (LORA_E_CAPTURE).
 */
int lora_plan_bytes(lora_table_t t, const lora_batch_t* b, size_t* bytes);
int lora_plan_create_reserved(lora_plan_t* out, lora_table_t t, const lora_batch_t* b, size_t min_bytes,
                              void* stream);
int lora_plan_update(lora_plan_t p, lora_table_t t, const lora_batch_t* b, void* stream);
int lora_plan_apply(lora_plan_t p, lora_table_t t, const void* x, int64_t ldx, void* y,
                    int64_t ldy, void* stream);
int lora_plan_shrink(lora_plan_t p, lora_table_t t, const void* x, int64_t ldx, void* stream);
int lora_plan_expand(lora_plan_t p, lora_table_t t, void* y, int64_t ldy, void* stream);
int lora_plan_destroy(lora_plan_t p);

/*
 * Projections that share their input (Section 4.1's adapter on several
 * weights of a layer: q, k and v on the attention input; gate and up on the
 * MLP input; q and gate when both read one input), run as one launch.
 * lora_plan_create_multi plans the batch on each tables[i] (n in [1, 4]) and
 * lays the n work lists out one after the other, each with its own partial
 * blocks and counters; every tables[i] must agree with tables[0] in h_in,
 * dtype and the ranks of the adapters the batch references (LORA_E_SHAPE,
 * LORA_E_RANK otherwise); h_out may differ.  lora_plan_apply_multi then runs,
 * in one grid,
 *
 *     ys[i][t, :] = round(ys[i][t, :] + s_g (x[t, :] . A_g^(i)) . B_g^(i))
 *
 * for every projection i < n (the plan's n) with the factors of tables[i]
 * (tables[0] NULL: the plan's own), which must have the h_out of projection i
 * at plan creation (LORA_E_SHAPE), each projection's items waiting only on
 * items of the same projection; ys[i] is [n_rows, ldys[i]] with ldys[i] >=
 * that h_out.  Results equal n lora_plan_apply launches bit for bit.  The ys
 * must not overlap x or each other.  Recordable in a HIP graph, like
 * lora_plan_apply; lora_plan_status reports its give-ups.  Such a plan is
 * refused by lora_plan_apply, _shrink, _expand and lora_plan_update
 * (LORA_E_ARG): create another for a new batch.
 */
int lora_plan_create_multi(lora_plan_t* out, int32_t n, const lora_table_t* tables, const lora_batch_t* b,
                           void* stream);
int lora_plan_apply_multi(lora_plan_t p, const lora_table_t* tables, const void* x, int64_t ldx, void* const* ys,
                          const int64_t* ldys, void* stream);

/*
 * Status of the plan's launches so far: waits for `stream`, then returns
 * LORA_OK; LORA_E_SYNC when a lora_plan_apply launch gave up waiting (its y is
 * invalid); or LORA_E_STALE when a recorded launch of an earlier batch ran
 * after lora_plan_update and did nothing.  The flag, the row block counters
 * and the sentinel are then reset, so the plan is usable again.
 * Host-synchronising: call it off the hot loop.
 */
int lora_plan_status(lora_plan_t p, void* stream);

/*
 * Polling rounds per thread after which a step launch's wait gives up (>= 0;
 * applies to later lora_plan_apply calls).  Returns LORA_E_ARG for a NULL
 * plan or a negative count.
 */
int lora_plan_set_spin_limit(lora_plan_t p, int32_t polls);

/*
 * The integer part of the plan, on the host only (no GPU needed): rows that
 * carry an adapter, grouped by adapter (Sections 2.3 C2 / 4.1 gather).  Groups
 * are ordered by the first row that uses the adapter; rows ascend within a
 * group; adapter -1 rows are dropped.  perm: [n_rows] capacity,
 * group_off: [n_rows + 1], group_adapter: [n_rows]; *n_groups receives G
 * and perm[0 .. group_off[G]) is filled.
 */
int lora_group_rows(const lora_batch_t* b, int32_t n_adapters, int32_t* perm, int32_t* group_off,
                    int32_t* group_adapter, int32_t* n_groups);

/*
 * The work list a plan of this batch would run, on the host only (no GPU, no
 * allocation): for adapters of ranks[0 .. n_adapters) on a projection
 * h_in -> h_out, and n_xcd XCDs (the grid of a step that fits one round of
 * workgroups is laid out per XCD; n_xcd = 1 keeps the list order).  For
 * inspection and tests of the planner.  items[0 .. *n_items) receives every
 * work item of the single launch in grid order (items of no kind included,
 * kind 0), then every reduce item of lora_shrink (kind 3, grid_pos -1);
 * capacity is the room in items.  Errors as lora_plan_create's, and
 * LORA_E_ARG when the list does not fit (*n_items then holds the size needed).
 */
typedef struct {
    int32_t kind;       /* 1 shrink, 2 expand, 3 reduce, 0 none                   */
    int32_t row_block;  /* row block index (rows of one adapter, at most 64)      */
    int32_t rank;
    int32_t nrows;      /* rows of the row block                                  */
    int32_t lo, len;    /* shrink: K range; expand: column tile; reduce: v slice  */
    int32_t sub;        /* shrink: K per pass; expand: 1 = adds the partial blocks itself; reduce: split groups */
    int32_t nsplit;     /* partial blocks (K ranges) of the row block             */
    int32_t pstride;    /* floats of one partial (or v) block                     */
    int32_t grid_pos;   /* position in the single launch's grid, -1 if not in it  */
} lora_item_info_t;
int lora_plan_inspect(const lora_batch_t* b, int32_t h_in, int32_t h_out, int32_t n_adapters,
                      const int32_t* ranks, int32_t n_xcd, lora_item_info_t* items, int32_t capacity,
                      int32_t* n_items);

/*
 * The schedule of the fused base GEMM (lora_base_apply) for this batch, on
 * the host only (no GPU, no allocation): for adapters of ranks[0 ..
 * n_adapters) on a projection h_in -> h_out and a device of n_cu compute
 * units in n_xcd XCDs.  For inspection and tests of the tiling.  Tiles are
 * square, of edge `tile`; K runs in n_stages stages of stage_k.  The tile
 * order runs over panels of `panel` row tiles, column by column inside a
 * panel; its first n_whole tiles run whole, workgroup p (p < n_xcd per_xcd)
 * taking the (p / n_xcd)-th tile of XCD p % n_xcd's share of per_xcd
 * consecutive tiles; each later tile runs as `split` workgroups over
 * consecutive ranges of `chunk` stages.  workspace_bytes is
 * lora_base_workspace_bytes'.  Errors as lora_plan_inspect's.
 */
typedef struct {
    int32_t tile;               /* tile edge: 256 or 128                          */
    int32_t n_mt, n_nt;         /* row tiles, column tiles                        */
    int32_t n_whole;            /* tiles run whole                                */
    int32_t split, chunk;       /* K ranges of each other tile, stages per range  */
    int32_t n_stages, stage_k;  /* stages of K (an even number), K per stage      */
    int32_t per_xcd;            /* whole-tile workgroups per XCD                  */
    int32_t grid;               /* workgroups of the GEMM launch                  */
    int32_t panel;              /* row tiles per panel of the tile order          */
    int32_t pad;
    uint64_t workspace_bytes;
} lora_base_info_t;
int lora_base_inspect(const lora_batch_t* b, int32_t h_in, int32_t h_out, int32_t n_adapters,
                      const int32_t* ranks, int32_t n_cu, int32_t n_xcd, lora_base_info_t* out);

/* Message of the last failed call on this thread ("" if none). */
const char* lora_last_error(void);

/* LORA_ABI_VERSION of the built library. */
int lora_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LORA_H */
