// gfx950 kernels of the batched, heterogeneous-rank LoRA delta
//   y[t,:] <- round(y[t,:] + s_g * (x[t,:] . A_g) . B_g)          (Eq. 1)
//
// Shrink: one workgroup per (row block of an adapter group, K range of A_g).
// A's rows k0..k0+len are one contiguous run of bytes, read once per step
// however many tokens use the adapter: tokens are gathered to their adapter
// instead of each token re-reading it (Section 4.1's gather, done once per
// distinct adapter).  Each lane loads eight consecutive K rows of eight
// ranks (16-byte loads, a wave covering whole rows), transposes the 8 x 8
// block in registers and writes eight 16-byte chunks of A^T to LDS; x goes to
// LDS as it is.  The pass runs on v_mfma_f32_16x16x32 (v^T[r, t] = sum_k
// A[k, r] x[t, k], float32 accumulation) while the next pass's loads are in
// flight.  When a rank has fewer tiles than waves, the waves split K and add
// their sums through LDS in wave order.  The workgroup writes its float32
// partial block.
//
// Reduce: one workgroup per slice of a row block's v.  Every position of the
// slice is the sum of the row block's partial blocks in a fixed order.
//
// Expand: one workgroup per (row block, column tile of B_g).  v is staged in
// LDS as MFMA operand fragments holding its high and low 16-bit parts, so v
// is never rounded to one 16-bit value.  Each wave streams B for its column
// blocks straight into registers: a lane loads four columns of eight
// consecutive ranks (8-byte loads, sixteen lanes covering a 128-byte row
// segment) and transposes them into four operand fragments; half-wave
// exchanges give every lane the fragment its MFMA slot needs.  y^T = B^T v^T
// runs on v_mfma_f32_16x16x32 whose 32 K slots hold 16 ranks twice, once with
// the high and once with the low 16-bit part of v (the 16x16x16 form costs
// the same per instruction on gfx950, measured, for half the work).  Each
// lane then holds 16 columns of one row; y + s*d is rounded once to the
// storage dtype.  Items of one 16-row subtile load and store each lane's y
// directly (16-byte accesses); larger items read and write y row by row and
// exchange it with the MFMA layout through LDS.  The B tile and the y values
// are requested before v is read.  A row block whose partial blocks are small
// has no reduce items: its expand items add the partial blocks up themselves.
//
// Masked loads and stores are buffer operations whose offset is moved out of
// the buffer's range: they read zeros or are dropped, with no branch.
//
// Rank is a runtime value: any rank in [1, 256] runs the same code (padded to
// a multiple of 16 inside LDS and registers only), so items of different
// ranks share one grid; the bodies are compiled for the number of rank tiles
// (or column blocks and rank steps) per wave and of 16-row subtiles, so the
// MFMA loops have no branches.
//
// Step launch: one grid holds every shrink item, then every reduce item, then
// every expand item (for a small step, laid out per XCD by the planner).  Its partial and v blocks live in two buffers used by
// alternate launches; the one a launch reads holds a sentinel bit pattern until
// it is written.  Producers write with device-coherent stores (the L2 caches
// of the XCDs are not coherent with each other; these stores write through to
// the common level instead of flushing a cache) and arm their block in the
// other buffer for the next launch.  A consumer requests what it can first (B
// tile, y values), then loads the values it waits for with device-coherent
// loads and loads again those that still hold the sentinel: the data is its
// own ready flag, so no counter or fence sits between producer and consumer.
// A workgroup only waits for workgroups earlier in the grid, which do not wait
// for later ones, so every wait ends; the number of rounds is bounded all the
// same (past it the wait gives up and sets the status flag).  The partial
// blocks are added in the same fixed order as in the separate launches, so
// both give bit-identical results whatever the timing.
#include <hip/hip_runtime.h>
#include <stddef.h>

#include <type_traits>

#include "lora_device.h"
#include "lora_internal.h"

namespace lora {

// The work item, field by field in scalar registers (the whole struct is
// never copied as one aggregate, which would send it to scratch memory).
struct Item {
    int64_t part;
    int kind, group, adapter, rank, nrows, lo, len, sub, nsplit, p0, pstride, rb, nexp, row0;
    int rows[kInlineRows];
    const void* fac;     // the factor this item streams: A_g (shrink) or B_g (expand)
    float scale;         // s_g
    int proj;            // the item's projection (launches of several projections)
    void* y;             // its y and h_out (such launches only)
    int64_t ldy;
    uint32_t y_bytes;
    int h_out;
};

// The item's two 64-byte halves are requested together (two scalar loads in
// flight), so its inline rows cost no second round trip.
typedef unsigned int u32x16 __attribute__((ext_vector_type(16)));
static_assert(offsetof(DevItem, rows) == 64 && offsetof(DevItem, row0) == 60, "DevItem halves");
__device__ __forceinline__ Item load_item(const DevItem* __restrict__ p) {
    const u32x16 w0 = ((const u32x16*)p)[0];
    const u32x16 w1 = ((const u32x16*)p)[1];
    Item it;
    it.part = (int64_t)(((uint64_t)w0[1] << 32) | w0[0]);
    it.kind = (int)(w0[2] & ((1u << kProjShift) - 1));
    it.proj = (int)(w0[2] >> kProjShift);
    it.group = (int)w0[3];
    it.adapter = (int)w0[4];
    it.rank = (int)w0[5];
    it.nrows = (int)w0[6];
    it.lo = (int)w0[7];
    it.len = (int)w0[8];
    it.sub = (int)w0[9];
    it.nsplit = (int)w0[10];
    it.p0 = (int)w0[11];
    it.pstride = (int)w0[12];
    it.rb = (int)w0[13];
    it.nexp = (int)w0[14];
    it.row0 = (int)w0[15];
#pragma unroll
    for (int q = 0; q < kInlineRows; ++q) it.rows[q] = (int)w1[q];
    it.fac = nullptr;
    it.scale = 0.f;
    it.y = nullptr;
    it.ldy = 0;
    it.y_bytes = 0;
    it.h_out = 0;
    return it;
}

// A launch whose arguments were made for another generation of the work
// list (recorded in a graph before the plan was re-planned) does nothing and
// reports itself in the status word.  The header sits at a fixed place, so
// this check is safe whatever the stale arguments hold.
__device__ __forceinline__ bool stale(const uint32_t* __restrict__ hdr, const KernelArgs& a) {
    if (hdr[0] == a.generation) return false;
    if (threadIdx.x == 0)
        __hip_atomic_store((int32_t*)(hdr + 1), (int32_t)kStatusStale, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
}

// Where the factor pointers and scales of a launch's groups are read.
enum : int {
    kLookupAuto = 0,     // the argument table for groups below kKargGroups, else the registry
    kLookupArgs = 1,     // the argument table only (the launch has at most kKargGroups groups)
    kLookupReg = 2,      // the device registry only
    kLookupMulti = 3,    // the registry of the item's projection (launches of several projections)
};

// The factor this item streams and the group's scale.  The step kernel fixes
// the source at compile time: a pointer that could point into either the
// kernel arguments or the registry makes the compiler copy the arguments to
// private memory.
constexpr int kArgsOffset = 16;   // every kernel: the item list and header pointers, then KernelArgs

template <int kLookup>
__device__ __forceinline__ void resolve(const KernelArgs& a, Item& it) {
    const bool shrink = it.kind == kItemShrink;
    if constexpr (kLookup == kLookupMulti) {
        // per-projection fields, read through the argument segment with the
        // item's (uniform) projection index
        const unsigned char* kp = (const unsigned char*)__builtin_amdgcn_kernarg_segment_ptr() + kArgsOffset;
        const int q = it.proj;
        const DevAdapter* d = *(const DevAdapter* const*)(kp + offsetof(KernelArgs, ptable) + 8 * q) + it.adapter;
        it.fac = shrink ? d->A : d->B;
        it.scale = d->scale;
        it.y = *(void* const*)(kp + offsetof(KernelArgs, py) + 8 * q);
        it.ldy = *(const int64_t*)(kp + offsetof(KernelArgs, pldy) + 8 * q);
        it.y_bytes = *(const uint32_t*)(kp + offsetof(KernelArgs, py_bytes) + 4 * q);
        it.h_out = *(const int32_t*)(kp + offsetof(KernelArgs, ph_out) + 4 * q);
        return;
    }
    if (kLookup == kLookupArgs || (kLookup == kLookupAuto && it.group < kKargGroups)) {
        it.fac = a.gfac[2 * it.group + (shrink ? 0 : 1)];
        it.scale = a.gscale[it.group];
    } else {
        const DevAdapter* d = a.table + it.adapter;
        it.fac = shrink ? d->A : d->B;
        it.scale = d->scale;
    }
}

// The launch's factor pointers and scales, striped over a wave's lanes: lane
// l holds gfac[l + 64 i] and gscale[l + 64 i].  Loaded at entry beside the
// work item, then picked with lane reads, so the pointer costs no second
// memory round trip after the item arrives.
struct LaneTable {
    uint64_t f[4];
    float s[2];
};
static_assert(2 * kKargGroups == 4 * 64 && kKargGroups == 2 * 64, "lane table shape");
// The table is read through the kernel argument segment (the step kernel's
// KernelArgs follow its 8-byte item pointer), not through the by-value
// parameter: a lane-dependent index into the parameter can make the compiler
// copy the whole argument block to private memory.
static_assert(alignof(KernelArgs) == 8, "kernel arguments: KernelArgs at offset 16");
__device__ __forceinline__ LaneTable load_lane_table() {
    const int l = threadIdx.x & 63;
    const unsigned char* kp = (const unsigned char*)__builtin_amdgcn_kernarg_segment_ptr() + kArgsOffset;
    const uint64_t* g = (const uint64_t*)(kp + offsetof(KernelArgs, gfac));
    const float* sc = (const float*)(kp + offsetof(KernelArgs, gscale));
    LaneTable t;
#pragma unroll
    for (int i = 0; i < 4; ++i) t.f[i] = g[l + 64 * i];
#pragma unroll
    for (int i = 0; i < 2; ++i) t.s[i] = sc[l + 64 * i];
    return t;
}
__device__ __forceinline__ void resolve_lanes(const LaneTable& t, Item& it) {
    const int e = 2 * it.group + (it.kind == kItemShrink ? 0 : 1);   // < 2 * kKargGroups
    const int slot = e >> 6, lane = e & 63;
    const uint64_t v = slot == 0 ? t.f[0] : (slot == 1 ? t.f[1] : (slot == 2 ? t.f[2] : t.f[3]));
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
    it.fac = (const void*)(((uint64_t)hi << 32) | lo);
    const float sv = (it.group >> 6) == 0 ? t.s[0] : t.s[1];
    it.scale = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sv), it.group & 63));
}

// v with lane Q replaced by the wave-uniform value s (one VALU lane write).
template <int Q>
__device__ __forceinline__ int write_lane(int v, int s) {
    const int su = __builtin_amdgcn_readfirstlane(s);   // the operand must be a scalar register
    asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(v) : "s"(su), "n"(Q));
    return v;
}
template <int Q>
__device__ __forceinline__ int write_rows(int v, const Item& it) {
    if constexpr (Q < kInlineRows) return write_rows<Q + 1>(write_lane<Q>(v, it.rows[Q]), it);
    return v;
}

// Lane l of every wave holds the item's row l (nrows <= 64): built from the
// inline rows with lane writes, counted from the first row when the rows are
// consecutive, or read from the grouped row order.  Must be called with
// every lane active.
__device__ __forceinline__ int lane_rows(const KernelArgs& a, const Item& it) {
    if (it.nrows <= kInlineRows) return write_rows<0>(0, it);
    const int lane = threadIdx.x & 63;
    if (it.row0 >= 0) return it.row0 + (lane < it.nrows ? lane : 0);
    return lane < it.nrows ? a.perm[it.p0 + lane] : 0;
}
// The item's r-th row, fetched from lane r (every lane active).
__device__ __forceinline__ int row_of(int rowv, int r) {
    return __builtin_amdgcn_ds_bpermute(r << 2, rowv);
}

// Step launch: between launches the partial and v blocks hold this bit
// pattern, a NaN whose low payload bits no 16-bit input can carry into a
// float32 sum.
constexpr uint32_t kSentinel = 0xffffffffu;
__device__ __forceinline__ bool unready4(const u32x4& v) {
    return (v.x == kSentinel) | (v.y == kSentinel) | (v.z == kSentinel) | (v.w == kSentinel);
}

// Step launch: a produced value is written with a device-coherent store and
// read back with device-coherent loads (measured here: a plain store polled
// through the producer's L2 is seen sooner, but a device-coherent store after
// it costs more than that saves, and without one a consumer on another XCD
// would depend on when the L2 writes the line back).
__device__ __forceinline__ u32x4 sync_load16(rsrc_t r, int off) { return bload16<kCoherent>(r, off); }
__device__ __forceinline__ void sync_store16(const u32x4& v, rsrc_t r, int off) { bstore16<kCoherent>(v, r, off); }

// Step launch: wait until none of the N 16-byte values v[i] (loaded from r at
// off[i]; masked ones read zeros) holds the sentinel, reloading those that
// do.  budget is the thread's remaining polling rounds; once it is spent the
// status flag is raised and values are used as they are.  (Compile-time
// recursion over the values: the indices stay constants.)
template <int I, int N>
__device__ __forceinline__ bool any_unready(const u32x4 (&v)[N]) {
    if constexpr (I < N) return unready4(v[I]) || any_unready<I + 1, N>(v);
    return false;
}
template <int I, int N>
__device__ __forceinline__ void reload_unready(u32x4 (&v)[N], rsrc_t r, const int (&off)[N]) {
    if constexpr (I < N) {
        if (unready4(v[I])) v[I] = sync_load16(r, off[I]);
        reload_unready<I + 1, N>(v, r, off);
    }
}
template <int N>
__device__ __forceinline__ void poll16(const KernelArgs& a, u32x4 (&v)[N], rsrc_t r, const int (&off)[N],
                                       int& budget) {
    while (any_unready<0, N>(v) && budget >= 0) {
        if (budget-- == 0) {
            __hip_atomic_store(a.status, (int32_t)kStatusGaveUp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
        __builtin_amdgcn_s_sleep(1);
        reload_unready<0, N>(v, r, off);
    }
}

// Step launch: the row block's two partial buffers.  Launches alternate
// between them, the parity coming from the row block's counter of finished
// expand items (it wraps at 2 nexp): below nexp -> buffer 0, else buffer 1.
// Within one launch every reader sees the same parity: every shrink and
// reduce item of a row block starts before any of its expand items can
// finish, and an expand item that reads late sees fewer than nexp increments
// of its own launch.  Each producer arms (sets to the sentinel) its block in
// the buffer the next launch will use, which no item of this launch reads.
// Read before the item's other loads: vector loads complete in order, so a
// wait for this one then waits for nothing else.
__device__ __forceinline__ uint32_t row_block_parity(const KernelArgs& a, const Item& it) {
    const uint32_t c = __hip_atomic_load(a.sync + (int64_t)it.rb * kSyncStride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return c >= (uint32_t)it.nexp ? 1u : 0u;
}

// ---------------------------------------------------------------------------
// Shrink
// ---------------------------------------------------------------------------
template <class Fmt, int TQ, int MS, bool kSync>
__device__ __forceinline__ void shrink_body(const KernelArgs& a, const Item& it,
                                            unsigned char* smem) {
    const int t = threadIdx.x;
    const int w = t >> 6;
    const int lr = t & 15;
    const int lg = (t >> 4) & 3;
    uint32_t parity = 0;                      // step launch: which partial buffer (read first, used last)
    if constexpr (kSync) parity = row_block_parity(a, it);
    const int R = it.rank;
    const int Rp = round_up_i(R, 16);
    const int Rv = rank_stride(R);
    const int NT = Rp / 16;
    const int sub = it.sub;                   // K staged per pass, multiple of 32
    const int KC = shrink_chunks(sub);        // 16-byte chunks per LDS row (odd)
    const int nk8 = sub / 8;
    const int nrows = it.nrows;
    const int WN = shrink_wn(R, nrows);
    const int WK = 4 / WN;
    const int wn = w % WN;
    const int wk = w / WN;
    u32x4* As = (u32x4*)smem;                 // [Rp][KC] chunks of A^T (8 consecutive K of one rank)
    u32x4* Xs = As + Rp * KC;                 // [MS*16][KC] chunks of x
    const rsrc_t ar = make_rsrc((const uint16_t*)it.fac + (int64_t)it.lo * R, (uint32_t)it.len * R * 2);
    const rsrc_t xr = make_rsrc(a.x, a.x_bytes);
    const int rowv = lane_rows(a, it);
    const u32x4 z4 = {0u, 0u, 0u, 0u};
    const bool vec = (R & 7) == 0;
    // A transpose unit of this thread: eight K rows (8 k8 .. 8 k8 + 7) of ranks
    // 8 jo .. 8 jo + 7.  Eight consecutive lanes take eight consecutive k8 of
    // one jo (their 16-byte LDS writes hit distinct banks); a wave covers whole
    // rows of A.
    const int VPR = vec ? R / 8 : 1;
    const int rest = t >> 3;
    const int jo = rest % VPR;
    const int k8 = (t & 7) + 8 * (rest / VPR);
    const bool aunit = vec && rest < VPR * (32 / VPR) && k8 < nk8;
    const int aoff0 = (8 * k8 * R + 8 * jo) * 2;   // bytes, pass start excluded
    // x chunks of this thread: chunk c of row r, p = t + 256 i
    int xoff[4], xc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int p = t + i * kThreads;
        const int r = p / nk8;
        xc[i] = p - r * nk8;
        const int row = row_of(rowv, r < nrows ? r : 0);
        xoff[i] = r < nrows ? (int)(((int64_t)row * a.ldx + it.lo + 8 * xc[i]) * 2) : kOut;
    }
    const int npass = (it.len + sub - 1) / sub;

    // the padding ranks of A^T stay zero for every pass
    for (int i = t; i < (Rp - (vec ? R : 0)) * KC; i += kThreads) As[(vec ? R : 0) * KC + i] = z4;

    u32x4 av[8], xv[4];
    auto load_pass = [&](int pass) __attribute__((always_inline)) {
        const int k0 = pass * sub;
        const int plen = min_i(sub, it.len - k0);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
            const bool ok = aunit && 8 * k8 + kk < plen;
            av[kk] = bload16(ar, ok ? aoff0 + ((k0 + kk) * R) * 2 : kOut);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) xv[i] = bload16(xr, 8 * xc[i] < plen && xoff[i] != kOut ? xoff[i] + 2 * k0 : kOut);
    };
    auto store_x = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = t + i * kThreads;
            if (p < MS * 16 * nk8) {
                const int r = p / nk8;
                Xs[r * KC + (p - r * nk8)] = xv[i];    // rows >= nrows: zero
            }
        }
    };
    auto store_a = [&]() __attribute__((always_inline)) {
        if (aunit) {
            u32x4 o[8];
            transpose8x8(av, o);
#pragma unroll
            for (int c = 0; c < 8; ++c) As[(8 * jo + c) * KC + k8] = o[c];
        }
    };
    // ranks that are not a multiple of 8: A^T element by element (correct, not tuned)
    auto store_a_generic = [&](int pass) __attribute__((always_inline)) {
        const int k0 = pass * sub;
        const int plen = min_i(sub, it.len - k0);
        for (int i = t; i < R * KC; i += kThreads) As[i] = z4;
        __syncthreads();
        uint16_t* As16 = (uint16_t*)As;
        gu16* src = (gu16*)it.fac + ((int64_t)it.lo + k0) * R;
        for (int e = t; e < plen * R; e += kThreads) {
            const int k = e / R;
            const int j = e - k * R;
            As16[j * KC * 8 + k] = src[e];
        }
    };

    f32x4 acc[MS][TQ];
#pragma unroll
    for (int m = 0; m < MS; ++m)
#pragma unroll
        for (int q = 0; q < TQ; ++q) acc[m][q] = f32x4{0.f, 0.f, 0.f, 0.f};

    load_pass(0);
    for (int pass = 0; pass < npass; ++pass) {
        if (pass > 0) __syncthreads();        // the previous pass's MFMA reads are done
        if (vec) store_a();
        else store_a_generic(pass);
        store_x();
        __syncthreads();
        const int plen = min_i(sub, it.len - pass * sub);
        if (pass + 1 < npass) load_pass(pass + 1);   // in flight during this pass's MFMA
        const int ks = (plen + 31) / 32;
        // U K-steps per round: every fragment of the round is read from LDS
        // before its MFMAs, so the reads overlap instead of each MFMA waiting
        // for its own
        auto step_frags = [&](int s, u32x4 (&af)[TQ], u32x4 (&xf)[MS]) __attribute__((always_inline)) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                af[q] = As[((tile < NT ? tile : 0) * 16 + lr) * KC + 4 * s + lg];
                if (tile >= NT) af[q] = z4;
            }
#pragma unroll
            for (int m = 0; m < MS; ++m) xf[m] = Xs[(m * 16 + lr) * KC + 4 * s + lg];
        };
        auto step_mma = [&](const u32x4 (&af)[TQ], const u32x4 (&xf)[MS]) __attribute__((always_inline)) {
#pragma unroll
            for (int m = 0; m < MS; ++m)
#pragma unroll
                for (int q = 0; q < TQ; ++q) acc[m][q] = Fmt::mma32(af[q], xf[m], acc[m][q]);
        };
        constexpr int U = TQ + MS <= 2 ? 4 : (TQ + MS <= 4 ? 2 : 1);
        int s = wn < NT ? wk : ks;            // a wave without a rank tile has no MFMA work
        for (; s + (U - 1) * WK < ks; s += U * WK) {
            u32x4 af[U][TQ], xf[U][MS];
#pragma unroll
            for (int u = 0; u < U; ++u) step_frags(s + u * WK, af[u], xf[u]);
#pragma unroll
            for (int u = 0; u < U; ++u) step_mma(af[u], xf[u]);
        }
        for (; s < ks; s += WK) {
            u32x4 af[TQ], xf[MS];
            step_frags(s, af, xf);
            step_mma(af, xf);
        }
    }

    // lane holds v[row m*16+lr][ranks tile*16 + 4lg .. +3]; the partial block
    // is [nrows][Rv] (ranks R..Rv-1 hold the zeros of the padded A^T)
    const float* pbase = a.partials + it.part + (kSync && parity ? a.pbuf : 0);
    const rsrc_t pr = make_rsrc(pbase, (uint32_t)it.pstride * 4);
    if (WK == 1) {
#pragma unroll
        for (int m = 0; m < MS; ++m) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                const int row = m * 16 + lr;
                const int r0 = tile * 16 + 4 * lg;
                const bool ok = tile < NT && row < nrows && r0 < Rv;
                if constexpr (kSync) sync_store16(as_u4(acc[m][q]), pr, ok ? (row * Rv + r0) * 4 : kOut);
                else bstore16(as_u4(acc[m][q]), pr, ok ? (row * Rv + r0) * 4 : kOut);
            }
        }
    } else {
        __syncthreads();                      // staging is read no more
        float* red = (float*)smem;            // [WK][MS*16][Rp + 4]
        const int RS = Rp + 4;
#pragma unroll
        for (int m = 0; m < MS; ++m) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                if (tile < NT)
                    *(f32x4*)(red + ((wk * MS + m) * 16 + lr) * RS + tile * 16 + 4 * lg) = acc[m][q];
            }
        }
        __syncthreads();
        const int n4 = nrows * Rv / 4;
        for (int o = t; o < n4; o += kThreads) {
            const int row = (4 * o) / Rv;
            const int r0 = 4 * o - row * Rv;
            f32x4 sum = *(const f32x4*)(red + row * RS + r0);
            for (int k = 1; k < WK; ++k) sum += *(const f32x4*)(red + (k * MS * 16 + row) * RS + r0);
            if constexpr (kSync) sync_store16(as_u4(sum), pr, 16 * o);
            else bstore16(as_u4(sum), pr, 16 * o);
        }
    }
    if constexpr (kSync) {
        // arm this block in the other buffer for the next launch.  Plain
        // stores: only the next launch reads them, and a kernel's end makes
        // its stores visible to the next.
        const rsrc_t orr = make_rsrc(a.partials + it.part + (parity ? 0 : a.pbuf), (uint32_t)it.pstride * 4);
        const u32x4 s4 = {kSentinel, kSentinel, kSentinel, kSentinel};
        for (int o = t; 4 * o < it.pstride; o += kThreads) bstore16(s4, orr, 16 * o);
    }
}

// ---------------------------------------------------------------------------
// Shrink with direct-to-LDS staging (ranks that are a multiple of 8).  Each
// pass brings `sub` K of the item's A rows and x rows into one of
// kShrinkStages LDS buffers by buffer-to-LDS loads (no registers, no VALU
// work), up to kShrinkStages passes ahead of the MFMAs.  A stays as stored,
// [K][rank] with ranks contiguous: its MFMA operand (8 consecutive K of one
// rank per lane) comes out of LDS through the transposing 64-bit read, two
// per fragment.  x rows keep their K order: one 16-byte read is a fragment.
//
// Buffer layout, in 16-byte chunks: A chunk (k, c) (ranks 8c .. 8c + 7 of K
// row k) at slot k cpr + (c ^ swa(k)), then, from the next multiple of 64,
// x chunk (r, c) (K 8c .. 8c + 7 of the item's row r) at slot r cpx +
// (c ^ (r & xmask)).  The swizzles spread a fragment read over the banks: the
// 16 lanes of a transposing read cover 4 K rows x 32 bytes, those of an x
// read 16 rows x 16 bytes.  Every slot a fragment read touches is rewritten
// by each pass (chunks past the pass's K, the item's rows or the region read
// as zeros), so nothing stale is ever used.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) unsigned char lds_u8;

// 16 bytes from buffer r at byte offset off (zeros when out of range) into
// LDS at lds + 16 * lane; lds is the same for every lane of the wave.
__device__ __forceinline__ void dma16(rsrc_t r, unsigned char* lds, int off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_u8*)lds, 16, off, 0, 0, 0);
}
// Transposing read: within each 16 lanes, lane j returns element j % 4 of the
// 8-byte values that lanes j / 4, 4 + j / 4, 8 + j / 4, 12 + j / 4 address.
// Written as inline assembly: for the builtin the compiler waits for every
// buffer-to-LDS load in flight (later passes' too) before the read.  The
// compiler does not count this read, so its value is used only after
// lgkm_wait() on it; the compiler's own LDS waits stay correct, as LDS
// operations complete in order and an uncounted one only makes them wait
// longer.
__device__ __forceinline__ u32x2 lds_read_tr16(const unsigned char* p) {
    u32x2 v;
    const uint32_t addr = (uint32_t)(uintptr_t)(lds_u8*)p;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
    return v;
}
// Every LDS read issued so far has completed, those of v among them.
template <int N>
__device__ __forceinline__ void lgkm_wait(u32x4 (&v)[N]) {
    static_assert(N == 1 || N == 2 || N == 4, "fragments");
    if constexpr (N == 1) asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]));
    else if constexpr (N == 2) asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1]));
    else asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
}
// s_waitcnt vmcnt(N), the other counters left free (gfx9 encoding: vmcnt
// bits 3:0 and 15:14).
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// LDS written by every wave (its own loads waited for) and read by none of
// the earlier pass's fragment reads any more; later LDS reads stay after it.
__device__ __forceinline__ void stage_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <class Fmt, int TQ, int MS, bool kSync>
__device__ __forceinline__ void shrink_dma_body(const KernelArgs& a, const Item& it, unsigned char* smem) {
    constexpr int S = kShrinkStages;
    constexpr int kStageBytes = kStageChunks * 16;
    constexpr int NL = kStageChunks / kThreads;   // loads per thread (and per wave) of one pass
    static_assert(NL * kThreads == kStageChunks && NL * (S - 1) < 64, "stage loads");
    const int t = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(t >> 6);
    const int lr = t & 15;
    const int lg = (t >> 4) & 3;
    uint32_t parity = 0;                      // step launch: which partial buffer (read first, used last)
    if constexpr (kSync) parity = row_block_parity(a, it);
    const int R = it.rank;                    // a multiple of 8: the partial row stride is R
    const int Rp = round_up_i(R, 16);
    const int NT = Rp / 16;
    const int sub = it.sub;                   // K per pass, a multiple of 32
    const int cpr = R / 8;
    const int cpx = sub / 8;
    const int nA = sub * cpr;
    const int nAr = round_up_i(nA, 64);
    const int nX = MS * 16 * cpx;
    const int nrows = it.nrows;
    const int WN = shrink_wn(R, nrows);
    const int WK = 4 / WN;
    const int wn = w % WN;
    const int wk = w / WN;
    // A swizzle swa(k) = ((k >> ash) << 1) & amask: 2 (k % 4) for 8 or more
    // chunks per row, 2 ((k / 2) % 2) for 4, none otherwise (and for a chunk
    // count that is not a power of two)
    const int ash = cpr >= 8 ? 0 : 1;
    const int amask = (cpr & (cpr - 1)) != 0 ? 0 : (cpr >= 8 ? 6 : (cpr == 4 ? 2 : 0));
    const int xmask = (cpx & 7) == 0 ? 7 : 3;
    // the loads take their resource from scalar registers: say that these
    // values are the same in every lane
    const uint64_t fa = (uint64_t)((const uint16_t*)it.fac + (int64_t)it.lo * R);
    const void* fau = (const void*)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(fa >> 32)) << 32) |
                                    (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)fa));
    const rsrc_t ar = make_rsrc(fau, (uint32_t)__builtin_amdgcn_readfirstlane(it.len * R * 2));
    const rsrc_t xr = make_rsrc(a.x, a.x_bytes);
    const int rowv = lane_rows(a, it);

    // This thread's NL loads of a pass: chunk q = 256 i + t of the buffer;
    // wave w's load i fills chunks 256 i + 64 w .. + 63 (one resource each).
    int lbase[NL], lk[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
        const int q = 256 * i + t;
        const int qx = q - nAr;
        const int r = qx >= 0 && qx < nX ? qx / cpx : 0;
        const int row = row_of(rowv, r < nrows ? r : 0);   // every lane active
        lbase[i] = kOut;
        lk[i] = 0;
        if (q < nA) {
            const int k = q / cpr;
            const int c = (q - k * cpr) ^ (((k >> ash) << 1) & amask);
            lbase[i] = (k * R + 8 * c) * 2;
            lk[i] = k;
        } else if (qx >= 0 && qx < nX && r < nrows) {
            const int c = (qx - r * cpx) ^ (r & xmask);
            lbase[i] = (int)(((int64_t)row * a.ldx + it.lo + 8 * c) * 2);
            lk[i] = 8 * c;
        }
    }
    auto issue = [&](int pass) __attribute__((always_inline)) {
        const int k0 = pass * sub;
        const int plen = min_i(sub, it.len - k0);
        unsigned char* st = smem + (pass % S) * kStageBytes;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            const int cb = 256 * i + 64 * w;  // wave-uniform
            const bool isA = cb < nAr;
            const int off = lbase[i] != kOut && lk[i] < plen ? lbase[i] + (isA ? k0 * R * 2 : k0 * 2) : kOut;
            dma16(isA ? ar : xr, st + cb * 16, off);
        }
    };

    f32x4 acc[MS][TQ];
#pragma unroll
    for (int m = 0; m < MS; ++m)
#pragma unroll
        for (int q = 0; q < TQ; ++q) acc[m][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    const u32x4 z4 = {0u, 0u, 0u, 0u};
    const int npass = (it.len + sub - 1) / sub;
    const int ksf = sub / 32;                 // K steps of a whole pass

    const int pre = min_i(npass, S);
    for (int p = 0; p < pre; ++p) issue(p);
    for (int pass = 0; pass < npass; ++pass) {
        // passes whose loads this wave issued after this one's
        const int after = min_i(npass - 1, pass == 0 ? S - 1 : pass + S - 2) - pass;
        if (after >= 3) wait_vm<(S > 3 ? 3 * NL : 0)>();
        else if (after == 2) wait_vm<(S > 2 ? 2 * NL : 0)>();
        else if (after == 1) wait_vm<NL>();
        else wait_vm<0>();
        stage_barrier();
        if (pass >= 1 && pass + S - 1 < npass) issue(pass + S - 1);   // into the buffer pass - 1 used
        const unsigned char* st = smem + (pass % S) * kStageBytes;
        const int plen = min_i(sub, it.len - pass * sub);
        const int ks = (plen + 31) / 32;
        // the fragment reads of K step s; af is usable after lgkm_wait(af)
        // and mask_a(af)
        auto frags = [&](int s, u32x4 (&af)[TQ], u32x4 (&xf)[MS]) __attribute__((always_inline)) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                const int col = tile * 16 + 4 * (lr & 3);     // the ranks this lane's reads address
                const int cc = tile < NT && col < R ? col >> 3 : 0;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int k = 32 * s + 8 * lg + 4 * h + (lr >> 2);
                    const int slot = k * cpr + (cc ^ (((k >> ash) << 1) & amask));
                    const u32x2 v = lds_read_tr16(st + slot * 16 + (lr & 1) * 8);
                    af[q][2 * h] = v.x;
                    af[q][2 * h + 1] = v.y;
                }
            }
#pragma unroll
            for (int m = 0; m < MS; ++m) {
                const int row = m * 16 + lr;
                const int c = (4 * s + lg) ^ (row & xmask);
                xf[m] = *(const u32x4*)(st + (nAr + row * cpx + c) * 16);
            }
        };
        auto mask_a = [&](u32x4 (&af)[TQ]) __attribute__((always_inline)) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                // this lane's operand is rank tile * 16 + lr
                if (!(tile < NT && tile * 16 + lr < R)) af[q] = z4;
            }
        };
        auto mmas = [&](const u32x4 (&af)[TQ], const u32x4 (&xf)[MS]) __attribute__((always_inline)) {
#pragma unroll
            for (int m = 0; m < MS; ++m)
#pragma unroll
                for (int q = 0; q < TQ; ++q) acc[m][q] = Fmt::mma32(af[q], xf[m], acc[m][q]);
        };
        if (wn < NT) {                        // a wave without a rank tile has no MFMA work
            // K steps of this wave: pass * ksf + s = wk (mod WK), so that the
            // waves that split K share every pass's steps in turn
            int s = ((wk - pass * ksf) % WK + WK) % WK;
            for (; s + WK < ks; s += 2 * WK) {
                u32x4 af[2][TQ], xf[2][MS];
                frags(s, af[0], xf[0]);
                frags(s + WK, af[1], xf[1]);
                lgkm_wait(af[0]);
                lgkm_wait(af[1]);
                mask_a(af[0]);
                mask_a(af[1]);
                mmas(af[0], xf[0]);
                mmas(af[1], xf[1]);
            }
            if (s < ks) {
                u32x4 af[TQ], xf[MS];
                frags(s, af, xf);
                lgkm_wait(af);
                mask_a(af);
                mmas(af, xf);
            }
        }
    }

    // lane holds v[row m*16+lr][ranks tile*16 + 4lg .. +3]; the partial block
    // is [nrows][R]
    const float* pbase = a.partials + it.part + (kSync && parity ? a.pbuf : 0);
    const rsrc_t pr = make_rsrc(pbase, (uint32_t)it.pstride * 4);
    if (WK == 1) {
#pragma unroll
        for (int m = 0; m < MS; ++m) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                const int row = m * 16 + lr;
                const int r0 = tile * 16 + 4 * lg;
                const bool ok = tile < NT && row < nrows && r0 < R;
                if constexpr (kSync) sync_store16(as_u4(acc[m][q]), pr, ok ? (row * R + r0) * 4 : kOut);
                else bstore16(as_u4(acc[m][q]), pr, ok ? (row * R + r0) * 4 : kOut);
            }
        }
    } else {
        __syncthreads();                      // the buffers are read no more
        float* red = (float*)smem;            // [WK][MS*16][Rp + 4]
        const int RS = Rp + 4;
#pragma unroll
        for (int m = 0; m < MS; ++m) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                if (tile < NT)
                    *(f32x4*)(red + ((wk * MS + m) * 16 + lr) * RS + tile * 16 + 4 * lg) = acc[m][q];
            }
        }
        __syncthreads();
        const int n4 = nrows * R / 4;
        for (int o = t; o < n4; o += kThreads) {
            const int row = (4 * o) / R;
            const int r0 = 4 * o - row * R;
            f32x4 sum = *(const f32x4*)(red + row * RS + r0);
            for (int k = 1; k < WK; ++k) sum += *(const f32x4*)(red + (k * MS * 16 + row) * RS + r0);
            if constexpr (kSync) sync_store16(as_u4(sum), pr, 16 * o);
            else bstore16(as_u4(sum), pr, 16 * o);
        }
    }
    if constexpr (kSync) {
        // arm this block in the other buffer for the next launch (plain
        // stores: only the next launch reads them)
        const rsrc_t orr = make_rsrc(a.partials + it.part + (parity ? 0 : a.pbuf), (uint32_t)it.pstride * 4);
        const u32x4 s4 = {kSentinel, kSentinel, kSentinel, kSentinel};
        for (int o = t; 4 * o < it.pstride; o += kThreads) bstore16(s4, orr, 16 * o);
    }
}

template <class Fmt, bool kSync>
__device__ __forceinline__ void shrink_item(const KernelArgs& a, const Item& it, unsigned char* smem) {
    const int tq = shrink_tq(it.rank, it.nrows);
    const int ms = msub_body(it.nrows);
    if (shrink_uses_dma(it.rank, it.nrows)) {     // ms is 2 or 4
        if (tq == 1) {
            if (ms == 2) shrink_dma_body<Fmt, 1, 2, kSync>(a, it, smem);
            else shrink_dma_body<Fmt, 1, 4, kSync>(a, it, smem);
        } else if (tq == 2) {
            if (ms == 2) shrink_dma_body<Fmt, 2, 2, kSync>(a, it, smem);
            else shrink_dma_body<Fmt, 2, 4, kSync>(a, it, smem);
        } else {
            if (ms == 2) shrink_dma_body<Fmt, 4, 2, kSync>(a, it, smem);
            else shrink_dma_body<Fmt, 4, 4, kSync>(a, it, smem);
        }
        return;
    }
    if (tq == 1) {
        if (ms == 1) shrink_body<Fmt, 1, 1, kSync>(a, it, smem);
        else if (ms == 2) shrink_body<Fmt, 1, 2, kSync>(a, it, smem);
        else shrink_body<Fmt, 1, 4, kSync>(a, it, smem);
    } else if (tq == 2) {
        if (ms == 1) shrink_body<Fmt, 2, 1, kSync>(a, it, smem);
        else if (ms == 2) shrink_body<Fmt, 2, 2, kSync>(a, it, smem);
        else shrink_body<Fmt, 2, 4, kSync>(a, it, smem);
    } else {
        if (ms == 1) shrink_body<Fmt, 4, 1, kSync>(a, it, smem);
        else if (ms == 2) shrink_body<Fmt, 4, 2, kSync>(a, it, smem);
        else shrink_body<Fmt, 4, 4, kSync>(a, it, smem);
    }
}

template <class Fmt>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) lora_shrink_kernel(const DevItem* __restrict__ items, const uint32_t* __restrict__ hdr, KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kShrinkLds];
    Item it = load_item(items + blockIdx.x);
    if (stale(hdr, a) || it.kind != kItemShrink) return;
    resolve<kLookupAuto>(a, it);
    shrink_item<Fmt, false>(a, it, smem);
}

// ---------------------------------------------------------------------------
// Reduce: floats [lo, lo + len) of the row block's v block (len a multiple
// of 4) are the sum of its nsplit partial blocks.  Thread (position p, group
// q) adds blocks q, q + G, q + 2G, ... in order (G = sub split groups, at
// most kMaxSplitLoads blocks per thread, all loads in flight together); the G
// sums are then added in order q = 0..G-1.  The order depends on the plan
// only, so every launch form adds identically.  With a caller v (lora_shrink)
// the sums go to its rows instead of the v block.
// ---------------------------------------------------------------------------
template <bool kSync>
__device__ __forceinline__ void reduce_body(const KernelArgs& a, const Item& it, unsigned char* smem) {
    const int t = threadIdx.x;
    uint32_t parity = 0;
    if constexpr (kSync) parity = row_block_parity(a, it);
    const int Rv = rank_stride(it.rank);
    const int np = it.len / 4;                // float4 positions of the slice
    const int G = it.sub;
    const int p = t % np;
    const int q = t / np;
    f32x4* red = (f32x4*)smem;                // [G][np]
    const float* P = a.partials + it.part + (kSync && parity ? a.pbuf : 0);
    const rsrc_t pr = make_rsrc(P, (uint32_t)(it.nsplit + 1) * it.pstride * 4);
    int budget = a.spin_limit;
    if (q < G) {
        int off[kMaxSplitLoads];
        u32x4 u[kMaxSplitLoads];
#pragma unroll
        for (int i = 0; i < kMaxSplitLoads; ++i) {
            const int c = q + i * G;
            off[i] = c < it.nsplit ? (c * it.pstride + it.lo + 4 * p) * 4 : kOut;
            u[i] = kSync ? sync_load16(pr, off[i]) : bload16(pr, off[i]);
        }
        if constexpr (kSync) poll16<kMaxSplitLoads>(a, u, pr, off, budget);
        f32x4 s = as_f4(u[0]);
#pragma unroll
        for (int i = 1; i < kMaxSplitLoads; ++i) s += as_f4(u[i]);
        red[q * np + p] = s;
    }
    __syncthreads();
    if (t < np) {
        f32x4 s = red[t];
        for (int g = 1; g < G; ++g) s += red[g * np + t];
        const int f = it.lo + 4 * t;          // flat index in the v block
        if (a.v) {
            const int row = f / Rv;
            const int r0 = f - row * Rv;
            float* dst = a.v + (int64_t)a.perm[it.p0 + row] * a.ldv + r0;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (r0 + i < it.rank) dst[i] = s[i];
        } else {
            const int vo = (it.nsplit * it.pstride + f) * 4;
            if constexpr (kSync) sync_store16(as_u4(s), pr, vo);
            else bstore16(as_u4(s), pr, vo);
            if constexpr (kSync) {
                // arm this slice in the other buffer for the next launch
                const rsrc_t orr = make_rsrc(a.partials + it.part + (parity ? 0 : a.pbuf),
                                             (uint32_t)(it.nsplit + 1) * it.pstride * 4);
                bstore16(u32x4{kSentinel, kSentinel, kSentinel, kSentinel}, orr, vo);
            }
        }
    }
}

__global__ void __launch_bounds__(kThreads) lora_reduce_kernel(const DevItem* __restrict__ items,
                                                              const uint32_t* __restrict__ hdr, KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kReduceLds];
    const Item it = load_item(items + blockIdx.x);
    if (stale(hdr, a) || it.kind != kItemReduce) return;
    reduce_body<false>(a, it, smem);
}

// ---------------------------------------------------------------------------
// Expand
// ---------------------------------------------------------------------------
// Column order inside a 64-column block: MFMA output row m of instruction c
// (c = 0..3) is column base(m) + c.  A lane then loads 4 consecutive columns
// of B (sixteen lanes: one 128-byte row segment) and ends up holding columns
// 8g .. 8g+7 and 32 + 8g .. 32 + 8g + 7 of its row (g = lane / 16).
__device__ __forceinline__ int col_base(int m) { return 8 * (m >> 2) + 32 * ((m >> 1) & 1) + 4 * (m & 1); }

template <class Fmt, int Q, int KSG, int MS, bool kSync, bool kMulti = false>
__device__ __forceinline__ void expand_body(const KernelArgs& a, const Item& it,
                                            unsigned char* smem) {
    // the item's y: the launch's, or its projection's in a launch of several
    void* const ybase = kMulti ? it.y : a.y;
    const int64_t ldy = kMulti ? it.ldy : a.ldy;
    const uint32_t ybytes = kMulti ? it.y_bytes : a.y_bytes;
    const int t = threadIdx.x;
    const int w = t >> 6;
    const int l = t & 63;
    const int lr = l & 15;
    const int lg = l >> 4;
    uint32_t parity = 0;                      // step launch (read first, see row_block_parity)
    if constexpr (kSync) parity = row_block_parity(a, it);
    const int R = it.rank;
    const int Rv = rank_stride(R);
    const int KS = round_up_i(R, 16) / 16;
    const int len = it.len;                   // columns of the item: one tile, or (prompt items) several
    constexpr int kTile = 256 * Q;            // columns of a tile
    int tl = 0;                               // the current tile's first column within the item
    const int nrows = it.nrows;
    const int h_out = kMulti ? it.h_out : a.h_out;
    u32x4* Vf = (u32x4*)smem;                 // [MS][KS][64] operand fragments of v
    const rsrc_t yr = make_rsrc(ybase, ybytes);
    const rsrc_t br = make_rsrc((const uint16_t*)it.fac + it.lo, (uint32_t)(R * h_out - it.lo) * 2);
    const int rowv = lane_rows(a, it);

    // --- y.  Items of one 16-row subtile (decode) load each lane's y directly:
    // rows m*16+lr, columns cb*64 + 32h + 8lg .. +7 of the wave's column blocks
    // cb = w + 4q.  Larger items read and write y row by row (whole 16-byte
    // chunks of consecutive columns across the lanes) and exchange it with the
    // MFMA layout through LDS: measured on a plain read-modify-write of y, 22.8
    // us against 29.3 us for the MFMA layout's access pattern.
    constexpr bool kStage = MS > 1;
    constexpr int TC = 32 * Q;                // 16-byte chunks per row of the tile
    constexpr int YS = kStage ? MS * 16 * TC / kThreads : 1;
    int yoff[kStage ? 1 : Q][MS][2];
    u32x4 yv[kStage ? 1 : Q][MS][2];
    // Larger items: the tile's y goes straight into LDS (buffer-to-LDS loads),
    // row r's chunk c at slot r TC + (c ^ (r % 8)); thread t moves slots
    // t + 256 i, wave w's load i slots 256 i + 64 w .. + 63.
    unsigned char* Ysb = smem + kExpandYsOff;
    int soff[YS];
    auto y_tile = [&]() __attribute__((always_inline)) {
        const int wu = __builtin_amdgcn_readfirstlane(w);
#pragma unroll
        for (int i = 0; i < YS; ++i) {
            const int p = t + i * kThreads;
            const int r = p / TC;
            const int c = (p - r * TC) ^ (r & 7);
            const int row = row_of(rowv, r < nrows ? r : 0);
            soff[i] = r < nrows && tl + 8 * c + 8 <= len ? (int)(((int64_t)row * ldy + it.lo + tl + 8 * c) * 2) : kOut;
            dma16(yr, Ysb + (i * kThreads + 64 * wu) * 16, soff[i]);
        }
    };
    if constexpr (kStage && kSync) {
        y_tile();                             // in flight while the item waits for its v
    } else if constexpr (kStage) {
        // separate launch (v is ready): y after the v loads, so that those
        // are not queued behind it
    } else {
#pragma unroll
        for (int m = 0; m < MS; ++m) {
            const int row = row_of(rowv, m * 16 + lr < nrows ? m * 16 + lr : 0);
#pragma unroll
            for (int q = 0; q < Q; ++q)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int c = (w + 4 * q) * 64 + 32 * h + 8 * lg;
                    const bool ok = m * 16 + lr < nrows && c + 8 <= len;
                    yoff[q][m][h] = ok ? (int)(((int64_t)row * ldy + it.lo + c) * 2) : kOut;
                }
        }
#pragma unroll
        for (int q = 0; q < Q; ++q)
#pragma unroll
            for (int m = 0; m < MS; ++m)
#pragma unroll
                for (int h = 0; h < 2; ++h) yv[q][m][h] = bload16(yr, yoff[q][m][h]);
    }

    // --- B.  A group is NU = Q * KSG units (column block q, rank step ks =
    // g0 + kl); units go in pairs: lanes 0-31 load the first, lanes 32-63 the
    // second, each lane rank octet 16ks + 8(lg & 1) (8 rows) of 4 columns
    // cb*64 + base(lr) .. +3.  After the transpose a half-wave exchange gives
    // every lane both units' fragments (the K slots hold each octet twice).
    constexpr int NU = Q * KSG;
    constexpr int NP = (NU + 1) / 2;
    const int mycol = col_base(lr);
    u32x2 bv[NP][8];
    auto load_group = [&](int g0) __attribute__((always_inline)) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int u = l < 32 ? 2 * p : (2 * p + 1 < NU ? 2 * p + 1 : 2 * p);
            const int q = u / KSG;
            const int kl = u - q * KSG;
            const int col = (w + 4 * q) * 64 + mycol;
            const int j0 = 16 * (g0 + kl) + 8 * (lg & 1);
#pragma unroll
            for (int kk = 0; kk < 8; ++kk) {
                const bool ok = j0 + kk < R && tl + col + 4 <= len;
                bv[p][kk] = bload8(br, ok ? ((j0 + kk) * h_out + tl + col) * 2 : kOut);
            }
        }
    };
    load_group(0);
    // MFMA operand fragments of the loaded group: column c of unit pair p, as
    // lanes 0-31 loaded it (fa) and as lanes 32-63 loaded it (fb), in every
    // lane.  The first group's are made right after the thread's v fill,
    // while other threads may still wait for theirs.
    u32x4 fa[NP][4], fb[NP][4];
    auto prepare = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int wd = c >> 1;
                u32x4 f;
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
                    const uint32_t x0 = bv[p][2 * qq][wd], x1 = bv[p][2 * qq + 1][wd];
                    f[qq] = (c & 1) ? pack_hi(x0, x1) : pack_lo(x0, x1);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const auto sw = __builtin_amdgcn_permlane32_swap(f[i], f[i], false, false);
                    fa[p][c][i] = sw[0];
                    fb[p][c][i] = sw[1];
                }
            }
    };

    // --- v fragments to LDS.  Entry (m, ks, lane): lanes 16g + n hold row
    // m*16 + n, ranks 16ks + 8(g & 1) .. +7, the high part for g < 2 and the
    // low part for g >= 2.  Task (m, ks, n, qq) fills ranks 16ks + 4qq .. +3:
    // half (qq & 1) of lanes n + 16(qq >> 1) (high) and n + 16((qq >> 1) + 2) (low).
    //
    // binary16 cannot hold a high part beyond 65504.  The fill keeps each
    // thread's largest |v| and every wave leaves its maximum in LDS; if the
    // item's maximum reaches 2^15, the fill runs again with v scaled by the
    // power of two 2^k that brings the maximum into [2^14, 2^15) and the
    // epilogue multiplies s_g by 2^-k.  Both scalings are exact, so the result
    // is the unscaled product's (bit for bit wherever the unscaled split was
    // finite and normal).
    const bool direct = it.sub != 0;          // add the partial blocks up here
    const float* vP = a.partials + it.part + (kSync && parity ? a.pbuf : 0);
    const rsrc_t pr = make_rsrc(vP, (uint32_t)(it.nsplit + 1) * it.pstride * 4);
    const int vbase = it.nsplit * it.pstride * 4;
    int budget = a.spin_limit;
    float vabs = 0.f;
    // kSerial: the rerun, when every value is known to be written; partial
    // blocks are then loaded one by one (the same additions in the same
    // order) so that the B fragments made meanwhile keep their registers
    auto fill = [&](auto serial, float mul) __attribute__((always_inline)) {
        constexpr bool kSerial = decltype(serial)::value;
        u32x2* Vh = (u32x2*)smem;             // Vf as 8-byte halves
        const int ntask = MS * KS * 64;
        for (int task = t; task < ntask; task += kThreads) {
            const int mk = task >> 6;                 // m * KS + ks
            const int ll = task & 63;
            const int n = ll & 15;
            const int qq = ll >> 4;
            const int m = mk / KS;
            const int ks = mk - m * KS;
            const int row = m * 16 + n;
            const int j0 = 16 * ks + 4 * qq;
            const bool ok = row < nrows && j0 < R;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (a.v) {
                if (ok) {
                    const float* src = a.v + (int64_t)a.perm[it.p0 + row] * a.ldv + j0;
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (j0 + i < R) v[i] = src[i];
                }
            } else if (direct && kSerial) {
                const int o = (row * Rv + j0) * 4;
                v = as_f4(kSync ? sync_load16(pr, ok ? o : kOut) : bload16(pr, ok ? o : kOut));
                for (int c = 1; c < it.nsplit; ++c) {
                    const int oc = ok ? c * it.pstride * 4 + o : kOut;
                    v += as_f4(kSync ? sync_load16(pr, oc) : bload16(pr, oc));
                }
            } else if (direct) {
                const int o = (row * Rv + j0) * 4;
                int off[kDirectSplits];
                u32x4 u[kDirectSplits];
#pragma unroll
                for (int c = 0; c < kDirectSplits; ++c) {
                    off[c] = ok && c < it.nsplit ? c * it.pstride * 4 + o : kOut;
                    u[c] = kSync ? sync_load16(pr, off[c]) : bload16(pr, off[c]);
                }
                if constexpr (kSync) poll16<kDirectSplits>(a, u, pr, off, budget);
                v = as_f4(u[0]);
#pragma unroll
                for (int c = 1; c < kDirectSplits; ++c) v += as_f4(u[c]);
            } else {
                int off[1] = {ok ? vbase + (row * Rv + j0) * 4 : kOut};
                u32x4 u[1] = {kSync ? sync_load16(pr, off[0]) : bload16(pr, off[0])};
                if constexpr (kSync && !kSerial) poll16<1>(a, u, pr, off, budget);
                v = as_f4(u[0]);
            }
            if constexpr (Fmt::kNarrowRange) {
                vabs = fmaxf(vabs, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
                v *= mul;
            }
            const uint32_t h01 = Fmt::pack2(v[0], v[1]), h23 = Fmt::pack2(v[2], v[3]);
            const uint32_t l01 = Fmt::pack2(v[0] - Fmt::to_f32(lo16(h01)), v[1] - Fmt::to_f32(hi16(h01)));
            const uint32_t l23 = Fmt::pack2(v[2] - Fmt::to_f32(lo16(h23)), v[3] - Fmt::to_f32(hi16(h23)));
            const int e = mk * 64 + n + 16 * (qq >> 1);
            Vh[2 * e + (qq & 1)] = u32x2{h01, h23};
            Vh[2 * (e + 32) + (qq & 1)] = u32x2{l01, l23};
        }
    };
    fill(std::false_type{}, 1.f);
    if constexpr (kStage && !kSync) y_tile();
    float* vmax = (float*)(smem + kExpandVmaxOff);   // one float per wave
    if constexpr (Fmt::kNarrowRange) {
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) vabs = fmaxf(vabs, __shfl_xor(vabs, d, 64));
        if (l == 0) vmax[w] = vabs;
    }
    prepare();                                // while other threads still wait for their v
    // decode items (one subtile) put the next rank group's B in flight from
    // here, during the barrier and this group's MFMAs (larger items, whose B
    // mostly comes from L2, keep the registers for their accumulators)
    constexpr bool kAhead = MS != 2;          // (items of two subtiles: registers)
    if (kAhead && KSG < KS) load_group(KSG);
    __syncthreads();
    float escale = it.scale;                  // s_g, times 2^-k when v was scaled
    if constexpr (Fmt::kNarrowRange) {
        const float m = fmaxf(fmaxf(vmax[0], vmax[1]), fmaxf(vmax[2], vmax[3]));
        if (m >= 32768.f) {                   // the same in every thread: a uniform branch
            const int E = (int)((__float_as_uint(m) >> 23) & 0xff) - 127;
            const int k = max_i(14 - E, -64);
            fill(std::true_type{}, __uint_as_float((uint32_t)(127 + k) << 23));
            escale = it.scale * __uint_as_float((uint32_t)(127 - k) << 23);
            __syncthreads();
        }
    }
    // step launch: this item has read its v; count it (no wait for the result)
    if constexpr (kSync)
        if (t == 0)
            (void)__builtin_amdgcn_atomic_inc32(a.sync + (int64_t)it.rb * kSyncStride, 2u * (uint32_t)it.nexp - 1u,
                                                __ATOMIC_RELAXED, "agent");

    // --- per tile: y^T = B^T v^T on MFMA (16x16x32: 16 ranks x high and low
    // part of v), then the epilogue.  A prompt item walks its tiles with the
    // v fragments made once; the next tile's B and y are loaded while this
    // tile's epilogue runs.
    for (;;) {
    if (tl > 0) {                             // a later tile: its group 0 was loaded in the last epilogue
        prepare();
        if (kAhead && KSG < KS) load_group(KSG);
    }
    f32x4 acc[Q][4][MS];
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int m = 0; m < MS; ++m) acc[q][c][m] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int g0 = 0; g0 < KS; g0 += KSG) {
        if (g0 > 0) {
            if (!kAhead) load_group(g0);
            prepare();
            if (kAhead && g0 + KSG < KS) load_group(g0 + KSG);
        }
        u32x4 vf[KSG][MS];
#pragma unroll
        for (int kl = 0; kl < KSG; ++kl)
#pragma unroll
            for (int m = 0; m < MS; ++m) {
                const int ks = g0 + kl < KS ? g0 + kl : KS - 1;
                vf[kl][m] = Vf[(m * KS + ks) * 64 + l];
                if (g0 + kl >= KS) vf[kl][m] = u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int ua = 2 * p, ub = 2 * p + 1;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
#pragma unroll
                for (int m = 0; m < MS; ++m)
                    acc[ua / KSG][c][m] = Fmt::mma32(fa[p][c], vf[ua % KSG][m], acc[ua / KSG][c][m]);
                if (ub < NU) {
#pragma unroll
                    for (int m = 0; m < MS; ++m)
                        acc[ub / KSG][c][m] = Fmt::mma32(fb[p][c], vf[ub % KSG][m], acc[ub / KSG][c][m]);
                }
            }
        }
    }

    const bool more = MS == 4 && tl + kTile < len;  // the item has another tile

    // --- epilogue: lane holds, for instruction c and output row 4lg + i,
    // column cb*64 + 8lg + 32(i >> 1) + 4(i & 1) + c of row m*16 + lr
    u32x4* Ys = (u32x4*)Ysb;
    if constexpr (kStage) {
        wait_vm<0>();                         // this thread's y loads have landed (and anything before them)
        stage_barrier();                      // every thread's have
        if (more) {                           // the next tile's B, during this epilogue
            tl += kTile;
            load_group(0);
            tl -= kTile;
        }
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
#pragma unroll
        for (int m = 0; m < MS; ++m) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int yr_ = m * 16 + lr;
                const int sidx = yr_ * TC + (((w + 4 * q) * 8 + 4 * h + lg) ^ (yr_ & 7));
                u32x4 yo;
                if constexpr (kStage) yo = Ys[sidx];
                else yo = yv[q][m][h];
                u32x4 o;
#pragma unroll
                for (int e2 = 0; e2 < 4; ++e2) {
                    // elements e = 2 e2, 2 e2 + 1: i = 2h + (e >> 2), c = e & 3
                    const int e = 2 * e2;
                    const int i = 2 * h + (e >> 2);
                    const float f0 = fmaf(escale, acc[q][e & 3][m][i], Fmt::to_f32(lo16(yo[e2])));
                    const float f1 = fmaf(escale, acc[q][(e + 1) & 3][m][i], Fmt::to_f32(hi16(yo[e2])));
                    o[e2] = Fmt::pack2(f0, f1);
                }
                if constexpr (kStage) Ys[sidx] = o;
                else bstore16(o, yr, yoff[q][m][h]);
            }
        }
    }
    if constexpr (kStage) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < YS; ++i) bstore16(Ys[t + i * kThreads], yr, soff[i]);
    }
    if (!more) break;
    tl += kTile;
    __syncthreads();                          // every thread has read Ys for its stores
    y_tile();                                 // the next tile's y, during its MFMAs
    }
}

template <class Fmt, bool kSync, bool kMulti = false>
__device__ __forceinline__ void expand_item(const KernelArgs& a, const Item& it, unsigned char* smem) {
    const int ms = msub_body(it.nrows);
    const int q = expand_q(it.rank, it.nrows);
    const int ksg = expand_ksg(it.rank, it.nrows);
    if (ms == 1) {
        if (q == 4) expand_body<Fmt, 4, 1, 1, kSync, kMulti>(a, it, smem);
        else if (q == 2) {
            if (ksg == 1) expand_body<Fmt, 2, 1, 1, kSync, kMulti>(a, it, smem);
            else expand_body<Fmt, 2, 2, 1, kSync, kMulti>(a, it, smem);
        } else {
            if (ksg == 2) expand_body<Fmt, 1, 2, 1, kSync, kMulti>(a, it, smem);
            else expand_body<Fmt, 1, 4, 1, kSync, kMulti>(a, it, smem);
        }
    } else if (ms == 2) {
        if (q == 2) {
            if (ksg == 1) expand_body<Fmt, 2, 1, 2, kSync, kMulti>(a, it, smem);
            else expand_body<Fmt, 2, 2, 2, kSync, kMulti>(a, it, smem);
        } else {
            if (ksg == 2) expand_body<Fmt, 1, 2, 2, kSync, kMulti>(a, it, smem);
            else expand_body<Fmt, 1, 4, 2, kSync, kMulti>(a, it, smem);
        }
    } else {
        if (ksg == 1) expand_body<Fmt, 1, 1, 4, kSync, kMulti>(a, it, smem);
        else expand_body<Fmt, 1, 2, 4, kSync, kMulti>(a, it, smem);   // ksg <= 2 with four subtiles
    }
}

template <class Fmt>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) lora_expand_kernel(const DevItem* __restrict__ items, const uint32_t* __restrict__ hdr, KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kExpandLds];
    Item it = load_item(items + blockIdx.x);
    if (stale(hdr, a) || it.kind != kItemExpand) return;
    resolve<kLookupAuto>(a, it);
    expand_item<Fmt, false>(a, it, smem);
}

// ---------------------------------------------------------------------------
// Step: shrink items, then reduce items, then expand items, in one grid (two
// workgroups per CU: the register budget is 256 per lane); in a grid laid out
// per XCD this order holds among the items each XCD runs, and slots holding an
// item of no kind end at once.  The item list is
// a kernel argument of its own, ahead of the argument block, so that it can
// be preloaded into scalar registers at wave launch.
// ---------------------------------------------------------------------------
template <class Fmt, int kLookup>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
lora_step_kernel(const DevItem* __restrict__ items, const uint32_t* __restrict__ hdr, KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kStepLds];
    Item it;
    if constexpr (kLookup == kLookupArgs) {
        const LaneTable lt = load_lane_table();       // in flight with the item and the header
        it = load_item(items + blockIdx.x);
        if (stale(hdr, a)) return;
        if (it.kind == kItemShrink || it.kind == kItemExpand) resolve_lanes(lt, it);
    } else {
        it = load_item(items + blockIdx.x);
        if (stale(hdr, a)) return;
        if (it.kind == kItemShrink || it.kind == kItemExpand) resolve<kLookup>(a, it);
    }
    constexpr bool kMulti = kLookup == kLookupMulti;
    if (it.kind == kItemShrink) shrink_item<Fmt, true>(a, it, smem);
    else if (it.kind == kItemExpand) expand_item<Fmt, true, kMulti>(a, it, smem);
    else if (it.kind == kItemReduce) reduce_body<true>(a, it, smem);
}

// ---------------------------------------------------------------------------
// launches (hdr: the plan's or workspace's header)
// ---------------------------------------------------------------------------
hipError_t launch_shrink(const KernelArgs& a, const uint32_t* hdr, int dtype, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    if (dtype == 0)
        hipLaunchKernelGGL(lora_shrink_kernel<FmtF16>, dim3(a.n_items), dim3(kThreads), 0, s, a.items, hdr, a);
    else
        hipLaunchKernelGGL(lora_shrink_kernel<FmtBF16>, dim3(a.n_items), dim3(kThreads), 0, s, a.items, hdr, a);
    return hipGetLastError();
}

hipError_t launch_expand(const KernelArgs& a, const uint32_t* hdr, int dtype, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    if (dtype == 0)
        hipLaunchKernelGGL(lora_expand_kernel<FmtF16>, dim3(a.n_items), dim3(kThreads), 0, s, a.items, hdr, a);
    else
        hipLaunchKernelGGL(lora_expand_kernel<FmtBF16>, dim3(a.n_items), dim3(kThreads), 0, s, a.items, hdr, a);
    return hipGetLastError();
}

hipError_t launch_step(const KernelArgs& a, const uint32_t* hdr, int dtype, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    const dim3 g(a.n_items), b(kThreads);
    const bool args = a.n_groups <= kKargGroups;
    if (a.n_proj > 1) {
        if (dtype == 0) hipLaunchKernelGGL((lora_step_kernel<FmtF16, kLookupMulti>), g, b, 0, s, a.items, hdr, a);
        else hipLaunchKernelGGL((lora_step_kernel<FmtBF16, kLookupMulti>), g, b, 0, s, a.items, hdr, a);
    } else if (dtype == 0) {
        if (args) hipLaunchKernelGGL((lora_step_kernel<FmtF16, kLookupArgs>), g, b, 0, s, a.items, hdr, a);
        else hipLaunchKernelGGL((lora_step_kernel<FmtF16, kLookupReg>), g, b, 0, s, a.items, hdr, a);
    } else {
        if (args) hipLaunchKernelGGL((lora_step_kernel<FmtBF16, kLookupArgs>), g, b, 0, s, a.items, hdr, a);
        else hipLaunchKernelGGL((lora_step_kernel<FmtBF16, kLookupReg>), g, b, 0, s, a.items, hdr, a);
    }
    return hipGetLastError();
}

hipError_t launch_reduce(const KernelArgs& a, const uint32_t* hdr, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    hipLaunchKernelGGL(lora_reduce_kernel, dim3(a.n_items), dim3(kThreads), 0, s, a.items, hdr, a);
    return hipGetLastError();
}

// Fill n 32-bit words at p with v (arming a plan's step buffers and counters:
// a kernel, not a memset, so that the sequence may be recorded in a graph).
__global__ void __launch_bounds__(kThreads) lora_fill_kernel(uint32_t* __restrict__ p, uint32_t v, uint64_t n) {
    const uint64_t stride = (uint64_t)gridDim.x * kThreads * 4;
    const u32x4 v4 = {v, v, v, v};
    for (uint64_t i = ((uint64_t)blockIdx.x * kThreads + threadIdx.x) * 4; i < n; i += stride) {
        if (i + 4 <= n) *(u32x4*)(p + i) = v4;
        else
            for (uint64_t j = i; j < n; ++j) p[j] = v;
    }
}

hipError_t launch_fill(uint32_t* p, uint32_t v, uint64_t n_words, hipStream_t s) {
    if (n_words == 0) return hipSuccess;
    const uint64_t want = (n_words + 4 * kThreads - 1) / (4 * kThreads);
    const unsigned grid = (unsigned)(want < 1024 ? want : 1024);
    hipLaunchKernelGGL(lora_fill_kernel, dim3(grid), dim3(kThreads), 0, s, p, v, n_words);
    return hipGetLastError();
}

}  // namespace lora
