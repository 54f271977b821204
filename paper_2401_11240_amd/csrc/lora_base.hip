// gfx950 kernel of Eq. 1 whole (Section 2.1): the base projection and the
// adapter delta of every row in one MFMA GEMM,
//
//     y[t, :] = round( x[t, :] . W  +  s_g (x[t, :] . A_g) . B_g ),
//
// where g is the adapter of row t's segment (rows of adapter -1 get x . W).
// The float32 v = x . A_g comes in beforehand (the shrink kernels); the
// delta s_g v . B_g is added in the epilogue of each output tile.  This is
// the shape of a prompt step of Section 4.1's GPU LoRA once the base
// projection is fused in: the base GEMM's arithmetic intensity is far above
// the MFMA ridge, so the tile runs at MFMA rate while the delta costs r_g/K of
// the base work.
//
// Tile: T rows of x (tokens) x T columns of y, T = 256 or 128, one
// workgroup of 4 wave64 (2 x 2 waves, each a T/2 x T/2 quarter of the tile:
// (T/64)^2 MFMA blocks of 32 x 32, one wave per SIMD).  The 256 tile carries
// 256 float32 accumulators per lane; the 128 tile serves launches whose big
// tiles would not fill the compute units (a 1024-token prompt), which it
// fills with whole tiles instead of K-split ones.  The contraction runs on
// v_mfma_f32_32x32x16 (measured here: about 34 cycles for its 32768 flop with
// four independent accumulators, against about 27 for the 16384 of a
// 16x16x32 even with sixteen) with the base weight as the A operand (rows =
// output columns) and x as the B operand, so each group of four accumulators
// holds four consecutive columns of one row of y (8-byte stores).
//
// The base weight is taken transposed, W^T [h_out, h_in] (row n = column n of
// W, the layout of a linear layer's weight), so that both operands run along
// K in memory: every 16-byte chunk of 8 consecutive K is one MFMA operand
// slice, with no transpose.
//
// Pipeline: K advances in stages of 64 KiB, the x and W slices of the tile:
// 64 of K for T = 256 (a row's slice is one whole 128-byte line), 128 for
// T = 128 (two lines).  Consecutive lanes load consecutive 16-byte chunks of
// one row slice, a wave whole rows per instruction.  (Loads of 32 bytes per
// row from 32 rows, in the operand's own order, measured about 9 bytes per
// cycle per CU and bounded the kernel.)  Each stage is loaded into registers
// two steps ahead and written, one step ahead, to the other of two 64 KiB LDS
// buffers in the order the MFMA operands are read: per 32-row block and K-16
// slice a 1 KiB region holding chunk c of row r at 32 (c % 2) + r % 32 with
// the bits 0..3 of the row flipped by 2 (c % 8) + c / 8, so the 64 lanes of an
// operand read one contiguous KiB, free of bank conflicts, and the 16 chunks
// a quarter wave writes fall in 16 different bank groups.  Rows past the
// batch, columns past h_out and K past h_in are loads out of the buffer's
// range, which read zeros.
//
// Epilogue: for every run of the tile's rows that share an adapter (at most
// a few for prompt segments), B_g's ranks are staged in LDS 64 at a time,
// transposed so that 8 consecutive ranks of one output column form an
// operand slice, with the tile's rows of v for the same ranks in the other
// stage buffer (all loads of a rank range issued before its LDS writes), and
// each wave adds s_g v . B_g for its rows into its base
// accumulators: s_g v is split into a high and a low 16-bit part that share
// one 32x32x16 MFMA (its 16 K slots hold 8 ranks twice), rows of other runs
// masked to zero.  binary16 cannot hold a high part past 65504, so for it each
// wave first takes the largest |s_g v| it will use and, past 2^15, scales v
// and its accumulators by a power of two around those MFMAs and back after
// (exact).  The sum is rounded once to the storage dtype.
//
// Tiles go to XCDs in blocks: workgroup p runs on XCD p % n_xcd and takes the
// (p / n_xcd)-th tile of that XCD's contiguous share of the tile order.  The
// order runs over panels of kBasePanel row tiles, column by column inside a
// panel, so that an XCD's share, and the part of it that runs at a time, is a
// block of tiles a few row tiles high and a few column tiles wide: they share
// rows of x and columns of W in the XCD's L2 (a 1024-token prompt in tiles of
// 128: each XCD all 8 row tiles x 4 column tiles, 12 MiB of x and W, where
// one row tile x all 32 column tiles would be 33 MiB).  Every XCD gets
// per_xcd workgroups (the whole tiles over n_xcd, rounded up); those past the
// last tile end at once.
//
// A last round of tiles that would leave compute units idle is split along
// K: each of its tiles runs as `split` workgroups over consecutive K ranges,
// which store their float32 partial tiles (in accumulator order, the first
// range with the adapter delta added) to the workspace; the reduction kernel
// adds a tile's ranges in order 0, 1, ..., rounds once and stores y, so the
// result does not depend on timing.
#include <hip/hip_runtime.h>
#include <stddef.h>

#include "lora_device.h"
#include "lora_internal.h"

namespace lora {

namespace {

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kStageChunks = kBaseStageBytes / 16;     // 4096 chunks of 16 bytes
constexpr int kRegionChunks = 64;                      // one operand fragment: 32 rows x 2 chunks (K 16)
static_assert(kBaseThreads == 256, "base tiling: 2 x 2 waves");

// Derived tiling of tile edge T.
template <int T>
struct BaseCfg {
    static constexpr int kBK = base_bk(T);                   // K per stage
    static constexpr int kKQ = kBK / 16;                     // K-16 slices per stage
    static constexpr int kWB = T / 64;                       // 32 x 32 blocks per wave and dimension
    static constexpr int kWRegion = kKQ * (T / 32);          // first region of the W slice in a stage
    static constexpr int kRowChunks = kBK / 8;               // 16-byte chunks per row of a stage
    static constexpr int kRowStep = kBaseThreads / kRowChunks;   // rows between a thread's staged chunks
    static constexpr int kLoads = T / kRowStep;              // chunks of x (and of W) a thread stages
    static constexpr int kTileQuads = T * T / 4;
    // K-16 slices whose fragments are read ahead of the MFMAs: the small
    // tile's 4 MFMAs per slice do not cover one LDS read's latency
    static constexpr int kAhead = T == 256 ? 1 : 2;
    static_assert(kLoads == 8 && kKQ % 4 == 0 && kRowStep % 16 == 0, "staging");
    static_assert(kWRegion * 2 * kRegionChunks == kStageChunks, "a stage fills its buffer");
    static_assert(kBaseLoraRanks * T * 2 <= kBaseStageBytes, "B_g staging fits one stage buffer");
};

// s_waitcnt lgkmcnt(0), vmcnt and expcnt left free (gfx9 encoding).
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// s_waitcnt with lgkmcnt(0) and vmcnt(0).
__device__ __forceinline__ void wait_vm0_lgkm0() { __builtin_amdgcn_s_waitcnt(0x0070); }

// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int kSchedMfma = 0x008, kSchedVmemRead = 0x020, kSchedDsRead = 0x100, kSchedDsWrite = 0x200;

// v_mfma_f32_32x32x16: A [32 x 16] lane l holds A[l % 32][8 (l / 32) .. +7];
// B [16 x 32] lane l holds B[8 (l / 32) .. +7][l % 32]; accumulator r of
// lane l is D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
template <class Fmt>
__device__ __forceinline__ f32x16 mma32x32(const u32x4& a, const u32x4& b, f32x16 c);
template <>
__device__ __forceinline__ f32x16 mma32x32<FmtF16>(const u32x4& a, const u32x4& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                  0, 0, 0);
}
template <>
__device__ __forceinline__ f32x16 mma32x32<FmtBF16>(const u32x4& a, const u32x4& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   c, 0, 0, 0);
}

// Row tile mt and column tile nt of tile index `tile` in the panel order.
__device__ __forceinline__ void tile_coords(const BaseArgs& a, int tile, int& mt, int& nt) {
    const int per_panel = kBasePanel * a.n_nt;
    const int panel = tile / per_panel;
    const int h = min_i(kBasePanel, a.n_mt - panel * kBasePanel);   // row tiles of this panel
    const int u = tile - panel * per_panel;
    nt = u / h;
    mt = panel * kBasePanel + (u - nt * h);
}

// Bits 0..3 of a staged row's place in its region are flipped by swz(c) for
// chunk c of the row.
__device__ __forceinline__ int swz(int c) { return 2 * (c & 7) + (c >> 3); }

template <class Fmt, int TILE>
struct BaseTile {
    using C = BaseCfg<TILE>;
    static constexpr int WB = C::kWB;
    const BaseArgs& a;
    const int t, w, l, wm, wn;
    const int m0, n0;
    rsrc_t xr, wr;
    // this thread stages chunk c = t % kRowChunks of rows r0 + kRowStep i
    // (i < 8) of x and of W
    int c;
    uint32_t xo[C::kLoads], wo[C::kLoads];   // byte offsets at K = 0; kOut for rows past the matrix
    int lpos;                                // LDS chunk of row r0 (region, swizzled lane)
    u32x4 st[2][C::kLoads][2];               // the next two stages, in flight: [stage parity][i][x, W]
    f32x16 acc[WB][WB];                      // [32-row block of x][32-column block of y]

    __device__ __forceinline__ BaseTile(const BaseArgs& args, int mt, int nt)
        : a(args), t(threadIdx.x), w(threadIdx.x >> 6), l(threadIdx.x & 63), wm((threadIdx.x >> 6) >> 1),
          wn((threadIdx.x >> 6) & 1), m0(mt * TILE), n0(nt * TILE) {
        xr = make_rsrc(a.x, a.x_bytes);
        wr = make_rsrc(a.wt, a.w_bytes);
        const int r0 = t / C::kRowChunks;
        c = t % C::kRowChunks;
#pragma unroll
        for (int i = 0; i < C::kLoads; ++i) {
            const int row = m0 + r0 + C::kRowStep * i, col = n0 + r0 + C::kRowStep * i;
            xo[i] = row < a.M ? (uint32_t)(((int64_t)row * a.ldx) * 2) + 16u * c : (uint32_t)kOut;
            wo[i] = col < a.N ? (uint32_t)(((int64_t)col * a.ldw) * 2) + 16u * c : (uint32_t)kOut;
        }
        // chunk c of row r goes to region (r / 32, c / 2) at 32 (c % 2) + r % 32
        // with bits 0..3 flipped by swz(c); row r0 + kRowStep i is kRowStep i
        // rows further (swz leaves bit 4 alone)
        lpos = (c >> 1) * kRegionChunks + ((32 * (c & 1) + r0) ^ swz(c));
#pragma unroll
        for (int i = 0; i < WB; ++i)
#pragma unroll
            for (int j = 0; j < WB; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    }

    // Chunks [I0, I1) of stage k of x (part 0) or W (part 1) into staging
    // set S: consecutive lanes read consecutive 16-byte chunks of one row
    // slice, a wave whole rows per instruction.  Stages past K read zeros.
    template <int S, int part, int I0 = 0, int I1 = C::kLoads>
    __device__ __forceinline__ void load(int k) {
        // one select per stage: K past the end moves every offset past the
        // buffer (offsets and kOut stay below 2^32 together, above its size)
        const uint32_t kb = k * C::kBK + 8 * c < a.K ? (uint32_t)k * (C::kBK * 2) : (uint32_t)kOut;
#pragma unroll
        for (int i = I0; i < I1; ++i) st[S][i][part] = bload16(part ? wr : xr, (int)((part ? wo[i] : xo[i]) + kb));
    }

    // Staged chunks [I0, I1) of part 0 (x) or 1 (W) into buf in the operand
    // order.  The 16 chunks a quarter wave writes fall in 16 different bank
    // groups; a reader's 16 consecutive lanes share c and stay in one aligned
    // group of 16 chunks.
    template <int S, int part, int I0 = 0, int I1 = C::kLoads>
    __device__ __forceinline__ void commit(u32x4* buf) {
#pragma unroll
        for (int i = I0; i < I1; ++i) {
            constexpr int kRegionRow = C::kKQ * kRegionChunks;   // chunks between 32-row blocks
            const int rr = C::kRowStep * i;
            buf[(part ? C::kWRegion : 0) * kRegionChunks + (rr / 32) * kRegionRow + rr % 32 + lpos] = st[S][i][part];
        }
    }

    // Operand fragments of K-16 slice q: W blocks WB wn + j into f[j], x
    // blocks WB wm + i into f[WB + i].
    __device__ __forceinline__ void frags(const u32x4* buf, int q, u32x4* f) {
        // lane l reads chunk 2q + l / 32 of row l % 32 of its blocks
        const int ls = l ^ (4 * (q & 3) + 2 * (l >> 5) + (q >> 2));
#pragma unroll
        for (int j = 0; j < WB; ++j) f[j] = buf[(C::kWRegion + C::kKQ * (WB * wn + j) + q) * kRegionChunks + ls];
#pragma unroll
        for (int i = 0; i < WB; ++i) f[WB + i] = buf[(C::kKQ * (WB * wm + i) + q) * kRegionChunks + ls];
    }

    __device__ __forceinline__ void mfmas(const u32x4* f) {
#pragma unroll
        for (int i = 0; i < WB; ++i)
#pragma unroll
            for (int j = 0; j < WB; ++j) acc[i][j] = mma32x32<Fmt>(f[j], f[WB + i], acc[i][j]);
    }

    // Slice s of step k: the fragment reads of slice s + kAhead, this
    // slice's share of the step's memory work, the slice's MFMAs.  The memory work is
    // in four parts, each over a quarter of the slices: the writes of stage
    // k + 1's x, then of its W (loaded during step k - 1) into nxt, whose
    // readers have passed the barrier, then the loads of stage k + 3's x,
    // then of its W.
    static constexpr int NF = C::kAhead + 1;       // fragment sets in registers
    template <int P, int s>
    __device__ __forceinline__ void slices(const u32x4* cur, u32x4* nxt, int k, u32x4 (&f)[NF][2 * WB]) {
        constexpr int NQ = C::kKQ / 4;
        constexpr int kind = s / NQ;
        constexpr int NO = C::kLoads / NQ;         // memory instructions of the slice
        constexpr int I0 = (s % NQ) * NO;
        constexpr bool reads = s + C::kAhead < C::kKQ;
        constexpr int NM = WB * WB / NO;           // MFMAs per memory instruction
        if constexpr (reads) frags(cur, s + C::kAhead, f[(s + C::kAhead) % NF]);
        if constexpr (kind == 0) commit<P ^ 1, 0, I0, I0 + NO>(nxt);
        else if constexpr (kind == 1) commit<P ^ 1, 1, I0, I0 + NO>(nxt);
        else if constexpr (kind == 2) load<P ^ 1, 0, I0, I0 + NO>(k + 3);
        else load<P ^ 1, 1, I0, I0 + NO>(k + 3);
        mfmas(f[s % NF]);
        constexpr int op = kind < 2 ? kSchedDsWrite : kSchedVmemRead;
        static_assert(NM >= 1 && (!reads || 2 * WB == NO), "slice schedule");
#pragma unroll
        for (int g = 0; g < NO; ++g) {
            if constexpr (reads) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
                if constexpr (NM > 1) __builtin_amdgcn_sched_group_barrier(kSchedMfma, NM - 1, 0);
            } else {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, NM, 0);
            }
            __builtin_amdgcn_sched_group_barrier(op, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (s + 1 < C::kKQ) slices<P, s + 1>(cur, nxt, k, f);
    }

    // Step k on buffer cur (stage k, written in step k-1).  Every wave's
    // writes of stage k and reads of stage k-1 are done at the barrier; then
    // the MFMAs run with, in their shadow, the fragment reads of the K slices
    // ahead and the step's memory work.
    template <int P>
    __device__ __forceinline__ void step(const u32x4* cur, u32x4* nxt, int k) {
        wait_lgkm0();
        __builtin_amdgcn_s_barrier();
        u32x4 f[NF][2 * WB];
#pragma unroll
        for (int q = 0; q < C::kAhead; ++q) frags(cur, q, f[q]);
        __builtin_amdgcn_sched_barrier(0);
        slices<P, 0>(cur, nxt, k, f);
    }
};

// The adapter delta of one run of rows [lo, hi) with adapter g, ranks staged
// 64 at a time: B_g's in bt, v's in vt (the two stage buffers).  Every load
// of a rank range is issued before any of its LDS writes, so that the range
// costs one round trip to memory, not one per loop turn.
template <class Fmt, int TILE>
__device__ __forceinline__ void tile_delta(BaseTile<Fmt, TILE>& T, const BasePiece& pc, u32x4* bt, u32x4* vt) {
    constexpr int WB = BaseTile<Fmt, TILE>::WB;
    constexpr int kBTasks = kBaseLoraRanks * (TILE / 8) / kBaseThreads;   // B_g loads per thread (64 ranks)
    constexpr int kVTasks = TILE * (kBaseLoraRanks / 4) / kBaseThreads;    // v loads per thread
    const BaseArgs& a = T.a;
    const DevAdapter ad = a.table[pc.adapter];
    const int R = ad.rank;
    const rsrc_t br = make_rsrc(ad.B, (uint32_t)R * (uint32_t)a.N * 2u);
    const rsrc_t vr = make_rsrc(a.v, a.v_bytes);
    const int l = T.l;
    for (int rc0 = 0; rc0 < R; rc0 += kBaseLoraRanks) {
        const int rr = min_i(kBaseLoraRanks, R - rc0);
        const int RC = (rr + 7) / 8;              // 8-rank chunks (one MFMA each)
        // B_g ranks [rc0, rc0 + 8 RC) of the tile's columns into bt: column n
        // of 32-column block nb, chunk c (ranks rc0 + 8c .. +7) at
        // nb * 32 RC + 32 c + (n % 32).  A thread loads 8 columns of one rank
        // (16 bytes) and writes each element to its place (2-byte LDS writes).
        // (the big tile, short of registers beside its accumulators, stages
        // B_g and v in two halves each: a half's loads after the previous
        // half's writes.  Binary16 in the big tile, whose range check keeps
        // more registers, stages B_g one load at a time and reads v from
        // memory per fragment: staged in bulk, it spills.)
        constexpr bool kLean = Fmt::kNarrowRange && TILE == kBaseBig;
        constexpr int kHalves = kLean ? kBTasks : (TILE == kBaseBig ? 2 : 1);
        constexpr bool kVLds = !kLean;
        constexpr int kBLoads = kBTasks / kHalves;
        u32x4 b8[kBLoads];
        auto bfetch = [&](int h) __attribute__((always_inline)) {
#pragma unroll
            for (int it = 0; it < kBLoads; ++it) {
                const int task = T.t + (h * kBLoads + it) * kBaseThreads;
                const int jr = task / (TILE / 8);     // rank within the staged range
                const int j = rc0 + jr;
                const int col = T.n0 + 8 * (task - jr * (TILE / 8));
                b8[it] = bload16(br, jr < 8 * RC && j < R && col < a.N ? (int)((((int64_t)j * a.N) + col) * 2) : kOut);
            }
        };
        uint16_t* bt16 = (uint16_t*)bt;
        auto bstore = [&](int h) __attribute__((always_inline)) {
#pragma unroll
            for (int it = 0; it < kBLoads; ++it) {
                const int task = T.t + (h * kBLoads + it) * kBaseThreads;
                const int jr = task / (TILE / 8);
                const int co = task - jr * (TILE / 8);
                if (jr < 8 * RC) {
#pragma unroll
                    for (int c = 0; c < 8; ++c) {
                        const int n = 8 * co + c;
                        const uint32_t word = b8[it][c >> 1];
                        bt16[((n >> 5) * (32 * RC) + 32 * (jr >> 3) + (n & 31)) * 8 + (jr & 7)] =
                            (uint16_t)((c & 1) ? hi16(word) : lo16(word));
                    }
                }
            }
        };
        // v of the tile's rows for ranks [rc0, rc0 + 64) into vt: float4 q
        // (ranks rc0 + 4q .. +3) of tile row r at 16 r + (q ^ (r % 16)), so
        // that 16 lanes reading one chunk of 16 rows hit 16 bank groups.
        // Rows outside [lo, hi) and ranks >= R are zeros.
        constexpr int kVLoads = kVTasks / kHalves;
        f32x4 vv[kVLoads];
        auto vfetch = [&](int h) __attribute__((always_inline)) {
#pragma unroll
            for (int it = 0; it < kVLoads; ++it) {
                const int e = T.t + (h * kVLoads + it) * kBaseThreads;
                const int m = T.m0 + (e >> 4);
                const int j = rc0 + 4 * (e & 15);
                const bool ok = m >= pc.lo && m < pc.hi && j < R;
                vv[it] = as_f4(bload16(vr, ok ? (int)((((int64_t)m * a.ldv) + j) * 4) : kOut));
            }
        };
        f32x4* vt4 = (f32x4*)vt;
        auto vstore = [&](int h) __attribute__((always_inline)) {
#pragma unroll
            for (int it = 0; it < kVLoads; ++it) {
                const int e = T.t + (h * kVLoads + it) * kBaseThreads;
                const int r = e >> 4, q = e & 15;
                f32x4 v = vv[it];
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (rc0 + 4 * q + k >= R) v[k] = 0.f;
                vt4[16 * r + (q ^ (r & 15))] = v;
            }
        };
        bfetch(0);
        if constexpr (kVLds) vfetch(0);
        __builtin_amdgcn_s_barrier();             // earlier readers of bt and vt are done (every wave waited lgkmcnt)
        bstore(0);
        if constexpr (kVLds) vstore(0);
#pragma unroll 1
        for (int h = 1; h < kHalves; ++h) {
            bfetch(h);
            if constexpr (kVLds) vfetch(h);
            bstore(h);
            if constexpr (kVLds) vstore(h);
        }
        __syncthreads();
        // v operand of block i, chunk c: lane l takes row TILE/2 wm + 32 i + (l % 32)
        // of the tile, ranks rc0 + 8 c .. +7, the high part of s_g v for l < 32
        // and the low part for l >= 32 (the B_g operand holds the same ranks in
        // both halves of K).
        auto vload = [&](int i, int c, f32x4& v0, f32x4& v1) __attribute__((always_inline)) {
            const int r = (TILE / 2) * T.wm + 32 * i + (l & 31);
            if constexpr (kVLds) {
                v0 = vt4[16 * r + ((2 * c) ^ (r & 15))];
                v1 = vt4[16 * r + ((2 * c + 1) ^ (r & 15))];
            } else {
                const int m = T.m0 + r;
                const int j = rc0 + 8 * c;
                const bool ok = m >= pc.lo && m < pc.hi && j < R;
                const int off = ok ? (int)((((int64_t)m * a.ldv) + j) * 4) : kOut;
                v0 = as_f4(bload16(vr, off));
                v1 = as_f4(bload16(vr, off + 16));
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (j + e >= R) v0[e] = 0.f;
                    if (j + 4 + e >= R) v1[e] = 0.f;
                }
            }
        };
        // v enters the MFMA pre-multiplied by s_g, so the delta adds straight
        // into the base accumulators.  binary16: past 2^15 the wave scales v
        // by 2^k (k < 0) and its accumulators by 2^k around these MFMAs, then
        // back by 2^-k; powers of two, exact for every accumulator at or above
        // 2^-126+|k| (far below the output's precision).
        float vmul = ad.scale;
        float unscale = 1.f;
        if constexpr (Fmt::kNarrowRange) {
            float vabs = 0.f;
            for (int i = 0; i < WB; ++i)
                for (int c = 0; c < RC; ++c) {
                    f32x4 v0, v1;
                    vload(i, c, v0, v1);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        vabs = fmaxf(vabs, fmaxf(fabsf(v0[e] * ad.scale), fabsf(v1[e] * ad.scale)));
                }
#pragma unroll
            for (int d = 32; d >= 1; d >>= 1) vabs = fmaxf(vabs, __shfl_xor(vabs, d, 64));
            if (vabs >= 32768.f) {
                const int E = (int)((__float_as_uint(vabs) >> 23) & 0xff) - 127;
                const int k = max_i(14 - E, -64);
                const float down = __uint_as_float((uint32_t)(127 + k) << 23);
                vmul = ad.scale * down;
                unscale = __uint_as_float((uint32_t)(127 - k) << 23);
#pragma unroll
                for (int i = 0; i < WB; ++i)
#pragma unroll
                    for (int jn = 0; jn < WB; ++jn) T.acc[i][jn] *= down;
            }
        }
        const bool hi_half = l < 32;
        for (int c = 0; c < RC; ++c) {
            u32x4 bf[WB];
#pragma unroll
            for (int jn = 0; jn < WB; ++jn) bf[jn] = bt[(WB * T.wn + jn) * (32 * RC) + 32 * c + (l & 31)];
#pragma unroll
            for (int i = 0; i < WB; ++i) {
                f32x4 v0, v1;
                vload(i, c, v0, v1);
                v0 *= vmul;
                v1 *= vmul;
                const uint32_t h0 = Fmt::pack2(v0[0], v0[1]), h1 = Fmt::pack2(v0[2], v0[3]);
                const uint32_t h2 = Fmt::pack2(v1[0], v1[1]), h3 = Fmt::pack2(v1[2], v1[3]);
                u32x4 vf;
                if (hi_half) {
                    vf = u32x4{h0, h1, h2, h3};
                } else {
                    vf = u32x4{Fmt::pack2(v0[0] - Fmt::to_f32(lo16(h0)), v0[1] - Fmt::to_f32(hi16(h0))),
                               Fmt::pack2(v0[2] - Fmt::to_f32(lo16(h1)), v0[3] - Fmt::to_f32(hi16(h1))),
                               Fmt::pack2(v1[0] - Fmt::to_f32(lo16(h2)), v1[1] - Fmt::to_f32(hi16(h2))),
                               Fmt::pack2(v1[2] - Fmt::to_f32(lo16(h3)), v1[3] - Fmt::to_f32(hi16(h3)))};
                }
#pragma unroll
                for (int jn = 0; jn < WB; ++jn) T.acc[i][jn] = mma32x32<Fmt>(bf[jn], vf, T.acc[i][jn]);
            }
        }
        if constexpr (Fmt::kNarrowRange) {
            if (unscale != 1.f) {
#pragma unroll
                for (int i = 0; i < WB; ++i)
#pragma unroll
                    for (int jn = 0; jn < WB; ++jn) T.acc[i][jn] *= unscale;
            }
        }
        wait_vm0_lgkm0();                         // this wave's reads of bt are done before the next staging
    }
}

template <class Fmt, int TILE>
__global__ void __launch_bounds__(kBaseThreads, 1) lora_base_kernel(BaseArgs a) {
    using C = BaseCfg<TILE>;
    constexpr int WB = C::kWB;
    __shared__ __attribute__((aligned(16))) u32x4 s0[kStageChunks];
    __shared__ __attribute__((aligned(16))) u32x4 s1[kStageChunks];
    // an even number of stages (a stage past K reads zeros and adds nothing),
    // so that the loop runs whole pairs of steps and has one exit
    const int nk = ((a.K + 2 * C::kBK - 1) / (2 * C::kBK)) * 2;
    const int p = blockIdx.x;
    const int slots = a.n_xcd * a.per_xcd;   // workgroups of the whole tiles, per_xcd for every XCD
    int tile, k0 = 0, k1 = nk, range = -1;
    if (p < slots) {
        const int q = p / a.n_xcd;
        tile = (p - q * a.n_xcd) * a.per_xcd + q;
        if (tile >= a.n_whole) return;
    } else {
        const int u = p - slots;
        tile = a.n_whole + u / a.split;
        range = u - (tile - a.n_whole) * a.split;
        k0 = range * a.chunk;
        k1 = min_i(nk, k0 + a.chunk);
        if (tile >= a.n_mt * a.n_nt || k0 >= k1) return;
    }
    int mt, nt;
    tile_coords(a, tile, mt, nt);
    BaseTile<Fmt, TILE> T(a, mt, nt);

    T.template load<0, 0>(k0);
    T.template load<0, 1>(k0);
    T.template load<1, 0>(k0 + 1);
    T.template load<1, 1>(k0 + 1);
    T.template commit<0, 0>(s0);
    T.template commit<0, 1>(s0);
    T.template load<0, 0>(k0 + 2);
    T.template load<0, 1>(k0 + 2);
    for (int k = k0; k < k1; k += 2) {
        T.template step<0>(s0, s1, k);
        T.template step<1>(s1, s0, k + 1);
    }
    wait_vm0_lgkm0();

    // the adapter delta of each run of rows that carries one (once per tile)
    if (range <= 0) {
        const int pe = a.piece_off[mt + 1];
        for (int pi = a.piece_off[mt]; pi < pe; ++pi) {
            const BasePiece pc = a.pieces[pi];
            tile_delta<Fmt, TILE>(T, pc, s0, s1);
        }
    }

    if (range >= 0) {
        // partial tile in accumulator order: float4 g of block (i, j) of wave
        // w, lane l at (((w WB + i) WB + j) 4 + g) 64 + l
        float4* dst = (float4*)a.part + (size_t)((tile - a.n_whole) * a.split + range) * C::kTileQuads;
#pragma unroll
        for (int i = 0; i < WB; ++i)
#pragma unroll
            for (int j = 0; j < WB; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x16& c = T.acc[i][j];
                    dst[(((T.w * WB + i) * WB + j) * 4 + g) * 64 + T.l] =
                        float4{c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]};
                }
        return;
    }

    // y: accumulator r of block (i, j) is column n0 + TILE/2 wn + 32 j + 8 (r / 4)
    // + 4 (l / 32) + r % 4 of row m0 + TILE/2 wm + 32 i + l % 32: four
    // consecutive columns per group of four registers (8-byte stores)
    const rsrc_t yr = make_rsrc(a.y, a.y_bytes);
#pragma unroll
    for (int i = 0; i < WB; ++i) {
        const int m = T.m0 + (TILE / 2) * T.wm + 32 * i + (T.l & 31);
#pragma unroll
        for (int j = 0; j < WB; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = T.n0 + (TILE / 2) * T.wn + 32 * j + 8 * g + 4 * (T.l >> 5);
                const bool ok = m < a.M && n < a.N;
                const f32x16& c = T.acc[i][j];
                bstore8(u32x2{Fmt::pack2(c[4 * g], c[4 * g + 1]), Fmt::pack2(c[4 * g + 2], c[4 * g + 3])}, yr,
                        ok ? (int)((((int64_t)m * a.ldy) + n) * 2) : kOut);
            }
    }
}

// The split tiles: the float32 partials of ranges 0 .. split-1 added in that
// order, rounded once and stored.  One thread per four consecutive columns of
// one row (one float4 of every partial).
constexpr int kReduceThreads = 256;

template <class Fmt, int TILE>
__global__ void __launch_bounds__(kReduceThreads) lora_base_reduce_kernel(BaseArgs a) {
    using C = BaseCfg<TILE>;
    constexpr int WB = C::kWB;
    static_assert(C::kTileQuads % kReduceThreads == 0, "reduce grid");
    const int gid = blockIdx.x * kReduceThreads + threadIdx.x;
    const int rt = gid / C::kTileQuads;
    const int e = gid - rt * C::kTileQuads;
    const int l = e & 63, g = (e >> 6) & 3, blk = e >> 8;
    const int j = blk % WB, i = (blk / WB) % WB, w = blk / (WB * WB);
    const int tile = a.n_whole + rt;
    if (tile >= a.n_mt * a.n_nt) return;
    int mt, nt;
    tile_coords(a, tile, mt, nt);
    const int m = mt * TILE + (TILE / 2) * (w >> 1) + 32 * i + (l & 31);
    const int n = nt * TILE + (TILE / 2) * (w & 1) + 32 * j + 8 * g + 4 * (l >> 5);
    const float4* src = (const float4*)a.part + (size_t)rt * a.split * C::kTileQuads + e;
    float4 sum = src[0];
    for (int r = 1; r < a.split; ++r) {
        const float4 v = src[(size_t)r * C::kTileQuads];
        sum.x += v.x;
        sum.y += v.y;
        sum.z += v.z;
        sum.w += v.w;
    }
    if (m < a.M && n < a.N) {
        const rsrc_t yr = make_rsrc(a.y, a.y_bytes);
        bstore8(u32x2{Fmt::pack2(sum.x, sum.y), Fmt::pack2(sum.z, sum.w)}, yr, (int)((((int64_t)m * a.ldy) + n) * 2));
    }
}

template <class Fmt, int TILE>
hipError_t launch_tiles(const BaseArgs& a, hipStream_t s) {
    const int n_split = a.split > 1 ? a.n_mt * a.n_nt - a.n_whole : 0;
    const int grid = a.n_xcd * a.per_xcd + n_split * a.split;
    if (grid <= 0) return hipSuccess;
    hipLaunchKernelGGL((lora_base_kernel<Fmt, TILE>), dim3(grid), dim3(kBaseThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n_split == 0) return e;
    const int rgrid = n_split * (BaseCfg<TILE>::kTileQuads / kReduceThreads);
    hipLaunchKernelGGL((lora_base_reduce_kernel<Fmt, TILE>), dim3(rgrid), dim3(kReduceThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_base(const BaseArgs& a, int dtype, hipStream_t s) {
    if (a.tile == kBaseBig)
        return dtype == 0 ? launch_tiles<FmtF16, kBaseBig>(a, s) : launch_tiles<FmtBF16, kBaseBig>(a, s);
    if (a.tile == kBaseSmall)
        return dtype == 0 ? launch_tiles<FmtF16, kBaseSmall>(a, s) : launch_tiles<FmtBF16, kBaseSmall>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace lora
