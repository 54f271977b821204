// gfx950 kernels of the batched, heterogeneous-rank LoRA delta
//   y[t,:] <- round(y[t,:] + s_g * (x[t,:] . A_g) . B_g)          (Eq. 1)
//
// Shrink: one workgroup per (row block of an adapter group, K range of A_g).
// A's rows k0..k0+len are one contiguous run of bytes, read once per step
// with 16-byte loads however many tokens use the adapter: tokens are gathered
// to their adapter instead of each token re-reading it (Section 4.1's gather,
// done once per distinct adapter).  The range is staged in passes: A goes to
// LDS transposed into words that hold two consecutive K elements of one rank,
// the row block's x columns go to LDS as they are, and the next pass's loads
// are in flight while the current pass runs on v_mfma_f32_16x16x32
// (v^T[r, t] = sum_k A[k, r] x[t, k], 16 ranks x 16 rows x 32 K per
// instruction, float32 accumulation).  When a rank has fewer tiles than waves,
// the waves split K and add their sums through LDS in wave order.  The
// workgroup writes its float32 partial block.
//
// Expand: one workgroup per (row block, column tile of B_g).  It adds the row
// block's partial blocks in a fixed order (v stays float32 up to here),
// splits each v into a high and a low 16-bit part so that v is never rounded
// to one 16-bit value, stages the B tile in LDS transposed into rank pairs and
// runs y^T[n, t] = sum_j B[j, n] v[t, j] on v_mfma_f32_16x16x16 (two
// instructions per step: high and low part).  Each lane then holds four
// consecutive columns of one row of y; y + s*d is rounded once to the storage
// dtype and written with 8-byte stores.  The B tile, the y values and the
// partial blocks are all requested before the first barrier.
//
// Rank is a runtime value: any rank in [1, 256] runs the same code (padded to
// a multiple of 16 inside LDS and registers only), so items of different
// ranks share one grid; the bodies are compiled for the number of rank tiles
// (or column tiles) per wave and of 16-row subtiles, so the MFMA loops have no
// branches.
//
// Step launch: one grid holds every shrink item, then every expand item.  Its
// partial blocks live in two buffers of their own, used by alternate
// launches; the one a launch reads holds a sentinel bit pattern until it is
// written.  A shrink workgroup writes its block with device-coherent stores
// (the L2 caches of the XCDs are not coherent with each other; these stores
// write through to the common level instead of flushing a cache) and arms its
// block in the other buffer for the next launch.  An expand workgroup requests its B tile and its y values, stages
// B^T, then loads the partial values it needs with device-coherent loads and
// loads again those that still hold the sentinel: the data is its own ready
// flag, so no counter or fence sits between a shrink and the expands that use
// it.  A workgroup only waits for workgroups earlier in the grid, which do not
// wait, so every wait ends; the number of rounds is bounded all the same (past
// it the wait gives up and sets the status flag).  The in the same fixed order as in the two-launch form, so both
// give bit-identical results whatever the timing.
#include <hip/hip_runtime.h>
#include <stddef.h>

#include "lora_internal.h"

namespace lora {

typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
// Native vectors (not HIP's struct vector types): selects stay in registers.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
// Adapter factors are reached through pointers read at run time; they are
// global memory, said explicitly so that the loads are global, not flat.
typedef __attribute__((address_space(1))) const uint16_t gu16;
typedef __attribute__((address_space(1))) const u32x4 gu32x4;

// ---------------------------------------------------------------------------
// 16-bit storage formats and their MFMA instructions
// ---------------------------------------------------------------------------
struct FmtF16 {
    static __device__ __forceinline__ float to_f32(uint32_t b16) {
        return (float)__builtin_bit_cast(_Float16, (uint16_t)b16);
    }
    static __device__ __forceinline__ uint32_t from_f32(float f) {
        return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
    }
    static __device__ __forceinline__ f32x4 mma32(const u32x4& a, const u32x4& b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    }
    static __device__ __forceinline__ f32x4 mma16(const u32x2& a, const u32x2& b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, a),
                                                     __builtin_bit_cast(f16x4, b), c, 0, 0, 0);
    }
};
struct FmtBF16 {
    static __device__ __forceinline__ float to_f32(uint32_t b16) { return __uint_as_float(b16 << 16); }
    static __device__ __forceinline__ uint32_t from_f32(float f) {
        return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
    }
    static __device__ __forceinline__ f32x4 mma32(const u32x4& a, const u32x4& b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
    static __device__ __forceinline__ f32x4 mma16(const u32x2& a, const u32x2& b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a),
                                                         __builtin_bit_cast(i16x4, b), c, 0, 0, 0);
    }
};

// The work item, field by field in scalar registers (the whole struct is
// never copied as one aggregate, which would send it to scratch memory).
struct Item {
    int64_t part;
    int kind, group, adapter, rank, nrows, lo, len, sub, nsplit, p0, pstride, rb, nexp, row0;
    int rows[kInlineRows];
    const void* fac;     // the factor this item streams: A_g (shrink) or B_g (expand)
    float scale;         // s_g
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
    it.kind = (int)w0[2];
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
    return it;
}

__device__ __forceinline__ uint32_t lo16(uint32_t w) { return w & 0xffffu; }
__device__ __forceinline__ uint32_t hi16(uint32_t w) { return w >> 16; }

// Where the factor pointers and scales of a launch's groups are read.
enum : int {
    kLookupAuto = 0,     // the argument table for groups below kKargGroups, else the registry
    kLookupArgs = 1,     // the argument table only (the launch has at most kKargGroups groups)
    kLookupReg = 2,      // the device registry only
};

// The factor this item streams and the group's scale.  The step kernel fixes
// the source at compile time: a pointer that could point into either the
// kernel arguments or the registry makes the compiler copy the arguments to
// private memory.
template <int kLookup>
__device__ __forceinline__ gu16* item_factor(const KernelArgs& a, const Item& it, bool shrink) {
    if (kLookup == kLookupArgs || (kLookup == kLookupAuto && it.group < kKargGroups))
        return (gu16*)a.gfac[2 * it.group + (shrink ? 0 : 1)];
    const DevAdapter* d = a.table + it.adapter;
    return (gu16*)(shrink ? d->A : d->B);
}
template <int kLookup>
__device__ __forceinline__ float item_scale(const KernelArgs& a, const Item& it) {
    if (kLookup == kLookupArgs || (kLookup == kLookupAuto && it.group < kKargGroups))
        return a.gscale[it.group];
    return a.table[it.adapter].scale;
}
template <int kLookup>
__device__ __forceinline__ void resolve(const KernelArgs& a, Item& it) {
    it.fac = (const void*)item_factor<kLookup>(a, it, it.kind == kItemShrink);
    it.scale = item_scale<kLookup>(a, it);
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
__device__ __forceinline__ LaneTable load_lane_table(const KernelArgs& a) {
    const int l = threadIdx.x & 63;
    const uint64_t* g = reinterpret_cast<const uint64_t*>(a.gfac);
    LaneTable t;
#pragma unroll
    for (int i = 0; i < 4; ++i) t.f[i] = g[l + 64 * i];
#pragma unroll
    for (int i = 0; i < 2; ++i) t.s[i] = a.gscale[l + 64 * i];
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

// Partial-block stores and loads: plain, or device-coherent (agent scope) in
// the step launch, where producer and consumer may sit on different XCDs.
template <bool kSync>
__device__ __forceinline__ void put_f32(float* p, float v) {
    if constexpr (kSync) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else *p = v;
}
template <bool kSync>
__device__ __forceinline__ void put_f32x4(float* p, const f32x4& v) {   // p 16-byte aligned
    if constexpr (kSync) {
        const uint64_t lo = (uint64_t)__float_as_uint(v[0]) | ((uint64_t)__float_as_uint(v[1]) << 32);
        const uint64_t hi = (uint64_t)__float_as_uint(v[2]) | ((uint64_t)__float_as_uint(v[3]) << 32);
        __hip_atomic_store((uint64_t*)p, lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store((uint64_t*)p + 1, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
        *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
    }
}
template <bool kSync>
__device__ __forceinline__ float get_f32(const float* p) {
    if constexpr (kSync) return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else return *p;
}

// Step launch: between launches the partial blocks hold this bit pattern, a
// NaN whose low payload bits no 16-bit input can carry into a float32 sum.
constexpr uint32_t kSentinel = 0xffffffffu;
__device__ __forceinline__ bool unready(float v) { return __float_as_uint(v) == kSentinel; }

// Part q of the ordered sums of a row block's partial blocks at two positions
// (two consecutive ranks): blocks q, q+P, q+2P, ... added in that order,
// sixteen loads in flight.  In the step launch a value that still holds the
// sentinel has not been written yet and is loaded again; budget is the
// thread's remaining polling rounds (spin_limit for the whole item): once it
// is spent the status flag is raised and values are used as they are.
template <bool kSync>
__device__ __forceinline__ float2 part_sum2(const KernelArgs& a, const float* src0, const float* src1,
                                            int64_t pstride, int nsplit, int P, int q, bool ok0, bool ok1,
                                            int& budget) {
    float s0 = 0.f, s1 = 0.f;
    for (int c0 = q; c0 < nsplit; c0 += 8 * P) {
        float u[8], w[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int c = c0 + i * P;
            const int64_t off = (int64_t)c * pstride;
            u[i] = (ok0 && c < nsplit) ? get_f32<kSync>(src0 + off) : 0.f;
            w[i] = (ok1 && c < nsplit) ? get_f32<kSync>(src1 + off) : 0.f;
        }
        if constexpr (kSync) {
            for (;;) {
                bool miss = false;
#pragma unroll
                for (int i = 0; i < 8; ++i) miss |= unready(u[i]) | unready(w[i]);
                if (!miss || budget < 0) break;
                if (budget-- == 0) {
                    __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
#pragma unroll
                for (int i = 0; i < 8; ++i) {     // only positions that were loaded can hold the sentinel
                    const int64_t off = (int64_t)(c0 + i * P) * pstride;
                    if (unready(u[i])) u[i] = get_f32<true>(src0 + off);
                    if (unready(w[i])) w[i] = get_f32<true>(src1 + off);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) s0 += u[i];
#pragma unroll
        for (int i = 0; i < 8; ++i) s1 += w[i];
    }
    return make_float2(s0, s1);
}

// The same ordered sum at one position (the reduce kernel's).
__device__ __forceinline__ float part_sum(const float* src, int64_t pstride, int nsplit, int P, int q) {
    float s = 0.f;
    for (int c0 = q; c0 < nsplit; c0 += 8 * P) {
        float u[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int c = c0 + i * P;
            u[i] = c < nsplit ? src[(int64_t)c * pstride] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) s += u[i];
    }
    return s;
}

// Step launch: the row block's two partial buffers.  Launches alternate
// between them, the parity coming from the row block's counter of finished
// expand items (it wraps at 2 nexp): below nexp -> buffer 0, else buffer 1.
// Within one launch every reader sees the same parity: all shrink items of a
// row block start before any of its expand items can finish, and an expand
// item that reads late sees fewer than nexp increments of its own launch.
// Each shrink item arms (sets to the sentinel) its block in the buffer the
// next launch will use, which no item of this launch reads.
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
    const int R = it.rank;
    const int Rp = round_up_i(R, 16);
    const int NT = Rp / 16;
    const int sub = it.sub;                   // K staged per pass, multiple of 32
    const int KP = shrink_kp(sub);            // words per A^T row, 4 (mod 8): conflict-free 16-byte reads
    const int KX = shrink_kx(sub);            // halves per x row
    const int nrows = it.nrows;
    const int WN = shrink_wn(R);
    const int WK = 4 / WN;
    const int wn = w % WN;
    const int wk = w / WN;
    uint32_t* As = (uint32_t*)smem;                               // [Rp][KP] words
    uint16_t* Xs = (uint16_t*)(smem + (size_t)Rp * KP * 4);       // [MS*16][KX]
    gu16* A = (gu16*)it.fac + (int64_t)it.lo * R;
    const uint16_t* X = (const uint16_t*)a.x + it.lo;
    const int rowv = lane_rows(a, it);
    const u32x4 z4 = {0u, 0u, 0u, 0u};
    const bool vec = (R & 7) == 0;
    const int VPR = max_i(R / 8, 1);
    const int npairs = vec ? (sub / 2) * VPR : 0;
    const int kv = sub / 8;
    const int nx = nrows * kv;
    const int npass = (it.len + sub - 1) / sub;
    uint32_t parity = 0;                       // step launch: which partial buffer (read early, used last)
    if constexpr (kSync) parity = row_block_parity(a, it);

    // the padding ranks of A^T stay zero for every pass
    for (int i = t; i < (Rp - R) * KP; i += kThreads) As[R * KP + i] = 0u;

    u32x4 v0[4], v1[4], xv[4];
    auto load_pass = [&](int pass) {
        const int k0 = pass * sub;
        const int plen = min_i(sub, it.len - k0);
        const int lv = plen / 8;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = t + i * kThreads;
            const int k2 = p / VPR;
            const int k = 2 * k2;
            const int jo = p - k2 * VPR;
            const bool ok0 = p < npairs && k < plen;
            const bool ok1 = p < npairs && k + 1 < plen;
            // addresses stay inside A even where the load is masked off
            gu16* src0 = A + (int64_t)(ok0 ? k0 + k : 0) * R + (ok0 ? jo * 8 : 0);
            gu16* src1 = A + (int64_t)(ok1 ? k0 + k + 1 : 0) * R + (ok1 ? jo * 8 : 0);
            v0[i] = ok0 ? *(gu32x4*)src0 : z4;
            v1[i] = ok1 ? *(gu32x4*)src1 : z4;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = t + i * kThreads;
            const int r = p < nx ? p / kv : 0;
            const int c = p - r * kv;
            const int row = row_of(rowv, r);
            const bool ok = p < nx && c < lv;
            xv[i] = ok ? *(const u32x4*)(X + (int64_t)row * a.ldx + k0 + (ok ? c * 8 : 0)) : z4;
        }
    };
    auto store_x = [&]() {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = t + i * kThreads;
            if (p < nx) {
                const int r = p / kv;
                *(u32x4*)(Xs + r * KX + (p - r * kv) * 8) = xv[i];
            }
        }
    };
    auto store_a = [&]() {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = t + i * kThreads;
            if (p < npairs) {
                const int k2 = p / VPR;
                const int jo = p - k2 * VPR;
                uint32_t* d = As + (jo * 8) * KP + k2;
                d[0 * KP] = lo16(v0[i].x) | (v1[i].x << 16);
                d[1 * KP] = hi16(v0[i].x) | (v1[i].x & 0xffff0000u);
                d[2 * KP] = lo16(v0[i].y) | (v1[i].y << 16);
                d[3 * KP] = hi16(v0[i].y) | (v1[i].y & 0xffff0000u);
                d[4 * KP] = lo16(v0[i].z) | (v1[i].z << 16);
                d[5 * KP] = hi16(v0[i].z) | (v1[i].z & 0xffff0000u);
                d[6 * KP] = lo16(v0[i].w) | (v1[i].w << 16);
                d[7 * KP] = hi16(v0[i].w) | (v1[i].w & 0xffff0000u);
            }
        }
    };
    // ranks that are not a multiple of 8: A^T element by element (correct, not tuned)
    auto store_a_generic = [&](int pass) {
        const int k0 = pass * sub;
        const int plen = min_i(sub, it.len - k0);
        for (int i = t; i < R * KP; i += kThreads) As[i] = 0u;
        __syncthreads();
        uint16_t* As16 = (uint16_t*)As;
        gu16* src = A + (int64_t)k0 * R;
        for (int e = t; e < plen * R; e += kThreads) {
            const int k = e / R;
            const int j = e - k * R;
            As16[(j * KP) * 2 + k] = src[e];
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
        auto step_frags = [&](int s, u32x4 (&af)[TQ], u32x4 (&xf)[MS]) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                af[q] = tile < NT ? *(const u32x4*)(As + (tile * 16 + lr) * KP + 16 * s + 4 * lg) : z4;
            }
#pragma unroll
            for (int m = 0; m < MS; ++m) {
                const int row = m * 16 + lr;
                xf[m] = row < nrows ? *(const u32x4*)(Xs + row * KX + 32 * s + 8 * lg) : z4;
            }
        };
        auto step_mma = [&](const u32x4 (&af)[TQ], const u32x4 (&xf)[MS]) {
#pragma unroll
            for (int m = 0; m < MS; ++m)
#pragma unroll
                for (int q = 0; q < TQ; ++q) acc[m][q] = Fmt::mma32(af[q], xf[m], acc[m][q]);
        };
        constexpr int U = TQ + MS <= 2 ? 4 : (TQ + MS <= 4 ? 2 : 1);
        int s = wk;
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

    // lane holds v[row m*16+lr][ranks tile*16 + 4lg .. +3]
    float* part = a.partials + it.part;
    if constexpr (kSync) part += parity ? a.pbuf : 0;
    if (WK == 1) {
#pragma unroll
        for (int m = 0; m < MS; ++m) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                const int row = m * 16 + lr;
                if (tile < NT && row < nrows) {
                    const int r0 = tile * 16 + 4 * lg;
                    float* dst = part + row * R + r0;
                    if ((R & 3) == 0 && r0 + 3 < R) {
                        put_f32x4<kSync>(dst, acc[m][q]);
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (r0 + i < R) put_f32<kSync>(dst + i, acc[m][q][i]);
                    }
                }
            }
        }
    } else {
        __syncthreads();                      // staging is read no more
        float* red = (float*)smem;            // [WK][MS*16][Rp]
#pragma unroll
        for (int m = 0; m < MS; ++m) {
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int tile = wn + WN * q;
                if (tile < NT)
                    *(float4*)(red + ((wk * MS + m) * 16 + lr) * Rp + tile * 16 + 4 * lg) =
                        make_float4(acc[m][q][0], acc[m][q][1], acc[m][q][2], acc[m][q][3]);
            }
        }
        __syncthreads();
        for (int o = t; o < nrows * R; o += kThreads) {
            const int row = o / R;
            const int rank = o - row * R;
            float s = red[row * Rp + rank];
            for (int k = 1; k < WK; ++k) s += red[(k * MS * 16 + row) * Rp + rank];
            put_f32<kSync>(part + o, s);
        }
    }
    if constexpr (kSync) {
        // arm this block in the other buffer for the next launch, after this
        // launch's block is out.  Plain stores: only the next launch reads
        // them, and a kernel's end makes its stores visible to the next.  The
        // block is reserved to a multiple of 4 floats, so whole 16-byte
        // stores stay inside it.
        u32x4* other = (u32x4*)(a.partials + (parity ? 0 : a.pbuf) + it.part);
        const u32x4 s4 = {kSentinel, kSentinel, kSentinel, kSentinel};
        for (int o = t; 4 * o < nrows * R; o += kThreads) other[o] = s4;
    }
}

template <class Fmt, bool kSync>
__device__ __forceinline__ void shrink_item(const KernelArgs& a, const Item& it, unsigned char* smem) {
    const int tq = shrink_tq(it.rank);
    const int ms = msub_body(it.nrows);
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

// Two workgroups per CU: the register budget is capped at 256 per lane.
template <class Fmt>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
lora_shrink_kernel(KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kShrinkLds];
    const Item it = load_item(a.items + blockIdx.x);
    if (it.kind != kItemShrink) return;
    Item r = it;
    resolve<kLookupAuto>(a, r);
    shrink_item<Fmt, false>(a, r, smem);
}

// ---------------------------------------------------------------------------
// Expand
// ---------------------------------------------------------------------------
template <class Fmt, int Q, int MS, bool kSync>
__device__ __forceinline__ void expand_body(const KernelArgs& a, const Item& it,
                                            unsigned char* smem) {
    const int t = threadIdx.x;
    const int w = t >> 6;
    const int lr = t & 15;
    const int lg = (t >> 4) & 3;
    const int R = it.rank;
    const int Rk = round_up_i(R, 16);
    const int KS = Rk / 16;
    const int half = Rk / 2;
    const int RP = expand_rp(R);              // words per row: two ranks each, 2 (mod 4)
    const int len = it.len;
    const int ncol = round_up_i(len, 16);
    const int NCT = ncol / 16;
    const int nrows = it.nrows;
    uint32_t* Bs = (uint32_t*)smem;           // [ncol][RP]  B^T, rank pairs
    uint32_t* Vh = Bs + ncol * RP;            // [MS*16][RP]  high part of v
    uint32_t* Vl = Vh + MS * 16 * RP;         // [MS*16][RP]  low part of v
    float2* red = (float2*)(Vl + MS * 16 * RP);   // [kThreads]
    gu16* B = (gu16*)it.fac;
    const float scale = it.scale;
    const int rowv = lane_rows(a, it);
    const u32x4 z4 = {0u, 0u, 0u, 0u};

    // --- requests: the B tile (<= 4 rank-pair loads per thread by the tiling) ...
    const int cv = ncol / 8;                  // column octets
    const int npairs = half * cv;
    u32x4 b0[4], b1[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int p = t + i * kThreads;
        const int jp = p / cv;
        const int co = p - jp * cv;
        const int j = 2 * jp;
        const bool ok0 = p < npairs && co * 8 < len && j < R;
        const bool ok1 = p < npairs && co * 8 < len && j + 1 < R;
        // addresses stay inside B even where the load is masked off
        gu16* src0 = B + (int64_t)(ok0 ? j : 0) * a.h_out + it.lo + (ok0 ? co * 8 : 0);
        gu16* src1 = B + (int64_t)(ok1 ? j + 1 : 0) * a.h_out + it.lo + (ok1 ? co * 8 : 0);
        b0[i] = ok0 ? *(gu32x4*)src0 : z4;
        b1[i] = ok1 ? *(gu32x4*)src1 : z4;
    }
    // ... this lane's y: rows m*16+lr, columns ct*16 + 4lg .. +3 of the wave's
    // column tiles ct = w, w+4, ...
    int yrow[MS];
#pragma unroll
    for (int m = 0; m < MS; ++m) yrow[m] = row_of(rowv, m * 16 + lr < nrows ? m * 16 + lr : 0);
    u32x2 yv[Q][MS];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int ct = w + 4 * q;
        const int c = ct * 16 + 4 * lg;
#pragma unroll
        for (int m = 0; m < MS; ++m) {
            const bool ok = ct < NCT && m * 16 + lr < nrows && c + 4 <= len;
            const uint16_t* src = (const uint16_t*)a.y + (int64_t)yrow[m] * a.ldy + it.lo + (ok ? c : 0);
            yv[q][m] = ok ? *(const u32x2*)src : u32x2{0u, 0u};
        }
    }
    // ... and v: rank pairs of every row, the sum of the row block's partial
    // blocks (or the caller's v).  With few slots, P threads share a slot,
    // each adding every P-th block; the P sums are then added in order.
    const int slots = nrows * half;
    const int nslot = MS * 16 * half;
    const int P = a.v ? 1 : partial_parts(nrows, R, it.nsplit);
    const float* Pb = a.partials + it.part;
    if constexpr (kSync) Pb += row_block_parity(a, it) ? a.pbuf : 0;
    int budget = a.spin_limit;                // step launch: polling rounds left to this thread
    auto sum_parts = [&]() {
        if (P > 1) {
            const int slot = t % slots;
            const int q = t / slots;
            if (q < P) {
                const int row = slot / half;
                const int j = 2 * (slot - row * half);
                const float* src = Pb + row * R;
                red[t] = part_sum2<kSync>(a, src + (j < R ? j : 0), src + (j + 1 < R ? j + 1 : 0), it.pstride,
                                          it.nsplit, P, q, j < R, j + 1 < R, budget);
            }
        }
    };
    // --- B^T to LDS
    auto store_bt = [&]() {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = t + i * kThreads;
            if (p < npairs) {
                const int jp = p / cv;
                const int co = p - jp * cv;
                uint32_t* d = Bs + (co * 8) * RP + jp;
                d[0 * RP] = lo16(b0[i].x) | (b1[i].x << 16);
                d[1 * RP] = hi16(b0[i].x) | (b1[i].x & 0xffff0000u);
                d[2 * RP] = lo16(b0[i].y) | (b1[i].y << 16);
                d[3 * RP] = hi16(b0[i].y) | (b1[i].y & 0xffff0000u);
                d[4 * RP] = lo16(b0[i].z) | (b1[i].z << 16);
                d[5 * RP] = hi16(b0[i].z) | (b1[i].z & 0xffff0000u);
                d[6 * RP] = lo16(b0[i].w) | (b1[i].w << 16);
                d[7 * RP] = hi16(b0[i].w) | (b1[i].w & 0xffff0000u);
            }
        }
    };
    if constexpr (kSync) {
        // the B tile and y are requested and B^T staged before the partial
        // blocks are polled
        store_bt();
        sum_parts();
    } else {
        sum_parts();
        store_bt();
    }
    if (P > 1) __syncthreads();               // the P-way sums are in red
    // --- v to LDS as high / low 16-bit parts (rows past nrows: zero)
    for (int o = t; o < nslot; o += kThreads) {
        const int row = o / half;
        const int jp = o - row * half;
        const int j = 2 * jp;
        float v0 = 0.f, v1 = 0.f;
        if (row < nrows) {
            if (a.v) {
                const float* src = a.v + (int64_t)a.perm[it.p0 + row] * a.ldv;
                if (j < R) v0 = src[j];
                if (j + 1 < R) v1 = src[j + 1];
            } else if (P > 1) {
                for (int q = 0; q < P; ++q) {
                    const float2 r2 = red[q * slots + o];
                    v0 += r2.x;
                    v1 += r2.y;
                }
            } else {
                const float* src = Pb + row * R;
                const float2 s2 = part_sum2<kSync>(a, src + (j < R ? j : 0), src + (j + 1 < R ? j + 1 : 0),
                                                   it.pstride, it.nsplit, 1, 0, j < R, j + 1 < R, budget);
                v0 += s2.x;
                v1 += s2.y;
            }
        }
        const uint32_t h0 = Fmt::from_f32(v0), h1 = Fmt::from_f32(v1);
        const uint32_t l0 = Fmt::from_f32(v0 - Fmt::to_f32(h0));
        const uint32_t l1 = Fmt::from_f32(v1 - Fmt::to_f32(h1));
        Vh[row * RP + jp] = h0 | (h1 << 16);
        Vl[row * RP + jp] = l0 | (l1 << 16);
    }
    __syncthreads();
    // step launch: this item has read its partial values; count it (no wait
    // for the result)
    if constexpr (kSync)
        if (t == 0)
            (void)__builtin_amdgcn_atomic_inc32(a.sync + (int64_t)it.rb * kSyncStride, 2u * (uint32_t)it.nexp - 1u, __ATOMIC_RELAXED,
                                                "agent");

    // --- y^T = B^T v^T on MFMA, then y + s*d rounded once
    f32x4 acc[Q][MS];
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int m = 0; m < MS; ++m) acc[q][m] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < KS; ++s) {
        u32x2 af[Q];
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int ct = w + 4 * q;
            af[q] = ct < NCT ? *(const u32x2*)(Bs + (ct * 16 + lr) * RP + 8 * s + 2 * lg) : u32x2{0u, 0u};
        }
#pragma unroll
        for (int m = 0; m < MS; ++m) {
            const u32x2 bh = *(const u32x2*)(Vh + (m * 16 + lr) * RP + 8 * s + 2 * lg);
            const u32x2 bl = *(const u32x2*)(Vl + (m * 16 + lr) * RP + 8 * s + 2 * lg);
#pragma unroll
            for (int q = 0; q < Q; ++q) {
                acc[q][m] = Fmt::mma16(af[q], bh, acc[q][m]);
                acc[q][m] = Fmt::mma16(af[q], bl, acc[q][m]);
            }
        }
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int ct = w + 4 * q;
        const int c = ct * 16 + 4 * lg;
#pragma unroll
        for (int m = 0; m < MS; ++m) {
            if (ct < NCT && m * 16 + lr < nrows && c + 4 <= len) {
                const u32x2 yo = yv[q][m];
                const float f0 = fmaf(scale, acc[q][m][0], Fmt::to_f32(lo16(yo.x)));
                const float f1 = fmaf(scale, acc[q][m][1], Fmt::to_f32(hi16(yo.x)));
                const float f2 = fmaf(scale, acc[q][m][2], Fmt::to_f32(lo16(yo.y)));
                const float f3 = fmaf(scale, acc[q][m][3], Fmt::to_f32(hi16(yo.y)));
                *(u32x2*)((uint16_t*)a.y + (int64_t)yrow[m] * a.ldy + it.lo + c) =
                    u32x2{Fmt::from_f32(f0) | (Fmt::from_f32(f1) << 16),
                          Fmt::from_f32(f2) | (Fmt::from_f32(f3) << 16)};
            }
        }
    }
}

template <class Fmt, bool kSync>
__device__ __forceinline__ void expand_item(const KernelArgs& a, const Item& it, unsigned char* smem) {
    const int q = (round_up_i(it.len, 16) / 16 + 3) / 4;   // column tiles per wave
    const int ms = msub_body(it.nrows);
    if (ms == 1) {
        if (q <= 1) expand_body<Fmt, 1, 1, kSync>(a, it, smem);
        else if (q <= 2) expand_body<Fmt, 2, 1, kSync>(a, it, smem);
        else if (q <= 4) expand_body<Fmt, 4, 1, kSync>(a, it, smem);
        else expand_body<Fmt, 8, 1, kSync>(a, it, smem);
    } else if (ms == 2) {
        if (q <= 1) expand_body<Fmt, 1, 2, kSync>(a, it, smem);
        else if (q <= 2) expand_body<Fmt, 2, 2, kSync>(a, it, smem);
        else if (q <= 4) expand_body<Fmt, 4, 2, kSync>(a, it, smem);
        else expand_body<Fmt, 8, 2, kSync>(a, it, smem);
    } else {
        if (q <= 1) expand_body<Fmt, 1, 4, kSync>(a, it, smem);
        else if (q <= 2) expand_body<Fmt, 2, 4, kSync>(a, it, smem);
        else expand_body<Fmt, 4, 4, kSync>(a, it, smem);
    }
}

template <class Fmt>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
lora_expand_kernel(KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kExpandLds];
    const Item it = load_item(a.items + blockIdx.x);
    if (it.kind != kItemExpand) return;
    Item r = it;
    resolve<kLookupAuto>(a, r);
    expand_item<Fmt, false>(a, r, smem);
}

// ---------------------------------------------------------------------------
// Step: shrink items, then expand items, in one grid (two workgroups per CU).
// The item list is a kernel argument of its own, ahead of the argument block,
// so that it can be preloaded into scalar registers at wave launch.
// ---------------------------------------------------------------------------
template <class Fmt, int kLookup>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
lora_step_kernel(const DevItem* __restrict__ items, KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kStepLds];
    Item it;
    if constexpr (kLookup == kLookupArgs) {
        const LaneTable lt = load_lane_table(a);      // in flight with the item
        it = load_item(items + blockIdx.x);
        resolve_lanes(lt, it);
    } else {
        it = load_item(items + blockIdx.x);
        resolve<kLookupReg>(a, it);
    }
    if (it.kind == kItemShrink) shrink_item<Fmt, true>(a, it, smem);
    else if (it.kind == kItemExpand) expand_item<Fmt, true>(a, it, smem);
}

// ---------------------------------------------------------------------------
// Reduce: v(rows, 0:r) = sum of the row block's partial blocks, in order (the
// standalone shrink's output).
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads) lora_reduce_kernel(KernelArgs a) {
    const Item it = load_item(a.items + blockIdx.x);
    if (it.kind != kItemReduce) return;
    const int R = it.rank;
    const int n = it.nrows * R;
    const float* Pb = a.partials + it.part;
    const int P = partial_parts(it.nrows, R, it.nsplit);   // the expand's order
    for (int o = threadIdx.x; o < n; o += kThreads) {
        float s = 0.f;
        for (int q = 0; q < P; ++q) s += part_sum(Pb + o, it.pstride, it.nsplit, P, q);
        const int i = o / R;
        a.v[(int64_t)a.perm[it.p0 + i] * a.ldv + (o - i * R)] = s;
    }
}

// ---------------------------------------------------------------------------
// launches
// ---------------------------------------------------------------------------
hipError_t launch_shrink(const KernelArgs& a, int dtype, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    if (dtype == 0)
        hipLaunchKernelGGL(lora_shrink_kernel<FmtF16>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(lora_shrink_kernel<FmtBF16>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_expand(const KernelArgs& a, int dtype, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    if (dtype == 0)
        hipLaunchKernelGGL(lora_expand_kernel<FmtF16>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(lora_expand_kernel<FmtBF16>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_step(const KernelArgs& a, int dtype, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    const dim3 g(a.n_items), b(kThreads);
    const bool args = a.n_groups <= kKargGroups;
    if (dtype == 0) {
        if (args) hipLaunchKernelGGL((lora_step_kernel<FmtF16, kLookupArgs>), g, b, 0, s, a.items, a);
        else hipLaunchKernelGGL((lora_step_kernel<FmtF16, kLookupReg>), g, b, 0, s, a.items, a);
    } else {
        if (args) hipLaunchKernelGGL((lora_step_kernel<FmtBF16, kLookupArgs>), g, b, 0, s, a.items, a);
        else hipLaunchKernelGGL((lora_step_kernel<FmtBF16, kLookupReg>), g, b, 0, s, a.items, a);
    }
    return hipGetLastError();
}

hipError_t launch_reduce(const KernelArgs& a, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    hipLaunchKernelGGL(lora_reduce_kernel, dim3(a.n_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace lora
