// gfx950 kernels of the batched, heterogeneous-rank LoRA delta
//   y[t,:] <- round(y[t,:] + s_g * (x[t,:] . A_g) . B_g)          (Eq. 1)
//
// Shrink: one workgroup per (adapter group, K-chunk of A_g).  The chunk of
// A_g (rows k0..k0+klen of the row-major [h_in, r] matrix) is one contiguous
// run of bytes, streamed once per step with 16-byte loads, whatever the
// number of tokens that use the adapter: tokens are gathered to their adapter
// instead of each token re-reading its adapter (the gather of Section 4.1
// done once per distinct adapter).  The group's x rows for the chunk sit in
// LDS; products accumulate in float32; lanes that share an output column
// reduce with cross-lane shuffles, then across the four waves through LDS in
// a fixed order.  When a group's h_in is split over several workgroups, each
// writes its partial sums; the last to arrive (atomic counter) adds them in
// chunk order, so results never depend on timing.
//
// Expand: one workgroup per (adapter group, column tile of B_g).  Each lane
// owns 8 consecutive output columns (16-byte loads and stores of B and y) and
// 8 consecutive ranks; the float32 intermediate v of the group's rows is read
// from LDS; partial sums over rank slices are added in a fixed order and
// y + s*d is rounded once to the storage dtype.
//
// Ranks 8, 16, 32, 64, 128 and 256 have compile-time specialised bodies;
// any other rank in [1, 256] takes a generic body.  All of them are
// selected per workgroup inside one grid, so items of different ranks run
// concurrently instead of queueing behind each other.
#include <hip/hip_runtime.h>

#include "lora_internal.h"

namespace lora {

// ---------------------------------------------------------------------------
// 16-bit storage formats
// ---------------------------------------------------------------------------
struct FmtF16 {
    static __device__ __forceinline__ float to_f32(uint32_t b16) {
        return (float)__builtin_bit_cast(_Float16, (uint16_t)b16);
    }
    static __device__ __forceinline__ uint32_t from_f32(float f) {
        return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
    }
};
struct FmtBF16 {
    static __device__ __forceinline__ float to_f32(uint32_t b16) {
        return __uint_as_float(b16 << 16);
    }
    static __device__ __forceinline__ uint32_t from_f32(float f) {
        return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
    }
};

template <class Fmt>
__device__ __forceinline__ void unpack8(const uint4& v, float f[8]) {
    f[0] = Fmt::to_f32(v.x & 0xffffu); f[1] = Fmt::to_f32(v.x >> 16);
    f[2] = Fmt::to_f32(v.y & 0xffffu); f[3] = Fmt::to_f32(v.y >> 16);
    f[4] = Fmt::to_f32(v.z & 0xffffu); f[5] = Fmt::to_f32(v.z >> 16);
    f[6] = Fmt::to_f32(v.w & 0xffffu); f[7] = Fmt::to_f32(v.w >> 16);
}

template <class Fmt>
__device__ __forceinline__ uint4 pack8(const float f[8]) {
    uint4 v;
    v.x = Fmt::from_f32(f[0]) | (Fmt::from_f32(f[1]) << 16);
    v.y = Fmt::from_f32(f[2]) | (Fmt::from_f32(f[3]) << 16);
    v.z = Fmt::from_f32(f[4]) | (Fmt::from_f32(f[5]) << 16);
    v.w = Fmt::from_f32(f[6]) | (Fmt::from_f32(f[7]) << 16);
    return v;
}

__device__ __forceinline__ int64_t v_row(const KernelArgs& a, int p) {
    return a.v_by_row ? (int64_t)a.perm[p] : (int64_t)p;
}

// Where the shrink result of (group-local row i, rank j) goes: the final v
// when the group's h_in is a single chunk, else this chunk's partial slot.
__device__ __forceinline__ void shrink_store(const KernelArgs& a, const DevItem& it, int R, int i,
                                             int j, float s) {
    const int nsplit = it.split & 0xffff;
    if (nsplit == 1) {
        a.v[v_row(a, it.p0 + i) * a.ldv + j] = s;
    } else {
        const int chunk = it.split >> 16;
        a.partials[a.part_off[it.group] + ((int64_t)chunk * it.nrows + i) * R + j] = s;
    }
}

// ---------------------------------------------------------------------------
// Shrink, rank R in {8,16,32,64,128,256}
// ---------------------------------------------------------------------------
constexpr int kShrinkLdsBytes = 32768;

template <class Fmt, int R>
__device__ __forceinline__ void shrink_fast(const KernelArgs& a, const DevItem& it,
                                            const DevAdapter& ad, unsigned char* smem) {
    constexpr int RT = kShrinkRowTile;
    constexpr int VPR = R / 8;               // 16-byte vectors per row of A
    constexpr int TPJ = kThreads / VPR;      // threads that share one octet of ranks
    constexpr int KMAX = kChunkElems / R;    // rows of A in a full chunk
    constexpr int M = KMAX / TPJ;            // vectors per thread (8)
    static_assert(M * TPJ == KMAX, "chunk tiling");
    static_assert(RT * KMAX * 2 <= kShrinkLdsBytes, "x tile fits");
    static_assert(4 * RT * R * 4 <= kShrinkLdsBytes, "reduction fits");

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int j0 = (t % VPR) * 8;
    const int kr0 = t / VPR;
    const int klen = it.len;
    const uint16_t* A = (const uint16_t*)ad.A + (int64_t)it.lo * R;

    // The whole chunk of A goes to registers first: every load in flight at once.
    uint4 av[M];
#pragma unroll
    for (int m = 0; m < M; ++m) {
        const int kr = kr0 + m * TPJ;
        av[m] = kr < klen ? *(const uint4*)(A + (int64_t)kr * R + j0) : make_uint4(0, 0, 0, 0);
    }

    uint16_t* xs = (uint16_t*)smem;    // [RT][KMAX]
    float* red = (float*)smem;         // [4][RT][R], reuses the x tile's bytes
    const uint16_t* X = (const uint16_t*)a.x;
    const int kv = klen / 8;
    auto load_x_tile = [&](int i0, int nr) {
        for (int idx = t; idx < nr * kv; idx += kThreads) {
            const int r = idx / kv;
            const int c = idx - r * kv;
            const int64_t row = a.perm[it.p0 + i0 + r];
            *(uint4*)(xs + r * KMAX + c * 8) = *(const uint4*)(X + row * a.ldx + it.lo + c * 8);
        }
    };

    // First x tile is requested while the A chunk is still in flight; A is
    // widened to float32 once, after which its packed copy is dead.
    load_x_tile(0, min(RT, it.nrows));
    float af[M][8];
#pragma unroll
    for (int m = 0; m < M; ++m) unpack8<Fmt>(av[m], af[m]);
    __syncthreads();

    for (int i0 = 0; i0 < it.nrows; i0 += RT) {
        const int nr = min(RT, it.nrows - i0);
        if (i0 > 0) {
            __syncthreads();
            load_x_tile(i0, nr);
            __syncthreads();
        }

        float acc[RT][8];
#pragma unroll
        for (int i = 0; i < RT; ++i)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[i][e] = 0.f;

#pragma unroll
        for (int m = 0; m < M; ++m) {
            const int kr = kr0 + m * TPJ;
            if (kr < klen) {
#pragma unroll
                for (int i = 0; i < RT; ++i) {
                    if (i < nr) {
                        const float xk = Fmt::to_f32(xs[i * KMAX + kr]);
#pragma unroll
                        for (int e = 0; e < 8; ++e) acc[i][e] = fmaf(xk, af[m][e], acc[i][e]);
                    }
                }
            }
        }

        // lanes with the same rank octet within a wave: butterfly
#pragma unroll
        for (int mask = VPR; mask < 64; mask <<= 1)
#pragma unroll
            for (int i = 0; i < RT; ++i)
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[i][e] += __shfl_xor(acc[i][e], mask);

        __syncthreads();   // x tile no longer read; its bytes become the reduction buffer
        if (lane < VPR) {
#pragma unroll
            for (int i = 0; i < RT; ++i)
                if (i < nr)
#pragma unroll
                    for (int e = 0; e < 8; ++e) red[(w * RT + i) * R + j0 + e] = acc[i][e];
        }
        __syncthreads();
        for (int o = t; o < nr * R; o += kThreads) {
            const int i = o / R;
            const int j = o - i * R;
            const float s = ((red[(0 * RT + i) * R + j] + red[(1 * RT + i) * R + j]) +
                             red[(2 * RT + i) * R + j]) + red[(3 * RT + i) * R + j];
            shrink_store(a, it, R, i0 + i, j, s);
        }
    }
}

// ---------------------------------------------------------------------------
// Shrink, any rank in [1, 256] (correct, not tuned)
// ---------------------------------------------------------------------------
constexpr int kGenericRowTile = 2;
constexpr int kGenericChunkElems = 8192;
constexpr int kGenericLdsBytes = 2 * kGenericChunkElems + 2 * kGenericRowTile * 8192 + 4 * kThreads;

template <class Fmt>
__device__ void shrink_generic(const KernelArgs& a, const DevItem& it, const DevAdapter& ad,
                               unsigned char* smem) {
    const int R = ad.rank;
    const int klen = it.len;
    const int t = threadIdx.x;
    // A chunk (klen*R <= kGenericChunkElems elements, a multiple of 8 and
    // 16-byte aligned since k0 % 8 == 0), then the x rows, then the reduction.
    uint16_t* as = (uint16_t*)smem;                                  // [kGenericChunkElems]
    uint16_t* xs = as + kGenericChunkElems;                          // [2][klen <= 8192]
    float* red = (float*)(smem + 2 * kGenericChunkElems + 2 * kGenericRowTile * 8192);   // [256]
    const uint16_t* A = (const uint16_t*)ad.A + (int64_t)it.lo * R;
    const int nvec = klen * R / 8;
    __syncthreads();
    for (int idx = t; idx < nvec; idx += kThreads) *(uint4*)(as + idx * 8) = *(const uint4*)(A + (int64_t)idx * 8);
    const uint16_t* X = (const uint16_t*)a.x;
    const int kv = klen / 8;
    for (int i0 = 0; i0 < it.nrows; i0 += kGenericRowTile) {
        const int nr = min(kGenericRowTile, it.nrows - i0);
        __syncthreads();
        for (int idx = t; idx < nr * kv; idx += kThreads) {
            const int r = idx / kv;
            const int c = idx - r * kv;
            const int64_t row = a.perm[it.p0 + i0 + r];
            *(uint4*)(xs + r * klen + c * 8) = *(const uint4*)(X + row * a.ldx + it.lo + c * 8);
        }
        __syncthreads();
        const int NO = nr * R;
        const int P = NO <= kThreads ? kThreads / NO : 1;   // threads per output
        for (int ob = 0; ob < NO; ob += kThreads / P) {
            const int o = ob + t % (kThreads / P);
            const int part = t / (kThreads / P);
            float acc = 0.f;
            if (o < NO && part < P) {
                const int i = o / R;
                const int j = o - i * R;
                for (int k = part; k < klen; k += P)
                    acc = fmaf(Fmt::to_f32(xs[i * klen + k]), Fmt::to_f32(as[k * R + j]), acc);
            }
            __syncthreads();
            red[t] = acc;
            __syncthreads();
            if (t < kThreads / P) {
                const int oo = ob + t;
                if (oo < NO) {
                    float s = 0.f;
                    for (int q = 0; q < P; ++q) s += red[q * (kThreads / P) + t];
                    const int i = oo / R;
                    shrink_store(a, it, R, i0 + i, oo - i * R, s);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Split-K completion: the last workgroup of a group adds the partials in
// chunk order into v and re-arms the group's counter for the next launch.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void shrink_finish(const KernelArgs& a, const DevItem& it, int R) {
    const int nsplit = it.split & 0xffff;
    if (nsplit == 1) return;
    __shared__ int s_last;
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const int old = atomicAdd(&a.counters[it.group], 1);
        s_last = (old == nsplit - 1);
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const float* P = a.partials + a.part_off[it.group];
    const int64_t per = (int64_t)it.nrows * R;
    for (int o = threadIdx.x; o < per; o += kThreads) {
        float s = 0.f;
        for (int c = 0; c < nsplit; ++c) s += P[c * per + o];
        const int i = o / R;
        a.v[v_row(a, it.p0 + i) * a.ldv + (o - i * R)] = s;
    }
    if (threadIdx.x == 0)
        __hip_atomic_store(&a.counters[it.group], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <class Fmt>
__global__ void __launch_bounds__(kThreads) lora_shrink_kernel(KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kGenericLdsBytes > kShrinkLdsBytes ? kGenericLdsBytes : kShrinkLdsBytes];
    const DevItem it = a.items[blockIdx.x];
    const DevAdapter ad = a.table[it.adapter];
    switch (ad.rank) {
        case 8: shrink_fast<Fmt, 8>(a, it, ad, smem); break;
        case 16: shrink_fast<Fmt, 16>(a, it, ad, smem); break;
        case 32: shrink_fast<Fmt, 32>(a, it, ad, smem); break;
        case 64: shrink_fast<Fmt, 64>(a, it, ad, smem); break;
        case 128: shrink_fast<Fmt, 128>(a, it, ad, smem); break;
        case 256: shrink_fast<Fmt, 256>(a, it, ad, smem); break;
        default: shrink_generic<Fmt>(a, it, ad, smem); break;
    }
    shrink_finish(a, it, ad.rank);
}

// ---------------------------------------------------------------------------
// Expand, rank R in {8,16,32,64,128,256}
// ---------------------------------------------------------------------------
template <class Fmt>
__device__ __forceinline__ void y_update8(const KernelArgs& a, int64_t row, int col, float scale,
                                          const float d[8]) {
    uint16_t* Y = (uint16_t*)a.y + row * a.ldy + col;
    const uint4 yv = *(const uint4*)Y;
    float f[8];
    unpack8<Fmt>(yv, f);
#pragma unroll
    for (int c = 0; c < 8; ++c) f[c] = fmaf(scale, d[c], f[c]);
    *(uint4*)Y = pack8<Fmt>(f);
}

template <class Fmt, int R>
__device__ __forceinline__ void expand_fast(const KernelArgs& a, const DevItem& it,
                                            const DevAdapter& ad, unsigned char* smem) {
    constexpr int RT = kExpandRowTile;
    constexpr int NMAX = kChunkElems / R;   // columns in a full tile
    constexpr int CB = NMAX / 8;            // column blocks of 8
    constexpr int JS = kThreads / CB;       // rank slices
    static_assert(JS * 8 == R, "8 ranks per thread");
    constexpr int WPC = CB >= 64 ? CB / 64 : 1;   // waves per column set
    constexpr int NW = 4 / WPC;                   // partial sums per output after the wave step

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int cb = t % CB;
    const int js = t / CB;
    const int nlen = it.len;
    const bool col_ok = cb * 8 < nlen;
    const int col = it.lo + cb * 8;
    const uint16_t* B = (const uint16_t*)ad.B;

    uint4 bv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        bv[e] = col_ok ? *(const uint4*)(B + (int64_t)(js * 8 + e) * a.h_out + col) : make_uint4(0, 0, 0, 0);
    float bf[8][8];
#pragma unroll
    for (int e = 0; e < 8; ++e) unpack8<Fmt>(bv[e], bf[e]);

    float* vs = (float*)smem;                 // [RT][R]
    float* red = vs + RT * kMaxRank;          // [NW][RT][NMAX]

    for (int i0 = 0; i0 < it.nrows; i0 += RT) {
        const int nr = min(RT, it.nrows - i0);
        __syncthreads();
        for (int o = t; o < nr * R; o += kThreads) {
            const int i = o / R;
            vs[o] = a.v[v_row(a, it.p0 + i0 + i) * a.ldv + (o - i * R)];
        }
        __syncthreads();
        float acc[RT][8];
#pragma unroll
        for (int i = 0; i < RT; ++i) {
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[i][c] = 0.f;
            if (i < nr) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float ve = vs[i * R + js * 8 + e];
#pragma unroll
                    for (int c = 0; c < 8; ++c) acc[i][c] = fmaf(ve, bf[e][c], acc[i][c]);
                }
            }
        }
        if constexpr (CB < 64) {
#pragma unroll
            for (int mask = CB; mask < 64; mask <<= 1)
#pragma unroll
                for (int i = 0; i < RT; ++i)
#pragma unroll
                    for (int c = 0; c < 8; ++c) acc[i][c] += __shfl_xor(acc[i][c], mask);
        }
        if constexpr (NW == 1) {
            if (col_ok) {
#pragma unroll
                for (int i = 0; i < RT; ++i)
                    if (i < nr) y_update8<Fmt>(a, a.perm[it.p0 + i0 + i], col, ad.scale, acc[i]);
            }
        } else {
            const int q = CB >= 64 ? w / WPC : w;
            const bool writer = CB >= 64 ? true : lane < CB;
            const int cbw = CB >= 64 ? (w % WPC) * 64 + lane : lane;
            if (writer) {
#pragma unroll
                for (int i = 0; i < RT; ++i)
                    if (i < nr)
#pragma unroll
                        for (int c = 0; c < 8; ++c) red[(q * RT + i) * NMAX + cbw * 8 + c] = acc[i][c];
            }
            __syncthreads();
            for (int o = t; o < nr * CB; o += kThreads) {
                const int i = o / CB;
                const int b = o - i * CB;
                if (b * 8 < nlen) {
                    float d[8];
#pragma unroll
                    for (int c = 0; c < 8; ++c) {
                        float s = red[(0 * RT + i) * NMAX + b * 8 + c];
#pragma unroll
                        for (int qq = 1; qq < NW; ++qq) s += red[(qq * RT + i) * NMAX + b * 8 + c];
                        d[c] = s;
                    }
                    y_update8<Fmt>(a, a.perm[it.p0 + i0 + i], it.lo + b * 8, ad.scale, d);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Expand, any rank in [1, 256] (correct, not tuned)
// ---------------------------------------------------------------------------
template <class Fmt>
__device__ void expand_generic(const KernelArgs& a, const DevItem& it, const DevAdapter& ad,
                               unsigned char* smem) {
    constexpr int RT = kExpandRowTile;
    const int R = ad.rank;
    const int t = threadIdx.x;
    float* vs = (float*)smem;   // [RT][R]
    const uint16_t* B = (const uint16_t*)ad.B;
    for (int i0 = 0; i0 < it.nrows; i0 += RT) {
        const int nr = min(RT, it.nrows - i0);
        __syncthreads();
        for (int o = t; o < nr * R; o += kThreads) {
            const int i = o / R;
            vs[o] = a.v[v_row(a, it.p0 + i0 + i) * a.ldv + (o - i * R)];
        }
        __syncthreads();
        for (int c = t; c < it.len; c += kThreads) {
            const int col = it.lo + c;
            float acc[RT];
#pragma unroll
            for (int i = 0; i < RT; ++i) acc[i] = 0.f;
            for (int j = 0; j < R; ++j) {
                const float b = Fmt::to_f32(B[(int64_t)j * a.h_out + col]);
#pragma unroll
                for (int i = 0; i < RT; ++i)
                    if (i < nr) acc[i] = fmaf(vs[i * R + j], b, acc[i]);
            }
#pragma unroll
            for (int i = 0; i < RT; ++i) {
                if (i < nr) {
                    uint16_t* Y = (uint16_t*)a.y + (int64_t)a.perm[it.p0 + i0 + i] * a.ldy + col;
                    *Y = (uint16_t)Fmt::from_f32(fmaf(ad.scale, acc[i], Fmt::to_f32(*Y)));
                }
            }
        }
    }
}

constexpr int kExpandLdsBytes = (kExpandRowTile * kMaxRank + 4 * kExpandRowTile * 512) * 4;

template <class Fmt>
__global__ void __launch_bounds__(kThreads) lora_expand_kernel(KernelArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[kExpandLdsBytes];
    const DevItem it = a.items[blockIdx.x];
    const DevAdapter ad = a.table[it.adapter];
    switch (ad.rank) {
        case 8: expand_fast<Fmt, 8>(a, it, ad, smem); break;
        case 16: expand_fast<Fmt, 16>(a, it, ad, smem); break;
        case 32: expand_fast<Fmt, 32>(a, it, ad, smem); break;
        case 64: expand_fast<Fmt, 64>(a, it, ad, smem); break;
        case 128: expand_fast<Fmt, 128>(a, it, ad, smem); break;
        case 256: expand_fast<Fmt, 256>(a, it, ad, smem); break;
        default: expand_generic<Fmt>(a, it, ad, smem); break;
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

}  // namespace lora
