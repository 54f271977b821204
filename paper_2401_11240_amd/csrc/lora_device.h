// Device-side building blocks shared by the gfx950 kernels: vector types,
// the two 16-bit storage formats with their MFMA instruction, 16-bit packing,
// buffer operations with out-of-range masking, and the 8 x 8 transpose of
// 16-bit values.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lora_internal.h"

namespace lora {

typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef float f32x2v __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
// Native vectors (not HIP's struct vector types): selects stay in registers.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
// Adapter factors are reached through pointers read at run time; they are
// global memory, said explicitly so that the loads are global, not flat.
typedef __attribute__((address_space(1))) const uint16_t gu16;

// ---------------------------------------------------------------------------
// 16-bit storage formats and their MFMA instruction
// ---------------------------------------------------------------------------
struct FmtF16 {
    // binary16 tops out at 65504: a float32 v beyond about 2^15 cannot be
    // split into a finite high part (see expand_body)
    static constexpr bool kNarrowRange = true;
    static __device__ __forceinline__ float to_f32(uint32_t b16) {
        return (float)__builtin_bit_cast(_Float16, (uint16_t)b16);
    }
    // two floats rounded (RNE) into one word: a low, b high
    static __device__ __forceinline__ uint32_t pack2(float a, float b) {
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2v{a, b}, f16x2v));
    }
    static __device__ __forceinline__ f32x4 mma32(const u32x4& a, const u32x4& b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    }
};
struct FmtBF16 {
    static constexpr bool kNarrowRange = false;   // the exponent range of float32
    static __device__ __forceinline__ float to_f32(uint32_t b16) { return __uint_as_float(b16 << 16); }
    static __device__ __forceinline__ uint32_t pack2(float a, float b) {
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2v{a, b}, bf16x2v));
    }
    static __device__ __forceinline__ f32x4 mma32(const u32x4& a, const u32x4& b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};

__device__ __forceinline__ uint32_t lo16(uint32_t w) { return w & 0xffffu; }
__device__ __forceinline__ uint32_t hi16(uint32_t w) { return w >> 16; }
// two 16-bit values (their low halves) in one word: a low, b high
__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

// ---------------------------------------------------------------------------
// Buffer operations.  A buffer resource covers [base, base + bytes); a load
// at an offset past bytes returns zeros and a store there is dropped, so a
// masked lane is an out-of-range offset, not a branch.  Every buffer this
// library builds spans less than kMaxSpan bytes, so kOut is past all of them.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer, 32-bit data format
constexpr int kOut = 0x7fffff00;
constexpr int kCoherent = 16;            // cache policy sc1: device-coherent (agent scope) access
static_assert((uint32_t)kOut > kMaxSpan, "out-of-range offset");

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}
template <int AUX = 0>
__device__ __forceinline__ u32x4 bload16(rsrc_t r, int off) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX));
}
template <int AUX = 0>
__device__ __forceinline__ u32x2 bload8(rsrc_t r, int off) {
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, AUX));
}
template <int AUX = 0>
__device__ __forceinline__ void bstore8(const u32x2& v, rsrc_t r, int off) {
    __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, AUX);
}
template <int AUX = 0>
__device__ __forceinline__ void bstore16(const u32x4& v, rsrc_t r, int off) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, AUX);
}

__device__ __forceinline__ u32x4 as_u4(const f32x4& v) { return __builtin_bit_cast(u32x4, v); }
__device__ __forceinline__ f32x4 as_f4(const u32x4& v) { return __builtin_bit_cast(f32x4, v); }

// The 8 x 8 transpose of 16-bit values: in[k] holds 8 consecutive elements
// of row k; out[c] gets element c of rows 0..7 (row k at position k).
__device__ __forceinline__ void transpose8x8(const u32x4 (&in)[8], u32x4 (&out)[8]) {
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const int w = c >> 1;
        u32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t a = in[2 * q][w], b = in[2 * q + 1][w];
            o[q] = (c & 1) ? pack_hi(a, b) : pack_lo(a, b);
        }
        out[c] = o;
    }
}
}  // namespace lora
