// Device helpers shared by the libtreewy kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "treewy.h"

namespace treewy {

constexpr int D = 128;          // d_k == d_v
constexpr int THREADS = 256;    // four wave64s per workgroup
constexpr int MAX_TREE = 256;   // most nodes per draft tree (one 64-bit ancestor word per 64 nodes)
constexpr int MASK_WORDS = MAX_TREE / 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// D(32x32) += A(32x16) B(16x32) on the matrix cores, bf16 in, fp32 accumulate.
// Lane l supplies row l%32 of A and column l%32 of B, each with the eight
// contraction indices of group l/32; lane l receives column l%32 of D at rows
// 8*(r/4) + 4*(l/32) + r%4 in accumulator element r.
__device__ __forceinline__ f32x16 mma(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row of the 32x32 accumulator tile held in element r by lanes of group hg.
__device__ __forceinline__ int acc_row(int r, int hg) { return 8 * (r >> 2) + 4 * hg + (r & 3); }

// Two floats -> a packed bf16 pair (element 0 in the low half), both rounded
// to nearest even by one conversion instruction.  (Element-wise casts became
// one conversion per element, at half the vector ALU's rate.)
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a, b}), bf16x2));
}

// fp32 -> bf16 pair with x ~= hi + lo (|x - hi - lo| <= 2^-16 |x|); both round to nearest even.
// Per pair of elements: hi by one conversion, each hi widened back to fp32 by a
// shift or a mask, lo = x - hi (exact), lo by one conversion.
__device__ __forceinline__ void split8(const float *x, bf16x8 &hi, bf16x8 &lo) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 h, l;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t hb = pack_bf2(x[2 * p], x[2 * p + 1]);
        const float h0 = __builtin_bit_cast(float, hb << 16), h1 = __builtin_bit_cast(float, hb & 0xffff0000u);
        h[p] = hb;
        l[p] = pack_bf2(x[2 * p] - h0, x[2 * p + 1] - h1);
    }
    hi = __builtin_bit_cast(bf16x8, h);
    lo = __builtin_bit_cast(bf16x8, l);
}

__device__ __forceinline__ bf16x8 round8(const float *x) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 h;
#pragma unroll
    for (int p = 0; p < 4; ++p) h[p] = pack_bf2(x[2 * p], x[2 * p + 1]);
    return __builtin_bit_cast(bf16x8, h);
}

// Raw buffer view of `bytes` bytes at `base` (the descriptor lives in SGPRs).
// Loads at offsets past the end return zero and stores there are dropped, so
// the ragged tail of a tile needs no branch.  The range check covers the
// per-lane offset plus the instruction offset.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// Cache policy of a buffer access.  STREAM sets the non-temporal bit: the line
// is not kept in L2 / MALL after use, which suits data each kernel touches
// once (the state, the node vectors, U and o) and lets a read+write stream
// run closer to the HBM rate than the default write-back policy does.
constexpr int CACHED = 0;
constexpr int STREAM = 2;

template <int P = CACHED> __device__ __forceinline__ f32x4 ld_f32x4(rsrc_t r, int off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, P));
}
template <int P = CACHED> __device__ __forceinline__ uint4 ld_u32x4(rsrc_t r, int off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, P));
}
template <int P = CACHED> __device__ __forceinline__ uint2 ld_u32x2(rsrc_t r, int off) {
    return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, P));
}
__device__ __forceinline__ float ld_f32(rsrc_t r, int off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ int ld_i32(rsrc_t r, int off) {
    return __builtin_bit_cast(int, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ __bf16 ld_bf16(rsrc_t r, int off) {
    return __builtin_bit_cast(__bf16, __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
}
template <typename T> __device__ __forceinline__ T ld_elem(rsrc_t r, int off);
template <> __device__ __forceinline__ float ld_elem<float>(rsrc_t r, int off) { return ld_f32(r, off); }
template <> __device__ __forceinline__ __bf16 ld_elem<__bf16>(rsrc_t r, int off) { return ld_bf16(r, off); }
template <int P = CACHED> __device__ __forceinline__ void st_u32x4(rsrc_t r, int off, uint4 x) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned int, x),
                                           r, off, 0, P);
}
template <int P = CACHED> __device__ __forceinline__ void st_u32x2(rsrc_t r, int off, uint2 x) {
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) unsigned int, x),
                                          r, off, 0, P);
}
template <int P = CACHED> __device__ __forceinline__ void st_f32(rsrc_t r, int off, float x) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, x), r, off, 0, P);
}

// One butterfly step of quad_transpose: lanes with `bit` clear exchange x[q]
// with x[p] of the lane `bit` away (DPP quad permutation CTRL).
template <int BIT, int CTRL>
__device__ __forceinline__ void quad_swap(f32x4 &xp, f32x4 &xq, int lane) {
    const bool hi = lane & BIT;
#pragma unroll
    for (int e = 0; e < 4; ++e) {                       // (value selects: a select of references goes through memory)
        const float a = xp[e], b = xq[e];
        const float got =
            __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, hi ? a : b), CTRL, 0xF, 0xF, false));
        xp[e] = hi ? got : a;
        xq[e] = hi ? b : got;
    }
}

// 4 x 4 transpose across the four lanes of each quad: afterwards lane i of a
// quad holds in x[r] what lane r held in x[i].  Two butterfly steps, each
// swapping one bit of the lane index with the same bit of the register index.
__device__ __forceinline__ void quad_transpose(f32x4 (&x)[4], int lane) {
    quad_swap<1, 0xB1>(x[0], x[1], lane);               // quad_perm [1, 0, 3, 2]
    quad_swap<1, 0xB1>(x[2], x[3], lane);
    quad_swap<2, 0x4E>(x[0], x[2], lane);               // quad_perm [2, 3, 0, 1]
    quad_swap<2, 0x4E>(x[1], x[3], lane);
}

// OR of a 32-bit value over the 64 lanes of a wave, returned wave-uniform:
// within each row of 16 lanes by DPP (two quad permutations, half-row and
// row mirrors), then row 0's total into row 1 and row 2's into row 3
// (row_bcast:15), rows 0-1 into rows 2-3 (row_bcast:31); lane 63 ends with all.
__device__ __forceinline__ uint32_t wave_or32(uint32_t v) {
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);    // quad_perm [1, 0, 3, 2]
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);    // quad_perm [2, 3, 0, 1]
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);   // row_half_mirror
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);   // row_mirror
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);   // row_bcast:15
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);   // row_bcast:31
    return __builtin_amdgcn_readlane(v, 63);
}
__device__ __forceinline__ uint64_t wave_or64(uint64_t v) {
    return (uint64_t)wave_or32((uint32_t)v) | ((uint64_t)wave_or32((uint32_t)(v >> 32)) << 32);
}

// The set bits of a wave-uniform word w, compacted: lane c (c < popcount(w))
// receives the position of the c-th set bit, lowest first.  Lane p, whose bit
// is set, sends p to lane rank(p) (one LDS-free permute); the lanes of clear
// bits all send to lane 63, so lanes at or past the count hold no position.
__device__ __forceinline__ int compact_bits(uint64_t w, int lane) {
    const bool set = (w >> lane) & 1ull;
    const int rank = __popcll(w & ((1ull << lane) - 1ull));
    return __builtin_amdgcn_ds_permute((set ? rank : 63) * 4, lane);
}

// A copy of x the compiler cannot see through (keeps derived values inside a loop).
__device__ __forceinline__ int opaque(int x) {
    asm volatile("" : "+v"(x));
    return x;
}

// Four bf16 held in a uint2 <-> four floats (exact widening; narrowing rounds
// to nearest even).
__device__ __forceinline__ f32x4 bf4_to_f32(uint2 x) {
    const bf16x4 h = __builtin_bit_cast(bf16x4, x);
    return f32x4{(float)h[0], (float)h[1], (float)h[2], (float)h[3]};
}
__device__ __forceinline__ uint2 f32_to_bf4(f32x4 x) {
    return uint2{pack_bf2(x[0], x[1]), pack_bf2(x[2], x[3])};
}

// Cumulative decays in extended range.  g_t, a product of up to 256 gates in
// (0, 1], is held as g = m 2^e with m in [0.5, 1) (m = e = 0 for a padding
// node): the product of many small gates cannot underflow, and a ratio
// g_t / g_i (i an ancestor of t, so at most 1) is formed as
// (m_t / m_i) 2^(e_t - e_i) and cannot overflow.  Scaling by a power of two
// is exact, so wherever the plain fp32 products stay normal these give the
// same bits as g_t * (1 / g_i).
struct DecayX {
    // a = a * b, renormalised
    static __device__ __forceinline__ void mul(float &m, int &e, float mb, int eb) {
        m *= mb;
        e += eb + __builtin_amdgcn_frexp_expf(m);
        m = __builtin_amdgcn_frexp_mantf(m);
    }
    static __device__ __forceinline__ float mant(float x) { return __builtin_amdgcn_frexp_mantf(x); }
    static __device__ __forceinline__ int expo(float x) { return __builtin_amdgcn_frexp_expf(x); }
    // the plain value (tiny values round to a denormal or zero, as they should)
    static __device__ __forceinline__ float value(float m, int e) { return __builtin_amdgcn_ldexpf(m, e); }
    // g_t / g_i from g_t = (mt, et) and 1 / m_i, e_i
    static __device__ __forceinline__ float ratio(float mt, int et, float inv_mi, int ei) {
        return __builtin_amdgcn_ldexpf(mt * inv_mi, et - ei);
    }
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(__bf16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ __bf16 from_f32<__bf16>(float x) { return (__bf16)x; }

__device__ __forceinline__ void flag_error(int32_t *err, int b, int flag) {
    if (err) atomicOr(err + b, flag);
}

}  // namespace treewy
