// device.h -- gfx950 device helpers shared by the sdattn kernels.
//
// 16-bit tensor elements travel as raw 32-bit words (two elements per word)
// and are reinterpreted as fp16 or bf16 only at the MFMA and at conversions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace sdattn {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

enum ElemType { kF16 = 0, kBF16 = 1, kF32 = 2 };

constexpr float kLog2e = 1.4426950408889634f;

// D = A * B + C on one 32x32x16 matrix-core tile.  A is 32 x 16 (lane l holds
// row l % 32, eight consecutive k of half l / 32), B is 16 x 32 (lane l holds
// column l % 32, the same eight k), C/D is 32 x 32 fp32 with lane l holding
// column l % 32 and rows 8*(r/4) + 4*(l/32) + r%4 in register r.
template <int ET>
__device__ __forceinline__ f32x16 mfma32x32x16(u32x4 a, u32x4 b, f32x16 c) {
    if constexpr (ET == kF16) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    } else {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
}

// Round two floats to the 16-bit type (nearest even) and pack them, x in the low half.
// (one v_cvt_pk_f16_f32 / v_cvt_pk_bf16_f32)
template <int ET>
__device__ __forceinline__ uint32_t pack2(float x, float y) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    const f2 v = {x, y};
    if constexpr (ET == kF16) {
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
    } else {
        typedef __bf16 b2 __attribute__((ext_vector_type(2)));
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b2));
    }
}

template <int ET>
__device__ __forceinline__ float to_float(uint16_t bits) {
    if constexpr (ET == kF16) {
        return (float)__builtin_bit_cast(_Float16, bits);
    } else {
        return __uint_as_float((uint32_t)bits << 16);
    }
}

template <int ET>
__device__ __forceinline__ uint16_t from_float(float x) {
    if constexpr (ET == kF16) {
        return __builtin_bit_cast(uint16_t, (_Float16)x);
    } else {
        return __builtin_bit_cast(uint16_t, (__bf16)x);
    }
}

// acc + the two 16-bit values packed in w (exact products with 1.0, fp32 sum):
// v_dot2_f32_f16 / v_dot2_f32_bf16.
template <int ET>
__device__ __forceinline__ float add_pair(uint32_t w, float acc) {
    if constexpr (ET == kF16) {
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
        const h2 one = {(_Float16)1.0f, (_Float16)1.0f};
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w), one, acc, false);
    } else {
        typedef __bf16 b2 __attribute__((ext_vector_type(2)));
        const b2 one = {(__bf16)1.0f, (__bf16)1.0f};
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(b2, w), one, acc, false);
    }
}

// s_waitcnt immediate that waits until at most n vector-memory loads are
// outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14; expcnt and
// lgkmcnt left at their maxima, i.e. not waited on).
constexpr int vm_wait(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
// s_waitcnt immediate that waits for every LDS operation (lgkmcnt = 0) only.
constexpr int lgkm_wait0() { return 15 | (3 << 14) | (7 << 4); }

// 2^x on the transcendental unit (v_exp_f32); exp2(-inf) = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Exchange a value between lane l and lane l ^ 32 with v_permlane32_swap.
// Returns {own, partner} in some order per lane; callers combine the two
// with a commutative operation, or pick with half_select().
struct HalfPair { float a, b; };
__device__ __forceinline__ HalfPair half_swap(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return HalfPair{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ float half_max(float x) {
    HalfPair p = half_swap(x);
    return fmaxf(p.a, p.b);
}
__device__ __forceinline__ float half_sum(float x) {
    HalfPair p = half_swap(x);
    return p.a + p.b;
}
// The value held by lane l ^ 32.  After the swap, lanes 0..31 see
// {own, partner} and lanes 32..63 see {partner, own}.
__device__ __forceinline__ float half_partner(float x, int half) {
    HalfPair p = half_swap(x);
    return half ? p.a : p.b;
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// 16-bit element groups for the transposing LDS read, and LDS address-space
// pointer types for the builtins that take them.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

// Logical tile for workgroup `bid` of `nblk`.  Workgroups are dealt
// round-robin over the 8 XCDs; this gives every XCD a contiguous run of
// logical tiles, so that tiles which read the same operands (the query blocks
// of one (batch, head), or the token tiles of one weight slice) share one L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
    const int per = nblk / 8, rem = nblk % 8;
    const int xcd = bid % 8, slot = bid / 8;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives the
// 16-bit element i % 4 of the 8 bytes that lanes i / 4 + {0, 4, 8, 12} point
// at -- four consecutive rows of one column of a row-major tile when each
// lane points at four consecutive columns of one row.
__device__ __forceinline__ u32x2 lds_read_tr(const char* p) {
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p);
    return __builtin_bit_cast(u32x2, v);
}

// Where query row i of head bh = b*H + h goes in O: out_base(O, ...) + i * out_stride.
// oh == 0: O is [B, H, Lq, D]; oh == H: O is [B, Lq, H*D] (the heads merged
// into token rows).
__device__ __forceinline__ uint16_t* out_base(uint16_t* O, int bh, int Lq, int D, int oh) {
    if (oh == 0) return O + (size_t)bh * Lq * D;
    const int b = bh / oh;
    return O + ((size_t)b * Lq * oh + (bh - b * oh)) * D;
}
__device__ __forceinline__ size_t out_stride(int D, int oh) { return oh == 0 ? (size_t)D : (size_t)oh * D; }

}  // namespace sdattn
