// Device helpers shared by the gfx950 kernels of libprox: wave64 reductions
// and scans, matrix-core and dot-product wrappers and 16-bit float
// conversions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layout.hpp"

namespace prox {

constexpr int kWave = 64;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// 16-bit float conversions (exact widening, round-to-nearest-even narrowing)
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float f16_bits_to_float(uint32_t h) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

template <int DT>
__device__ __forceinline__ float lo_to_float(uint32_t w) {
    if constexpr (DT == kBF16) return bf16_lo(w);
    else return f16_bits_to_float(w & 0xFFFFu);
}
template <int DT>
__device__ __forceinline__ float hi_to_float(uint32_t w) {
    if constexpr (DT == kBF16) return bf16_hi(w);
    else return f16_bits_to_float(w >> 16);
}
template <int DT>
__device__ __forceinline__ float half_to_float(uint16_t h) {
    return lo_to_float<DT>((uint32_t)h);
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t float_to_bf16_rne(float v) {
    uint32_t u = __float_as_uint(v);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
// fp32 -> fp16 bits; the hardware conversion rounds to nearest even.
__device__ __forceinline__ uint16_t float_to_f16_rne(float v) {
    return __builtin_bit_cast(uint16_t, (_Float16)v);
}
template <int DT>
__device__ __forceinline__ uint16_t float_to_half(float v) {
    if constexpr (DT == kBF16) return float_to_bf16_rne(v);
    else return float_to_f16_rne(v);
}

// Two-term dot product with fp32 accumulation: a.lo*b.lo + a.hi*b.hi + c.
template <int DT>
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    if constexpr (DT == kBF16)
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                               __builtin_bit_cast(bf16x2, b), c, false);
    else
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b),
                                      c, false);
}

// INT4 dequant by exponent OR: a nibble n under the bits of M (128.0 in bf16,
// 1024.0 in fp16) is exactly the 16-bit value M + n, so a code q stored as
// n = q + 8 reads back as q after subtracting offset = M + 8 once per sum.
template <int DT>
struct Int4Magic;
template <>
struct Int4Magic<kBF16> {
    static constexpr uint32_t pair = 0x43004300u;   // (128.0, 128.0)
    static constexpr uint32_t one = 0x3F803F80u;    // (1.0, 1.0)
    static constexpr float offset = 136.0f;
};
template <>
struct Int4Magic<kF16> {
    static constexpr uint32_t pair = 0x64006400u;   // (1024.0, 1024.0)
    static constexpr uint32_t one = 0x3C003C00u;
    static constexpr float offset = 1032.0f;
};

// (v & mask) | bits.  FUSED: one v_and_or_b32 (the compiler otherwise emits
// two VOP2 instructions with literals); the asm form lengthens live ranges, so
// it is used only where registers are not tight.
template <bool FUSED>
__device__ __forceinline__ uint32_t and_or(uint32_t v, uint32_t mask, uint32_t bits) {
    if constexpr (FUSED) {
        uint32_t r;
        asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(v), "s"(mask), "v"(bits));
        return r;
    } else {
        return (v & mask) | bits;
    }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

typedef short v4s __attribute__((ext_vector_type(4)));
typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

// D += A B on the matrix cores, 16 x 16 x 16 with fp32 accumulation.  Lane l
// holds A[l % 16][4 (l / 16) + e] and B[4 (l / 16) + e][l % 16] for e = 0..3
// (four 16-bit values in a uint2) and gets D[4 (l / 16) + e][l % 16].
template <int DT>
__device__ __forceinline__ v4f mfma16(uint2 a, uint2 b, v4f c) {
    if constexpr (DT == kBF16)
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(v4s, a),
                                                         __builtin_bit_cast(v4s, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(v4h, a),
                                                     __builtin_bit_cast(v4h, b), c, 0, 0, 0);
}

// 16- and 8-byte streaming loads (non-temporal hint: weights are read once
// per call).
__device__ __forceinline__ uint4 load_stream16(const void *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint2 load_stream8(const void *p) {
    const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(p));
    return make_uint2(v.x, v.y);
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// Gate activation of the gated FFN: SiLU (act 0) or GELU z * Phi(z) (act 1),
// with Phi(z) = erfc(-z / sqrt 2) / 2 (no cancellation in the negative tail).
__device__ __forceinline__ float gate_act(float z, int act) {
    return act == 0 ? silu(z) : 0.5f * z * erfcf(-z * 0.70710678118654752f);
}

// ---------------------------------------------------------------------------
// Wave64 collectives
// ---------------------------------------------------------------------------

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Cross-lane moves on the VALU (no LDS round trip): DPP within 16-lane rows,
// and the gfx950 row / half swaps.  swap16(v) is v + lane^16's v, swap32(v)
// is v + lane^32's v; both lanes of a pair get the same bits.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppRor4 = 0x124;    // row_ror:4
constexpr int kDppRor8 = 0x128;    // row_ror:8 (lane ^ 8 within a row)
__device__ __forceinline__ float add_swap16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_swap32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sum over the wave in a fixed order, returned in every lane (lane 0's value).
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_move<kDppXor1>(v);
    v += dpp_move<kDppXor2>(v);    // quads uniform
    v += dpp_move<kDppRor4>(v);
    v += dpp_move<kDppRor8>(v);    // rows summed
    v = add_swap16(v);
    v = add_swap32(v);
    return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
}

// Number of set bits of `mask` in lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Inclusive prefix sum over the wave (every lane active).  Shifts of 1, 2, 4
// and 8 inside each 16-lane row (lanes shifted in from outside the row read
// 0), then each row adds the totals of the rows below it.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);   // row_shr:8
    const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
              r2 = __builtin_amdgcn_readlane(v, 47);
    const int row = lane_id() >> 4;
    return v + (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
}

// Maximum over the wave (every lane active), in every lane.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppXor1, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppXor2, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppRor4, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppRor8, 0xF, 0xF, false));
    const auto a = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    v = max(a[0], a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return max(b[0], b[1]);
}

// Sum over each quad of lanes (lanes 4j .. 4j+3), in every lane of the quad.
__device__ __forceinline__ uint32_t quad_sum_u32(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppXor1, 0xF, 0xF, false);
    return v + (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppXor2, 0xF, 0xF, false);
}

// Block-wide exclusive prefix sum of one int per thread (NT threads); also
// returns the block total.  `sh` is LDS scratch of NT/64 + 1 ints.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int *sh, int &total) {
    constexpr int NW = NT / kWave;
    const int lane = lane_id(), wid = threadIdx.x / kWave;
    int incl = wave_inclusive_scan(v);
    if (lane == kWave - 1) sh[wid] = incl;
    __syncthreads();
    if (wid == 0) {
        int wv = lane < NW ? sh[lane] : 0;
        int wi = wave_inclusive_scan(wv);
        if (lane < NW) sh[lane] = wi - wv;
        if (lane == NW - 1) sh[NW] = wi;
    }
    __syncthreads();
    int res = sh[wid] + incl - v;
    total = sh[NW];
    __syncthreads();
    return res;
}

}  // namespace prox
