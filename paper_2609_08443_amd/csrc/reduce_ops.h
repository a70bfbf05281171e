// Cross-lane reductions for the matrix-core kernels (gfx950, wave64): DPP inside
// rows of 16 lanes, v_permlane16_swap between the two rows of a 32-lane half and
// v_permlane32_swap between the halves; no LDS.
#pragma once

#include "tile_ops.h"

namespace sa {
namespace tile {

__device__ inline float sumsq8(uint4 v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float a = bf16_lo(w[i]), b = bf16_hi(w[i]);
        s = __builtin_fmaf(a, a, s);
        s = __builtin_fmaf(b, b, s);
    }
    return s;
}

// Cross-lane moves without LDS: DPP inside rows of 16 lanes, then
// v_permlane16_swap between the two rows of each 32-lane half.
template <int CTRL>
__device__ inline float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadXor1 = 0xB1;      // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;      // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;
constexpr int kRowRor4 = 0x124;
constexpr int kRowRor8 = 0x128;

// reduce across the 32 lanes of each half-wave; every lane gets the result
__device__ inline float half_max(float v) {
    v = fmaxf(v, dpp<kQuadXor1>(v));
    v = fmaxf(v, dpp<kQuadXor2>(v));
    v = fmaxf(v, dpp<kRowRor4>(v));
    v = fmaxf(v, dpp<kRowRor8>(v));
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float half_sum(float v) {
    v += dpp<kQuadXor1>(v);
    v += dpp<kQuadXor2>(v);
    v += dpp<kRowRor4>(v);
    v += dpp<kRowRor8>(v);
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// sum over aligned groups of G = 8 or 16 consecutive lanes; every lane gets it
template <int G>
__device__ inline float group_sum(float v) {
    v += dpp<kQuadXor1>(v);
    v += dpp<kQuadXor2>(v);
    v += dpp<kRowHalfMirror>(v);
    if constexpr (G == 16) v += dpp<kRowMirror>(v);
    return v;
}
// Sums of 16 values across the 32 lanes of each half-wave, one value kept per
// lane: the lanes exchange halves of their remaining values at each level
// (partners l ^ 16, l ^ 8, l ^ 7, l ^ 2, l ^ 1), so 38 instructions do what 16
// full reductions (96) would.  Afterwards lanes 2 t and 2 t + 1 of the half hold
// the total of value t.  Every value is summed over the same tree of lanes (the
// pairings are xor masks), whatever its index.
__device__ inline float half_sum16(const float (&v)[16], int l32) {
    float u[8], w[4], x[2];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        // lanes 0-15 keep value i, lanes 16-31 value i + 8
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]), __float_as_uint(v[i + 8]), false,
                                                        false);
        u[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    const bool b3 = (l32 & 8) != 0, b2 = (l32 & 4) != 0, b1 = (l32 & 2) != 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = (b3 ? u[j + 4] : u[j]) + dpp<kRowRor8>(b3 ? u[j] : u[j + 4]);
#pragma unroll
    for (int k = 0; k < 2; ++k) x[k] = (b2 ? w[k + 2] : w[k]) + dpp<kRowHalfMirror>(b2 ? w[k] : w[k + 2]);
    const float y = (b1 ? x[1] : x[0]) + dpp<kQuadXor2>(b1 ? x[0] : x[1]);
    return y + dpp<kQuadXor1>(y);
}

__device__ inline float wave_max(float v) {
    v = half_max(v);
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

}  // namespace tile
}  // namespace sa
