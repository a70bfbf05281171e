// Device helpers shared by the matrix-core kernels (gfx950): bf16 packing, the
// LDS tile layout, and operand loads for v_mfma_f32_32x32x16_bf16.
//
// MFMA 32x32x16 bf16 register layouts (checked on the device):
//   A operand: lane l holds row l%32, k = (l/32)*8 + 0..7
//   B operand: lane l holds col l%32, k = (l/32)*8 + 0..7
//   C/D      : lane l holds col l%32, rows 8*(r/4) + 4*(l/32) + r%4, r = 0..15
// A C tile read back as the k slots of a following contraction visits its rows
// in the order perm16 (swap bits 2 and 3 of the row index inside each 16-group).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {
namespace tile {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// two fp32 -> packed bf16x2 (round to nearest even), first value in the low half
__device__ inline uint32_t pack_bf16x2(float a, float b) {
    bf16x2 v = __builtin_convertvector((f32x2){a, b}, bf16x2);
    return __builtin_bit_cast(uint32_t, v);
}
__device__ inline uint16_t to_bf16(float a) { return (uint16_t)(pack_bf16x2(a, 0.f) & 0xffffu); }

__device__ inline bf16x8 pack8(const float* e) {
    uint4 pk;
    pk.x = pack_bf16x2(e[0], e[1]);
    pk.y = pack_bf16x2(e[2], e[3]);
    pk.z = pack_bf16x2(e[4], e[5]);
    pk.w = pack_bf16x2(e[6], e[7]);
    return __builtin_bit_cast(bf16x8, pk);
}

// 8 bf16 (one 16-byte chunk) times a scalar, rounded back to bf16
__device__ inline uint4 scale8(uint4 v, float f) {
    uint4 r;
    r.x = pack_bf16x2(bf16_lo(v.x) * f, bf16_hi(v.x) * f);
    r.y = pack_bf16x2(bf16_lo(v.y) * f, bf16_hi(v.y) * f);
    r.z = pack_bf16x2(bf16_lo(v.z) * f, bf16_hi(v.z) * f);
    r.w = pack_bf16x2(bf16_lo(v.w) * f, bf16_hi(v.w) * f);
    return r;
}

// Work-list range of workgroup b out of n.  The dispatcher deals workgroups to
// the 8 XCDs round-robin (b % 8), each with its own L2; this gives the
// workgroups of one XCD consecutive ranges (same head, mostly the same users), so
// the prototype and dY blocks they stream are shared in that L2.  XCD x takes
// ranges [x*q + min(x, n%8), ...) with q = n/8, one more when x < n%8: a
// bijection of [0, n).
__device__ inline int64_t xcd_range(int64_t b, int64_t n) {
    const int64_t q = n / 8, rem = n % 8, x = b % 8, i = b / 8;
    return x * q + (x < rem ? x : rem) + i;
}

__device__ inline int perm16(int t) { return (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1); }

// row of a C tile held by register r of lane-half hl
__device__ inline int srow(int r, int hl) { return 8 * (r >> 2) + 4 * hl + (r & 3); }

// LDS element offset of 16-byte chunk c of row r of a row-major bf16 tile with
// COLS columns.  The chunk index is XORed with a permutation of the low row bits
// such that an operand read (32 consecutive rows, one chunk each, ds_read_b128)
// and the transposing 8-byte reads of lds_tr_tokens touch each bank once per 16
// lanes; a plain row layout costs two passes per read.
template <int COLS>
__device__ inline int swz_x(int r) {
    if constexpr (COLS == 32) {
        return (r >> 2) & 3;
    } else if constexpr (COLS == 64) {
        return (r & 6) | ((r >> 3) & 1);
    } else {
        static_assert(COLS == 128, "tile width");
        return ((r & 3) << 1) | ((r & 4) << 1) | ((r >> 3) & 1);
    }
}
template <int COLS>
__device__ inline int swz(int r, int c) {
    return r * COLS + ((c ^ swz_x<COLS>(r)) << 3);
}

// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4): lane l
// of the wave writes LDS bytes [16 l, 16 l + 16) after `lds_base` (wave-uniform).
// Completion is tracked by vmcnt; wait for it before the barrier that publishes
// the data.
__device__ inline void load_lds16(const void* src, void* lds_base) {
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)(src),
                                     (void __attribute__((address_space(3)))*)(lds_base), 16, 0, 0);
}
__device__ inline void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations,
// then s_barrier.  Unlike __syncthreads(), which also waits for every
// outstanding global load (vmcnt(0)), loads issued into registers ahead of time
// stay in flight across it; their uses wait for them as usual.  Not for data
// that global_load_lds writes into LDS (wait_vmem() first for that).
__device__ inline void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Lanes of one wave reading LDS words that other lanes of the same wave wrote
// just before: the wave's LDS operations execute in program order, so only the
// compiler has to be kept from moving the reads above the (lane-predicated)
// writes or forwarding a lane's own stored values past them.
__device__ inline void wave_lds_order() { asm volatile("" ::: "memory"); }

__device__ inline bf16x8 lds_b128(const uint16_t* base, int off) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(base + off));
}

// B operand (k = 16 tokens, n = 32 columns) of a contraction over the tokens of
// a row-major [32 tokens][D] LDS tile (layout swz<D>): column block jt, token half
// h2 (tokens 16*h2 .. 16*h2+15), k slots in the perm16 token order of an A operand
// built from a C tile.  It uses the gfx950 transposing load ds_read_b64_tr_b16:
// inside each group of 16 lanes, lane i receives element i%4 of the 8-byte rows
// addressed by lanes 4e + i/4, e = 0..3.  Two such loads (token rows 4*hl + s/4
// and 8 further) give the 8 k slots of the lane.
template <int D>
__device__ inline bf16x8 lds_tr_tokens(const uint16_t* tile, int lane, int jt, int h2) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    typedef __attribute__((address_space(3))) short lds_short;
    const int s = lane & 15, jg = (lane >> 4) & 1, hl = lane >> 5;
    const int col = jt * 32 + 16 * jg + 4 * (s & 3);
    const int row = 16 * h2 + 4 * hl + (s >> 2);
    lds_short* base = (lds_short*)(const_cast<uint16_t*>(tile));
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_s16x4*)(base + swz<D>(row, col >> 3) + (col & 7)));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_s16x4*)(base + swz<D>(row + 8, col >> 3) + (col & 7)));
    const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
}

}  // namespace tile
}  // namespace sa
