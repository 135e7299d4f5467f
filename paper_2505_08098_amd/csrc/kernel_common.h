// Device helpers shared by the forward and backward kernels (CDNA4, gfx950).
#pragma once

#include "f3s_internal.h"

namespace f3s {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s4 lds_s4;

// D(16x16, fp32) += A(16x32, fp16) * B(32x16, fp16).  Lane l holds A row
// l%16 and B column l%16 with 8 reduction slots chosen by l/16, and D rows
// 4(l/16)..+3 of column l%16 (layout probed on the GPU).
__device__ __forceinline__ f4 mfma16x16x32(h8 a, h8 b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// The same product with bfloat16 operands (raw 16-bit patterns in h8).
__device__ __forceinline__ f4 mfma16x16x32_bf16(h8 a, h8 b, f4 c)
{
    typedef __bf16 b8 __attribute__((ext_vector_type(8)));
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8, a),
                                                   __builtin_bit_cast(b8, b), c, 0, 0, 0);
}

__device__ __forceinline__ h8 load16(const _Float16 *p)
{
    return *reinterpret_cast<const h8 *>(p);
}

__device__ __forceinline__ h8 load16_off(const _Float16 *base, uint32_t byte_off)
{
    return *reinterpret_cast<const h8 *>(reinterpret_cast<const char *>(base) + byte_off);
}

// Transposed LDS read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane j of the group returns element k = 0..3 taken from the 8-byte chunk
// addressed by group lane 4k + j/4, at position j%4 of that chunk.  So if
// group lane s points at row (R + s/4), columns C + 4(s%4) .. +3 of a
// row-major fp16 tile, lane j receives rows R..R+3 of column C + j: one
// column of a 4 x 16 sub-tile, i.e. 4 reduction slots of an MFMA operand.
__device__ __forceinline__ h4 lds_read_tr(const _Float16 *p)
{
    return __builtin_bit_cast(h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)p));
}

// Max / sum of v over lanes l and l ^ 16, and over l and l ^ 32, with the
// cross-row swap instructions (VALU, no LDS round trip): called with the
// same value twice, v_permlane16_swap / v_permlane32_swap leave in each lane
// the pair {v[l], v[l ^ 16]} / {v[l], v[l ^ 32]} (checked on the GPU).
__device__ __forceinline__ float max_xor16(float v)
{
    const int b = __builtin_bit_cast(int, v);
    const auto r = __builtin_amdgcn_permlane16_swap(b, b, false, false);
    return fmaxf(__builtin_bit_cast(float, (int)r[0]), __builtin_bit_cast(float, (int)r[1]));
}
__device__ __forceinline__ float max_xor32(float v)
{
    const int b = __builtin_bit_cast(int, v);
    const auto r = __builtin_amdgcn_permlane32_swap(b, b, false, false);
    return fmaxf(__builtin_bit_cast(float, (int)r[0]), __builtin_bit_cast(float, (int)r[1]));
}

// Orders this wave's LDS accesses (one wave per workgroup).
__device__ __forceinline__ void wave_lds_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Orders one wave's accesses to its LDS tile.  With one wave per workgroup
// the workgroup barrier of wave_lds_fence does it; with several waves per
// workgroup (which run different numbers of block pairs) only this wave may
// take part: fences at wavefront scope around a wave barrier (a wave's LDS
// operations run in issue order, so only the compiler has to be held).
template <int NW>
__device__ __forceinline__ void tile_fence()
{
    if constexpr (NW == 1) {
        wave_lds_fence();
    } else {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
    }
}

// Position of this workgroup in the launch order: window-major (item * nh
// + head) or, with kOrderHead, head-major (head * items + item).
// Workgroups reach the 8 XCDs round-robin (workgroup b on XCD b mod 8).
// With kOrderXcd the XCDs cut a work list into consecutive ranges, so that
// neighbouring windows -- which share K/V rows on banded and block-diagonal
// patterns -- meet in one XCD's L2:
// - window-major with nh dividing 8: XCD x serves head x mod nh only, and the
//   8 / nh XCDs of a head split its list: XCD x takes items (its range's
//   first) + b / 8;
// - head-major (any nh): the heads' lists follow one another in launch
//   order, and within head h's list the workgroup with index t = b - h *
//   items takes item (range t mod 8's first) + t / 8: whatever XCD t mod 8
//   maps to for that head, each XCD walks one consecutive range per head.
// Each range gets exactly as many workgroups as it holds items, so the map is
// one-to-one.
__device__ __forceinline__ int workgroup_position(uint32_t order, int nh)
{
    int wg = (int)blockIdx.x;
    if (!(order & kOrderXcd) || nh < 1) return wg;
    const int n_it = (int)gridDim.x / nh;
    if (order & kOrderHead) {
        const int h = wg / n_it, t = wg - h * n_it;
        const int q = n_it >> 3, r = n_it & 7, y = t & 7;
        return h * n_it + y * q + min(y, r) + (t >> 3);
    }
    if (8 % nh != 0) return wg;
    const int x = wg & 7, per = 8 / nh, h = x % nh, k = x / nh;
    const int q = n_it / per, r = n_it % per;
    return (k * q + min(k, r) + (wg >> 3)) * nh + h;
}

__device__ __forceinline__ h8 cat44(h4 lo, h4 hi)
{
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

}  // namespace f3s
