// wave_ops.h -- lane reductions and broadcasts inside aligned groups of
// 2..32 lanes of a 64-wide wavefront, on DPP where the pattern stays within a
// row of 16 lanes (no LDS round trip) and ds_bpermute otherwise.
//
// The reductions are butterflies over lane pairs that are symmetric (each
// pair adds the same two operands), so every lane of a group ends with a
// bitwise identical result.
#pragma once

#include <hip/hip_runtime.h>

namespace rgnn {

// DPP controls (gfx9 encoding)
constexpr int kDppQuadXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141; // lane i <-> 7 - i within each 8
constexpr int kDppRowMirror = 0x140;     // lane i <-> 15 - i within each 16

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum over the aligned group of W lanes containing this lane (W a power of 2, <= 32).
template <int W>
__device__ __forceinline__ float gsum(float x)
{
    static_assert(W >= 1 && W <= 32 && (W & (W - 1)) == 0, "group width");
    if (W >= 2) x += dpp_f<kDppQuadXor1>(x);
    if (W >= 4) x += dpp_f<kDppQuadXor2>(x);
    if (W >= 8) x += dpp_f<kDppRowHalfMirror>(x);
    if (W >= 16) x += dpp_f<kDppRowMirror>(x);
    if (W >= 32) x += __shfl_xor(x, 16, 32);
    return x;
}

template <int W>
__device__ __forceinline__ float gmax(float x)
{
    static_assert(W >= 1 && W <= 32 && (W & (W - 1)) == 0, "group width");
    if (W >= 2) x = fmaxf(x, dpp_f<kDppQuadXor1>(x));
    if (W >= 4) x = fmaxf(x, dpp_f<kDppQuadXor2>(x));
    if (W >= 8) x = fmaxf(x, dpp_f<kDppRowHalfMirror>(x));
    if (W >= 16) x = fmaxf(x, dpp_f<kDppRowMirror>(x));
    if (W >= 32) x = fmaxf(x, __shfl_xor(x, 16, 32));
    return x;
}

// Value of lane J (0..3) of this lane's quad.
template <int J>
__device__ __forceinline__ float quad_bcast(float x)
{
    return dpp_f<J * 0x55>(x);
}

}  // namespace rgnn
