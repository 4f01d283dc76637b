// wave_impl.h -- wavefront-wide scans, reductions and broadcasts of the
// 64-lane wave on the DPP lane network (row shifts within 16-lane rows, the
// row-15 and row-31 broadcasts of the GFX9 encoding) and scalar lane reads,
// in place of LDS-routed permutes: each step is a register move with a lane
// pattern, a few cycles instead of an LDS round trip.
//
// Inclusive sum (Hillis-Steele within each row, then across rows): after
// row shifts by 1, 2, 4 and 8 every lane holds the sum of its row up to
// itself; broadcasting lane 15 into row 1 and lane 47 into row 3 extends
// rows 0-1 and 2-3 to 32-lane scans, and broadcasting lane 31 into rows 2
// and 3 completes the 64-lane scan.  Lanes that the pattern gives no
// source (or whose row it leaves out) take the `old` value: 0 for sums,
// the lane's own value for max and min (x op x = x).  Reductions end in
// lane 63 and are read from there into a scalar register, so every lane
// receives the same value.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gbt {

constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;

template <int kCtrl, int kRowMask>
__device__ inline uint32_t dpp32(uint32_t old, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, kCtrl, kRowMask, 0xf, false);
}

template <int kCtrl, int kRowMask>
__device__ inline uint64_t dpp64(uint64_t old, uint64_t v)
{
    const uint32_t lo = dpp32<kCtrl, kRowMask>((uint32_t)old, (uint32_t)v);
    const uint32_t hi = dpp32<kCtrl, kRowMask>((uint32_t)(old >> 32), (uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// A DPP move of a 32- or 64-bit value (integers, doubles).
template <int kCtrl, int kRowMask, typename T>
__device__ inline T dpp_move(T old, T v)
{
    static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit lane values");
    if constexpr (sizeof(T) == 8) {
        return __builtin_bit_cast(T, dpp64<kCtrl, kRowMask>(__builtin_bit_cast(uint64_t, old),
                                                             __builtin_bit_cast(uint64_t, v)));
    } else {
        return __builtin_bit_cast(T, dpp32<kCtrl, kRowMask>(__builtin_bit_cast(uint32_t, old),
                                                             __builtin_bit_cast(uint32_t, v)));
    }
}

// Lane `lane`'s value (lane uniform across the wave) in every lane.
template <typename T>
__device__ inline T wave_read(T v, int lane)
{
    static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit lane values");
    if constexpr (sizeof(T) == 8) {
        const uint64_t b = __builtin_bit_cast(uint64_t, v);
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
        return __builtin_bit_cast(T, ((uint64_t)hi << 32) | lo);
    } else {
        return __builtin_bit_cast(T, (uint32_t)__builtin_amdgcn_readlane((int)__builtin_bit_cast(uint32_t, v), lane));
    }
}

// Inclusive prefix sum over the wave's 64 lanes (all lanes active).
template <typename T>
__device__ inline T wave_incl_sum(T x)
{
    const T z = 0;
    x += dpp_move<kDppRowShr1, 0xf>(z, x);
    x += dpp_move<kDppRowShr2, 0xf>(z, x);
    x += dpp_move<kDppRowShr4, 0xf>(z, x);
    x += dpp_move<kDppRowShr8, 0xf>(z, x);
    x += dpp_move<kDppRowBcast15, 0xa>(z, x);
    x += dpp_move<kDppRowBcast31, 0xc>(z, x);
    return x;
}

// Sum over the wave, in every lane.
template <typename T>
__device__ inline T wave_total(T x)
{
    return wave_read(wave_incl_sum(x), 63);
}

// Maximum / minimum over the wave, in every lane (op(x, x) == x).
template <typename T, typename Op>
__device__ inline T wave_fold(T x, Op op)
{
    x = op(x, dpp_move<kDppRowShr1, 0xf>(x, x));
    x = op(x, dpp_move<kDppRowShr2, 0xf>(x, x));
    x = op(x, dpp_move<kDppRowShr4, 0xf>(x, x));
    x = op(x, dpp_move<kDppRowShr8, 0xf>(x, x));
    x = op(x, dpp_move<kDppRowBcast15, 0xa>(x, x));
    x = op(x, dpp_move<kDppRowBcast31, 0xc>(x, x));
    return wave_read(x, 63);
}

__device__ inline double wave_max_f64(double x)
{
    return wave_fold(x, [](double a, double b) { return fmax(a, b); });
}

template <typename T>
__device__ inline T wave_max(T x)
{
    return wave_fold(x, [](T a, T b) { return a > b ? a : b; });
}

template <typename T>
__device__ inline T wave_min(T x)
{
    return wave_fold(x, [](T a, T b) { return a < b ? a : b; });
}

}  // namespace gbt
