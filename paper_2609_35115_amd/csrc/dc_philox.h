// Counter-based generator shared by the device code: Philox4x64-10 and the
// map of 64 random bits to a uniform in (0, 1).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dc {

// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of two
// 64x64 -> 128-bit products, the key advanced by two Weyl constants between
// rounds.
struct Philox4 {
    uint64_t v[4];
};
__device__ __forceinline__ Philox4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0,
                                                 uint64_t k1)
{
    constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        const uint64_t p0_hi = __umul64hi(M0, c0), p0_lo = M0 * c0;
        const uint64_t p1_hi = __umul64hi(M1, c2), p1_lo = M1 * c2;
        const uint64_t n0 = p1_hi ^ c1 ^ k0, n2 = p0_hi ^ c3 ^ k1;
        c0 = n0;
        c1 = p1_lo;
        c2 = n2;
        c3 = p0_lo;
        k0 += W0;
        k1 += W1;
    }
    return Philox4{{c0, c1, c2, c3}};
}

// 64 random bits -> uniform in (0, 1): the top 53 bits, centred in their cell.
__device__ __forceinline__ double to_u01(uint64_t x) { return ((double)(x >> 11) + 0.5) * 0x1.0p-53; }

}  // namespace dc
