// Wave-wide digit match for the stable ranking of the radix sorts and the
// bucketed tile order: for each item, the lanes whose item holds the same
// digit.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tgs {

// peers[g] enters as the lanes taking part (a subset of the active lanes)
// and leaves as those of them whose digit dg[g] equals this lane's, matched
// over the low nbits bits (nbits block-uniform, at most 8; every digit below
// 2^nbits).  Per bit and item, one ballot z of the lanes whose bit is clear:
// the lanes sharing this lane's bit are z, or its complement where the bit is
// set (z xor the bit spread over 32 bits, one three-input bit operation per
// half with the and).  The G items' ballots are independent, so they issue
// back to back.
template <int G>
__device__ inline void match_digits(const uint32_t (&dg)[G], int nbits, uint64_t (&peers)[G]) {
    uint32_t pl[G], ph[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        pl[g] = (uint32_t)peers[g];
        ph[g] = (uint32_t)(peers[g] >> 32);
    }
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        if (b < nbits) {   // uniform
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const uint32_t sb = (uint32_t)((int32_t)(dg[g] << (31 - b)) >> 31);
                const uint64_t z = __ballot(sb == 0u);
                pl[g] &= (uint32_t)z ^ sb;
                ph[g] &= (uint32_t)(z >> 32) ^ sb;
            }
        }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) peers[g] = (uint64_t)ph[g] << 32 | pl[g];
}

}  // namespace tgs
