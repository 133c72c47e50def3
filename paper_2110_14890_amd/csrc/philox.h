// philox.h -- Philox4x32-10 counter-based generator for gfx950 kernels.
//
// Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3",
// SC'11: a 4x32-bit counter is mixed by ten rounds, each two 32x32->64
// products (multipliers 0xD2511F53 and 0xCD9E8D57) whose high halves are
// XORed with the other counter words and the round key; the 2x32-bit key is
// bumped by the Weyl constants (0x9E3779B9, 0xBB67AE85) between rounds.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace smore {

enum : uint32_t { TAG_POS = 1u, TAG_NEG = 2u, TAG_SHARED = 3u };

struct U4 {
    uint32_t x, y, z, w;
};

__device__ __forceinline__ U4 philox4x32_10(U4 c, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        // one 32x32->64 product per multiplier (a single v_mad_u64_u32)
        const uint64_t pa = (uint64_t)0xD2511F53u * c.x;
        const uint64_t pb = (uint64_t)0xCD9E8D57u * c.z;
        U4 n;
        n.x = (uint32_t)(pb >> 32) ^ c.y ^ k0;
        n.y = (uint32_t)pb;
        n.z = (uint32_t)(pa >> 32) ^ c.w ^ k1;
        n.w = (uint32_t)pa;
        c = n;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c;
}

// 64-bit draw of stream `tag` for query id q, attempt t, index j: the first
// two output words of counter (j, t, q, tag) under key (seed low, seed high),
// first word low.
__device__ __forceinline__ uint64_t draw64(uint64_t seed, uint32_t tag, uint32_t q, uint32_t t,
                                           uint32_t j)
{
    const U4 o = philox4x32_10(U4{j, t, q, tag}, (uint32_t)seed, (uint32_t)(seed >> 32));
    return ((uint64_t)o.y << 32) | o.x;
}

// Reduce a 64-bit draw to [0, n): the high word of the 128-bit product u*n.
__device__ __forceinline__ uint32_t reduce_range(uint64_t u, uint32_t n)
{
    return (uint32_t)__umul64hi(u, (uint64_t)n);
}

}  // namespace smore
