// Seed-expanded switching keys: the uniform half a_j of a key is a function of a 128-bit seed, generated where a
// kernel needs it instead of being read from HBM.  The generator is Philox-4x64-10 (Salmon, Moraes, Dror and Shaw,
// "Parallel random numbers: as easy as 1, 2, 3", SC 2011), counter-based, so any residue is computed on its own:
//
//   residue n (NTT-domain position) of prime index k in digit j: over the attempts t = 0, 1, ..., the word j mod 4
//   of the block Philox-4x64-10(counter (n, k, j / 4, t), key seed), w, gives the candidate w >> (64 - b), b the
//   bit length of q_k; the first candidate below q_k is the residue (rejection sampling), and after 64 rejections
//   (each of probability 1 - q/2^b < 1/2) the residue is w mod q_k.
//
// With the benchmark's primes (the largest b-bit primes that are 1 mod 2N) a rejection has probability below
// 2^-30, so the retries never run in practice; they are kept out of line.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace seedk {

__device__ __forceinline__ void philox4x64_10(uint64_t (&x)[4], uint64_t k0, uint64_t k1)
{
    constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t hi0 = __umul64hi(M0, x[0]), lo0 = M0 * x[0];
        const uint64_t hi1 = __umul64hi(M1, x[2]), lo1 = M1 * x[2];
        const uint64_t y0 = hi1 ^ x[1] ^ k0, y2 = hi0 ^ x[3] ^ k1;
        x[0] = y0;
        x[1] = lo1;
        x[2] = y2;
        x[3] = lo0;
    }
}

// word j of the attempts t >= 1 of block (n, k, jb): the rejection path
static __device__ __attribute__((noinline)) uint64_t retry_word(uint64_t s0, uint64_t s1, uint32_t n, uint32_t k,
                                                         uint32_t jb, int j, uint64_t q, uint32_t shift)
{
    uint64_t w = 0;
    for (uint64_t t = 1; t < 64; t++) {
        uint64_t x[4] = {n, k, jb, t};
        philox4x64_10(x, s0, s1);
        w = j == 0 ? x[0] : j == 1 ? x[1] : j == 2 ? x[2] : x[3];
        if ((w >> shift) < q) return w >> shift;
    }
    return w % q;
}

// The four residues of digits 4 jb .. 4 jb + 3 at position n of prime index k (modulus q); shift = 64 - bit length.
__device__ __forceinline__ void block_residues(uint64_t s0, uint64_t s1, uint32_t n, uint32_t k, uint32_t jb,
                                               uint64_t q, uint32_t shift, uint64_t (&a)[4])
{
    uint64_t x[4] = {n, k, jb, 0};
    philox4x64_10(x, s0, s1);
#pragma unroll
    for (int j = 0; j < 4; j++) {
        const uint64_t v = x[j] >> shift;
        a[j] = v < q ? v : retry_word(s0, s1, n, k, jb, j, q, shift);
    }
}

__device__ __forceinline__ uint32_t shift_of(uint64_t q) { return (uint32_t)__clzll((long long)q); }

}  // namespace seedk
