// Device-side modular arithmetic for primes q < 2^62 on gfx950.
//
// CDNA4 has no 64-bit integer multiplier: a 64x64-bit product is composed from
// 32x32-bit multiplies (v_mad_u64_u32 / v_mul_hi_u32 / v_mul_lo_u32).  The
// routines below are written so that each partial product maps onto one such
// instruction.
//
// * Shoup multiplication by a precomputed constant w (twiddles, conversion
//   constants): w' = floor(w 2^64 / q); for any a < 2^64,
//   a*w - floor(a*w'/2^64)*q lies in [0, 2q)  (Shoup 2007; Harvey 2014).
// * Products of two variables are accumulated exactly in 128 bits and reduced
//   once: x = hi*2^64 + lo = hi*[2^64]_q + lo (mod q), each term by a Shoup
//   multiplication, so a dot product of k terms costs one reduction.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

struct ModQ {
    uint64_t q;
    uint64_t twoq;
    uint64_t r64, r64s;   // 2^64 mod q and its Shoup companion
    uint64_t one_s;       // floor(2^64 / q): the Shoup companion of 1
    uint64_t ninv, ninvs; // N^-1 mod q and its Shoup companion
    uint64_t iw1n, iw1ns; // psi^-brev(1) N^-1 mod q (the inverse transform's last twiddle, N^-1 folded in), Shoup
    double qd, qinvd;     // q and fl(1/q) for the fp64 arithmetic (q < 2^50)
    double ninvd;         // N^-1 mod q as a double
};

__device__ __forceinline__ uint64_t mulhi64(uint64_t a, uint64_t b)
{
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t p00h = __umulhi(a0, b0);
    const uint64_t p01 = (uint64_t)a0 * b1 + p00h;              // < 2^64
    const uint64_t p10 = (uint64_t)a1 * b0 + (uint32_t)p01;     // < 2^64
    return (uint64_t)a1 * b1 + (p01 >> 32) + (p10 >> 32);       // < 2^64
}

__device__ __forceinline__ uint64_t csub(uint64_t x, uint64_t m) { return x >= m ? x - m : x; }

// a*w mod q in [0, 2q); any a < 2^64, w < q, ws = floor(w 2^64 / q).
__device__ __forceinline__ uint64_t shoup_lazy(uint64_t a, uint64_t w, uint64_t ws, uint64_t q)
{
    return a * w - mulhi64(a, ws) * q;
}
__device__ __forceinline__ uint64_t shoup(uint64_t a, uint64_t w, uint64_t ws, uint64_t q)
{
    return csub(shoup_lazy(a, w, ws, q), q);
}

struct acc128 {
    uint64_t lo, hi;
};
__device__ __forceinline__ void mac(acc128 &acc, uint64_t a, uint64_t b)
{
    const uint64_t lo = a * b;
    const uint64_t hi = mulhi64(a, b);
    acc.lo += lo;
    acc.hi += hi + (acc.lo < lo ? 1u : 0u);
}
// Exact x mod q for a 128-bit x, canonical result.
__device__ __forceinline__ uint64_t reduce128(acc128 x, const ModQ &m)
{
    const uint64_t a = shoup_lazy(x.hi, m.r64, m.r64s, m.q);   // [0, 2q)
    const uint64_t b = x.lo - mulhi64(x.lo, m.one_s) * m.q;     // [0, 2q)
    return csub(csub(a + b, m.twoq), m.q);
}
__device__ __forceinline__ uint64_t mulmod(uint64_t a, uint64_t b, const ModQ &m)
{
    acc128 x{0, 0};
    mac(x, a, b);
    return reduce128(x, m);
}
__device__ __forceinline__ uint64_t addmod(uint64_t a, uint64_t b, uint64_t q) { return csub(a + b, q); }
__device__ __forceinline__ uint64_t submod(uint64_t a, uint64_t b, uint64_t q) { return csub(a + q - b, q); }
