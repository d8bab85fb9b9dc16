// Building blocks of the two-pass negacyclic NTT shared by the transform
// kernels and the fused projection kernel: the two exact butterfly arithmetics
// (integer Shoup, fp64 for primes below 2^50), the register-resident radix-16
// stage groups and the padded LDS transpose.  The transform itself, its
// factorisation N = N1 * N2 and the exactness bounds are described at the top
// of ntt.hip.
#pragma once
#include <hip/hip_runtime.h>

#include "modarith.h"

namespace nttc {

constexpr int kE = 16;  // residues per thread

template <bool F>
struct Ar;

template <>
struct Ar<false> {
    using E = uint64_t;
    using W = ulonglong2;
    uint64_t q, twoq, ninv, ninvs;
    __device__ explicit Ar(const ModQ &m) : q(m.q), twoq(m.twoq), ninv(m.ninv), ninvs(m.ninvs) {}
    __device__ E from_u64(uint64_t v) const { return v; }
    __device__ E from_raw(uint64_t v) const { return v; }
    __device__ uint64_t to_raw(E x) const { return x; }
    __device__ uint64_t to_canon(E x) const { return csub(csub(x, twoq), q); }  // from [0, 4q)
    __device__ E from_i64(int64_t v, const ModQ &m) const
    {
        const bool neg = v < 0;
        const uint64_t mag = neg ? (uint64_t)(-(v + 1)) + 1u : (uint64_t)v;
        const uint64_t r = csub(mag - mulhi64(mag, m.one_s) * m.q, m.q);
        return (neg && r) ? m.q - r : r;
    }
    // X, Y in [0, 4q) -> [0, 4q)
    __device__ void ct(E &X, E &Y, W w) const
    {
        const uint64_t x = csub(X, twoq);
        const uint64_t t = shoup_lazy(Y, w.x, w.y, q);
        X = x + t;
        Y = x + twoq - t;
    }
    // X, Y in [0, 2q) -> [0, 2q)
    __device__ void gs(E &X, E &Y, W w) const
    {
        const uint64_t x = X, y = Y;
        X = csub(x + y, twoq);
        Y = shoup_lazy(x + twoq - y, w.x, w.y, q);
    }
    __device__ E scale_n(E x) const { return shoup(x, ninv, ninvs, q); }
};

template <>
struct Ar<true> {
    using E = double;
    using W = double;
    double q, qinv, ninv;
    __device__ explicit Ar(const ModQ &m) : q(m.qd), qinv(m.qinvd), ninv(m.ninvd) {}
    __device__ static E from_u64(uint64_t v)
    {
        return (double)(uint32_t)(v >> 32) * 4294967296.0 + (double)(uint32_t)v;
    }
    __device__ static E from_raw(uint64_t v) { return __longlong_as_double((long long)v); }
    __device__ static uint64_t to_raw(E x) { return (uint64_t)__double_as_longlong(x); }
    // |x| < 2^52 -> |result| <= q/2 + 1
    __device__ E red(E x) const { return fma(-rint(x * qinv), q, x); }
    // |a| < 4q, 0 <= w < q -> a w mod q, exact, |result| < 2q
    __device__ E mul(E a, E w) const
    {
        const double h = a * w;
        const double l = fma(a, w, -h);
        const double c = rint(h * qinv);
        return fma(-c, q, h) + l;
    }
    __device__ uint64_t to_canon(E x) const
    {
        double t = fma(-floor(x * qinv), q, x);
        t = t < 0.0 ? t + q : t;
        t = t >= q ? t - q : t;
        const double hi = floor(t * (1.0 / 4294967296.0));
        const double lo = fma(-hi, 4294967296.0, t);
        return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
    }
    // exact for any int64: |v| <= 2^52 converts exactly; larger values are reduced as integers first
    __device__ E from_i64(int64_t v, const ModQ &m) const
    {
        if (v >= -(1ll << 52) && v <= (1ll << 52)) return red((double)v);
        const bool neg = v < 0;
        const uint64_t mag = neg ? (uint64_t)(-(v + 1)) + 1u : (uint64_t)v;
        const uint64_t r = csub(mag - mulhi64(mag, m.one_s) * m.q, m.q);
        return neg ? -(double)r : (double)r;
    }
    // |X|, |Y| < 2q -> |X'|, |Y'| < 2q
    __device__ void ct(E &X, E &Y, W w) const
    {
        const double x = red(X);
        const double r = mul(Y, w);
        X = x + r;
        Y = x - r;
    }
    __device__ void gs(E &X, E &Y, W w) const
    {
        const double u = X + Y, v = X - Y;
        X = red(u);
        Y = mul(v, w);
    }
    __device__ E scale_n(E x) const { return mul(x, ninv); }
};

// Forward, top 4 stages of a sub-transform: x[k] is point u = r + TS*k.
template <bool F>
__device__ __forceinline__ void fwd_top(typename Ar<F>::E (&x)[kE], const typename Ar<F>::W *tw, uint32_t B,
                                        const Ar<F> &ar)
{
#pragma unroll
    for (int lm = 0; lm < 4; lm++) {
        const int mp = 1 << lm, tk = 8 >> lm;
#pragma unroll
        for (int g = 0; g < mp; g++) {
            const typename Ar<F>::W w = tw[B * mp + g];
#pragma unroll
            for (int j = 0; j < tk; j++) ar.ct(x[g * 2 * tk + j], x[g * 2 * tk + j + tk], w);
        }
    }
}
// Forward, remaining LOGS-4 stages: x[k] is point u = 16 r + k.
template <int LOGS, bool F>
__device__ __forceinline__ void fwd_low(typename Ar<F>::E (&x)[kE], const typename Ar<F>::W *tw, uint32_t B,
                                        uint32_t r, const Ar<F> &ar)
{
#pragma unroll
    for (int l = 0; l < LOGS - 4; l++) {
        const int mp = 16 << l, t = (1 << LOGS) / (2 * mp), gpt = 8 / t;
#pragma unroll
        for (int g = 0; g < gpt; g++) {
            const typename Ar<F>::W w = tw[B * mp + r * gpt + g];
#pragma unroll
            for (int j = 0; j < t; j++) ar.ct(x[g * 2 * t + j], x[g * 2 * t + j + t], w);
        }
    }
}
template <int LOGS, bool F>
__device__ __forceinline__ void inv_low(typename Ar<F>::E (&x)[kE], const typename Ar<F>::W *tw, uint32_t B,
                                        uint32_t r, const Ar<F> &ar)
{
#pragma unroll
    for (int l = LOGS - 5; l >= 0; l--) {
        const int mp = 16 << l, t = (1 << LOGS) / (2 * mp), gpt = 8 / t;
#pragma unroll
        for (int g = 0; g < gpt; g++) {
            const typename Ar<F>::W w = tw[B * mp + r * gpt + g];
#pragma unroll
            for (int j = 0; j < t; j++) ar.gs(x[g * 2 * t + j], x[g * 2 * t + j + t], w);
        }
    }
}
template <bool F>
__device__ __forceinline__ void inv_top(typename Ar<F>::E (&x)[kE], const typename Ar<F>::W *tw, uint32_t B,
                                        const Ar<F> &ar)
{
#pragma unroll
    for (int lm = 3; lm >= 0; lm--) {
        const int mp = 1 << lm, tk = 8 >> lm;
#pragma unroll
        for (int g = 0; g < mp; g++) {
            const typename Ar<F>::W w = tw[B * mp + g];
#pragma unroll
            for (int j = 0; j < tk; j++) ar.gs(x[g * 2 * tk + j], x[g * 2 * tk + j + tk], w);
        }
    }
}

// padded LDS index of point u of sub-transform `sub`
template <int LOGS>
__device__ __forceinline__ uint32_t lidx(uint32_t sub, uint32_t u)
{
    return sub * ((1u << LOGS) + (1u << LOGS) / 16 + 1) + u + (u >> 4);
}

// write x[k] at points ua(k), barrier, read x[k] from points ub(k)
template <int LOGS, bool A_TOP, typename E>
__device__ __forceinline__ void transpose(E (&x)[kE], E *lds, uint32_t sub, uint32_t r)
{
    constexpr uint32_t TS = (1u << LOGS) / 16;
#pragma unroll
    for (int k = 0; k < kE; k++) lds[lidx<LOGS>(sub, A_TOP ? r + TS * k : 16 * r + k)] = x[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kE; k++) x[k] = lds[lidx<LOGS>(sub, A_TOP ? 16 * r + k : r + TS * k)];
    __syncthreads();
}

template <bool F>
__device__ __forceinline__ const typename Ar<F>::W *twp(const void *tw_all, uint32_t prime, uint32_t log_n)
{
    return (const typename Ar<F>::W *)tw_all + ((size_t)prime << log_n);
}

template <int LOGS>
size_t lds_bytes(uint32_t subs)
{
    return (size_t)subs * ((1u << LOGS) + (1u << LOGS) / 16 + 1) * sizeof(uint64_t);
}

}  // namespace nttc
