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

// Global accesses of data that a pass reads or writes exactly once, with the nontemporal hint: streamed rows do
// not displace reused data (twiddle tables, keys) from the caches, and a copy kernel moves measurably more bytes
// per second on gfx950 with the hint than without it.
__device__ __forceinline__ uint64_t ld_stream(const uint64_t *p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_stream(uint64_t *p, uint64_t v) { __builtin_nontemporal_store(v, p); }

template <bool F>
struct Ar;

template <>
struct Ar<false> {
    using E = uint64_t;
    using W = ulonglong2;
    uint64_t q, twoq, ninv, ninvs, iw1n, iw1ns;
    __device__ explicit Ar(const ModQ &m)
        : q(m.q), twoq(m.twoq), ninv(m.ninv), ninvs(m.ninvs), iw1n(m.iw1n), iw1ns(m.iw1ns)
    {
    }
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
    // the last Gentleman-Sande stage of an inverse transform (its twiddle is psi^-brev(1)) times N^-1, canonical:
    // X' = (X + Y) N^-1, Y' = (X - Y) psi^-brev(1) N^-1, from X, Y in [0, 2q)
    __device__ void gs_scaled(E &X, E &Y) const
    {
        const uint64_t x = X, y = Y;
        X = shoup(x + y, ninv, ninvs, q);
        Y = shoup(x + twoq - y, iw1n, iw1ns, q);
    }
};

template <>
struct Ar<true> {
    using E = double;
    using W = double;
    double q, qinv, ninv;
    __device__ explicit Ar(const ModQ &m) : q(m.qd), qinv(m.qinvd), ninv(m.ninvd) {}
    __device__ Ar() : q(0.0), qinv(0.0), ninv(0.0) {}
    // v < 2^52 (every residue): 2^52 + v has the bits of 2^52 with v in its mantissa
    __device__ static E from_u64(uint64_t v)
    {
        return __longlong_as_double((long long)(v | 0x4330000000000000ull)) - 4503599627370496.0;
    }
    __device__ static E from_raw(uint64_t v) { return __longlong_as_double((long long)v); }
    __device__ static uint64_t to_raw(E x) { return (uint64_t)__double_as_longlong(x); }
    // |x| < 2^53 -> x mod q, exact, |result| <= q/2 + 2^-52 |x| + 1
    __device__ E red(E x) const { return fma(-rint(x * qinv), q, x); }
    // 0 <= w < q, |a| <= 8q -> a w mod q, exact, |result| <= q/2 + 0.375 |a| (< 2q for |a| < 4q): the
    // estimate h/q of the quotient is at most |a| in size with relative error 2^-52, and |l| <= ulp(h)/2
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
        // the integer t in [0, q) is the mantissa of 2^52 + t (exact below 2^52)
        return (uint64_t)__double_as_longlong(t + 4503599627370496.0) & 0x000FFFFFFFFFFFFFull;
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
    // |X|, |Y| < 2q -> |X'|, |Y'| < 2q; in general |X'|, |Y'| <= q + 0.375 |Y|
    __device__ void ct(E &X, E &Y, W w) const
    {
        const double x = red(X);
        const double r = mul(Y, w);
        X = x + r;
        Y = x - r;
    }
    // the same without the range reduction of X: |X'|, |Y'| <= |X| + |mul(Y, w)|
    __device__ void ct_lazy(E &X, E &Y, W w) const
    {
        const double r = mul(Y, w);
        const double x = X;
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
    // w * N^-1 mod q in [0, q), for the last inverse stage with the scaling folded in (w canonical)
    __device__ double scaled_twiddle(double w) const
    {
        double t = mul(w, ninv);
        t = t < 0.0 ? t + q : t;
        return t >= q ? t - q : t;
    }
    // the last Gentleman-Sande stage times N^-1: X' = (X + Y) N^-1, Y' = (X - Y) w N^-1 with wn = w N^-1 mod q
    __device__ void gs_scaled(E &X, E &Y, W wn) const
    {
        const double u = X + Y, v = X - Y;
        X = mul(u, ninv);
        Y = mul(v, wn);
    }
};

// One forward butterfly of stage s: with fp64 arithmetic a stage whose bit in RMASK is clear skips the range
// reduction of X (ct_lazy); the integer arithmetic keeps its own lazy range [0, 4q) and ignores the mask.
template <bool F, unsigned RMASK>
__device__ __forceinline__ void ct_stage(const Ar<F> &ar, int s, typename Ar<F>::E &X, typename Ar<F>::E &Y,
                                         typename Ar<F>::W w)
{
    if constexpr (F) {
        if ((RMASK >> s) & 1u)
            ar.ct(X, Y, w);
        else
            ar.ct_lazy(X, Y, w);
    } else {
        ar.ct(X, Y, w);
    }
}
// Forward, top 4 stages of a sub-transform: x[k] is point u = r + TS*k.
template <bool F, unsigned RMASK = 0xFFFFu>
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
            for (int j = 0; j < tk; j++) ct_stage<F, RMASK>(ar, lm, x[g * 2 * tk + j], x[g * 2 * tk + j + tk], w);
        }
    }
}
// Forward, remaining LOGS-4 stages: x[k] is point u = 16 r + k.
template <int LOGS, bool F, unsigned RMASK = 0xFFFFu>
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
            for (int j = 0; j < t; j++)
                ct_stage<F, RMASK>(ar, 4 + l, x[g * 2 * t + j], x[g * 2 * t + j + t], w);
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
// SCALED: the last stage also multiplies by N^-1 (gs_scaled), so the caller skips scale_n.  Only the last pass
// of an inverse transform passes SCALED, where B = 1 (its last stage's twiddle is psi^-brev(1)).
template <bool F, bool SCALED = false>
__device__ __forceinline__ void inv_top(typename Ar<F>::E (&x)[kE], const typename Ar<F>::W *tw, uint32_t B,
                                        const Ar<F> &ar)
{
#pragma unroll
    for (int lm = 3; lm >= 0; lm--) {
        const int mp = 1 << lm, tk = 8 >> lm;
#pragma unroll
        for (int g = 0; g < mp; g++) {
            const typename Ar<F>::W w = tw[B * mp + g];
            if constexpr (F && SCALED) {
                if (lm == 0) {
                    const double wn = ar.scaled_twiddle(w);
#pragma unroll
                    for (int j = 0; j < tk; j++) ar.gs_scaled(x[g * 2 * tk + j], x[g * 2 * tk + j + tk], wn);
                    continue;
                }
            }
            if constexpr (!F && SCALED) {
                if (lm == 0) {
#pragma unroll
                    for (int j = 0; j < tk; j++) ar.gs_scaled(x[g * 2 * tk + j], x[g * 2 * tk + j + tk]);
                    continue;
                }
            }
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

// ---- 256-point sub-transforms with 8 residues per thread (fp64 arithmetic) ----
//
// 32 threads hold one 256-point sub-transform, 8 points each, in three layouts
// (t: thread index within the sub-transform, k: register index):
//   A: u = t + 32 k                              register bits u7 u6 u5: stages 0-2
//   C: u = (t >> 2) << 5 | k << 2 | (t & 3)      register bits u4 u3 u2: stages 3-5
//   B: u = (k >> 2) << 7 | t << 2 | (k & 3)      register bits u7 u1 u0: stages 6-7
// Stage s pairs the points that differ in bit 7 - s, exactly as the 16-residue
// code above; group g of stage s (the top s bits of u) takes the twiddle
// tws[2^s + g], where tws is the sub-transform's table Psi[B 2^s + g] staged in
// LDS.  Half the residues of the 16-per-thread layout halve the registers a
// thread needs, so twice the waves fit on a SIMD.
// LDS addresses: the A -> C transpose XOR-swizzles u (conflict-free for both
// patterns), the C -> B one pads a word every 8 (C conflict-free, B at most
// two-way); kTr8 doubles per sub-transform.
//
// Lazy range reduction: a stage whose bit is clear in RMASK skips the
// reduction of X (ct_lazy).  Magnitudes, in units of q (q < 2^50): mul(a, w)
// returns |r| <= 0.5 + 0.375 |a| (the quotient estimate h/q, up to |a| q in
// size, carries a relative error of 2^-52, and |l| <= ulp(h)/2); red(x) returns
// <= 0.5 + 2^-52 |x|.  So a reducing stage maps a bound b on its inputs to
// 1 + 0.375 b and a lazy one to 1.375 b + 0.5.  The projection uses RMASK =
// 0x50 for the column pass (inputs reduced, <= 0.5; largest value 5.3, output
// <= 4.3) and 0xAA for the row pass (inputs <= 4.3; largest 6.4, output <= 2.6),
// then accumulates products of the outputs (each <= 1.5) four at a time onto a
// reduced sum: every value stays below 6.4 q < 2^53, so all arithmetic is exact
// integer arithmetic on doubles.  No pair of masks with fewer reducing stages
// in total keeps these bounds below 7.9 q.
constexpr int kE8 = 8;
constexpr uint32_t kTr8 = 287;
constexpr unsigned kColMask8 = 0x50, kRowMask8 = 0xAA;

template <int LAY>
__device__ __forceinline__ uint32_t u8(uint32_t t, int k)
{
    if (LAY == 0) return t + 32u * (uint32_t)k;
    if (LAY == 1) return ((t >> 2) << 5) | ((uint32_t)k << 2) | (t & 3u);
    return ((uint32_t)(k >> 2) << 7) | (t << 2) | (uint32_t)(k & 3);
}

// forward stage S on layout LAY (S in 0-2 for A, 3-5 for C, 6-7 for B)
template <int LAY, int S, bool RED = true>
__device__ __forceinline__ void fwd8_stage(double (&x)[kE8], const double *tws, uint32_t t, const Ar<true> &ar,
                                           uint32_t Bm = 1)
{
    constexpr int b = 7 - S;
    constexpr int rb = LAY == 0 ? b - 5 : LAY == 1 ? b - 2 : (b == 7 ? 2 : b);
    static_assert(rb >= 0 && rb < 3, "stage not in this layout");
#pragma unroll
    for (int k = 0; k < kE8; k++) {
        if (k & (1 << rb)) continue;
        const double w = tws[(1u << S) * Bm + (u8<LAY>(t, k) >> (b + 1))];
        if (RED)
            ar.ct(x[k], x[k | (1 << rb)], w);
        else
            ar.ct_lazy(x[k], x[k | (1 << rb)], w);
    }
}

__device__ __forceinline__ uint32_t pad_ac(uint32_t u) { return u ^ (((u >> 5) & 7u) << 2); }
__device__ __forceinline__ uint32_t pad_cb(uint32_t u) { return u + (u >> 3); }

struct NoHook {
    __device__ void operator()() const {}
};

// all eight forward stages of the sub-transform held by thread t (layout A in,
// layout B out), reducing X at the stages set in RMASK; tr: this sub-transform's
// kTr8 doubles of LDS; every thread of the block must call it (block barriers).
// hook() runs right after the first barrier: every thread has then finished the
// previous call's reads of the twiddle table, so a hook may refill a second
// table for the next call (three more barriers follow before this call returns).
template <unsigned RMASK, typename Hook = NoHook>
__device__ __forceinline__ void fwd8_256(double (&x)[kE8], const double *tws, double *tr, uint32_t t,
                                         const Ar<true> &ar, uint32_t Bm = 1, Hook hook = Hook())
{
    fwd8_stage<0, 0, (RMASK >> 0) & 1>(x, tws, t, ar, Bm);
    fwd8_stage<0, 1, (RMASK >> 1) & 1>(x, tws, t, ar, Bm);
    fwd8_stage<0, 2, (RMASK >> 2) & 1>(x, tws, t, ar, Bm);
#pragma unroll
    for (int k = 0; k < kE8; k++) tr[pad_ac(u8<0>(t, k))] = x[k];
    __syncthreads();
    hook();
#pragma unroll
    for (int k = 0; k < kE8; k++) x[k] = tr[pad_ac(u8<1>(t, k))];
    __syncthreads();
    fwd8_stage<1, 3, (RMASK >> 3) & 1>(x, tws, t, ar, Bm);
    fwd8_stage<1, 4, (RMASK >> 4) & 1>(x, tws, t, ar, Bm);
    fwd8_stage<1, 5, (RMASK >> 5) & 1>(x, tws, t, ar, Bm);
#pragma unroll
    for (int k = 0; k < kE8; k++) tr[pad_cb(u8<1>(t, k))] = x[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kE8; k++) x[k] = tr[pad_cb(u8<2>(t, k))];
    __syncthreads();
    fwd8_stage<2, 6, (RMASK >> 6) & 1>(x, tws, t, ar, Bm);
    fwd8_stage<2, 7, (RMASK >> 7) & 1>(x, tws, t, ar, Bm);
}

// layout B -> layout A through LDS (a word of padding every 32), so that
// consecutive lanes hold consecutive points again
__device__ __forceinline__ void b_to_a8(double (&x)[kE8], double *tr, uint32_t t)
{
#pragma unroll
    for (int k = 0; k < kE8; k++) tr[u8<2>(t, k) + (u8<2>(t, k) >> 5)] = x[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kE8; k++) x[k] = tr[u8<0>(t, k) + (u8<0>(t, k) >> 5)];
    __syncthreads();
}

// layout A -> layout B through LDS (the padding of b_to_a8)
__device__ __forceinline__ void a_to_b8(double (&x)[kE8], double *tr, uint32_t t)
{
#pragma unroll
    for (int k = 0; k < kE8; k++) tr[u8<0>(t, k) + (u8<0>(t, k) >> 5)] = x[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kE8; k++) x[k] = tr[u8<2>(t, k) + (u8<2>(t, k) >> 5)];
    __syncthreads();
}

// The inverse of fwd8_256 without the factor 1/256: Gentleman-Sande butterflies with a staged table of inverse
// twiddles (itws[2^s + g], as fwd8_256's table), stages 7 .. 0; layout B in, layout A out; every stage reduces,
// so inputs below 2q stay below 2q.  Every thread of the block must call it (block barriers).
template <int LAY, int S>
__device__ __forceinline__ void inv8_stage(double (&x)[kE8], const double *itws, uint32_t t, const Ar<true> &ar)
{
    constexpr int b = 7 - S;
    constexpr int rb = LAY == 0 ? b - 5 : LAY == 1 ? b - 2 : (b == 7 ? 2 : b);
    static_assert(rb >= 0 && rb < 3, "stage not in this layout");
#pragma unroll
    for (int k = 0; k < kE8; k++) {
        if (k & (1 << rb)) continue;
        ar.gs(x[k], x[k | (1 << rb)], itws[(1u << S) + (u8<LAY>(t, k) >> (b + 1))]);
    }
}

__device__ __forceinline__ void inv8_256(double (&x)[kE8], const double *itws, double *tr, uint32_t t,
                                         const Ar<true> &ar)
{
    inv8_stage<2, 7>(x, itws, t, ar);
    inv8_stage<2, 6>(x, itws, t, ar);
#pragma unroll
    for (int k = 0; k < kE8; k++) tr[pad_cb(u8<2>(t, k))] = x[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kE8; k++) x[k] = tr[pad_cb(u8<1>(t, k))];
    __syncthreads();
    inv8_stage<1, 5>(x, itws, t, ar);
    inv8_stage<1, 4>(x, itws, t, ar);
    inv8_stage<1, 3>(x, itws, t, ar);
#pragma unroll
    for (int k = 0; k < kE8; k++) tr[pad_ac(u8<1>(t, k))] = x[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kE8; k++) x[k] = tr[pad_ac(u8<0>(t, k))];
    __syncthreads();
    inv8_stage<0, 2>(x, itws, t, ar);
    inv8_stage<0, 1>(x, itws, t, ar);
    inv8_stage<0, 0>(x, itws, t, ar);
}

// twiddle table of a 256-point sub-transform with base B: tws[2^s + g] = Psi[B 2^s + g]
// for 1 <= 2^s + g < 256; filled by `nthreads` threads starting at thread `tid`
__device__ __forceinline__ void stage_twiddles8(double *tws, const double *tw, uint32_t B, uint32_t tid,
                                                uint32_t nthreads)
{
    for (uint32_t e = tid + 1; e < 256; e += nthreads) {
        const uint32_t m = 1u << (31 - __clz(e));
        tws[e] = tw[(size_t)B * m + (e - m)];
    }
}

}  // namespace nttc
