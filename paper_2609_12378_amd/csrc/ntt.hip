// Negacyclic NTT / INTT over rows of N = 2^log_n residues, batched over rows.
//
// Transform (textbook Cooley-Tukey with psi folded into the twiddles,
// Longa-Naehrig 2016): stage with m groups (m = 1, 2, ..., N/2), distance
// t = N/(2m), group i uses Psi[m + i] = psi^brev(m + i).  Output index j holds
// a(psi^(2 brev(j) + 1)).  The inverse runs Gentleman-Sande stages with
// psi^-brev(m + i) in the opposite order and multiplies by N^-1.
//
// MI355X mapping.  A 2^16-point row of uint64 is 512 KiB, more than a CU's
// LDS (160 KiB), so a row is split N = N1 * N2 (index x = h*N2 + c):
//  * column pass: the first log2(N1) stages only mix the high index bits h, so
//    each column c is an N1-point sub-transform with twiddles Psi[m' + i'];
//  * row pass: the remaining stages mix only c inside a row h, with twiddles
//    Psi[(N1 + h) m' + i'].
// Each sub-transform of S = 2^LOGS points is held by S/16 threads with 16
// residues each in registers: the top 4 stages run in registers, one LDS
// transpose (padded one word per 16 against bank conflicts) regroups 16
// consecutive points per thread, and the remaining LOGS-4 stages finish in
// registers.  Global loads and stores are arranged so that consecutive lanes
// touch consecutive words.
//
// Two exact arithmetics implement the butterflies:
//  * integer (any q < 2^62): Shoup products by the twiddles, values kept lazily
//    in [0, 4q) (Harvey 2014); about 37 VALU instructions per butterfly on
//    gfx950, where a 64-bit product is ten 32-bit multiplies;
//  * fp64 (q < 2^50): residues held as exact integer-valued doubles in (-2q, 2q).
//    a*w = h + l exactly (h = fl(a w), l = fma(a, w, -h)); c = rint(h / q) is
//    within 1.5 of a w / q, so r = fma(-c, q, h) + l = a w - c q is exact and
//    |r| < 2q; a range reduction x - q rint(x / q) keeps every stage input below
//    2q.  About 11 full-rate fp64 instructions per butterfly.  Exactness: with
//    |a| < 4q < 2^52 and w < q < 2^50, |a w| < 2^102 so |l| <= 2^49, and
//    |h - c q| <= 2q + 2^49 < 2^52: every intermediate is an integer below 2^53.
// Between the two passes the row holds lazy values (integer) or raw double
// bits (fp64); the last pass writes canonical residues in [0, q).
#include <type_traits>

#include "ckks_internal.h"
#include "ops.h"

namespace {

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

__device__ __forceinline__ size_t row_of_block(uint32_t blk_row, uint32_t batch, uint32_t bstride,
                                               uint32_t *prime_slot)
{
    // blocks are ordered limb-major so that concurrent blocks share one twiddle table
    const uint32_t limb = blk_row / batch, b = blk_row % batch;
    *prime_slot = limb;
    return (size_t)b * bstride + limb;
}

template <bool F>
__device__ __forceinline__ const typename Ar<F>::W *twp(const void *tw_all, uint32_t prime, uint32_t log_n)
{
    return (const typename Ar<F>::W *)tw_all + ((size_t)prime << log_n);
}

// Column pass over N1 = 2^LOGS points at stride N2 = 2^(log_n - LOGS).
// Forward: first pass (canonical input).  Inverse: last pass (N^-1, canonical output).
template <int LOGS, bool INV, bool F>
__global__ __launch_bounds__(256) void ntt_col(uint64_t *data, LimbMap map, uint32_t batch, uint32_t bstride,
                                               const ModQ *mods, const void *tw_all, uint32_t log_n,
                                               uint32_t cols_per_block, uint32_t blocks_per_row)
{
    using E = typename Ar<F>::E;
    constexpr uint32_t TS = (1u << LOGS) / 16;
    extern __shared__ uint64_t lds_raw[];
    E *lds = (E *)lds_raw;
    uint32_t slot;
    const size_t row = row_of_block(blockIdx.x / blocks_per_row, batch, bstride, &slot);
    const uint32_t blk = blockIdx.x % blocks_per_row;
    const uint32_t prime = map.prime[slot];
    const Ar<F> ar(mods[prime]);
    const typename Ar<F>::W *tw = twp<F>(tw_all, prime, log_n);
    const uint32_t n2 = 1u << (log_n - LOGS);
    uint64_t *base = data + (row << log_n) + (size_t)blk * cols_per_block;
    const uint32_t col = threadIdx.x % cols_per_block, r = threadIdx.x / cols_per_block;
    E x[kE];
    if (!INV) {
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = ar.from_u64(base[(size_t)(r + TS * k) * n2 + col]);
        fwd_top<F>(x, tw, 1, ar);
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, col, r);
            fwd_low<LOGS, F>(x, tw, 1, r, ar);
        }
#pragma unroll
        for (int k = 0; k < kE; k++) base[(size_t)(LOGS > 4 ? 16 * r + k : k) * n2 + col] = ar.to_raw(x[k]);
    } else {
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = ar.from_raw(base[(size_t)(LOGS > 4 ? 16 * r + k : k) * n2 + col]);
        if (LOGS > 4) {
            inv_low<LOGS, F>(x, tw, 1, r, ar);
            transpose<LOGS, false>(x, lds, col, r);
        }
        inv_top<F>(x, tw, 1, ar);
#pragma unroll
        for (int k = 0; k < kE; k++) base[(size_t)(r + TS * k) * n2 + col] = ar.to_canon(ar.scale_n(x[k]));
    }
}

// Forward column pass that starts from signed integer coefficients: block (b,
// column slice) loads its slice of m[b] once and, for each limb l < limbs in
// turn, reduces it modulo q_l and runs the column sub-transforms, writing
// out[b][l].  The RNS reduction of an encoded plaintext is thereby fused into
// the first NTT pass: the residues of all limbs never go through HBM before the
// transform.
template <int LOGS, bool F>
__global__ __launch_bounds__(256) void ntt_col_from_i64(const int64_t *__restrict__ m, uint64_t *out, uint32_t limbs,
                                                        const ModQ *mods, const void *tw_all, uint32_t log_n,
                                                        uint32_t cols_per_block, uint32_t blocks_per_row)
{
    using E = typename Ar<F>::E;
    constexpr uint32_t TS = (1u << LOGS) / 16;
    extern __shared__ uint64_t lds_raw[];
    E *lds = (E *)lds_raw;
    const uint32_t b = blockIdx.x / blocks_per_row, blk = blockIdx.x % blocks_per_row;
    const uint32_t n2 = 1u << (log_n - LOGS);
    const uint32_t col = threadIdx.x % cols_per_block, r = threadIdx.x / cols_per_block;
    const size_t coff = (size_t)blk * cols_per_block + col;
    const int64_t *src = m + ((size_t)b << log_n) + coff;
    int64_t v[kE];
#pragma unroll
    for (int k = 0; k < kE; k++) v[k] = src[(size_t)(r + TS * k) * n2];
    for (uint32_t l = 0; l < limbs; l++) {
        const ModQ md = mods[l];
        const Ar<F> ar(md);
        const typename Ar<F>::W *tw = twp<F>(tw_all, l, log_n);
        E x[kE];
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = ar.from_i64(v[k], md);
        fwd_top<F>(x, tw, 1, ar);
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, col, r);
            fwd_low<LOGS, F>(x, tw, 1, r, ar);
        }
        uint64_t *dst = out + (((size_t)b * limbs + l) << log_n) + coff;
#pragma unroll
        for (int k = 0; k < kE; k++) dst[(size_t)(LOGS > 4 ? 16 * r + k : k) * n2] = ar.to_raw(x[k]);
    }
}

// Row pass over N2 = 2^LOGS contiguous points of row h, twiddle base N1 + h.
// FIRST: input is canonical residues; LAST: write canonical residues (and, for
// the inverse, multiply by N^-1).
template <int LOGS, bool INV, bool FIRST, bool LAST, bool F>
__global__ __launch_bounds__(256) void ntt_row(uint64_t *data, LimbMap map, uint32_t batch, uint32_t bstride,
                                               const ModQ *mods, const void *tw_all, uint32_t log_n,
                                               uint32_t rows_per_block, uint32_t blocks_per_poly)
{
    using E = typename Ar<F>::E;
    constexpr uint32_t S = 1u << LOGS, TS = S / 16;
    extern __shared__ uint64_t lds_raw[];
    E *lds = (E *)lds_raw;
    uint32_t slot;
    const size_t poly = row_of_block(blockIdx.x / blocks_per_poly, batch, bstride, &slot);
    const uint32_t blk = blockIdx.x % blocks_per_poly;
    const uint32_t prime = map.prime[slot];
    const Ar<F> ar(mods[prime]);
    const typename Ar<F>::W *tw = twp<F>(tw_all, prime, log_n);
    const uint32_t n1 = 1u << (log_n - LOGS);
    const uint32_t sub = threadIdx.x / TS, r = threadIdx.x % TS;
    const uint32_t h = blk * rows_per_block + sub;
    uint64_t *base = data + (poly << log_n) + (size_t)h * S;
    const uint32_t B = n1 + h;
    E x[kE];
#pragma unroll
    for (int k = 0; k < kE; k++) {
        const uint64_t raw = base[r + TS * k];
        x[k] = FIRST ? ar.from_u64(raw) : ar.from_raw(raw);
    }
    if (!INV) {
        fwd_top<F>(x, tw, B, ar);
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, sub, r);
            fwd_low<LOGS, F>(x, tw, B, r, ar);
            transpose<LOGS, false>(x, lds, sub, r);
        }
    } else {
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, sub, r);
            inv_low<LOGS, F>(x, tw, B, r, ar);
            transpose<LOGS, false>(x, lds, sub, r);
        }
        inv_top<F>(x, tw, B, ar);
        if (LAST) {
#pragma unroll
            for (int k = 0; k < kE; k++) x[k] = ar.scale_n(x[k]);
        }
    }
#pragma unroll
    for (int k = 0; k < kE; k++) base[r + TS * k] = LAST ? ar.to_canon(x[k]) : ar.to_raw(x[k]);
}

template <int LOGS>
size_t lds_bytes(uint32_t subs)
{
    return (size_t)subs * ((1u << LOGS) + (1u << LOGS) / 16 + 1) * sizeof(uint64_t);
}

template <bool F>
const void *fwd_table(const ckks_ctx *c)
{
    return F ? (const void *)c->d_twf : (const void *)c->d_tw;
}
template <bool F>
const void *inv_table(const ckks_ctx *c)
{
    return F ? (const void *)c->d_itwf : (const void *)c->d_itw;
}

template <int LOGS, bool INV, bool F>
hipError_t launch_col(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map)
{
    const uint32_t n2 = 1u << (ctx->log_n - LOGS);
    const uint32_t TS = (1u << LOGS) / 16;
    uint32_t cols = 4096u >> LOGS;
    if (cols > n2) cols = n2;
    const uint32_t bpr = n2 / cols;
    const dim3 grid(batch * map.n * bpr), block(cols * TS);
    hipLaunchKernelGGL((ntt_col<LOGS, INV, F>), grid, block, lds_bytes<LOGS>(cols), ctx->stream, data, map, batch,
                       bstride, ctx->d_mod, INV ? inv_table<F>(ctx) : fwd_table<F>(ctx), ctx->log_n, cols, bpr);
    return hipGetLastError();
}

template <int LOGS, bool INV, bool FIRST, bool LAST, bool F>
hipError_t launch_row(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map)
{
    const uint32_t n1 = 1u << (ctx->log_n - LOGS);
    const uint32_t TS = (1u << LOGS) / 16;
    uint32_t rows = 4096u >> LOGS;
    if (rows > n1) rows = n1;
    const uint32_t bpp = n1 / rows;
    const dim3 grid(batch * map.n * bpp), block(rows * TS);
    hipLaunchKernelGGL((ntt_row<LOGS, INV, FIRST, LAST, F>), grid, block, lds_bytes<LOGS>(rows), ctx->stream, data,
                       map, batch, bstride, ctx->d_mod, INV ? inv_table<F>(ctx) : fwd_table<F>(ctx), ctx->log_n, rows,
                       bpp);
    return hipGetLastError();
}

template <int LOGS, bool F>
hipError_t launch_col_i64(ckks_ctx *ctx, const int64_t *m, uint64_t *out, uint32_t batch, uint32_t limbs)
{
    const uint32_t n2 = 1u << (ctx->log_n - LOGS);
    const uint32_t TS = (1u << LOGS) / 16;
    uint32_t cols = 4096u >> LOGS;
    if (cols > n2) cols = n2;
    const uint32_t bpr = n2 / cols;
    const dim3 grid(batch * bpr), block(cols * TS);
    hipLaunchKernelGGL((ntt_col_from_i64<LOGS, F>), grid, block, lds_bytes<LOGS>(cols), ctx->stream, m, out, limbs,
                       ctx->d_mod, fwd_table<F>(ctx), ctx->log_n, cols, bpr);
    return hipGetLastError();
}

#define NTT_SWITCH(s, CALL4, CALL5, CALL6, CALL7, CALL8)                                                            \
    switch (s) {                                                                                                   \
    case 4: return CALL4;                                                                                          \
    case 5: return CALL5;                                                                                          \
    case 6: return CALL6;                                                                                          \
    case 7: return CALL7;                                                                                          \
    case 8: return CALL8;                                                                                          \
    }                                                                                                              \
    return hipErrorInvalidValue;

template <bool INV, bool F>
hipError_t dispatch_col(int s1, ckks_ctx *ctx, uint64_t *d, uint32_t b, uint32_t bs, const LimbMap &m)
{
    NTT_SWITCH(s1, (launch_col<4, INV, F>(ctx, d, b, bs, m)), (launch_col<5, INV, F>(ctx, d, b, bs, m)),
               (launch_col<6, INV, F>(ctx, d, b, bs, m)), (launch_col<7, INV, F>(ctx, d, b, bs, m)),
               (launch_col<8, INV, F>(ctx, d, b, bs, m)))
}
template <bool INV, bool FIRST, bool LAST, bool F>
hipError_t dispatch_row(int s2, ckks_ctx *ctx, uint64_t *d, uint32_t b, uint32_t bs, const LimbMap &m)
{
    NTT_SWITCH(s2, (launch_row<4, INV, FIRST, LAST, F>(ctx, d, b, bs, m)),
               (launch_row<5, INV, FIRST, LAST, F>(ctx, d, b, bs, m)),
               (launch_row<6, INV, FIRST, LAST, F>(ctx, d, b, bs, m)),
               (launch_row<7, INV, FIRST, LAST, F>(ctx, d, b, bs, m)),
               (launch_row<8, INV, FIRST, LAST, F>(ctx, d, b, bs, m)))
}
template <bool F>
hipError_t dispatch_col_i64(int s1, ckks_ctx *ctx, const int64_t *m, uint64_t *out, uint32_t b, uint32_t limbs)
{
    NTT_SWITCH(s1, (launch_col_i64<4, F>(ctx, m, out, b, limbs)), (launch_col_i64<5, F>(ctx, m, out, b, limbs)),
               (launch_col_i64<6, F>(ctx, m, out, b, limbs)), (launch_col_i64<7, F>(ctx, m, out, b, limbs)),
               (launch_col_i64<8, F>(ctx, m, out, b, limbs)))
}

void split_log(int log_n, int *s1, int *s2)
{
    int a = log_n > 8 ? log_n - 8 : 0;
    if (a > 0 && a < 4) a = 4;
    *s1 = a;
    *s2 = log_n - a;
}

// the fp64 butterflies need every prime of the launch below 2^50
bool use_f64(const ckks_ctx *ctx, const LimbMap &map)
{
    if (ctx->int_only) return false;
    for (uint32_t i = 0; i < map.n; i++)
        if (!ctx->f64_ok[map.prime[i]]) return false;
    return true;
}

template <bool F>
hipError_t ntt_passes(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map,
                      bool inverse)
{
    int s1, s2;
    split_log((int)ctx->log_n, &s1, &s2);
    const double bytes = 16.0 * batch * map.n * ctx->n;  // each pass reads and writes every residue
    hipError_t e = hipSuccess;
    if (!inverse) {
        if (s1) {
            prof_begin(ctx, K_NTT_FWD_COL, bytes);
            e = dispatch_col<false, F>(s1, ctx, data, batch, bstride, map);
            prof_end(ctx, K_NTT_FWD_COL);
        }
        if (e == hipSuccess) {
            prof_begin(ctx, K_NTT_FWD_ROW, bytes);
            e = s1 ? dispatch_row<false, false, true, F>(s2, ctx, data, batch, bstride, map)
                   : dispatch_row<false, true, true, F>(s2, ctx, data, batch, bstride, map);
            prof_end(ctx, K_NTT_FWD_ROW);
        }
    } else {
        prof_begin(ctx, K_NTT_INV_ROW, bytes);
        e = s1 ? dispatch_row<true, true, false, F>(s2, ctx, data, batch, bstride, map)
               : dispatch_row<true, true, true, F>(s2, ctx, data, batch, bstride, map);
        prof_end(ctx, K_NTT_INV_ROW);
        if (e == hipSuccess && s1) {
            prof_begin(ctx, K_NTT_INV_COL, bytes);
            e = dispatch_col<true, F>(s1, ctx, data, batch, bstride, map);
            prof_end(ctx, K_NTT_INV_COL);
        }
    }
    return e;
}

}  // namespace

LimbMap limb_range(uint32_t first, uint32_t count)
{
    LimbMap m{};
    m.n = count;
    for (uint32_t i = 0; i < count && i < (uint32_t)kMaxLimbMap; i++) m.prime[i] = (uint8_t)(first + i);
    return m;
}

ckks_status launch_ntt(ckks_ctx *ctx, uint64_t *data, uint32_t rows, const LimbMap &map, bool inverse)
{
    if (rows == 0) return CKKS_OK;
    CK_REQUIRE(map.n > 0 && map.n <= (uint32_t)kMaxLimbMap && rows % map.n == 0, CKKS_EINVAL,
               "ntt: %u rows do not split into limb groups of %u", rows, map.n);
    return launch_ntt_strided(ctx, data, rows / map.n, map.n, map, inverse);
}

ckks_status launch_ntt_strided(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map,
                               bool inverse)
{
    if (batch == 0 || map.n == 0) return CKKS_OK;
    CK_REQUIRE(map.n <= (uint32_t)kMaxLimbMap && bstride >= map.n, CKKS_EINVAL, "ntt: bad limb map");
    const hipError_t e = use_f64(ctx, map) ? ntt_passes<true>(ctx, data, batch, bstride, map, inverse)
                                           : ntt_passes<false>(ctx, data, batch, bstride, map, inverse);
    if (e != hipSuccess) return set_error(CKKS_EHIP, "ntt launch failed: %s", hipGetErrorString(e));
    return CKKS_OK;
}

// Forward NTT of signed coefficient rows m[batch][N] into out[batch][limbs][N]
// over primes 0..limbs-1 (reduction fused into the first pass).
ckks_status launch_ntt_from_i64(ckks_ctx *ctx, const int64_t *m, uint64_t *out, uint32_t batch, uint32_t limbs)
{
    if (!batch || !limbs) return CKKS_OK;
    int s1, s2;
    split_log((int)ctx->log_n, &s1, &s2);
    if (s1 == 0) {
        // single-pass sizes: reduce, then transform
        CK_TRY(enc_to_rns(ctx, m, batch, limbs, out));
        return launch_ntt(ctx, out, batch * limbs, limb_range(0, limbs), false);
    }
    const LimbMap map = limb_range(0, limbs);
    const bool f = use_f64(ctx, map);
    hipError_t e;
    prof_begin(ctx, K_NTT_FWD_COL, 8.0 * batch * ctx->n * (1 + limbs));
    e = f ? dispatch_col_i64<true>(s1, ctx, m, out, batch, limbs) : dispatch_col_i64<false>(s1, ctx, m, out, batch, limbs);
    prof_end(ctx, K_NTT_FWD_COL);
    if (e == hipSuccess) {
        prof_begin(ctx, K_NTT_FWD_ROW, 16.0 * batch * limbs * ctx->n);
        e = f ? dispatch_row<false, false, true, true>(s2, ctx, out, batch, limbs, map)
              : dispatch_row<false, false, true, false>(s2, ctx, out, batch, limbs, map);
        prof_end(ctx, K_NTT_FWD_ROW);
    }
    if (e != hipSuccess) return set_error(CKKS_EHIP, "ntt launch failed: %s", hipGetErrorString(e));
    return CKKS_OK;
}
