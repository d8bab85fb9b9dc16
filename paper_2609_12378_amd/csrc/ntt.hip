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
// touch consecutive words.  Butterflies keep values lazily in [0, 4q)
// (Harvey 2014), so the only reductions are the Shoup products and one final
// correction; intermediate rows between the passes stay lazy.
#include "ckks_internal.h"

namespace {

constexpr int kE = 16;  // residues per thread

__device__ __forceinline__ void ct_bfly(uint64_t &X, uint64_t &Y, ulonglong2 w, uint64_t q, uint64_t twoq)
{
    const uint64_t x = csub(X, twoq);
    const uint64_t t = shoup_lazy(Y, w.x, w.y, q);
    X = x + t;
    Y = x + twoq - t;
}
__device__ __forceinline__ void gs_bfly(uint64_t &X, uint64_t &Y, ulonglong2 w, uint64_t q, uint64_t twoq)
{
    const uint64_t x = X, y = Y;
    X = csub(x + y, twoq);
    Y = shoup_lazy(x + twoq - y, w.x, w.y, q);
}

// Forward, top 4 stages of a sub-transform: x[k] is point u = r + TS*k.
__device__ __forceinline__ void fwd_top(uint64_t (&x)[kE], const ulonglong2 *tw, uint32_t B, uint64_t q, uint64_t twoq)
{
#pragma unroll
    for (int lm = 0; lm < 4; lm++) {
        const int mp = 1 << lm, tk = 8 >> lm;
#pragma unroll
        for (int g = 0; g < mp; g++) {
            const ulonglong2 w = tw[B * mp + g];
#pragma unroll
            for (int j = 0; j < tk; j++) ct_bfly(x[g * 2 * tk + j], x[g * 2 * tk + j + tk], w, q, twoq);
        }
    }
}
// Forward, remaining LOGS-4 stages: x[k] is point u = 16 r + k.
template <int LOGS>
__device__ __forceinline__ void fwd_low(uint64_t (&x)[kE], const ulonglong2 *tw, uint32_t B, uint32_t r, uint64_t q,
                                        uint64_t twoq)
{
#pragma unroll
    for (int l = 0; l < LOGS - 4; l++) {
        const int mp = 16 << l, t = (1 << LOGS) / (2 * mp), gpt = 8 / t;
#pragma unroll
        for (int g = 0; g < gpt; g++) {
            const ulonglong2 w = tw[B * mp + r * gpt + g];
#pragma unroll
            for (int j = 0; j < t; j++) ct_bfly(x[g * 2 * t + j], x[g * 2 * t + j + t], w, q, twoq);
        }
    }
}
template <int LOGS>
__device__ __forceinline__ void inv_low(uint64_t (&x)[kE], const ulonglong2 *tw, uint32_t B, uint32_t r, uint64_t q,
                                        uint64_t twoq)
{
#pragma unroll
    for (int l = LOGS - 5; l >= 0; l--) {
        const int mp = 16 << l, t = (1 << LOGS) / (2 * mp), gpt = 8 / t;
#pragma unroll
        for (int g = 0; g < gpt; g++) {
            const ulonglong2 w = tw[B * mp + r * gpt + g];
#pragma unroll
            for (int j = 0; j < t; j++) gs_bfly(x[g * 2 * t + j], x[g * 2 * t + j + t], w, q, twoq);
        }
    }
}
__device__ __forceinline__ void inv_top(uint64_t (&x)[kE], const ulonglong2 *tw, uint32_t B, uint64_t q, uint64_t twoq)
{
#pragma unroll
    for (int lm = 3; lm >= 0; lm--) {
        const int mp = 1 << lm, tk = 8 >> lm;
#pragma unroll
        for (int g = 0; g < mp; g++) {
            const ulonglong2 w = tw[B * mp + g];
#pragma unroll
            for (int j = 0; j < tk; j++) gs_bfly(x[g * 2 * tk + j], x[g * 2 * tk + j + tk], w, q, twoq);
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
template <int LOGS, bool A_TOP>
__device__ __forceinline__ void transpose(uint64_t (&x)[kE], uint64_t *lds, uint32_t sub, uint32_t r)
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

// Column pass over N1 = 2^LOGS points at stride N2 = 2^(log_n - LOGS).
template <int LOGS, bool INV>
__global__ __launch_bounds__(256) void ntt_col(uint64_t *data, LimbMap map, uint32_t batch, uint32_t bstride,
                                               const ModQ *mods,
                                               const ulonglong2 *tw_all, uint32_t log_n, uint32_t cols_per_block,
                                               uint32_t blocks_per_row)
{
    constexpr uint32_t TS = (1u << LOGS) / 16;
    extern __shared__ uint64_t lds[];
    uint32_t slot;
    const size_t row = row_of_block(blockIdx.x / blocks_per_row, batch, bstride, &slot);
    const uint32_t blk = blockIdx.x % blocks_per_row;
    const uint32_t prime = map.prime[slot];
    const ModQ m = mods[prime];
    const ulonglong2 *tw = tw_all + ((size_t)prime << log_n);
    const uint32_t n2 = 1u << (log_n - LOGS);
    uint64_t *base = data + (row << log_n) + (size_t)blk * cols_per_block;
    const uint32_t col = threadIdx.x % cols_per_block, r = threadIdx.x / cols_per_block;
    uint64_t x[kE];
    if (!INV) {
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = base[(size_t)(r + TS * k) * n2 + col];
        fwd_top(x, tw, 1, m.q, m.twoq);
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, col, r);
            fwd_low<LOGS>(x, tw, 1, r, m.q, m.twoq);
        }
#pragma unroll
        for (int k = 0; k < kE; k++) base[(size_t)(LOGS > 4 ? 16 * r + k : k) * n2 + col] = x[k];
    } else {
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = base[(size_t)(LOGS > 4 ? 16 * r + k : k) * n2 + col];
        if (LOGS > 4) {
            inv_low<LOGS>(x, tw, 1, r, m.q, m.twoq);
            transpose<LOGS, false>(x, lds, col, r);
        }
        inv_top(x, tw, 1, m.q, m.twoq);
        // the column pass is the last inverse pass: scale by N^-1 and make canonical
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = shoup(x[k], m.ninv, m.ninvs, m.q);
#pragma unroll
        for (int k = 0; k < kE; k++) base[(size_t)(r + TS * k) * n2 + col] = x[k];
    }
}

// Row pass over N2 = 2^LOGS contiguous points of row h, twiddle base N1 + h.
template <int LOGS, bool INV, bool LAST>
__global__ __launch_bounds__(256) void ntt_row(uint64_t *data, LimbMap map, uint32_t batch, uint32_t bstride,
                                               const ModQ *mods,
                                               const ulonglong2 *tw_all, uint32_t log_n, uint32_t rows_per_block,
                                               uint32_t blocks_per_poly)
{
    constexpr uint32_t S = 1u << LOGS, TS = S / 16;
    extern __shared__ uint64_t lds[];
    uint32_t slot;
    const size_t poly = row_of_block(blockIdx.x / blocks_per_poly, batch, bstride, &slot);
    const uint32_t blk = blockIdx.x % blocks_per_poly;
    const uint32_t prime = map.prime[slot];
    const ModQ m = mods[prime];
    const ulonglong2 *tw = tw_all + ((size_t)prime << log_n);
    const uint32_t n1 = 1u << (log_n - LOGS);
    const uint32_t sub = threadIdx.x / TS, r = threadIdx.x % TS;
    const uint32_t h = blk * rows_per_block + sub;
    uint64_t *base = data + (poly << log_n) + (size_t)h * S;
    const uint32_t B = n1 + h;
    uint64_t x[kE];
#pragma unroll
    for (int k = 0; k < kE; k++) x[k] = base[r + TS * k];
    if (!INV) {
        fwd_top(x, tw, B, m.q, m.twoq);
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, sub, r);
            fwd_low<LOGS>(x, tw, B, r, m.q, m.twoq);
        }
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = csub(csub(x[k], m.twoq), m.q);
        if (LOGS > 4) transpose<LOGS, false>(x, lds, sub, r);
    } else {
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, sub, r);
            inv_low<LOGS>(x, tw, B, r, m.q, m.twoq);
            transpose<LOGS, false>(x, lds, sub, r);
        }
        inv_top(x, tw, B, m.q, m.twoq);
        if (LAST) {
#pragma unroll
            for (int k = 0; k < kE; k++) x[k] = shoup(x[k], m.ninv, m.ninvs, m.q);
        }
    }
#pragma unroll
    for (int k = 0; k < kE; k++) base[r + TS * k] = x[k];
}

template <int LOGS>
size_t lds_bytes(uint32_t subs)
{
    return (size_t)subs * ((1u << LOGS) + (1u << LOGS) / 16 + 1) * sizeof(uint64_t);
}

template <int LOGS, bool INV>
hipError_t launch_col(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map,
                      const ulonglong2 *tw)
{
    const uint32_t n2 = 1u << (ctx->log_n - LOGS);
    const uint32_t TS = (1u << LOGS) / 16;
    uint32_t cols = 4096u >> LOGS;
    if (cols > n2) cols = n2;
    const uint32_t bpr = n2 / cols;
    const dim3 grid(batch * map.n * bpr), block(cols * TS);
    hipLaunchKernelGGL((ntt_col<LOGS, INV>), grid, block, lds_bytes<LOGS>(cols), ctx->stream, data, map, batch,
                       bstride, ctx->d_mod, tw, ctx->log_n, cols, bpr);
    return hipGetLastError();
}

template <int LOGS, bool INV, bool LAST>
hipError_t launch_row(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map,
                      const ulonglong2 *tw)
{
    const uint32_t n1 = 1u << (ctx->log_n - LOGS);
    const uint32_t TS = (1u << LOGS) / 16;
    uint32_t rows = 4096u >> LOGS;
    if (rows > n1) rows = n1;
    const uint32_t bpp = n1 / rows;
    const dim3 grid(batch * map.n * bpp), block(rows * TS);
    hipLaunchKernelGGL((ntt_row<LOGS, INV, LAST>), grid, block, lds_bytes<LOGS>(rows), ctx->stream, data, map,
                       batch, bstride, ctx->d_mod, tw, ctx->log_n, rows, bpp);
    return hipGetLastError();
}

template <bool INV>
hipError_t dispatch_col(int s1, ckks_ctx *ctx, uint64_t *d, uint32_t b, uint32_t bs, const LimbMap &m,
                        const ulonglong2 *tw)
{
    switch (s1) {
    case 4: return launch_col<4, INV>(ctx, d, b, bs, m, tw);
    case 5: return launch_col<5, INV>(ctx, d, b, bs, m, tw);
    case 6: return launch_col<6, INV>(ctx, d, b, bs, m, tw);
    case 7: return launch_col<7, INV>(ctx, d, b, bs, m, tw);
    case 8: return launch_col<8, INV>(ctx, d, b, bs, m, tw);
    }
    return hipErrorInvalidValue;
}
template <bool INV, bool LAST>
hipError_t dispatch_row(int s2, ckks_ctx *ctx, uint64_t *d, uint32_t b, uint32_t bs, const LimbMap &m,
                        const ulonglong2 *tw)
{
    switch (s2) {
    case 4: return launch_row<4, INV, LAST>(ctx, d, b, bs, m, tw);
    case 5: return launch_row<5, INV, LAST>(ctx, d, b, bs, m, tw);
    case 6: return launch_row<6, INV, LAST>(ctx, d, b, bs, m, tw);
    case 7: return launch_row<7, INV, LAST>(ctx, d, b, bs, m, tw);
    case 8: return launch_row<8, INV, LAST>(ctx, d, b, bs, m, tw);
    }
    return hipErrorInvalidValue;
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
    const int log_n = (int)ctx->log_n;
    int s1 = log_n > 8 ? log_n - 8 : 0;
    if (s1 > 0 && s1 < 4) s1 = 4;
    const int s2 = log_n - s1;
    hipError_t e = hipSuccess;
    const double bytes = 16.0 * batch * map.n * ctx->n;  // each pass reads and writes every residue
    if (!inverse) {
        if (s1) {
            prof_begin(ctx, K_NTT_FWD_COL, bytes);
            e = dispatch_col<false>(s1, ctx, data, batch, bstride, map, ctx->d_tw);
            prof_end(ctx, K_NTT_FWD_COL);
        }
        if (e == hipSuccess) {
            prof_begin(ctx, K_NTT_FWD_ROW, bytes);
            e = dispatch_row<false, true>(s2, ctx, data, batch, bstride, map, ctx->d_tw);
            prof_end(ctx, K_NTT_FWD_ROW);
        }
    } else {
        prof_begin(ctx, K_NTT_INV_ROW, bytes);
        if (s1)
            e = dispatch_row<true, false>(s2, ctx, data, batch, bstride, map, ctx->d_itw);
        else
            e = dispatch_row<true, true>(s2, ctx, data, batch, bstride, map, ctx->d_itw);
        prof_end(ctx, K_NTT_INV_ROW);
        if (e == hipSuccess && s1) {
            prof_begin(ctx, K_NTT_INV_COL, bytes);
            e = dispatch_col<true>(s1, ctx, data, batch, bstride, map, ctx->d_itw);
            prof_end(ctx, K_NTT_INV_COL);
        }
    }
    if (e != hipSuccess) return set_error(CKKS_EHIP, "ntt launch failed: %s", hipGetErrorString(e));
    return CKKS_OK;
}
