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
//    |r| < 2q; a range reduction x - q rint(x / q) keeps the stage inputs small.
//    About 11 full-rate fp64 instructions per butterfly, 8 where a forward stage
//    skips the reduction of X (fwd_col_mask, fwd_row_mask: values stay below 5q).
//    Exactness: with |a| < 8q < 2^53 and w < q < 2^50, |a w| < 2^103 so
//    |l| <= 2^50, and |h - c q| is a few q: every intermediate is an integer
//    below 2^53.  The inverse's last stage carries N^-1 (Ar<true>::gs_scaled).
// Between the two passes the row holds lazy values (integer) or raw double
// bits (fp64); the last pass writes canonical residues in [0, q).
#include <type_traits>

#include "ckks_internal.h"
#include "ntt_core.h"
#include "ops.h"

namespace {

using namespace nttc;

// Rows in memory order: consecutive blocks take consecutive limbs of one polynomial, then the next polynomial
// (limb-major order, which keeps one twiddle table hot, measured slower: its concurrent blocks touch rows a
// whole polynomial apart).
__device__ __forceinline__ size_t row_of_block(uint32_t blk_row, uint32_t limbs, uint32_t bstride,
                                               uint32_t *prime_slot)
{
    const uint32_t b = blk_row / limbs, limb = blk_row % limbs;
    *prime_slot = limb;
    return (size_t)b * bstride + limb;
}

// fp64 forward stages that skip the range reduction of X (bit s of the mask clear: stage s lazy).  In units of
// q a reducing stage maps a bound b on its values to 1 + 0.375 b and a lazy one to 1.375 b + 0.5 (Ar<true>).
// Column pass (canonical input, b = 1): every value below 3.7 q, output below 1.9 q (below 2 q for every LOGS,
// which the fused key-switching kernels that take a first pass's rows also assume); row pass after it (input
// below 2 q): values below 5 q before the canonical output; a single-pass transform (canonical input): below
// 4.8 q.  All stay below 8 q < 2^53, where the fp64 products are exact.  Half the stages or more are lazy at
// N = 2^16, 3 instructions saved per lazy butterfly.
// Indexed by log2 of the sub-transform size (4..8; smaller sizes do not occur).
constexpr unsigned kFwdColMask[9] = {0xff, 0xff, 0xff, 0xff, 0x0c, 0x1c, 0x34, 0x74, 0xd4};
constexpr unsigned kFwdRowMask[9] = {0xff, 0xff, 0xff, 0xff, 0x04, 0x14, 0x14, 0x54, 0x54};
constexpr unsigned kFwdSingleMask[9] = {0xff, 0xff, 0xff, 0xff, 0x08, 0x08, 0x28, 0x28, 0xa8};
constexpr unsigned fwd_col_mask(int logs) { return kFwdColMask[logs]; }
constexpr unsigned fwd_row_mask(int logs, bool first) { return first ? kFwdSingleMask[logs] : kFwdRowMask[logs]; }

// Sub-transforms per block of the column pass (16 columns of 256 points) and of the row pass (8 rows of 256).
constexpr uint32_t col_subs(int logs, int log_n)
{
    return (4096u >> logs) < (1u << (log_n - logs)) ? (4096u >> logs) : (1u << (log_n - logs));
}
constexpr uint32_t row_subs(int logs, int log_n)
{
    return (2048u >> logs) < (1u << (log_n - logs)) ? (2048u >> logs) : (1u << (log_n - logs));
}

// Column pass over N1 = 2^LOGS points at stride N2 = 2^(log_n - LOGS).
// Forward: first pass (canonical input).  Inverse: last pass (N^-1, canonical output).
// LOGN > 0: the ring degree is 2^LOGN at compile time (log_n, cols_per_block and blocks_per_row are then
// ignored), so every stride is a constant; 0: all from the arguments.
template <int LOGS, bool INV, bool F, int LOGN = 0>
__global__ __launch_bounds__(256) void ntt_col(uint64_t *data, LimbMap map, uint32_t bstride,
                                               const ModQ *mods, const void *tw_all, uint32_t log_n_arg,
                                               uint32_t cols_arg, uint32_t bpr_arg)
{
    using E = typename Ar<F>::E;
    constexpr uint32_t TS = (1u << LOGS) / 16;
    const uint32_t log_n = LOGN ? LOGN : log_n_arg;
    const uint32_t cols_per_block = LOGN ? col_subs(LOGS, LOGN) : cols_arg;
    const uint32_t blocks_per_row = LOGN ? (1u << (LOGN - LOGS)) / col_subs(LOGS, LOGN) : bpr_arg;
    extern __shared__ uint64_t lds_raw[];
    E *lds = (E *)lds_raw;
    uint32_t slot;
    const size_t row = row_of_block(blockIdx.x / blocks_per_row, map.n, bstride, &slot);
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
        for (int k = 0; k < kE; k++) x[k] = ar.from_u64(ld_stream(base + (size_t)(r + TS * k) * n2 + col));
        constexpr unsigned kMask = fwd_col_mask(LOGS);
        fwd_top<F, kMask>(x, tw, 1, ar);
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, col, r);
            fwd_low<LOGS, F, kMask>(x, tw, 1, r, ar);
        }
#pragma unroll
        for (int k = 0; k < kE; k++) st_stream(base + (size_t)(LOGS > 4 ? 16 * r + k : k) * n2 + col, ar.to_raw(x[k]));
    } else {
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = ar.from_raw(ld_stream(base + (size_t)(LOGS > 4 ? 16 * r + k : k) * n2 + col));
        if (LOGS > 4) {
            inv_low<LOGS, F>(x, tw, 1, r, ar);
            transpose<LOGS, false>(x, lds, col, r);
        }
        // N^-1 folded into the last stage
        inv_top<F, true>(x, tw, 1, ar);
#pragma unroll
        for (int k = 0; k < kE; k++) st_stream(base + (size_t)(r + TS * k) * n2 + col, ar.to_canon(x[k]));
    }
}

// Forward column pass that starts from signed integer coefficients: block (b,
// column slice) loads its slice of m[b] once and, for each limb l < limbs in
// turn, reduces it modulo q_l and runs the column sub-transforms, writing
// out[b][l].  The RNS reduction of an encoded plaintext is thereby fused into
// the first NTT pass: the residues of all limbs never go through HBM before the
// transform.
// Integer arithmetic: below every limb's prime in magnitude (weights at the usual scales), a wave's coefficients
// are their own residues (or q plus them), so the general reduction is skipped; `small` is the smallest q - 1.
template <int LOGS, bool F>
__global__ __launch_bounds__(256) void ntt_col_from_i64(const int64_t *__restrict__ m, uint64_t *out, uint32_t limbs,
                                                        const ModQ *mods, const void *tw_all, uint32_t log_n,
                                                        uint32_t cols_per_block, uint32_t blocks_per_row,
                                                        int64_t small)
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
    // fp64: coefficients within 2^52 are converted once for all limbs; a thread holding a larger one takes the
    // exact integer reduction for every limb, re-reading its coefficients
    double vd[kE];
    bool big = false;
    if constexpr (F) {
#pragma unroll
        for (int k = 0; k < kE; k++) {
            big |= v[k] > (1ll << 52) || v[k] < -(1ll << 52);
            vd[k] = (double)v[k];
        }
    }
    bool wide = false;
    if constexpr (!F) {
#pragma unroll
        for (int k = 0; k < kE; k++) wide |= v[k] > small || v[k] < -small;
    }
    const bool reduce = __any(wide);
    for (uint32_t l = 0; l < limbs; l++) {
        const ModQ md = mods[l];
        const Ar<F> ar(md);
        const typename Ar<F>::W *tw = twp<F>(tw_all, l, log_n);
        E x[kE];
        if constexpr (F) {
            if (!big) {
#pragma unroll
                for (int k = 0; k < kE; k++) x[k] = ar.red(vd[k]);
            } else {
                // an opaque copy of the pointer: the 16 addresses are formed here, not kept live across the loop
                auto sg = (const __attribute__((address_space(1))) int64_t *)src;
                asm volatile("" : "+v"(sg));
#pragma unroll
                for (int k = 0; k < kE; k++) x[k] = ar.from_i64(sg[(size_t)(r + TS * k) * n2], md);
            }
        } else if (!reduce) {
#pragma unroll
            for (int k = 0; k < kE; k++) x[k] = v[k] < 0 ? (uint64_t)v[k] + md.q : (uint64_t)v[k];
        } else {
#pragma unroll
            for (int k = 0; k < kE; k++) x[k] = ar.from_i64(v[k], md);
        }
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

// The same first pass for 256-point columns (N = 2^16) with 8 residues per
// thread and fp64 butterflies (nttc::fwd8_256): a block of 512 threads holds 16
// adjacent columns (consecutive lanes take consecutive columns, so every load
// and store moves 128-byte segments).  The twiddles of limb l+1 (Psi[1..255],
// shared by all columns) are staged into the idle half of a double-buffered LDS
// table while limb l is transformed.
__global__ __launch_bounds__(512) void ntt_col8_from_i64(const int64_t *__restrict__ m, uint64_t *out,
                                                         uint32_t limbs, const ModQ *mods, const double *twf,
                                                         uint32_t log_n, uint32_t blocks_per_row, int64_t small)
{
    using nttc::kE8;
    __shared__ double tws[2][256];
    __shared__ double tr[16][nttc::kTr8];
    const uint32_t b = blockIdx.x / blocks_per_row, blk = blockIdx.x % blocks_per_row;
    const uint32_t n2 = 1u << (log_n - 8);
    const uint32_t col = threadIdx.x & 15, t = threadIdx.x >> 4;
    const size_t coff = (size_t)blk * 16 + col;
    const int64_t *src = m + ((size_t)b << log_n) + coff;
    int64_t v[kE8];
#pragma unroll
    for (int k = 0; k < kE8; k++) v[k] = src[(size_t)nttc::u8<0>(t, k) * n2];
    double vd[kE8];
    bool big = false, wide = false;
#pragma unroll
    for (int k = 0; k < kE8; k++) {
        big |= v[k] > (1ll << 52) || v[k] < -(1ll << 52);
        wide |= v[k] > small || v[k] < -small;
        vd[k] = (double)v[k];
    }
    // coefficients below every limb's q/2 throughout the wave: the range reduction is the identity, skipped
    const bool reduce = __any(wide);
    if (threadIdx.x < 255) tws[0][threadIdx.x + 1] = twf[threadIdx.x + 1];
    __syncthreads();
    for (uint32_t l = 0; l < limbs; l++) {
        const ModQ md = mods[l];
        const Ar<true> ar(md);
        // next limb's twiddle, written to the other table after the first barrier of this limb (when every
        // thread has finished reading it for limb l - 1)
        double wnext = 0.0;
        if (l + 1 < limbs && threadIdx.x < 255) wnext = twf[((size_t)(l + 1) << log_n) + threadIdx.x + 1];
        double x[kE8];
        if (!reduce) {
#pragma unroll
            for (int k = 0; k < kE8; k++) x[k] = vd[k];
        } else if (!big) {
#pragma unroll
            for (int k = 0; k < kE8; k++) x[k] = ar.red(vd[k]);
        } else {
            auto sg = (const __attribute__((address_space(1))) int64_t *)src;
            asm volatile("" : "+v"(sg));
#pragma unroll
            for (int k = 0; k < kE8; k++) x[k] = ar.from_i64(sg[(size_t)nttc::u8<0>(t, k) * n2], md);
        }
        const double *tw = tws[l & 1];
        double *trc = tr[col];
        nttc::fwd8_stage<0, 0, (nttc::kColMask8 >> 0) & 1>(x, tw, t, ar);
        nttc::fwd8_stage<0, 1, (nttc::kColMask8 >> 1) & 1>(x, tw, t, ar);
        nttc::fwd8_stage<0, 2, (nttc::kColMask8 >> 2) & 1>(x, tw, t, ar);
#pragma unroll
        for (int k = 0; k < kE8; k++) trc[nttc::pad_ac(nttc::u8<0>(t, k))] = x[k];
        __syncthreads();
        if (l + 1 < limbs && threadIdx.x < 255) tws[(l + 1) & 1][threadIdx.x + 1] = wnext;
#pragma unroll
        for (int k = 0; k < kE8; k++) x[k] = trc[nttc::pad_ac(nttc::u8<1>(t, k))];
        __syncthreads();
        nttc::fwd8_stage<1, 3, (nttc::kColMask8 >> 3) & 1>(x, tw, t, ar);
        nttc::fwd8_stage<1, 4, (nttc::kColMask8 >> 4) & 1>(x, tw, t, ar);
        nttc::fwd8_stage<1, 5, (nttc::kColMask8 >> 5) & 1>(x, tw, t, ar);
#pragma unroll
        for (int k = 0; k < kE8; k++) trc[nttc::pad_cb(nttc::u8<1>(t, k))] = x[k];
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kE8; k++) x[k] = trc[nttc::pad_cb(nttc::u8<2>(t, k))];
        __syncthreads();
        nttc::fwd8_stage<2, 6, (nttc::kColMask8 >> 6) & 1>(x, tw, t, ar);
        nttc::fwd8_stage<2, 7, (nttc::kColMask8 >> 7) & 1>(x, tw, t, ar);
        uint64_t *dst = out + (((size_t)b * limbs + l) << log_n) + coff;
#pragma unroll
        for (int k = 0; k < kE8; k++) dst[(size_t)nttc::u8<2>(t, k) * n2] = Ar<true>::to_raw(x[k]);
    }
}

// Row pass over N2 = 2^LOGS contiguous points of row h, twiddle base N1 + h.
// FIRST: input is canonical residues; LAST: write canonical residues (and, for
// the inverse, multiply by N^-1).
// SHARE (N = 2^16, integer arithmetic): the block's 8 sub-transforms are the same row h of 8 consecutive batch
// entries of one limb, so they use the same twiddles (one table row read per block instead of eight); blocks run
// (batch octet, limb, h) in memory order.
template <int LOGS, bool INV, bool FIRST, bool LAST, bool F, int LOGN = 0, bool SHARE = false>
__global__ __launch_bounds__(LOGN ? 128 : 256) void ntt_row(uint64_t *data, LimbMap map, uint32_t bstride,
                                                             const ModQ *mods, const void *tw_all,
                                                             uint32_t log_n_arg, uint32_t rows_arg, uint32_t bpp_arg)
{
    using E = typename Ar<F>::E;
    constexpr uint32_t S = 1u << LOGS, TS = S / 16;
    const uint32_t log_n = LOGN ? LOGN : log_n_arg;
    const uint32_t rows_per_block = LOGN ? row_subs(LOGS, LOGN) : rows_arg;
    const uint32_t blocks_per_poly = LOGN ? (1u << (LOGN - LOGS)) / row_subs(LOGS, LOGN) : bpp_arg;
    // compile-time ring degree: the LDS of the block's rows is static (row_subs rows, padded)
    constexpr uint32_t kStatic = LOGN ? row_subs(LOGS, LOGN) * (S + S / 16 + 1) : 1;
    __shared__ E lds_static[kStatic];
    extern __shared__ uint64_t lds_raw[];
    E *lds = LOGN ? lds_static : (E *)lds_raw;
    uint32_t slot;
    size_t poly;
    uint32_t h;
    const uint32_t n1 = 1u << (log_n - LOGS);
    const uint32_t sub = threadIdx.x / TS, r = threadIdx.x % TS;
    if constexpr (SHARE) {
        static_assert(!SHARE || (LOGN == 16 && LOGS == 8), "shared-twiddle rows: N = 2^16 only");
        h = blockIdx.x % n1;
        const uint32_t rest = blockIdx.x / n1;
        slot = rest % map.n;
        poly = (size_t)(8 * (rest / map.n) + sub) * bstride + slot;
    } else {
        poly = row_of_block(blockIdx.x / blocks_per_poly, map.n, bstride, &slot);
        h = (blockIdx.x % blocks_per_poly) * rows_per_block + sub;
    }
    const uint32_t prime = map.prime[slot];
    const Ar<F> ar(mods[prime]);
    const typename Ar<F>::W *tw = twp<F>(tw_all, prime, log_n);
    uint64_t *base = data + (poly << log_n) + (size_t)h * S;
    const uint32_t B = n1 + h;
    E x[kE];
#pragma unroll
    for (int k = 0; k < kE; k++) {
        const uint64_t raw = ld_stream(base + r + TS * k);
        x[k] = FIRST ? ar.from_u64(raw) : ar.from_raw(raw);
    }
    if (!INV) {
        constexpr unsigned kMask = fwd_row_mask(LOGS, FIRST);
        fwd_top<F, kMask>(x, tw, B, ar);
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, sub, r);
            fwd_low<LOGS, F, kMask>(x, tw, B, r, ar);
            transpose<LOGS, false>(x, lds, sub, r);
        }
    } else {
        if (LOGS > 4) {
            transpose<LOGS, true>(x, lds, sub, r);
            inv_low<LOGS, F>(x, tw, B, r, ar);
            transpose<LOGS, false>(x, lds, sub, r);
        }
        // the last pass of an inverse folds N^-1 into its last stage (B = 1 there: a single-pass transform)
        inv_top<F, LAST>(x, tw, B, ar);
    }
#pragma unroll
    for (int k = 0; k < kE; k++) st_stream(base + r + TS * k, LAST ? ar.to_canon(x[k]) : ar.to_raw(x[k]));
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

// N = 2^16 (256 x 256) takes the variants with compile-time strides
template <int LOGS, bool INV, bool F>
hipError_t launch_col(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map)
{
    const uint32_t n2 = 1u << (ctx->log_n - LOGS);
    const uint32_t TS = (1u << LOGS) / 16;
    const uint32_t cols = col_subs(LOGS, (int)ctx->log_n);
    const uint32_t bpr = n2 / cols;
    const dim3 grid(batch * map.n * bpr), block(cols * TS);
    const void *tw = INV ? inv_table<F>(ctx) : fwd_table<F>(ctx);
    if (LOGS == 8 && ctx->log_n == 16)
        hipLaunchKernelGGL((ntt_col<LOGS, INV, F, 16>), grid, block, lds_bytes<LOGS>(cols), ctx->stream, data, map,
                           bstride, ctx->d_mod, tw, ctx->log_n, cols, bpr);
    else
        hipLaunchKernelGGL((ntt_col<LOGS, INV, F>), grid, block, lds_bytes<LOGS>(cols), ctx->stream, data, map,
                           bstride, ctx->d_mod, tw, ctx->log_n, cols, bpr);
    return hipGetLastError();
}

template <int LOGS, bool INV, bool FIRST, bool LAST, bool F>
hipError_t launch_row(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map)
{
    const uint32_t n1 = 1u << (ctx->log_n - LOGS);
    const uint32_t TS = (1u << LOGS) / 16;
    // 128 threads: smaller blocks stream measurably faster than 256
    const uint32_t rows = row_subs(LOGS, (int)ctx->log_n);
    const uint32_t bpp = n1 / rows;
    const dim3 grid(batch * map.n * bpp), block(rows * TS);
    const void *tw = INV ? inv_table<F>(ctx) : fwd_table<F>(ctx);
    if constexpr (LOGS == 8 && !F) {
        // integer arithmetic, batches of whole octets: each block's 8 rows share their (16-byte) twiddle pairs
        // (with the fp64 arithmetic the rows of one polynomial measured as fast, with 6% less fetch)
        if (ctx->log_n == 16 && batch % 8 == 0) {
            hipLaunchKernelGGL((ntt_row<LOGS, INV, FIRST, LAST, F, 16, true>), grid, block, 0, ctx->stream, data, map,
                               bstride, ctx->d_mod, tw, ctx->log_n, rows, bpp);
            return hipGetLastError();
        }
    }
    if (LOGS == 8 && ctx->log_n == 16)
        hipLaunchKernelGGL((ntt_row<LOGS, INV, FIRST, LAST, F, 16>), grid, block, 0, ctx->stream, data, map, bstride,
                           ctx->d_mod, tw, ctx->log_n, rows, bpp);
    else
        hipLaunchKernelGGL((ntt_row<LOGS, INV, FIRST, LAST, F>), grid, block, lds_bytes<LOGS>(rows), ctx->stream,
                           data, map, bstride, ctx->d_mod, tw, ctx->log_n, rows, bpp);
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
    uint64_t qmin = ~0ull;
    for (uint32_t l = 0; l < limbs; l++) qmin = ctx->primes[l] < qmin ? ctx->primes[l] : qmin;
    hipLaunchKernelGGL((ntt_col_from_i64<LOGS, F>), grid, block, lds_bytes<LOGS>(cols), ctx->stream, m, out, limbs,
                       ctx->d_mod, fwd_table<F>(ctx), ctx->log_n, cols, bpr, (int64_t)(qmin - 1));
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
    const double res = (double)batch * map.n * ctx->n;
    const double bytes = 16.0 * res;  // each pass reads and writes every residue
    // butterflies per residue: half the stages of the pass
    const double bf = F ? kOpsButterflyF64 : kOpsButterflyInt, ops1 = res * bf * s1 / 2, ops2 = res * bf * s2 / 2;
    hipError_t e = hipSuccess;
    if (!inverse) {
        if (s1) {
            prof_begin(ctx, K_NTT_FWD_COL, bytes, ops1);
            e = dispatch_col<false, F>(s1, ctx, data, batch, bstride, map);
            prof_end(ctx, K_NTT_FWD_COL);
        }
        if (e == hipSuccess) {
            prof_begin(ctx, K_NTT_FWD_ROW, bytes, ops2);
            e = s1 ? dispatch_row<false, false, true, F>(s2, ctx, data, batch, bstride, map)
                   : dispatch_row<false, true, true, F>(s2, ctx, data, batch, bstride, map);
            prof_end(ctx, K_NTT_FWD_ROW);
        }
    } else {
        prof_begin(ctx, K_NTT_INV_ROW, bytes, ops2);
        e = s1 ? dispatch_row<true, true, false, F>(s2, ctx, data, batch, bstride, map)
               : dispatch_row<true, true, true, F>(s2, ctx, data, batch, bstride, map);
        prof_end(ctx, K_NTT_INV_ROW);
        if (e == hipSuccess && s1) {
            prof_begin(ctx, K_NTT_INV_COL, bytes, ops1);
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

void ntt_split(uint32_t log_n, int *s1, int *s2) { split_log((int)log_n, s1, s2); }

// First (column) pass only of the forward transform of `batch` groups of map.n rows, fp64 butterflies; the rows
// are left as raw doubles for a fused second pass.  Needs a two-pass size and primes below 2^50.
ckks_status launch_ntt_fwd_first_pass(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride,
                                      const LimbMap &map)
{
    if (!batch || !map.n) return CKKS_OK;
    int s1, s2;
    split_log((int)ctx->log_n, &s1, &s2);
    CK_REQUIRE(s1 > 0 && use_f64(ctx, map), CKKS_EINVAL, "ntt: first pass alone needs two passes and fp64 primes");
    const double res = (double)batch * map.n * ctx->n;
    prof_begin(ctx, K_NTT_FWD_COL, 16.0 * res, res * kOpsButterflyF64 * s1 / 2);
    const hipError_t e = dispatch_col<false, true>(s1, ctx, data, batch, bstride, map);
    prof_end(ctx, K_NTT_FWD_COL);
    if (e != hipSuccess) return set_error(CKKS_EHIP, "ntt launch failed: %s", hipGetErrorString(e));
    return CKKS_OK;
}

// Second (column) pass only of the inverse transform of `batch` groups of map.n rows left by a fused first pass
// as raw doubles below 2q (fp64 primes, two-pass size): canonical coefficients out.
ckks_status launch_ntt_inv_second_pass(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride,
                                       const LimbMap &map)
{
    if (!batch || !map.n) return CKKS_OK;
    int s1, s2;
    split_log((int)ctx->log_n, &s1, &s2);
    CK_REQUIRE(s1 > 0 && use_f64(ctx, map), CKKS_EINVAL, "ntt: second pass alone needs two passes and fp64 primes");
    const double res = (double)batch * map.n * ctx->n;
    prof_begin(ctx, K_NTT_INV_COL, 16.0 * res, res * kOpsButterflyF64 * s1 / 2);
    const hipError_t e = dispatch_col<true, true>(s1, ctx, data, batch, bstride, map);
    prof_end(ctx, K_NTT_INV_COL);
    if (e != hipSuccess) return set_error(CKKS_EHIP, "ntt launch failed: %s", hipGetErrorString(e));
    return CKKS_OK;
}

bool ntt_uses_f64(const ckks_ctx *ctx, uint32_t limbs) { return use_f64(ctx, limb_range(0, limbs)); }

// The largest s such that the fp64 range reduction x - q rint(x / q) returns x itself for every |x| <= s and every
// prime q_0 .. q_{limbs-1}: |x| <= q/2 - 1.5 keeps |x / q| below 1/2 (with the rounding of 1/q), so rint gives 0.
int64_t identity_reduction_bound(const ckks_ctx *ctx, uint32_t limbs)
{
    uint64_t qmin = ~0ull;
    for (uint32_t l = 0; l < limbs; l++) qmin = ctx->primes[l] < qmin ? ctx->primes[l] : qmin;
    return limbs ? (int64_t)((qmin - 3) / 2) : 0;
}

// First (column) pass only of the forward NTT of m[batch][N] into out[batch][limbs][N]; the rows are left in the
// inter-pass form of the arithmetic ntt_uses_f64 selects.  Needs a two-pass size (s1 > 0).
ckks_status launch_ntt_col_i64(ckks_ctx *ctx, const int64_t *m, uint64_t *out, uint32_t batch, uint32_t limbs)
{
    if (!batch || !limbs) return CKKS_OK;
    int s1, s2;
    split_log((int)ctx->log_n, &s1, &s2);
    CK_REQUIRE(s1 > 0, CKKS_EINVAL, "ntt: a single-pass size has no column pass");
    const bool f = use_f64(ctx, limb_range(0, limbs));
    // butterflies of s1 stages plus the reduction of each coefficient (fp64: one range reduction); the 8-residue
    // kernel skips the reduction of X in 6 of its 8 stages (8 instead of 11 instructions)
    const double res = (double)batch * limbs * ctx->n;
    const double bf_ops = f && s1 == 8 ? (2 * kOpsButterflyF64 + 6 * (kOpsButterflyF64 - 3)) / 2
                                       : (f ? kOpsButterflyF64 : kOpsButterflyInt) * s1 / 2;
    prof_begin(ctx, K_NTT_FWD_COL, 8.0 * batch * ctx->n * (1 + limbs), res * (bf_ops + (f ? 3.0 : 8.0)));
    hipError_t e;
    if (f && s1 == 8) {
        const uint32_t bpr = (ctx->n >> 8) / 16;
        hipLaunchKernelGGL(ntt_col8_from_i64, dim3(batch * bpr), dim3(512), 0, ctx->stream, m, out, limbs,
                           ctx->d_mod, ctx->d_twf, ctx->log_n, bpr, identity_reduction_bound(ctx, limbs));
        e = hipGetLastError();
    } else {
        e = f ? dispatch_col_i64<true>(s1, ctx, m, out, batch, limbs)
              : dispatch_col_i64<false>(s1, ctx, m, out, batch, limbs);
    }
    prof_end(ctx, K_NTT_FWD_COL);
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
    CK_TRY(launch_ntt_col_i64(ctx, m, out, batch, limbs));
    const LimbMap map = limb_range(0, limbs);
    const bool f = use_f64(ctx, map);
    const double res = (double)batch * limbs * ctx->n, bf = f ? kOpsButterflyF64 : kOpsButterflyInt;
    prof_begin(ctx, K_NTT_FWD_ROW, 16.0 * batch * limbs * ctx->n, res * bf * s2 / 2);
    const hipError_t e = f ? dispatch_row<false, false, true, true>(s2, ctx, out, batch, limbs, map)
                           : dispatch_row<false, false, true, false>(s2, ctx, out, batch, limbs, map);
    prof_end(ctx, K_NTT_FWD_ROW);
    if (e != hipSuccess) return set_error(CKKS_EHIP, "ntt launch failed: %s", hipGetErrorString(e));
    return CKKS_OK;
}
