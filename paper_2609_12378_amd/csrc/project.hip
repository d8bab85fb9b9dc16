// The packed ciphertext x plaintext projection Y = X W in the feature-major
// layout, evaluated with the slot-diagonal identity Ax = sum_k D_k(A) * rho^k(x)
// (Section "Matrix Representations and Linear Computation in CKKS", Eq.
// slot-diagonal-matvec) under a baby-step/giant-step split k = n1 g + b:
//
//   out_j = Rescale( sum_g Rot_{T n1 g}( sum_{i,b} pt_{j,i,g,b} * Rot_{T b}(x_i) ) ),
//   pt_{j,i,g,b} = Encode_{q_l}( p[f T + t] = D_{n1 g + b}(A_{j,i})[(f - n1 g) mod D] ).
//
// Schedule on the GPU:
//  1. hoisted baby-step rotations: one ModUp per input ciphertext, n1 - 1
//     key switches each, into xrot[i][b] (b = 0 is a copy of x_i);
//  2. for a tile of J output blocks (28 on the fp64 path, 4 on the integer one) and one giant step g, the weight
//     plaintexts of a sub-batch of (i, b) pairs are encoded on the fly from W
//     (slot generation fused into the fp64 FFT -> round -> NTT column pass with
//     the RNS reduction fused in) and consumed by k_row_mac, which finishes
//     each plaintext's transform (the row pass) in registers and accumulates
//     pt * xrot there, so the plaintexts' NTT values never reach HBM.  With the
//     integer transform arithmetic (primes of 50 bits or more) the row pass
//     writes the plaintexts and k_mac accumulates them exactly in 128 bits,
//     loading each xrot residue once for all J output blocks;
//  3. giant-step rotation of each partial sum at level l, summation, rescale.
// The plaintext scale is q_l, so the rescale returns the input scale exactly.
#include <algorithm>
#include <cstring>
#include <vector>

#include "ckks_internal.h"
#include "ntt_core.h"
#include "ops.h"

namespace {

constexpr int kThreads = 256;

// acc[jj][c][l][n] (+)= sum_{p<P} pt[jj][p][l][n] * xrot[pair(p)][c][l][n]
template <int J>
__global__ __launch_bounds__(kThreads) void k_mac(uint64_t *acc, const uint64_t *__restrict__ pt,
                                                   const uint64_t *__restrict__ xrot, uint32_t P, uint32_t jc,
                                                   uint32_t ib0, uint32_t bcount, uint32_t n1, uint32_t L,
                                                   uint32_t log_n, int accumulate, const ModQ *__restrict__ mods)
{
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t l = blockIdx.y;
    if (col >= n) return;
    const ModQ m = mods[l];
    const size_t ct_words = (size_t)2 * L << log_n, pt_words = (size_t)L << log_n;
    const size_t off = ((size_t)l << log_n) + col;
    acc128 a[J][2];
#pragma unroll
    for (int jj = 0; jj < J; jj++) a[jj][0] = a[jj][1] = acc128{0, 0};
    for (uint32_t p = 0; p < P; p++) {
        const uint32_t pair = ib0 + p;
        const uint32_t xi = (pair / bcount) * n1 + pair % bcount;
        const uint64_t *xr = xrot + xi * ct_words + off;
        const uint64_t x0 = xr[0], x1 = xr[pt_words];
#pragma unroll
        for (int jj = 0; jj < J; jj++) {
            if (jj < (int)jc) {
                const uint64_t w = pt[((size_t)jj * P + p) * pt_words + off];
                mac(a[jj][0], w, x0);
                mac(a[jj][1], w, x1);
            }
        }
    }
#pragma unroll
    for (int jj = 0; jj < J; jj++) {
        if (jj < (int)jc) {
            uint64_t *dst = acc + (size_t)jj * ct_words + off;
            uint64_t r0 = reduce128(a[jj][0], m), r1 = reduce128(a[jj][1], m);
            if (accumulate) {
                r0 = addmod(r0, dst[0], m.q);
                r1 = addmod(r1, dst[pt_words], m.q);
            }
            dst[0] = r0;
            dst[pt_words] = r1;
        }
    }
}

// output blocks per tile: the blocks of one tile share each xrot read.  On the integer path k_mac keeps a tile's
// 128-bit accumulators in registers: 4 blocks (60 VGPRs, 8 waves per SIMD) read each xrot residue three and a half
// times as often as 14 (140 VGPRs, 3 waves) but hide the plaintext loads better: 0.65 -> 0.43 s of
// multiply-accumulate per 4096 x 14336 projection at the paper's moduli (7 blocks: 0.47 s)
constexpr uint32_t kJ = 4;    // output blocks per tile on the integer path (k_mac keeps them in registers)
constexpr uint32_t kJF = 28;  // on the fused fp64 path (one block per output: the tile only sets xrot reuse)

// Row pass of the forward NTT fused with the multiply-accumulate (fp64
// arithmetic, primes below 2^50).  Block (jj, tile) owns rows_per_block rows of
// 2^LOGS residues of limb l for output block jj; for each (i, b) pair p of the
// sub-batch it loads the column-pass output of plaintext (jj, p), finishes its
// transform in registers and LDS, and accumulates pt * xrot[pair] for both
// ciphertext components into registers.  The plaintexts' NTT values never go
// to HBM; only the column-pass rows are read, once.  The jc blocks of one tile
// read the same xrot rows at about the same time: with xcd set they are
// numbered so that all of them land on one XCD (blocks are dealt to the 8 XCDs
// round robin) and share those reads in its L2.
//
// Accumulators hold exact integer-valued doubles: a product of a transform
// output (|x| < 2q) and a canonical residue is reduced to |r| <= 1.25 q, the
// running sum is range-reduced to |a| <= q/2 + 1 every 4 pairs, so it stays
// below 5.5 q < 2^53.
template <int LOGS>
__global__ __launch_bounds__(64) void k_row_mac(uint64_t *acc, const uint64_t *__restrict__ colout,
                                                 const double *__restrict__ xrot, uint32_t P, uint32_t jc,
                                                 uint32_t ib0, uint32_t bcount, uint32_t n1, uint32_t L,
                                                 uint32_t log_n, int accumulate, const ModQ *__restrict__ mods,
                                                 const double *__restrict__ twf, uint32_t rows_per_block,
                                                 uint32_t blocks_per_limb, int xcd)
{
    using nttc::kE;
    constexpr uint32_t S = 1u << LOGS, TS = S / 16;
    extern __shared__ uint64_t lds_raw[];
    double *lds = (double *)lds_raw;
    const uint32_t bid = blockIdx.x;
    uint32_t jj, tile;
    if (xcd) {
        const uint32_t k = bid >> 3;
        jj = k % jc;
        tile = (k / jc) * 8 + (bid & 7);
    } else {
        jj = bid % jc;
        tile = bid / jc;
    }
    const uint32_t l = tile / blocks_per_limb, blk = tile % blocks_per_limb;
    const nttc::Ar<true> ar(mods[l]);
    const double *tw = twf + ((size_t)l << log_n);
    const uint32_t rows = 1u << (log_n - LOGS);
    const uint32_t sub = threadIdx.x / TS, r = threadIdx.x % TS;
    const uint32_t h = blk * rows_per_block + sub;
    const uint32_t B = rows + h;
    const size_t pt_words = (size_t)L << log_n, ct_words = 2 * pt_words;
    const size_t off = ((size_t)l << log_n) + (size_t)h * S + r;
    double a0[kE], a1[kE];
#pragma unroll
    for (int k = 0; k < kE; k++) a0[k] = a1[k] = 0.0;
    for (uint32_t p = 0; p < P; p++) {
        const uint64_t *src = colout + ((size_t)jj * P + p) * pt_words + off;
        double x[kE];
#pragma unroll
        for (int k = 0; k < kE; k++) x[k] = nttc::Ar<true>::from_raw(src[TS * k]);
        // an opaque copy of the table pointer keeps the compiler from hoisting the twiddle loads (cache hits) out
        // of the loop into ~60 registers that would halve the occupancy
        auto twg = (const __attribute__((address_space(1))) double *)tw;
        asm volatile("" : "+v"(twg));
        const double *twl = (const double *)twg;
        nttc::fwd_top<true>(x, twl, B, ar);
        if (LOGS > 4) {
            nttc::transpose<LOGS, true>(x, lds, sub, r);
            nttc::fwd_low<LOGS, true>(x, twl, B, r, ar);
            nttc::transpose<LOGS, false>(x, lds, sub, r);
        }
        const uint32_t pair = ib0 + p;
        const double *xr = xrot + (size_t)((pair / bcount) * n1 + pair % bcount) * ct_words + off;
#pragma unroll
        for (int k = 0; k < kE; k++) {
            a0[k] += ar.mul(x[k], xr[TS * k]);
            a1[k] += ar.mul(x[k], xr[pt_words + TS * k]);
        }
        if ((p & 3) == 3) {
#pragma unroll
            for (int k = 0; k < kE; k++) {
                a0[k] = ar.red(a0[k]);
                a1[k] = ar.red(a1[k]);
            }
        }
    }
    uint64_t *dst = acc + (size_t)jj * ct_words + off;
    const uint64_t q = mods[l].q;
#pragma unroll
    for (int k = 0; k < kE; k++) {
        uint64_t r0 = ar.to_canon(a0[k]), r1 = ar.to_canon(a1[k]);
        if (accumulate) {
            r0 = addmod(r0, dst[TS * k], q);
            r1 = addmod(r1, dst[pt_words + TS * k], q);
        }
        dst[TS * k] = r0;
        dst[pt_words + TS * k] = r1;
    }
}

// The same for 256-point rows with 8 residues per thread (nttc::fwd8_256): a
// block is one wave holding 2 rows, whose twiddle tables are staged in LDS once
// for all P pairs.  The transform ends in a layout where each lane holds runs of
// 4 points; one more LDS transpose returns the values to consecutive lanes
// before xrot is read, since the 16-byte strided reads of that layout measured
// 30% slower than the extra transpose.  Half the registers of the 16-residue
// kernel (126 VGPRs): 4 waves per SIMD instead of 3.
__global__ __launch_bounds__(64) void k_row_mac8(uint64_t *acc, const uint64_t *__restrict__ colout,
                                                 const double *__restrict__ xrot, uint32_t P, uint32_t jc,
                                                 uint32_t ib0, uint32_t bcount, uint32_t n1, uint32_t L,
                                                 uint32_t log_n, int accumulate, const ModQ *__restrict__ mods,
                                                 const double *__restrict__ twf, uint32_t blocks_per_limb, int xcd)
{
    using nttc::kE8;
    __shared__ double tws[2][257];
    __shared__ double tr[2][nttc::kTr8];
    const uint32_t bid = blockIdx.x;
    uint32_t jj, tile;
    if (xcd) {
        const uint32_t k = bid >> 3;
        jj = k % jc;
        tile = (k / jc) * 8 + (bid & 7);
    } else {
        jj = bid % jc;
        tile = bid / jc;
    }
    const uint32_t l = tile / blocks_per_limb, blk = tile % blocks_per_limb;
    const nttc::Ar<true> ar(mods[l]);
    const uint32_t sub = threadIdx.x >> 5, t = threadIdx.x & 31;
    const uint32_t h = blk * 2 + sub;
    nttc::stage_twiddles8(tws[sub], twf + ((size_t)l << log_n), (1u << (log_n - 8)) + h, t, 32);
    __syncthreads();
    const size_t pt_words = (size_t)L << log_n, ct_words = 2 * pt_words;
    const size_t row = ((size_t)l << log_n) + (size_t)h * 256;
    double a0[kE8], a1[kE8];
#pragma unroll
    for (int k = 0; k < kE8; k++) a0[k] = a1[k] = 0.0;
    for (uint32_t p = 0; p < P; p++) {
        const uint64_t *src = colout + ((size_t)jj * P + p) * pt_words + row;
        double x[kE8];
#pragma unroll
        for (int k = 0; k < kE8; k++) x[k] = nttc::Ar<true>::from_raw(nttc::ld_stream(src + nttc::u8<0>(t, k)));
        nttc::fwd8_256<nttc::kRowMask8>(x, tws[sub], tr[sub], t, ar);
        nttc::b_to_a8(x, tr[sub], t);
        const uint32_t pair = ib0 + p;
        const double *xr = xrot + (size_t)((pair / bcount) * n1 + pair % bcount) * ct_words + row;
#pragma unroll
        for (int k = 0; k < kE8; k++) {
            a0[k] += ar.mul(x[k], xr[nttc::u8<0>(t, k)]);
            a1[k] += ar.mul(x[k], xr[pt_words + nttc::u8<0>(t, k)]);
        }
        if ((p & 3) == 3) {
#pragma unroll
            for (int k = 0; k < kE8; k++) {
                a0[k] = ar.red(a0[k]);
                a1[k] = ar.red(a1[k]);
            }
        }
    }
    const uint64_t q = mods[l].q;
    uint64_t *dst = acc + (size_t)jj * ct_words + row;
#pragma unroll
    for (int k = 0; k < kE8; k++) {
        const uint32_t u = nttc::u8<0>(t, k);
        uint64_t r0 = ar.to_canon(a0[k]), r1 = ar.to_canon(a1[k]);
        if (accumulate) {
            r0 = addmod(r0, dst[u], q);
            r1 = addmod(r1, dst[pt_words + u], q);
        }
        dst[u] = r0;
        dst[pt_words + u] = r1;
    }
}

// W (d_in x d_out, row-major) -> its cyclic diagonals per block pair:
// Wd[((jb * n_in + i) * D + k) * D + o] = D_k(A_{jb,i})[o] = W[(i D + (k + o) mod D) * d_out + jb D + o]
__global__ __launch_bounds__(kThreads) void k_diag_layout(double *Wd, const double *__restrict__ W, uint32_t D,
                                                          uint32_t n_in, uint32_t d_out, size_t total)
{
    const size_t e = (size_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= total) return;
    const uint32_t o = (uint32_t)(e % D), k = (uint32_t)((e / D) % D);
    const size_t bi = e / ((size_t)D * D);
    const uint32_t i = (uint32_t)(bi % n_in), jb = (uint32_t)(bi / n_in);
    Wd[e] = W[((size_t)i * D + (k + o) % D) * d_out + (size_t)jb * D + o];
}

// canonical residues -> the same values as doubles (exact below 2^53), in place
__global__ __launch_bounds__(kThreads) void k_to_f64(uint64_t *v, size_t n)
{
    const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) v[i] = (uint64_t)__double_as_longlong((double)v[i]);
}

template <int LOGS>
hipError_t launch_row_mac_t(ckks_ctx *ctx, uint64_t *acc, const uint64_t *colout, const double *xrot, uint32_t P,
                            uint32_t jc, uint32_t ib0, uint32_t bcount, uint32_t n1, uint32_t L, bool accumulate)
{
    const uint32_t rows = 1u << (ctx->log_n - LOGS), TS = (1u << LOGS) / 16;
    // one wave per block: 64 / TS rows
    uint32_t rpb = 64 / TS;
    if (rpb > rows) rpb = rows;
    const uint32_t bpl = rows / rpb, tiles = L * bpl;
    const int xcd = tiles % 8 == 0;
    const dim3 grid(jc * tiles), block(rpb * TS);
    hipLaunchKernelGGL(k_row_mac<LOGS>, grid, block, nttc::lds_bytes<LOGS>(rpb), ctx->stream, acc, colout, xrot, P,
                       jc, ib0, bcount, n1, L, ctx->log_n, (int)accumulate, ctx->d_mod, ctx->d_twf, rpb, bpl, xcd);
    return hipGetLastError();
}

ckks_status launch_row_mac(ckks_ctx *ctx, uint64_t *acc, const uint64_t *colout, const double *xrot, uint32_t P,
                           uint32_t jc, uint32_t ib0, uint32_t bcount, uint32_t n1, uint32_t L, bool accumulate)
{
    int s1, s2;
    ntt_split(ctx->log_n, &s1, &s2);
    // column-pass rows (jc x P), rotated inputs (P ciphertexts), accumulators written (and read when accumulating)
    const double w = 8.0 * L * ctx->n;
    // per plaintext residue: the row pass's butterflies (the 8-residue kernel skips the reduction of X in half
    // of its stages), two exact products and additions (14), and the range reduction of both sums every 4 pairs
    // (1.5)
    const double res = (double)jc * P * L * ctx->n;
    const double bf_ops = s2 == 8 ? (4 * kOpsButterflyF64 + 4 * (kOpsButterflyF64 - 3)) / 2 : kOpsButterflyF64 * s2 / 2;
    prof_begin(ctx, K_ROW_MAC, w * ((double)jc * P + 2.0 * P + 2.0 * jc * (accumulate ? 2 : 1)),
               res * (bf_ops + 15.5));
    hipError_t e = hipErrorInvalidValue;
    if (s2 == 8) {
        const uint32_t bpl = 1u << (ctx->log_n - 9), tiles = L * bpl;  // two rows per block
        hipLaunchKernelGGL(k_row_mac8, dim3(jc * tiles), dim3(64), 0, ctx->stream, acc, colout, xrot, P, jc, ib0,
                           bcount, n1, L, ctx->log_n, (int)accumulate, ctx->d_mod, ctx->d_twf, bpl,
                           (int)(tiles % 8 == 0));
        e = hipGetLastError();
    } else switch (s2) {
    case 5: e = launch_row_mac_t<5>(ctx, acc, colout, xrot, P, jc, ib0, bcount, n1, L, accumulate); break;
    case 6: e = launch_row_mac_t<6>(ctx, acc, colout, xrot, P, jc, ib0, bcount, n1, L, accumulate); break;
    case 7: e = launch_row_mac_t<7>(ctx, acc, colout, xrot, P, jc, ib0, bcount, n1, L, accumulate); break;
    }
    prof_end(ctx, K_ROW_MAC);
    if (e != hipSuccess) return set_error(CKKS_EHIP, "row/mac launch failed: %s", hipGetErrorString(e));
    return CKKS_OK;
}

ckks_status launch_mac(ckks_ctx *ctx, uint64_t *acc, const uint64_t *pt, const uint64_t *xrot, uint32_t P,
                       uint32_t jc, uint32_t ib0, uint32_t bcount, uint32_t n1, uint32_t L, bool accumulate)
{
    const dim3 grid((ctx->n + kThreads - 1) / kThreads, L), block(kThreads);
    // plaintexts (jc x P), rotated inputs (P ciphertexts), accumulators written (and read when accumulating)
    const double w = 8.0 * L * ctx->n;
    prof_begin(ctx, K_MAC, w * ((double)jc * P + 2.0 * P + 2.0 * jc * (accumulate ? 2 : 1)));
    if (jc <= 1)
        hipLaunchKernelGGL(k_mac<1>, grid, block, 0, ctx->stream, acc, pt, xrot, P, jc, ib0, bcount, n1, L,
                           ctx->log_n, (int)accumulate, ctx->d_mod);
    else if (jc <= 2)
        hipLaunchKernelGGL(k_mac<2>, grid, block, 0, ctx->stream, acc, pt, xrot, P, jc, ib0, bcount, n1, L,
                           ctx->log_n, (int)accumulate, ctx->d_mod);
    else if (jc <= 4)
        hipLaunchKernelGGL(k_mac<4>, grid, block, 0, ctx->stream, acc, pt, xrot, P, jc, ib0, bcount, n1, L,
                           ctx->log_n, (int)accumulate, ctx->d_mod);
    else
        hipLaunchKernelGGL(k_mac<kJ>, grid, block, 0, ctx->stream, acc, pt, xrot, P, jc, ib0, bcount, n1, L,
                           ctx->log_n, (int)accumulate, ctx->d_mod);
    prof_end(ctx, K_MAC);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

// Scratch words of one ckks_linear_project call, by region (every region a multiple of N words).
struct ProjScratch {
    uint32_t Jt;  // output blocks per tile (kJ on the integer path, kJF on the fused fp64 one)
    uint32_t Pb;  // (input, baby step) pairs per plaintext sub-batch
    bool diag;    // W re-laid as its cyclic diagonals (radix-8 FFT pass A)
    size_t xrot_w, acc_w, tot_w, rot_w, pt_w, m_w, fft_w, ks_w, wd_w, fop_w, ua_w, total;
};

ProjScratch proj_scratch(const ckks_ctx *ctx, uint32_t L, uint32_t D, uint32_t d_in, uint32_t d_out, uint32_t n1)
{
    ProjScratch ps{};
    const uint32_t level = L - 1, n_in = d_in / D;
    const size_t N = ctx->n, ctw = 2 * (size_t)L * N;
    const uint32_t maxpairs = n_in * n1;
    int s1, s2;
    ntt_split(ctx->log_n, &s1, &s2);
    const uint32_t kJt = (s1 > 0 && ntt_uses_f64(ctx, L)) ? kJF : kJ;
    ps.Jt = kJt;
    // plaintext sub-batch of at most 24 GiB (128 pairs of 28 output blocks at the benchmark shape: each launch
    // reads and writes the accumulators once, so fewer, larger launches move less; 22 -> 128 pairs measured
    // 1092 -> 1039 ms)
    const size_t budget = size_t(24) << 30;
    uint32_t Pmax = std::min<uint32_t>(maxpairs, std::max<uint32_t>(1, (uint32_t)(budget / ((size_t)kJt * L * N * 8))));
    if (ctx->proj_max_pairs) Pmax = std::min(Pmax, ctx->proj_max_pairs);
    // k_mac sums one product per pair in each exact 128-bit accumulator
    if (kJt == kJ) Pmax = std::min(Pmax, ctx->sum128_terms);
    ps.Pb = Pmax;
    ps.xrot_w = (size_t)n_in * n1 * ctw;
    ps.acc_w = ps.tot_w = ps.rot_w = (size_t)kJt * ctw;
    ps.pt_w = (size_t)kJt * ps.Pb * L * N;
    ps.m_w = (size_t)kJt * ps.Pb * N;               // int64 coefficients
    ps.fft_w = (size_t)kJt * ps.Pb * (N / 2) * 2;   // double2 per slot
    // key switching: hoisted baby steps of one input, or the giant step of a tile's partial sums
    ps.ks_w = std::max(ks_scratch_words(ctx, level, ks_rot_batch(n1 > 1 ? n1 - 1 : 1)),
                       ks_scratch_words(ctx, level, ks_rot_batch(kJt), kJt));
    // W re-laid as its cyclic diagonals, and the feature index of every FFT position, for the radix-8 FFT pass
    ps.diag = D <= 256 && ctx->log_n >= 12;
    ps.wd_w = ps.diag ? (size_t)d_in * d_out : 0;
    ps.fop_w = ps.diag ? N / 4 : 0;
    // lazy ModDown: the tile's key-switching sums over Q u P
    ps.ua_w = ctx->lazy_moddown ? (size_t)kJt * 2 * (L + ctx->n_p) * N : 0;
    ps.total = ps.xrot_w + ps.acc_w + ps.tot_w + ps.rot_w + ps.pt_w + ps.m_w + ps.fft_w + ps.ks_w + ps.wd_w +
               ps.fop_w + ps.ua_w;
    return ps;
}

}  // namespace

ckks_status launch_diag_layout(ckks_ctx *ctx, double *Wd, const double *W, uint32_t D, uint32_t n_in,
                               uint32_t d_out)
{
    const size_t tot_e = (size_t)n_in * D * d_out;
    prof_begin(ctx, K_ELEM, 16.0 * tot_e);
    hipLaunchKernelGGL(k_diag_layout, dim3((unsigned)((tot_e + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                       ctx->stream, Wd, W, D, n_in, d_out, tot_e);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_to_f64(ckks_ctx *ctx, uint64_t *v, size_t words)
{
    prof_begin(ctx, K_ELEM, 16.0 * words);
    hipLaunchKernelGGL(k_to_f64, dim3((unsigned)((words + kThreads - 1) / kThreads)), dim3(kThreads), 0, ctx->stream,
                       v, words);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

size_t proj_workspace_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t tokens, uint32_t d_in, uint32_t d_out,
                            uint32_t n1)
{
    const uint32_t slots = ctx->n / 2;
    if (tokens < 1 || slots % tokens) return SIZE_MAX;
    const uint32_t D = slots / tokens;
    if (!d_in || !d_out || d_in % D || d_out % D || n1 < 1 || n1 > D || L < 2 || L > ctx->n_q) return SIZE_MAX;
    return proj_scratch(ctx, L, D, d_in, d_out, n1).total * 8;
}

extern "C" ckks_status ckks_linear_project(ckks_ctx *ctx, const ckks_buf *in, const double *W,
                                           const ckks_proj_shape *shape, const int32_t *key_steps,
                                           const uint64_t *const *keys, uint32_t n_keys, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx && in && W && shape && out, CKKS_EINVAL, "linear_project: null argument");
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "linear_project: the context has no special primes");
    const uint32_t T = shape->tokens, slots = ctx->n / 2;
    CK_REQUIRE(T >= 1 && slots % T == 0, CKKS_EINVAL, "linear_project: %u tokens do not divide %u slots", T, slots);
    const uint32_t D = slots / T;
    CK_REQUIRE(shape->d_in > 0 && shape->d_out > 0 && shape->d_in % D == 0 && shape->d_out % D == 0, CKKS_EINVAL,
               "linear_project: d_in %u and d_out %u must be positive multiples of %u features per ciphertext",
               shape->d_in, shape->d_out, D);
    const uint32_t n1 = shape->n1;
    CK_REQUIRE(n1 >= 1 && n1 <= D, CKKS_EINVAL, "linear_project: n1 %u outside [1, %u]", n1, D);
    const uint32_t n_in = shape->d_in / D, n_out = shape->d_out / D, n2 = (D + n1 - 1) / n1;
    const uint32_t L = in[0].n_limbs, level = L - 1;
    CK_REQUIRE(L >= 2 && L <= ctx->n_q, CKKS_ELEVEL, "linear_project: inputs need 2..%u limbs", ctx->n_q);
    for (uint32_t i = 0; i < n_in; i++) {
        CK_REQUIRE(in[i].data && in[i].n_polys == 2, CKKS_EINVAL, "linear_project: input %u is not a ciphertext", i);
        CK_REQUIRE(in[i].n_limbs == L, CKKS_ELEVEL, "linear_project: input %u has %u limbs, expected %u", i,
                   in[i].n_limbs, L);
        CK_REQUIRE(in[i].scale == in[0].scale, CKKS_ESCALE, "linear_project: input scales differ");
    }
    for (uint32_t j = 0; j < n_out; j++) {
        CK_REQUIRE(out[j].data && out[j].n_polys == 2 && out[j].n_limbs == level, CKKS_EINVAL,
                   "linear_project: output %u must be a ciphertext with %u limbs", j, level);
    }
    auto find_key = [&](int32_t st) -> const uint64_t * {
        for (uint32_t r = 0; r < n_keys; r++)
            if (key_steps[r] == st) return keys[r];
        return nullptr;
    };
    std::vector<int32_t> bsteps;
    std::vector<const uint64_t *> bkeys;
    for (uint32_t b = 1; b < n1; b++) {
        const uint64_t *k = find_key((int32_t)(T * b));
        CK_REQUIRE(k, CKKS_ENOKEY, "linear_project: no key for baby step %u", T * b);
        bsteps.push_back((int32_t)(T * b));
        bkeys.push_back(k);
    }
    std::vector<const uint64_t *> gkeys(n2, nullptr);
    for (uint32_t g = 1; g < n2; g++) {
        gkeys[g] = find_key((int32_t)(T * n1 * g));
        CK_REQUIRE(gkeys[g], CKKS_ENOKEY, "linear_project: no key for giant step %u", T * n1 * g);
    }

    // ---- scratch layout
    const size_t N = ctx->n, ctw = 2 * (size_t)L * N;
    const ProjScratch ps = proj_scratch(ctx, L, D, shape->d_in, shape->d_out, n1);
    const uint32_t Jt = ps.Jt, Pb = ps.Pb;
    const size_t xrot_w = ps.xrot_w, acc_w = ps.acc_w, tot_w = ps.tot_w, rot_w = ps.rot_w, pt_w = ps.pt_w;
    const size_t m_w = ps.m_w, fft_w = ps.fft_w, ks_w = ps.ks_w, wd_w = ps.wd_w, total = ps.total;
    const bool diag = ps.diag;
    void *w;
    CK_TRY(ctx_scratch(ctx, total * 8, &w));
    uint64_t *xrot = (uint64_t *)w;
    uint64_t *acc = xrot + xrot_w;
    uint64_t *tot = acc + acc_w;
    uint64_t *rot = tot + tot_w;
    uint64_t *pts = rot + rot_w;
    int64_t *mint = (int64_t *)(pts + pt_w);
    double2 *fft = (double2 *)(mint + m_w);
    uint64_t *ksw = (uint64_t *)(fft) + fft_w;
    double *Wd = (double *)(ksw + ks_w);
    uint32_t *fop = (uint32_t *)(ksw + ks_w + wd_w);
    uint64_t *uacc = ksw + ks_w + wd_w + ps.fop_w;  // [Jt][2][L + K][N] when the ModDown is lazy
    const bool lazy = ctx->lazy_moddown;
    if (diag) {
        CK_TRY(launch_diag_layout(ctx, Wd, W, D, n_in, shape->d_out));
        CK_TRY(enc_feat_of_pos(ctx, T, fop));
    }

    // ---- 1. baby-step rotations, hoisted per input ciphertext
    for (uint32_t i = 0; i < n_in; i++) {
        uint64_t *xi = xrot + (size_t)i * n1 * ctw;
        HIP_TRY(hipMemcpyAsync(xi, in[i].data, ctw * 8, hipMemcpyDeviceToDevice, ctx->stream));
        if (n1 > 1) {
            std::vector<uint64_t *> outs(n1 - 1);
            for (uint32_t b = 1; b < n1; b++) outs[b - 1] = xi + (size_t)b * ctw;
            CK_TRY(rotate_core(ctx, in[i].data, level, bsteps.data(), bkeys.data(), n1 - 1, outs.data(), ksw));
        }
    }
    // fp64 two-pass transforms: the row pass runs inside the multiply-accumulate, which reads xrot as doubles
    int s1, s2;
    ntt_split(ctx->log_n, &s1, &s2);
    const bool fused = s1 > 0 && ntt_uses_f64(ctx, L);
    if (fused) CK_TRY(launch_to_f64(ctx, xrot, xrot_w));

    // ---- 2./3. tiles of output blocks
    const double delta_w = (double)ctx->primes[level];
    for (uint32_t j0 = 0; j0 < n_out; j0 += Jt) {
        const uint32_t jc = std::min<uint32_t>(Jt, n_out - j0);
        for (uint32_t g = 0; g < n2; g++) {
            const uint32_t bcount = std::min<uint32_t>(n1, D - n1 * g);
            const uint32_t pairs = n_in * bcount;
            // sub-batches of equal size (within one pair): no short tail launch
            const uint32_t nsub = (pairs + Pb - 1) / Pb;
            for (uint32_t sb = 0, pb0 = 0; sb < nsub; sb++) {
                const uint32_t P = pairs / nsub + (sb < pairs % nsub ? 1 : 0);
                SlotSource src;
                src.W = W;
                src.d_out = shape->d_out;
                src.tokens = T;
                src.feats = D;
                src.n1g = n1 * g;
                src.bcount = bcount;
                src.j0 = j0;
                src.ib0 = pb0;
                src.pairs = P;
                if (diag) {
                    src.Wd = Wd;
                    src.feat_of_pos = fop;
                    src.n_in = n_in;
                }
                const uint32_t batch = jc * P;
                if (fused && enc_fused_ok(ctx, L)) {
                    CK_TRY(enc_ntt_first_pass(ctx, src, batch, delta_w, fft, L, pts));
                    CK_TRY(launch_row_mac(ctx, acc, pts, (const double *)xrot, P, jc, pb0, bcount, n1, L, pb0 > 0));
                } else if (fused) {
                    CK_TRY(enc_coeffs(ctx, src, batch, delta_w, fft, mint));
                    CK_TRY(launch_ntt_col_i64(ctx, mint, pts, batch, L));
                    CK_TRY(launch_row_mac(ctx, acc, pts, (const double *)xrot, P, jc, pb0, bcount, n1, L, pb0 > 0));
                } else {
                    CK_TRY(enc_coeffs(ctx, src, batch, delta_w, fft, mint));
                    CK_TRY(launch_ntt_from_i64(ctx, mint, pts, batch, L));
                    CK_TRY(launch_mac(ctx, acc, pts, xrot, P, jc, pb0, bcount, n1, L, pb0 > 0));
                }
                pb0 += P;
            }
            // giant step: the tile's jc partial sums rotated together, then added to the totals (lazy: their
            // key-switching sums accumulated over Q u P, divided by P once after the last giant step)
            if (g == 0) {
                HIP_TRY(hipMemcpyAsync(tot, acc, jc * ctw * 8, hipMemcpyDeviceToDevice, ctx->stream));
            } else if (lazy) {
                CK_TRY(rotate_many_lazy(ctx, acc, ctw, jc, level, (int32_t)(T * n1 * g), gkeys[g], uacc, g > 1, ksw));
            } else {
                std::vector<uint64_t *> outs(jc);
                for (uint32_t jj = 0; jj < jc; jj++) outs[jj] = rot + (size_t)jj * ctw;
                CK_TRY(rotate_many(ctx, acc, ctw, jc, level, (int32_t)(T * n1 * g), gkeys[g], outs.data(), ksw));
                CK_TRY(launch_binary(ctx, tot, tot, rot, jc * 2 * L, limb_range(0, L), EW_ADD));
            }
        }
        if (lazy && n2 > 1) {
            CK_TRY(ks_moddown(ctx, uacc, 2 * jc, level, nullptr, 1, nullptr, rot, ksw));
            CK_TRY(launch_binary(ctx, tot, tot, rot, jc * 2 * L, limb_range(0, L), EW_ADD));
        }
        for (uint32_t jj = 0; jj < jc; jj++) {
            CK_TRY(rescale_core(ctx, tot + (size_t)jj * ctw, level, out[j0 + jj].data, rot));
            out[j0 + jj].scale = in[0].scale;
        }
    }
    return CKKS_OK;
}
