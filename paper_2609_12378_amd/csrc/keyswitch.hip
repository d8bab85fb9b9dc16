// Hybrid key switching (Han-Ki 2020) in the RNS form of CKKS:
//
//   ModUp of digit j:  INTT of the digit's limbs, fast basis conversion to the
//                      other q-limbs and the special primes P, NTT;
//   inner product:     (u0, u1) = sum_j sigma_g(d_j) * (b_j, a_j) over Q_l u P,
//                      with the Galois automorphism folded into the digit loads;
//   ModDown:           u -> (u - NTT(Conv_{P->Q}(INTT([u]_P)))) * P^-1, fused
//                      with the final additions of the rotation or relinearisation.
//
// The fast basis conversion (Cheon-Han-Kim-Kim-Song 2018) is
//   Conv(x)_t = sum_i y_i * [Qhat_i]_t  (mod t),  y_i = [x_i * Qhat_i^-1]_{q_i} in (-q_i/2, q_i/2],
// without overflow correction.  Centred digits give the ModUp digits and the
// ModDown rounding a zero mean: with [0, q_i) digits every digit carries a
// constant offset of about |I|/2 * Q_I whose product with the key error piles
// up in the slots next to X = +-1.  Every constant multiplier is a Shoup
// product, so a conversion with ns source limbs and nt targets costs
// ns + ns*nt + nt Shoup multiplications per coefficient.  The inner dimension
// (ns <= 8 at the benchmark parameters) is far too small and too wide-integer
// for the matrix cores, so it runs on the vector ALUs.
#include <algorithm>

#include "ckks_internal.h"
#include "ntt_core.h"
#include "ops.h"
#include "philox.h"

namespace {

constexpr int kThreads = 256;
constexpr int kRotBatch = 32;  // rotations per batched launch

__device__ __forceinline__ uint32_t auto_index(uint32_t j, uint32_t g, uint32_t log_n)
{
    const uint32_t two_n_mask = (2u << log_n) - 1;
    const uint32_t k = 2u * (__brev(j) >> (32 - log_n)) + 1u;
    const uint32_t kg = (uint32_t)(((uint64_t)k * g) & two_n_mask);
    return __brev((kg - 1u) >> 1) >> (32 - log_n);
}

struct ConvArgs {
    int ns, nt;
    uint8_t src[kMaxPrimes];
    uint8_t dst[kMaxPrimes];
};

// in: [polys][ns][N] (stride in_stride rows between polys), coefficient form;
// out row for target ti: out + (poly*out_stride + (ti < split ? ti : ti + skip)) * N.
// A digit y_i > q_i/2 stands for y_i - q_i, so the centred sum is the sum of the
// canonical digits plus neg * [-Q_I]_t, neg the number of such digits.  Each
// target's sum is accumulated exactly in 128 bits (products below 2^124; eight of
// them and a residue below 2^128) and reduced once per eight sources, which costs
// fewer 32-bit multiplies than a Shoup product and a conditional subtraction per
// term.  The constants and the target moduli are staged in LDS once per block, so
// the per-target loop reads them at LDS latency instead of waiting on scalar
// memory loads.
template <int NS_MAX>
__global__ __launch_bounds__(kThreads) void k_conv(const uint64_t *in, uint32_t in_stride, uint64_t *out,
                                                    uint32_t out_stride, uint32_t split, uint32_t skip, ConvArgs a,
                                                    const ulonglong2 *__restrict__ qhat_inv,
                                                    const ulonglong2 *__restrict__ qhat_mod,
                                                    const ulonglong2 *__restrict__ neg_q,
                                                    const ModQ *__restrict__ mods, uint32_t log_n)
{
    __shared__ uint64_t s_mod[NS_MAX * kMaxPrimes];
    __shared__ uint64_t s_neg[kMaxPrimes];
    __shared__ ModQ s_tm[kMaxPrimes];
    const int ns = a.ns, nt = a.nt;
    for (int k = threadIdx.x; k < ns * nt; k += kThreads) s_mod[k] = qhat_mod[k].x;
    for (int k = threadIdx.x; k < nt; k += kThreads) {
        s_tm[k] = mods[a.dst[k]];
        s_neg[k] = neg_q[k].x;
    }
    __syncthreads();
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t poly = blockIdx.y;
    if (col >= n) return;
    const uint64_t *src = in + ((size_t)poly * in_stride << log_n) + col;
    uint64_t y[NS_MAX];
    uint64_t neg = 0;
#pragma unroll
    for (int i = 0; i < NS_MAX; i++) {
        if (i < ns) {
            const uint64_t q = mods[a.src[i]].q;
            const ulonglong2 w = qhat_inv[i];
            y[i] = shoup(src[(size_t)i << log_n], w.x, w.y, q);
            neg += y[i] > (q >> 1);
        }
    }
    uint64_t *dst = out + ((size_t)poly * out_stride << log_n) + col;
    for (int t = 0; t < nt; t++) {
        const ModQ mt = s_tm[t];
        acc128 acc{0, 0};
        mac(acc, neg, s_neg[t]);
#pragma unroll
        for (int i = 0; i < NS_MAX; i++) {
            if (i < ns) {
                mac(acc, y[i], s_mod[i * nt + t]);
                if ((i & 7) == 7 && i + 1 < ns) acc = acc128{reduce128(acc, mt), 0};
            }
        }
        const uint32_t row = t < (int)split ? t : t + skip;
        dst[(size_t)row << log_n] = reduce128(acc, mt);
    }
}

// The same conversion in fp64 (every prime below 2^50): y_i = x_i * qhat_inv_i mod s_i (|mul| < 0.875 s_i for
// canonical operands) is moved into (-s_i/2, s_i/2] by one add or subtract of s_i, then each target sums the
// products y_i * [Qhat_i]_t (each below 0.875 t in magnitude, since |y_i| < s_i/2 < t) with a range reduction
// after every eight terms that more follow (sums stay below 7.5 t < 2^53) and writes the canonical residue: the
// same integers as k_conv.
// C coefficients per thread (kThreads apart, so every load and store stays coalesced): the per-target constants
// come from LDS once for all C, and the C product chains are independent.  All source loads issue before the
// first is used (EXACT: ns == NS_MAX, no guards in the source loop).  blockIdx.z splits the target limbs into
// groups of t_per when a few polynomials alone would leave most SIMDs idle.
template <int NS_MAX, int C, bool EXACT = false>
__global__ __launch_bounds__(kThreads) void k_conv_f64(const uint64_t *in, uint32_t in_stride, uint64_t *out,
                                                        uint32_t out_stride, uint32_t split, uint32_t skip,
                                                        ConvArgs a, const double *__restrict__ qhat_inv,
                                                        const double *__restrict__ qhat_mod,
                                                        const ModQ *__restrict__ mods, uint32_t log_n,
                                                        uint32_t t_per)
{
    __shared__ double s_mod[NS_MAX * kMaxPrimes];
    __shared__ double2 s_tq[kMaxPrimes];
    const int ns = EXACT ? NS_MAX : a.ns, nt = a.nt;
    for (int k = threadIdx.x; k < ns * nt; k += kThreads) s_mod[k] = qhat_mod[k];
    for (int k = threadIdx.x; k < nt; k += kThreads) s_tq[k] = make_double2(mods[a.dst[k]].qd, mods[a.dst[k]].qinvd);
    __syncthreads();
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * (kThreads * C) + threadIdx.x;
    const uint32_t poly = blockIdx.y;
    if (col >= n) return;  // n is a multiple of kThreads * C
    const uint64_t *src = in + ((size_t)poly * in_stride << log_n) + col;
    // every source load issued before any is used: with fewer than NS_MAX sources the extra loads repeat the last
    // source row (no branch, so the loads stay together) and are ignored
    double y[C][NS_MAX];
    uint64_t raw[C][NS_MAX];
#pragma unroll
    for (int i = 0; i < NS_MAX; i++) {
        const int ii = EXACT ? i : min(i, ns - 1);
#pragma unroll
        for (int c = 0; c < C; c++) raw[c][i] = src[((size_t)ii << log_n) + c * kThreads];
    }
#pragma unroll
    for (int i = 0; i < NS_MAX; i++) {
        if (EXACT || i < ns) {
            const nttc::Ar<true> ar(mods[a.src[i]]);
            const double h = 0.5 * ar.q;
#pragma unroll
            for (int c = 0; c < C; c++) {
                const double v = ar.mul(nttc::Ar<true>::from_u64(raw[c][i]), qhat_inv[i]);
                y[c][i] = v > h ? v - ar.q : (v < -h ? v + ar.q : v);
            }
        }
    }
    uint64_t *dst = out + ((size_t)poly * out_stride << log_n) + col;
    // blockIdx.z: this block's group of t_per target limbs (several groups when one polynomial alone would leave
    // the chip mostly idle; each group recomputes the ns centred digits)
    const int t0 = (int)(blockIdx.z * t_per), t1 = min(nt, t0 + (int)t_per);
    for (int t = t0; t < t1; t++) {
        nttc::Ar<true> ar;
        ar.q = s_tq[t].x;
        ar.qinv = s_tq[t].y;
        double acc[C];
#pragma unroll
        for (int c = 0; c < C; c++) acc[c] = 0.0;
#pragma unroll
        for (int i = 0; i < NS_MAX; i++) {
            if (EXACT || i < ns) {
                const double w = s_mod[i * nt + t];
#pragma unroll
                for (int c = 0; c < C; c++) {
                    acc[c] += ar.mul(y[c][i], w);
                    if ((i & 7) == 7 && i + 1 < ns) acc[c] = ar.red(acc[c]);
                }
            }
        }
        const uint32_t row = t < (int)split ? t : t + skip;
#pragma unroll
        for (int c = 0; c < C; c++) dst[((size_t)row << log_n) + c * kThreads] = ar.to_canon(acc[c]);
    }
}

// The fp64 conversion (at most 8 source limbs) fused with the first forward column pass, N = 2^16: block
// (poly, 16 adjacent columns), 512 threads, 8 points of one 256-point column per thread.  The centred source
// digits y_i of the block's 4096 coefficients stay in registers; for each target limb in turn the block forms
// the converted residues with the products and range reductions of k_conv_f64 (reduced to |x| <= t/2 rather
// than made canonical), runs that limb's column sub-transforms on them (nttc::fwd8_256 with the column pass's
// lazy-reduction mask) and writes the rows as raw doubles, the inter-pass form the fused row passes read.  The
// converted rows thus cross HBM once instead of three times (written, read and written by a separate column
// pass, read by the ModDown).  Target t + 1's twiddles (Psi[1..255]) are staged into the idle half of a
// double-buffered table while target t is transformed.  EXACT: ns == 8 (no guards on the source loop, all
// source loads issued first).
struct StageNext {
    double *dst;
    double v;
    bool on;
    __device__ void operator()() const
    {
        if (on) dst[threadIdx.x + 1] = v;
    }
};

template <bool EXACT>
__global__ __launch_bounds__(512) void k_conv_col8(const uint64_t *__restrict__ in, uint32_t in_stride,
                                                   uint64_t *out, uint32_t out_stride, uint32_t split, uint32_t skip,
                                                   ConvArgs a, const double *__restrict__ qhat_inv,
                                                   const double *__restrict__ qhat_mod,
                                                   const ModQ *__restrict__ mods, const double *__restrict__ twf,
                                                   uint32_t log_n, uint32_t blocks_per_row)
{
    using nttc::Ar;
    using nttc::kE8;
    __shared__ double s_mod[8 * kMaxPrimes];
    __shared__ double tws[2][256];
    __shared__ double tr[16][nttc::kTr8];
    const int ns = EXACT ? 8 : a.ns, nt = a.nt;
    for (int k = threadIdx.x; k < ns * nt; k += 512) s_mod[k] = qhat_mod[k];
    if (threadIdx.x < 255) tws[0][threadIdx.x + 1] = twf[((size_t)a.dst[0] << log_n) + threadIdx.x + 1];
    const uint32_t poly = blockIdx.x / blocks_per_row, blk = blockIdx.x % blocks_per_row;
    const uint32_t n2 = 1u << (log_n - 8);
    const uint32_t col = threadIdx.x & 15, t = threadIdx.x >> 4;
    const size_t coff = (size_t)blk * 16 + col;
    const uint64_t *src = in + ((size_t)poly * in_stride << log_n) + coff;
    uint64_t raw[8][kE8];
#pragma unroll
    for (int i = 0; i < 8; i++)
#pragma unroll
        for (int k = 0; k < kE8; k++)
            if (EXACT || i < ns) raw[i][k] = src[((size_t)i << log_n) + (size_t)nttc::u8<0>(t, k) * n2];
    double y[kE8][8];
#pragma unroll
    for (int i = 0; i < 8; i++) {
        if (EXACT || i < ns) {
            const Ar<true> ar(mods[a.src[i]]);
            const double h = 0.5 * ar.q, w = qhat_inv[i];
#pragma unroll
            for (int k = 0; k < kE8; k++) {
                const double v = ar.mul(Ar<true>::from_u64(raw[i][k]), w);
                y[k][i] = v > h ? v - ar.q : (v < -h ? v + ar.q : v);
            }
        }
    }
    __syncthreads();
    for (int tt = 0; tt < nt; tt++) {
        const Ar<true> ar(mods[a.dst[tt]]);
        StageNext next{tws[(tt + 1) & 1], 0.0, tt + 1 < nt && threadIdx.x < 255};
        if (next.on) next.v = twf[((size_t)a.dst[tt + 1] << log_n) + threadIdx.x + 1];
        double x[kE8];
#pragma unroll
        for (int k = 0; k < kE8; k++) {
            double acc = 0.0;
#pragma unroll
            for (int i = 0; i < 8; i++) {
                if (EXACT || i < ns) {
                    acc += ar.mul(y[k][i], s_mod[i * nt + tt]);
                    if ((i & 7) == 7 && i + 1 < ns) acc = ar.red(acc);
                }
            }
            x[k] = ar.red(acc);
        }
        nttc::fwd8_256<nttc::kColMask8>(x, tws[tt & 1], tr[col], t, ar, 1, next);
        const uint32_t row = tt < (int)split ? tt : tt + skip;
        uint64_t *dst = out + (((size_t)poly * out_stride + row) << log_n) + coff;
#pragma unroll
        for (int k = 0; k < kE8; k++) nttc::st_stream(dst + (size_t)nttc::u8<2>(t, k) * n2, Ar<true>::to_raw(x[k]));
    }
}

// u[k][r][n] = sum_{j<nd} d_j[r][sigma(n)] * key[j][k][krow(r)][n], rows r over Q_level u P
__global__ __launch_bounds__(kThreads) void k_key_ip(const uint64_t *__restrict__ digits,
                                                      const uint64_t *__restrict__ key, uint64_t *u, uint32_t nd,
                                                      uint32_t ext, uint32_t level, uint32_t n_q, uint32_t key_rows,
                                                      uint32_t g, const ModQ *__restrict__ mods, uint32_t log_n)
{
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t r = blockIdx.y;
    if (col >= n) return;
    const uint32_t prime = r <= level ? r : n_q + (r - level - 1);
    const ModQ m = mods[prime];
    const uint32_t sc = g == 1 ? col : auto_index(col, g, log_n);
    acc128 a0{0, 0}, a1{0, 0};
    for (uint32_t j = 0; j < nd; j++) {
        const uint64_t d = digits[(((size_t)j * ext + r) << log_n) + sc];
        const size_t kb = ((size_t)j * 2 * key_rows + prime) << log_n;
        mac(a0, d, key[kb + col]);
        mac(a1, d, key[kb + ((size_t)key_rows << log_n) + col]);
    }
    u[((size_t)r << log_n) + col] = reduce128(a0, m);
    u[(((size_t)ext + r) << log_n) + col] = reduce128(a1, m);
}

// out[k][i][n] = (u[k][i][n] - c[k][i][n]) * P^-1 + add_k[i][sigma_k(n)], i <= level
__global__ __launch_bounds__(kThreads) void k_moddown_finish(uint64_t *out, const uint64_t *u, const uint64_t *c,
                                                              const uint64_t *add0, uint32_t add0_g,
                                                              const uint64_t *add1, uint32_t ext, uint32_t level,
                                                              const ulonglong2 *__restrict__ pinv,
                                                              const ModQ *__restrict__ mods, uint32_t log_n)
{
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t i = blockIdx.y, k = blockIdx.z;
    if (col >= n) return;
    const uint32_t L = level + 1;
    const uint64_t q = mods[i].q;
    const uint64_t x = u[(((size_t)k * ext + i) << log_n) + col];
    const uint64_t cv = c[(((size_t)k * L + i) << log_n) + col];
    const ulonglong2 w = pinv[i];
    uint64_t r = shoup(submod(x, cv, q), w.x, w.y, q);
    const uint64_t *add = k == 0 ? add0 : add1;
    if (add) {
        const uint32_t sc = (k == 0 && add0_g != 1) ? auto_index(col, add0_g, log_n) : col;
        r = addmod(r, add[((size_t)i << log_n) + sc], q);
    }
    out[(((size_t)k * L + i) << log_n) + col] = r;
}

// Batched rotations: rotation r of the batch uses Galois element g[r], key
// key[r], the ModUp digits dig[r] and c0[r] of its input, and writes out[r];
// hoisted rotations of one ciphertext share dig and c0.
struct RotArgs {
    uint32_t count;
    uint32_t g[kRotBatch];
    const uint64_t *key[kRotBatch];
    uint64_t *out[kRotBatch];
    const uint64_t *dig[kRotBatch];  // ModUp digits [nd][ext][N] of the rotated ciphertext
    const uint64_t *c0[kRotBatch];   // its c0 [level+1][N]
    // seed-expanded keys (the SEEDED kernels): key[r] is the b half [nd][key_rows][N] and seed[r] the seed of a
    uint64_t seed[kRotBatch][2];
};

// Where rotation r's key words for digit j, key row `krow`, position `pos` come from: b (and, stored, a) from the
// key; a seed-expanded key computes a (q = the row's modulus) from its seed, four digits per Philox block.
template <bool SEEDED>
struct KeyRow {
    const uint64_t *key;
    size_t kstride;      // words between the b and a halves (stored keys)
    uint32_t key_rows, log_n, prime, pos, shift;
    uint64_t q, s0, s1;
    uint64_t blk[4];
    __device__ KeyRow(const RotArgs &ra, uint32_t r, uint32_t key_rows_, uint32_t log_n_, uint32_t prime_,
                      uint32_t pos_, uint64_t q_)
        : key(ra.key[r]), kstride((size_t)key_rows_ << log_n_), key_rows(key_rows_), log_n(log_n_), prime(prime_),
          pos(pos_), shift(seedk::shift_of(q_)), q(q_), s0(ra.seed[r][0]), s1(ra.seed[r][1])
    {
    }
    __device__ uint64_t b(uint32_t j) const
    {
        const size_t row = SEEDED ? (size_t)j * key_rows + prime : (size_t)j * 2 * key_rows + prime;
        return nttc::ld_stream(key + (row << log_n) + pos);
    }
    __device__ uint64_t a(uint32_t j)
    {
        if (!SEEDED) return nttc::ld_stream(key + (((size_t)j * 2 * key_rows + prime) << log_n) + kstride + pos);
        const uint32_t m = j & 3;
        if (m == 0) seedk::block_residues(s0, s1, pos, prime, j >> 2, q, shift, blk);
        return m == 0 ? blk[0] : m == 1 ? blk[1] : m == 2 ? blk[2] : blk[3];
    }
};

// The key inner products of the 8 positions pos[e] of one thread (fp64, primes below 2^50):
//   u0[e], u1[e] = sum_j sigma_{g_r}(d_j)[row][pos[e]] * (b_j, a_j)[prime][pos[e]],  sc[e] = sigma^-1 position,
// each product reduced to <= 0.875 q and the sums range-reduced every 4 digits (so |u| <= 4 q).  With stored keys
// the gathers and key words of one digit for all 8 positions are issued together (24 loads in flight), so a wave
// waits on memory once per digit rather than once per digit and position; ND > 0 fixes the digit count at compile
// time (fully unrolled), ND = 0 takes nd.  Sums are formed in the same order either way.
template <bool SEEDED, int ND>
__device__ __forceinline__ void key_ip8(const RotArgs &ra, uint32_t r, uint32_t nd, uint32_t ext, uint32_t row,
                                        uint32_t prime, uint32_t key_rows, uint32_t log_n, uint64_t q,
                                        const nttc::Ar<true> &ar, const uint32_t (&pos)[nttc::kE8],
                                        const uint32_t (&sc)[nttc::kE8], double (&u0)[nttc::kE8],
                                        double (&u1)[nttc::kE8])
{
    using nttc::kE8;
    using A = nttc::Ar<true>;
    const uint32_t ndv = ND > 0 ? (uint32_t)ND : nd;
    constexpr int kUnroll = ND > 0 ? ND : 1;
    const uint64_t *dig = ra.dig[r] + ((size_t)row << log_n);
    const size_t dstride = (size_t)ext << log_n;
#pragma unroll
    for (int e = 0; e < kE8; e++) u0[e] = u1[e] = 0.0;
    if constexpr (!SEEDED) {
        const size_t kstride = (size_t)key_rows << log_n;   // from a digit's b rows to its a rows
        const uint64_t *key = ra.key[r] + ((size_t)prime << log_n);
#pragma unroll kUnroll
        for (uint32_t j = 0; j < ndv; j++) {
            const uint64_t *dj = dig + j * dstride, *kb = key + 2 * j * kstride, *ka = kb + kstride;
            uint64_t dv[kE8], bv[kE8], av[kE8];
#pragma unroll
            for (int e = 0; e < kE8; e++) {
                dv[e] = dj[sc[e]];
                bv[e] = nttc::ld_stream(kb + pos[e]);
                av[e] = nttc::ld_stream(ka + pos[e]);
            }
#pragma unroll
            for (int e = 0; e < kE8; e++) {
                const double d = A::from_u64(dv[e]);
                u0[e] += ar.mul(d, A::from_u64(bv[e]));
                u1[e] += ar.mul(d, A::from_u64(av[e]));
            }
            if ((j & 3) == 3) {
#pragma unroll
                for (int e = 0; e < kE8; e++) {
                    u0[e] = ar.red(u0[e]);
                    u1[e] = ar.red(u1[e]);
                }
            }
        }
    } else {
        // a regenerated per position (one Philox block per 4 digits), so positions run one after another
#pragma unroll
        for (int e = 0; e < kE8; e++) {
            KeyRow<true> kr(ra, r, key_rows, log_n, prime, pos[e], q);
#pragma unroll kUnroll
            for (uint32_t j = 0; j < ndv; j++) {
                const double d = A::from_u64(dig[j * dstride + sc[e]]);
                u0[e] += ar.mul(d, A::from_u64(kr.b(j)));
                u1[e] += ar.mul(d, A::from_u64(kr.a(j)));
                if ((j & 3) == 3) {
                    u0[e] = ar.red(u0[e]);
                    u1[e] = ar.red(u1[e]);
                }
            }
        }
    }
}

// u[r][k][row - row0][n] = sum_j d_j[row][sigma_{g_r}(n)] * key_r[j][k][krow][n] for rows row0 .. row0 + rows - 1
// of Q_level u P (u holds `rows` rows per polynomial).  ND > 0 (stored keys): the digit count at compile time, and
// every digit's gather and key words are loaded before the first product (3 ND loads in flight per thread instead
// of 3); the products are summed in the same order either way.
template <bool SEEDED, int ND = 0>
__global__ __launch_bounds__(kThreads) void k_key_ip_batch(RotArgs ra, uint64_t *u, uint32_t nd, uint32_t ext,
                                                            uint32_t level,
                                                            uint32_t n_q, uint32_t key_rows, uint32_t row0,
                                                            uint32_t rows, const ModQ *__restrict__ mods,
                                                            uint32_t log_n)
{
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t row = row0 + blockIdx.y, r = blockIdx.z;
    if (col >= n) return;
    const uint32_t prime = row <= level ? row : n_q + (row - level - 1);
    const ModQ m = mods[prime];
    const uint32_t sc = auto_index(col, ra.g[r], log_n);
    KeyRow<SEEDED> kr(ra, r, key_rows, log_n, prime, col, m.q);
    const uint64_t *digits = ra.dig[r];
    acc128 a0{0, 0}, a1{0, 0};
    if constexpr (ND > 0 && !SEEDED) {
        uint64_t dv[ND], bv[ND], av[ND];
#pragma unroll
        for (int j = 0; j < ND; j++) {
            dv[j] = digits[(((size_t)j * ext + row) << log_n) + sc];
            bv[j] = kr.b(j);
            av[j] = kr.a(j);
        }
#pragma unroll
        for (int j = 0; j < ND; j++) {
            mac(a0, dv[j], bv[j]);
            mac(a1, dv[j], av[j]);
        }
    } else {
        for (uint32_t j = 0; j < nd; j++) {
            const uint64_t d = digits[(((size_t)j * ext + row) << log_n) + sc];
            mac(a0, d, kr.b(j));
            mac(a1, d, kr.a(j));
        }
    }
    uint64_t *ur = u + (((size_t)r * 2 * rows + (row - row0)) << log_n) + col;
    ur[0] = reduce128(a0, m);
    ur[(size_t)rows << log_n] = reduce128(a1, m);
}

// k_key_ip_batch with stored keys: the digit count as a template argument for 1..6 digits, the loop beyond
template <int ND>
void launch_key_ip_batch_nd(dim3 grid, dim3 block, hipStream_t st, const RotArgs &ra, uint64_t *u, uint32_t nd,
                            uint32_t ext, uint32_t level, uint32_t n_q, uint32_t key_rows, uint32_t row0,
                            uint32_t rows, const ModQ *mods, uint32_t log_n)
{
    hipLaunchKernelGGL((k_key_ip_batch<false, ND>), grid, block, 0, st, ra, u, nd, ext, level, n_q, key_rows, row0,
                       rows, mods, log_n);
}

void launch_key_ip_batch_stored(dim3 grid, dim3 block, hipStream_t st, const RotArgs &ra, uint64_t *u, uint32_t nd,
                                uint32_t ext, uint32_t level, uint32_t n_q, uint32_t key_rows, uint32_t row0,
                                uint32_t rows, const ModQ *mods, uint32_t log_n)
{
#define CK_IPB(K) launch_key_ip_batch_nd<K>(grid, block, st, ra, u, nd, ext, level, n_q, key_rows, row0, rows, mods, log_n)
    switch (nd) {
    case 1: CK_IPB(1); break;
    case 2: CK_IPB(2); break;
    case 3: CK_IPB(3); break;
    case 4: CK_IPB(4); break;
    case 5: CK_IPB(5); break;
    case 6: CK_IPB(6); break;
    default: CK_IPB(0); break;
    }
#undef CK_IPB
}

// Lazy ModDown: the key inner products of several rotations summed over Q_level u P before one division by P.
// For rotation r: t_k = sum_j sigma_{g_r}(d_j) * key_r[j][k] on every row, plus P * sigma_{g_r}(c0_r) on the q rows of
// component 0 (P is 0 modulo the special primes, and ModDown(x + P y) = ModDown(x) + y, so the c0 term passes the
// division unchanged).  sum_all: one accumulator ra.out[0] takes the sum over all r of the batch; else ra.out[r]
// takes rotation r's.  Accumulators [2][ext][N], added to when `accumulate`.  The 128-bit sums hold at most
// 32 (nd + 1) products below 2^100.
template <int ND>
__global__ __launch_bounds__(kThreads) void k_key_ip_acc(RotArgs ra, uint32_t nd, uint32_t ext, uint32_t level,
                                                         uint32_t n_q, uint32_t key_rows,
                                                         const ulonglong2 *__restrict__ pmodq,
                                                         const ModQ *__restrict__ mods, uint32_t log_n, int sum_all,
                                                         int accumulate)
{
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t row = blockIdx.y;
    if (col >= n) return;
    const uint32_t r0 = sum_all ? 0 : blockIdx.z, r1 = sum_all ? ra.count : blockIdx.z + 1;
    const uint32_t prime = row <= level ? row : n_q + (row - level - 1);
    const ModQ m = mods[prime];
    const uint64_t pq = row <= level ? pmodq[row].x : 0;
    acc128 a0{0, 0}, a1{0, 0};
    if constexpr (ND > 0) {
        // every word rotation r needs (its digits' gathers, key words and c0) loaded in one go, and rotation
        // r + 1's loads issued before rotation r's products: one memory wait per rotation, overlapped
        struct Words {
            uint64_t d[ND], b[ND], a[ND], c;
        };
        const size_t kstride = (size_t)key_rows << log_n;
        auto load = [&](uint32_t r, Words &w) {
            const uint32_t sc = auto_index(col, ra.g[r], log_n);
            const uint64_t *key = ra.key[r] + ((size_t)prime << log_n) + col;
            const uint64_t *digits = ra.dig[r] + ((size_t)row << log_n) + sc;
#pragma unroll
            for (int j = 0; j < ND; j++) {
                w.d[j] = digits[(size_t)j * ext << log_n];
                w.b[j] = nttc::ld_stream(key + 2 * j * kstride);
                w.a[j] = nttc::ld_stream(key + (2 * j + 1) * kstride);
            }
            // loaded on every row (row 0 of c0 for the P rows, unused there) so that every path issues the same
            // loads and the waits stay partial
            w.c = ra.c0[r][((size_t)(pq ? row : 0) << log_n) + sc];
        };
        auto use = [&](const Words &w) {
#pragma unroll
            for (int j = 0; j < ND; j++) {
                mac(a0, w.d[j], w.b[j]);
                mac(a1, w.d[j], w.a[j]);
            }
            if (pq) mac(a0, w.c, pq);
        };
        // two register sets used in turn, with no copies between them and no loads under a condition inside the
        // loop: either would make the compiler wait for the newer loads as well
        Words w0, w1;
        load(r0, w0);
        uint32_t r = r0;
        for (; r + 2 < r1; r += 2) {
            load(r + 1, w1);
            use(w0);
            load(r + 2, w0);
            use(w1);
        }
        if (r + 1 < r1) {
            load(r + 1, w1);
            use(w0);
            use(w1);
        } else {
            use(w0);
        }
    } else {
        for (uint32_t r = r0; r < r1; r++) {
            const uint32_t sc = auto_index(col, ra.g[r], log_n);
            const uint64_t *key = ra.key[r];
            const uint64_t *digits = ra.dig[r];
            for (uint32_t j = 0; j < nd; j++) {
                const uint64_t d = digits[(((size_t)j * ext + row) << log_n) + sc];
                const size_t kb = ((size_t)j * 2 * key_rows + prime) << log_n;
                mac(a0, d, nttc::ld_stream(key + kb + col));
                mac(a1, d, nttc::ld_stream(key + kb + ((size_t)key_rows << log_n) + col));
            }
            if (pq) mac(a0, ra.c0[r][((size_t)row << log_n) + sc], pq);
        }
    }
    uint64_t *u = ra.out[r0] + ((size_t)row << log_n) + col;
    uint64_t v0 = reduce128(a0, m), v1 = reduce128(a1, m);
    if (accumulate) {
        v0 = addmod(v0, u[0], m.q);
        v1 = addmod(v1, u[(size_t)ext << log_n], m.q);
    }
    u[0] = v0;
    u[(size_t)ext << log_n] = v1;
}

// The key inner products of a rotation batch's P rows fused with the first (row) pass of their inverse
// transform (fp64, 256-point rows): block (r, P limb i, two rows h), one wave, 8 positions per thread as in
// k_ks_finish8.  u_k = sum_j sigma_{g_r}(d_j)[L + i] * key_r[j][k][n_q + i] (the products and range reductions
// of k_ks_finish8's inner product), reduced below q/2 + 1, then the row's Gentleman-Sande stages with its inverse
// twiddles; written as raw doubles below 2q to up[r][k][i], the inter-pass form the inverse column pass reads.
// The P rows of u thus never go to HBM in canonical form to be read back by a separate row pass.
template <bool SEEDED, int ND>
__global__ __launch_bounds__(64) void k_key_ip_intt8(RotArgs ra, uint64_t *up, uint32_t nd, uint32_t ext,
                                                     uint32_t L, uint32_t K, uint32_t n_q, uint32_t key_rows,
                                                     const ModQ *__restrict__ mods, const double *__restrict__ itwf,
                                                     uint32_t log_n, uint32_t blocks_per_limb)
{
    using nttc::kE8;
    __shared__ double tws[2][257];
    __shared__ double tr[2][nttc::kTr8];
    const uint32_t per_rot = K * blocks_per_limb;
    const uint32_t r = blockIdx.x / per_rot, rem = blockIdx.x % per_rot;
    const uint32_t i = rem / blocks_per_limb, blk = rem % blocks_per_limb;
    const uint32_t prime = n_q + i, row = L + i;
    const nttc::Ar<true> ar(mods[prime]);
    const uint32_t sub = threadIdx.x >> 5, t = threadIdx.x & 31;
    const uint32_t h = blk * 2 + sub;
    nttc::stage_twiddles8(tws[sub], itwf + ((size_t)prime << log_n), (1u << (log_n - 8)) + h, t, 32);
    const uint32_t g = ra.g[r];
    uint32_t pos[kE8], sc[kE8];
#pragma unroll
    for (int e = 0; e < kE8; e++) {
        pos[e] = h * 256 + nttc::u8<0>(t, e);
        sc[e] = auto_index(pos[e], g, log_n);
    }
    double u[2][kE8];
    key_ip8<SEEDED, ND>(ra, r, nd, ext, row, prime, key_rows, log_n, mods[prime].q, ar, pos, sc, u[0], u[1]);
#pragma unroll
    for (int e = 0; e < kE8; e++) {
        u[0][e] = ar.red(u[0][e]);
        u[1][e] = ar.red(u[1][e]);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 2; k++) {
        double x[kE8];
#pragma unroll
        for (int e = 0; e < kE8; e++) x[e] = u[k][e];
        nttc::a_to_b8(x, tr[sub], t);
        nttc::inv8_256(x, tws[sub], tr[sub], t, ar);
        uint64_t *out = up + ((((size_t)r * 2 + k) * K + i) << log_n) + (size_t)h * 256;
#pragma unroll
        for (int e = 0; e < kE8; e++) nttc::st_stream(out + nttc::u8<0>(t, e), nttc::Ar<true>::to_raw(x[e]));
    }
}

// ModDown of a batch of rotations, fused (fp64, 256-point rows)// ModDown of a batch of rotations, fused (fp64, 256-point rows): block (r, q-limb i, two rows h) finishes the
// forward transform of the converted P part cw[r][k][i] (its first pass already done), computes the q-limb part
// of the key inner product u_k = sum_j sigma_{g_r}(d_j)[i] * key_r[j][k][i] in registers, and writes
//   out_r[k][i] = (u_k - NTT(cw[r][k][i])) * P^-1 (+ sigma_{g_r}(c0)[i] for k = 0),
// so neither the q-limb rows of u nor the transformed conversion ever go to HBM.  Magnitudes (units of q):
// column-pass outputs <= 4.3 (from inputs reduced to q/2), transform outputs <= 2.6, each product <= 0.875 and the
// sum range-reduced every 4 digits (<= 4), differences <= 6.6, P^-1 products <= 3, plus c0 < 1: all below 8 q = 2^53.
__global__ __launch_bounds__(64) void k_ks_finish8(RotArgs ra, const uint64_t *__restrict__ cw, uint32_t nd,
                                                   uint32_t ext,
                                                   uint32_t L, uint32_t key_rows, const ModQ *__restrict__ mods,
                                                   const double *__restrict__ twf,
                                                   const ulonglong2 *__restrict__ pinv, uint32_t log_n,
                                                   uint32_t blocks_per_limb)
{
    using nttc::kE8;
    __shared__ double tws[2][257];
    __shared__ double tr[2][nttc::kTr8];
    const uint32_t per_rot = L * blocks_per_limb;
    const uint32_t r = blockIdx.x / per_rot, rem = blockIdx.x % per_rot;
    const uint32_t i = rem / blocks_per_limb, blk = rem % blocks_per_limb;
    const nttc::Ar<true> ar(mods[i]);
    const uint32_t sub = threadIdx.x >> 5, t = threadIdx.x & 31;
    const uint32_t h = blk * 2 + sub;
    nttc::stage_twiddles8(tws[sub], twf + ((size_t)i << log_n), (1u << (log_n - 8)) + h, t, 32);
    __syncthreads();
    const size_t row = ((size_t)i << log_n) + (size_t)h * 256;
    double v[2][kE8];
#pragma unroll
    for (int k = 0; k < 2; k++) {
        const uint64_t *src = cw + (((size_t)r * 2 + k) * L << log_n) + row;
        double x[kE8];
#pragma unroll
        for (int e = 0; e < kE8; e++) x[e] = nttc::Ar<true>::from_raw(nttc::ld_stream(src + nttc::u8<0>(t, e)));
        nttc::fwd8_256<nttc::kRowMask8>(x, tws[sub], tr[sub], t, ar);
        nttc::b_to_a8(x, tr[sub], t);
#pragma unroll
        for (int e = 0; e < kE8; e++) v[k][e] = x[e];
    }
    const uint32_t g = ra.g[r];
    uint64_t *out = ra.out[r];
    const uint64_t *digits = ra.dig[r], *c0 = ra.c0[r];
    const double pi = (double)pinv[i].x;
    const uint64_t qi = mods[i].q;
#pragma unroll
    for (int e = 0; e < kE8; e++) {
        const uint32_t pos = h * 256 + nttc::u8<0>(t, e);
        const uint32_t sc = auto_index(pos, g, log_n);
        KeyRow<false> kr(ra, r, key_rows, log_n, i, pos, qi);
        double u0 = 0.0, u1 = 0.0;
        for (uint32_t j = 0; j < nd; j++) {
            const double d = nttc::Ar<true>::from_u64(digits[(((size_t)j * ext + i) << log_n) + sc]);
            u0 += ar.mul(d, nttc::Ar<true>::from_u64(kr.b(j)));
            u1 += ar.mul(d, nttc::Ar<true>::from_u64(kr.a(j)));
            if ((j & 3) == 3) {
                u0 = ar.red(u0);
                u1 = ar.red(u1);
            }
        }
        const double r0 = ar.mul(u0 - v[0][e], pi) + nttc::Ar<true>::from_u64(c0[((size_t)i << log_n) + sc]);
        const double r1 = ar.mul(u1 - v[1][e], pi);
        nttc::st_stream(out + ((size_t)i << log_n) + pos, ar.to_canon(r0));
        nttc::st_stream(out + (((size_t)L + i) << log_n) + pos, ar.to_canon(r1));
    }
}

// k_ks_finish8 for seed-expanded keys: the inner products (with their Philox blocks) first, every position's
// loads issued before the transforms, and c0's gathers at the start.  (With stored keys the same order, 160 VGPRs
// and 3 waves per SIMD, measured 5% slower than k_ks_finish8's one position at a time after the transforms, 88
// VGPRs and 5 waves: that kernel streams ~5 TB/s of keys, converted rows and outputs.)
template <int ND>
__global__ __launch_bounds__(64) void k_ks_finish8_seeded(RotArgs ra, const uint64_t *__restrict__ cw, uint32_t nd,
                                                          uint32_t ext, uint32_t L, uint32_t key_rows,
                                                          const ModQ *__restrict__ mods,
                                                          const double *__restrict__ twf,
                                                          const ulonglong2 *__restrict__ pinv, uint32_t log_n,
                                                          uint32_t blocks_per_limb)
{
    using nttc::kE8;
    __shared__ double tws[2][257];
    __shared__ double tr[2][nttc::kTr8];
    const uint32_t per_rot = L * blocks_per_limb;
    const uint32_t r = blockIdx.x / per_rot, rem = blockIdx.x % per_rot;
    const uint32_t i = rem / blocks_per_limb, blk = rem % blocks_per_limb;
    const nttc::Ar<true> ar(mods[i]);
    const uint32_t sub = threadIdx.x >> 5, t = threadIdx.x & 31;
    const uint32_t h = blk * 2 + sub;
    nttc::stage_twiddles8(tws[sub], twf + ((size_t)i << log_n), (1u << (log_n - 8)) + h, t, 32);
    const uint32_t g = ra.g[r];
    const uint64_t *c0 = ra.c0[r] + ((size_t)i << log_n);
    uint32_t pos[kE8], sc[kE8];
    uint64_t c0v[kE8];
#pragma unroll
    for (int e = 0; e < kE8; e++) {
        pos[e] = h * 256 + nttc::u8<0>(t, e);
        sc[e] = auto_index(pos[e], g, log_n);
        c0v[e] = c0[sc[e]];
    }
    double u0[kE8], u1[kE8];
    key_ip8<true, ND>(ra, r, nd, ext, i, i, key_rows, log_n, mods[i].q, ar, pos, sc, u0, u1);
    __syncthreads();
    const size_t row = ((size_t)i << log_n) + (size_t)h * 256;
    double v[2][kE8];
#pragma unroll
    for (int k = 0; k < 2; k++) {
        const uint64_t *src = cw + (((size_t)r * 2 + k) * L << log_n) + row;
        double x[kE8];
#pragma unroll
        for (int e = 0; e < kE8; e++) x[e] = nttc::Ar<true>::from_raw(nttc::ld_stream(src + nttc::u8<0>(t, e)));
        nttc::fwd8_256<nttc::kRowMask8>(x, tws[sub], tr[sub], t, ar);
        nttc::b_to_a8(x, tr[sub], t);
#pragma unroll
        for (int e = 0; e < kE8; e++) v[k][e] = x[e];
    }
    uint64_t *out = ra.out[r];
    const double pi = (double)pinv[i].x;
#pragma unroll
    for (int e = 0; e < kE8; e++) {
        const double r0 = ar.mul(u0[e] - v[0][e], pi) + nttc::Ar<true>::from_u64(c0v[e]);
        const double r1 = ar.mul(u1[e] - v[1][e], pi);
        nttc::st_stream(out + ((size_t)i << log_n) + pos[e], ar.to_canon(r0));
        nttc::st_stream(out + (((size_t)L + i) << log_n) + pos[e], ar.to_canon(r1));
    }
}

// out_r[k][i][n] = (u[r][k][i][n] - c[r][k][i][n]) * P^-1 (+ c0[i][sigma_{g_r}(n)] for k = 0)
__global__ __launch_bounds__(kThreads) void k_moddown_finish_batch(RotArgs ra, const uint64_t *u, const uint64_t *c,
                                                                    uint32_t ext, uint32_t level,
                                                                    const ulonglong2 *__restrict__ pinv,
                                                                    const ModQ *__restrict__ mods, uint32_t log_n)
{
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t i = blockIdx.y, rk = blockIdx.z, r = rk >> 1, k = rk & 1;
    if (col >= n) return;
    const uint32_t L = level + 1;
    const uint64_t q = mods[i].q;
    const uint64_t x = u[(((size_t)rk * ext + i) << log_n) + col];
    const uint64_t cv = c[(((size_t)rk * L + i) << log_n) + col];
    const ulonglong2 w = pinv[i];
    uint64_t res = shoup(submod(x, cv, q), w.x, w.y, q);
    if (k == 0) res = addmod(res, ra.c0[r][((size_t)i << log_n) + auto_index(col, ra.g[r], log_n)], q);
    ra.out[r][(((size_t)k * L + i) << log_n) + col] = res;
}

ckks_status launch_conv(ckks_ctx *ctx, const ConvDev *cd, const uint64_t *in, uint32_t in_stride, uint64_t *out,
                        uint32_t out_stride, uint32_t split, uint32_t skip, uint32_t polys)
{
    ConvArgs a;
    a.ns = cd->ns;
    a.nt = cd->nt;
    for (int i = 0; i < cd->ns; i++) a.src[i] = cd->src[i];
    for (int t = 0; t < cd->nt; t++) a.dst[t] = cd->dst[t];
    const dim3 grid((ctx->n + kThreads - 1) / kThreads, polys), block(kThreads);
    // fp64 kernels: two coefficients per thread where the ring has at least 512 of them and that still leaves
    // 4096 waves (4 per SIMD); with fewer polynomials one coefficient per thread, and the target limbs split over
    // blockIdx.z until the grid has that many waves
    const size_t waves1 = (size_t)((ctx->n + 63) / 64) * polys;
    const bool two = ctx->n % (2 * kThreads) == 0 && waves1 / 2 >= 4096;
    uint32_t groups = 1;
    const uint32_t ntg = a.nt > 0 ? (uint32_t)a.nt : 1u;
    if (!two && waves1 < 4096) groups = (uint32_t)std::min<size_t>(ntg, (4096 + waves1 - 1) / waves1);
    const uint32_t t_per = (ntg + groups - 1) / groups;
    groups = (ntg + t_per - 1) / t_per;
    const dim3 grid1(grid.x, polys, groups);
    const dim3 grid2(two ? (uint32_t)(ctx->n / (2 * kThreads)) : grid.x, polys, two ? 1 : groups);
    prof_begin(ctx, K_CONV, 8.0 * polys * (a.ns + a.nt) * ctx->n);
#define CK_CONVF(NSM)                                                                                              \
    do {                                                                                                           \
        if (two && a.ns == NSM)                                                                                    \
            hipLaunchKernelGGL((k_conv_f64<NSM, 2, true>), grid2, block, 0, ctx->stream, in, in_stride, out,        \
                               out_stride, split, skip, a, cd->d_qhat_inv_f, cd->d_qhat_mod_f, ctx->d_mod,          \
                               ctx->log_n, (uint32_t)a.nt);                                                        \
        else if (a.ns == NSM)                                                                                      \
            hipLaunchKernelGGL((k_conv_f64<NSM, 1, true>), grid1, block, 0, ctx->stream, in, in_stride, out,        \
                               out_stride, split, skip, a, cd->d_qhat_inv_f, cd->d_qhat_mod_f, ctx->d_mod,          \
                               ctx->log_n, t_per);                                                                 \
        else if (two)                                                                                              \
            hipLaunchKernelGGL((k_conv_f64<NSM, 2>), grid2, block, 0, ctx->stream, in, in_stride, out, out_stride,  \
                               split, skip, a, cd->d_qhat_inv_f, cd->d_qhat_mod_f, ctx->d_mod, ctx->log_n,         \
                               (uint32_t)a.nt);                                                                    \
        else                                                                                                       \
            hipLaunchKernelGGL((k_conv_f64<NSM, 1>), grid1, block, 0, ctx->stream, in, in_stride, out, out_stride,  \
                               split, skip, a, cd->d_qhat_inv_f, cd->d_qhat_mod_f, ctx->d_mod, ctx->log_n, t_per); \
    } while (0)
    if (cd->f64 && !ctx->int_only && a.ns <= 16) {
        if (a.ns <= 8)
            CK_CONVF(8);
        else
            CK_CONVF(16);
    } else if (a.ns <= 4)
        hipLaunchKernelGGL(k_conv<4>, grid, block, 0, ctx->stream, in, in_stride, out, out_stride, split, skip, a,
                           cd->d_qhat_inv, cd->d_qhat_mod, cd->d_neg_q, ctx->d_mod, ctx->log_n);
    else if (a.ns <= 8)
        hipLaunchKernelGGL(k_conv<8>, grid, block, 0, ctx->stream, in, in_stride, out, out_stride, split, skip, a,
                           cd->d_qhat_inv, cd->d_qhat_mod, cd->d_neg_q, ctx->d_mod, ctx->log_n);
    else if (a.ns <= 16)
        hipLaunchKernelGGL(k_conv<16>, grid, block, 0, ctx->stream, in, in_stride, out, out_stride, split, skip, a,
                           cd->d_qhat_inv, cd->d_qhat_mod, cd->d_neg_q, ctx->d_mod, ctx->log_n);
    else if (a.ns <= 32)
        hipLaunchKernelGGL(k_conv<32>, grid, block, 0, ctx->stream, in, in_stride, out, out_stride, split, skip, a,
                           cd->d_qhat_inv, cd->d_qhat_mod, cd->d_neg_q, ctx->d_mod, ctx->log_n);
    else {
        prof_end(ctx, K_CONV);
        return set_error(CKKS_EUNSUPPORTED, "basis conversion from %d limbs (at most 32)", a.ns);
    }
#undef CK_CONVF
    prof_end(ctx, K_CONV);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

// The raw fp64 conversion of `polys` polynomials followed by the first forward column pass of its output rows
// (N = 2^16, at most 8 source limbs), in one kernel: out rows as launch_conv writes them, in the inter-pass form.
ckks_status launch_conv_col8(ckks_ctx *ctx, const ConvDev *cd, const uint64_t *in, uint32_t in_stride, uint64_t *out,
                             uint32_t out_stride, uint32_t split, uint32_t skip, uint32_t polys)
{
    CK_REQUIRE(ctx->log_n == 16 && cd->f64 && !ctx->int_only && cd->ns >= 1 && cd->ns <= 8 && cd->nt >= 1,
               CKKS_EINVAL, "fused conversion needs N = 2^16, the fp64 tables and 1..8 source limbs");
    CK_REQUIRE(split <= (uint32_t)cd->nt && (uint32_t)cd->nt + skip <= out_stride && cd->ns <= (int)in_stride,
               CKKS_EINVAL, "fused conversion: target rows outside the output");
    ConvArgs a;
    a.ns = cd->ns;
    a.nt = cd->nt;
    for (int i = 0; i < cd->ns; i++) a.src[i] = cd->src[i];
    for (int t = 0; t < cd->nt; t++) a.dst[t] = cd->dst[t];
    const uint32_t bpr = 1u << (ctx->log_n - 12);
    const double res = (double)polys * ctx->n;
    // the sources once, the converted rows once; the conversion products and the column pass's butterflies
    prof_begin(ctx, K_CONV, 8.0 * res * (a.ns + a.nt), res * a.nt * (a.ns * 5.0 + kOpsButterflyF64 * 4));
    if (a.ns == 8)
        hipLaunchKernelGGL(k_conv_col8<true>, dim3(polys * bpr), dim3(512), 0, ctx->stream, in, in_stride, out,
                           out_stride, split, skip, a, cd->d_qhat_inv_f, cd->d_qhat_mod_f, ctx->d_mod, ctx->d_twf,
                           ctx->log_n, bpr);
    else
        hipLaunchKernelGGL(k_conv_col8<false>, dim3(polys * bpr), dim3(512), 0, ctx->stream, in, in_stride, out,
                           out_stride, split, skip, a, cd->d_qhat_inv_f, cd->d_qhat_mod_f, ctx->d_mod, ctx->d_twf,
                           ctx->log_n, bpr);
    prof_end(ctx, K_CONV);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

// The a half [dnum][R][N] of a seed-expanded key: thread (prime k, position n) draws the Philox blocks of every
// group of four digits (philox.h).
__global__ __launch_bounds__(256) void k_expand_key_a(uint64_t *a, uint64_t s0, uint64_t s1, uint32_t dnum,
                                                      uint32_t R, const ModQ *__restrict__ mods, uint32_t log_n)
{
    const uint32_t col = blockIdx.x * 256 + threadIdx.x, k = blockIdx.y;
    if (col >= (1u << log_n)) return;
    const uint64_t q = mods[k].q;
    const uint32_t shift = seedk::shift_of(q);
    uint64_t blk[4];
    for (uint32_t j = 0; j < dnum; j++) {
        const uint32_t m = j & 3;
        if (m == 0) seedk::block_residues(s0, s1, col, k, j >> 2, q, shift, blk);
        a[(((size_t)j * R + k) << log_n) + col] = m == 0 ? blk[0] : m == 1 ? blk[1] : m == 2 ? blk[2] : blk[3];
    }
}

}  // namespace

ckks_status launch_expand_key_a(ckks_ctx *ctx, uint64_t s0, uint64_t s1, uint64_t *a)
{
    const uint32_t R = ctx->n_primes();
    const dim3 grid((ctx->n + 255) / 256, R), block(256);
    prof_begin(ctx, K_ELEM, 8.0 * ctx->dnum * R * ctx->n);
    hipLaunchKernelGGL(k_expand_key_a, grid, block, 0, ctx->stream, a, s0, s1, ctx->dnum, R, ctx->d_mod, ctx->log_n);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

uint32_t ks_rot_batch(uint32_t count) { return count < (uint32_t)kRotBatch ? count : (uint32_t)kRotBatch; }

size_t ks_scratch_words(const ckks_ctx *ctx, uint32_t level, uint32_t batch, uint32_t n_ct)
{
    const size_t ext = level + 1 + ctx->n_p;
    const size_t nd = n_digits(ctx, level);
    if (batch < 1) batch = 1;
    if (n_ct < 1) n_ct = 1;
    // per input ciphertext: digits + INTT staging [alpha]; per rotation of a batch: u[2][ext] and the converted
    // rows [2][level+1]
    return ((size_t)n_ct * (nd * ext + ctx->alpha) + (size_t)batch * (2 * ext + 2 * (level + 1))) << ctx->log_n;
}

// The fused kernels take the digit count as a template argument for 1..4 digits (dnum up to 4 at any level,
// and the low levels of larger dnum), fully unrolled; more digits take the run-time loop.
#define CK_ND_DISPATCH(nd, LAUNCH, SD)                                                                             \
    do {                                                                                                           \
        switch (nd) {                                                                                              \
        case 1: LAUNCH(SD, 1); break;                                                                              \
        case 2: LAUNCH(SD, 2); break;                                                                              \
        case 3: LAUNCH(SD, 3); break;                                                                              \
        case 4: LAUNCH(SD, 4); break;                                                                              \
        default: LAUNCH(SD, 0); break;                                                                             \
        }                                                                                                          \
    } while (0)

ckks_status ks_rotate_batch(ckks_ctx *ctx, uint32_t level, uint32_t count, const uint64_t *const *c0s,
                            const uint64_t *const *digs, const uint32_t *g, const uint64_t *const *keys,
                            uint64_t *const *outs, uint64_t *work, const uint64_t *seeds)
{
    CK_REQUIRE(count >= 1 && count <= (uint32_t)kRotBatch, CKKS_EINVAL, "rotation batch of %u", count);
    const uint32_t L = level + 1, K = ctx->n_p, ext = L + K, nd = n_digits(ctx, level);
    const size_t N = ctx->n;
    const bool seeded = seeds != nullptr;
    RotArgs ra{};
    ra.count = count;
    for (uint32_t r = 0; r < count; r++) {
        ra.g[r] = g[r];
        ra.key[r] = keys[r];
        ra.out[r] = outs[r];
        ra.dig[r] = digs[r];
        ra.c0[r] = c0s[r];
        if (seeded) {
            ra.seed[r][0] = seeds[2 * r];
            ra.seed[r][1] = seeds[2 * r + 1];
        }
    }
    // a seeded key holds its b half only: key_rows rows per digit instead of 2 key_rows
    const uint32_t kp = ctx->n_primes();
    int s1, s2;
    ntt_split(ctx->log_n, &s1, &s2);
    if (s2 == 8 && ntt_uses_f64(ctx, L)) {
        // fused ModDown: only the P rows of u are formed in HBM
        uint64_t *up = work;                             // [count][2][K][N]
        uint64_t *cw = up + (size_t)count * 2 * K * N;   // [count][2][L][N]
        bool p_f64 = !ctx->int_only;
        for (uint32_t i = 0; i < K; i++) p_f64 = p_f64 && ctx->f64_ok[ctx->n_q + i];
        if (s1 == 8 && p_f64) {
            // the P rows' inner products with the first pass of their inverse transform, then its second pass
            const uint32_t bpl = 1u << (ctx->log_n - 9);
            const double res = (double)count * 2 * K * N;
            prof_begin(ctx, K_KEYIP, 8.0 * res * (nd + 1.0) + 8.0 * (double)nd * K * N,
                       res * (nd * 10.0 + 4 * kOpsButterflyF64 + 8.0));
#define CK_IPI(SD, ND)                                                                                             \
    hipLaunchKernelGGL((k_key_ip_intt8<SD, ND>), dim3(count * K * bpl), dim3(64), 0, ctx->stream, ra, up, nd, ext, L, \
                       K, ctx->n_q, kp, ctx->d_mod, ctx->d_itwf, ctx->log_n, bpl)
            if (seeded)
                CK_ND_DISPATCH(nd, CK_IPI, true);
            else
                CK_ND_DISPATCH(nd, CK_IPI, false);
#undef CK_IPI
            prof_end(ctx, K_KEYIP);
            HIP_TRY(hipGetLastError());
            CK_TRY(launch_ntt_inv_second_pass(ctx, up, 2 * count, K, limb_range(ctx->n_q, K)));
        } else {
            const dim3 grid((ctx->n + kThreads - 1) / kThreads, K, count), block(kThreads);
            prof_begin(ctx, K_KEYIP, 8.0 * ctx->n * K * (count * (2.0 * nd + 2.0) + nd));
            if (seeded)
                hipLaunchKernelGGL(k_key_ip_batch<true>, grid, block, 0, ctx->stream, ra, up, nd, ext, level,
                                   ctx->n_q, kp, L, K, ctx->d_mod, ctx->log_n);
            else
                launch_key_ip_batch_stored(grid, block, ctx->stream, ra, up, nd, ext, level, ctx->n_q, kp, L, K,
                                           ctx->d_mod, ctx->log_n);
            prof_end(ctx, K_KEYIP);
            HIP_TRY(hipGetLastError());
            CK_TRY(launch_ntt_strided(ctx, up, 2 * count, K, limb_range(ctx->n_q, K), true));
        }
        const ConvDev *cd;
        CK_TRY(ctx_conv(ctx, (int)level, -1, &cd));
        if (s1 == 8 && cd->f64 && !ctx->int_only && cd->ns <= 8) {
            // the conversion and the first forward pass of the converted rows in one kernel
            CK_TRY(launch_conv_col8(ctx, cd, up, K, cw, L, L, 0, 2 * count));
        } else {
            CK_TRY(launch_conv(ctx, cd, up, K, cw, L, L, 0, 2 * count));
            CK_TRY(launch_ntt_fwd_first_pass(ctx, cw, 2 * count, L, limb_range(0, L)));
        }
        const uint32_t bpl = 1u << (ctx->log_n - 9);
        // cw rows once, the key's q rows, the outputs; digits and c0 are cache-resident gathers
        const double res = (double)count * L * N;
        prof_begin(ctx, K_MODDOWN, 8.0 * res * (2.0 + 2.0 * nd + 2.0),
                   res * (2 * (4 * kOpsButterflyF64 + 4 * (kOpsButterflyF64 - 3)) / 2 + nd * 2 * 10.0 + 40.0));
#define CK_FIN(SD, ND)                                                                                             \
    hipLaunchKernelGGL((k_ks_finish8_seeded<ND>), dim3(count * L * bpl), dim3(64), 0, ctx->stream, ra, cw, nd, ext, \
                       L, kp, ctx->d_mod, ctx->d_twf, ctx->d_pinv, ctx->log_n, bpl)
        if (seeded)
            CK_ND_DISPATCH(nd, CK_FIN, true);
        else
            hipLaunchKernelGGL(k_ks_finish8, dim3(count * L * bpl), dim3(64), 0, ctx->stream, ra, cw, nd, ext, L, kp,
                               ctx->d_mod, ctx->d_twf, ctx->d_pinv, ctx->log_n, bpl);
#undef CK_FIN
        prof_end(ctx, K_MODDOWN);
        HIP_TRY(hipGetLastError());
        return CKKS_OK;
    }
    uint64_t *u = work;                              // [count][2][ext][N]
    uint64_t *cw = u + (size_t)count * 2 * ext * N;  // [count][2][L][N]
    {
        const dim3 grid((ctx->n + kThreads - 1) / kThreads, ext, count), block(kThreads);
        prof_begin(ctx, K_KEYIP, 8.0 * ctx->n * ext * (count * (2.0 * nd + 2.0) + nd));
        if (seeded)
            hipLaunchKernelGGL(k_key_ip_batch<true>, grid, block, 0, ctx->stream, ra, u, nd, ext, level, ctx->n_q,
                               kp, 0u, ext, ctx->d_mod, ctx->log_n);
        else
            launch_key_ip_batch_stored(grid, block, ctx->stream, ra, u, nd, ext, level, ctx->n_q, kp, 0u, ext,
                                       ctx->d_mod, ctx->log_n);
        prof_end(ctx, K_KEYIP);
        HIP_TRY(hipGetLastError());
    }
    CK_TRY(launch_ntt_strided(ctx, u + (size_t)L * N, 2 * count, ext, limb_range(ctx->n_q, K), true));
    const ConvDev *cd;
    CK_TRY(ctx_conv(ctx, (int)level, -1, &cd));
    CK_TRY(launch_conv(ctx, cd, u + (size_t)L * N, ext, cw, L, L, 0, 2 * count));
    CK_TRY(launch_ntt(ctx, cw, 2 * count * L, limb_range(0, L), false));
    {
        const dim3 grid((ctx->n + kThreads - 1) / kThreads, L, 2 * count), block(kThreads);
        prof_begin(ctx, K_MODDOWN, 8.0 * ctx->n * L * count * 7.0);
        hipLaunchKernelGGL(k_moddown_finish_batch, grid, block, 0, ctx->stream, ra, u, cw, ext, level,
                           ctx->d_pinv, ctx->d_mod, ctx->log_n);
        prof_end(ctx, K_MODDOWN);
        HIP_TRY(hipGetLastError());
    }
    return CKKS_OK;
}

ckks_status ks_ip_accumulate(ckks_ctx *ctx, uint32_t level, uint32_t count, const uint64_t *const *c0s,
                             const uint64_t *const *digs, const uint32_t *g, const uint64_t *const *keys,
                             uint64_t *const *accs, bool sum_all, bool accumulate)
{
    CK_REQUIRE(count >= 1 && count <= (uint32_t)kRotBatch, CKKS_EINVAL, "rotation batch of %u", count);
    const uint32_t L = level + 1, ext = L + ctx->n_p, nd = n_digits(ctx, level);
    // one accumulator summing every rotation takes count (nd + 1) products in its exact 128-bit sum: with large
    // primes, fewer rotations per launch, the later launches adding to the reduced sum
    const uint32_t per = std::max(1u, ctx->sum128_terms / (nd + 1));
    if (sum_all && count > per) {
        for (uint32_t r0 = 0; r0 < count; r0 += per) {
            const uint32_t cnt = std::min(per, count - r0);
            CK_TRY(ks_ip_accumulate(ctx, level, cnt, c0s + r0, digs + r0, g + r0, keys + r0, accs, true,
                                    accumulate || r0 > 0));
        }
        return CKKS_OK;
    }
    RotArgs ra{};
    ra.count = count;
    for (uint32_t r = 0; r < count; r++) {
        ra.g[r] = g[r];
        ra.key[r] = keys[r];
        ra.out[r] = accs[sum_all ? 0 : r];
        ra.dig[r] = digs[r];
        ra.c0[r] = c0s[r];
    }
    const dim3 grid((ctx->n + kThreads - 1) / kThreads, ext, sum_all ? 1 : count), block(kThreads);
    const double outs = sum_all ? 1.0 : count;
    // digits and keys of every rotation, c0, the accumulators read (when accumulating) and written
    prof_begin(ctx, K_KEYIP, 8.0 * ctx->n * ext * (count * (3.0 * nd) + (double)L / ext * count +
                                                   outs * 2.0 * (accumulate ? 2 : 1)));
#define CK_ACC(SD, ND)                                                                                             \
    hipLaunchKernelGGL(k_key_ip_acc<ND>, grid, block, 0, ctx->stream, ra, nd, ext, level, ctx->n_q,                  \
                       ctx->n_primes(), ctx->d_pmodq, ctx->d_mod, ctx->log_n, (int)sum_all, (int)accumulate)
    CK_ND_DISPATCH(nd, CK_ACC, 0);
#undef CK_ACC
    prof_end(ctx, K_KEYIP);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status ks_modup_batch(ckks_ctx *ctx, const uint64_t *c1, size_t in_stride, uint32_t count, uint32_t level,
                           uint64_t *digits)
{
    if (!count) return CKKS_OK;
    const uint32_t K = ctx->n_p, ext = level + 1 + K, nd = n_digits(ctx, level), alpha = ctx->alpha;
    const size_t N = ctx->n, dig_ct = (size_t)nd * ext * N;
    const size_t cstride = count == 1 ? 0 : in_stride;
    // A few ciphertexts leave each digit's transforms of its converted rows too small to fill the chip: then one
    // forward transform runs over all ext rows of every digit (each digit's own rows are transformed along and
    // overwritten with their NTT-domain values afterwards): 2 launches in place of 2 nd.  With more ciphertexts
    // the per-digit launches are large, and transforming the own rows too would only add work.
    const bool one_ntt = count < 4;
    // coefficient form of a digit's limbs, staged in alpha rows per ciphertext after all the digits
    uint64_t *coef = digits + (size_t)count * dig_ct;
    LimbMap m{};
    for (uint32_t j = 0; j < nd; j++) {
        const uint32_t lo = digit_lo(ctx, j), hi = digit_hi(ctx, j, level), ns = hi - lo;
        uint64_t *dj = digits + (size_t)j * ext * N;
        // the digit's own limbs to the staging rows (and, unless they are written after the transform, into the
        // digit with their NTT-domain values), read once
        CK_TRY(launch_copy_rows(ctx, coef, (size_t)alpha * N, one_ntt ? nullptr : dj + lo * N, dig_ct, c1 + lo * N,
                                cstride, (size_t)ns * N, count));
        CK_TRY(launch_ntt_strided(ctx, coef, count, alpha, limb_range(lo, ns), true));
        const ConvDev *cd;
        CK_TRY(ctx_conv(ctx, (int)level, (int)j, &cd));
        CK_TRY(launch_conv(ctx, cd, coef, alpha, dj, (uint32_t)(dig_ct / N), lo, ns, count));
        if (one_ntt) continue;
        // NTT of the converted rows: [0, lo) and [hi, ext)
        if (lo) CK_TRY(launch_ntt_strided(ctx, dj, count, (uint32_t)(dig_ct / N), limb_range(0, lo), false));
        m.n = ext - hi;
        for (uint32_t r = hi; r < ext; r++) m.prime[r - hi] = (uint8_t)(r <= level ? r : ctx->n_q + (r - level - 1));
        CK_TRY(launch_ntt_strided(ctx, dj + (size_t)hi * N, count, (uint32_t)(dig_ct / N), m, false));
    }
    if (one_ntt) {
        m.n = ext;
        for (uint32_t r = 0; r < ext; r++) m.prime[r] = (uint8_t)(r <= level ? r : ctx->n_q + (r - level - 1));
        CK_TRY(launch_ntt_strided(ctx, digits, nd * count, ext, m, false));
        for (uint32_t j = 0; j < nd; j++) {
            const uint32_t lo = digit_lo(ctx, j), hi = digit_hi(ctx, j, level);
            CK_TRY(launch_copy_rows(ctx, digits + ((size_t)j * ext + lo) * N, dig_ct, nullptr, 0, c1 + lo * N,
                                    cstride, (size_t)(hi - lo) * N, count));
        }
    }
    return CKKS_OK;
}

ckks_status ks_modup(ckks_ctx *ctx, const uint64_t *c, uint32_t level, uint64_t *digits)
{
    return ks_modup_batch(ctx, c, 0, 1, level, digits);
}

ckks_status ks_inner_product(ckks_ctx *ctx, const uint64_t *digits, uint32_t nd, const uint64_t *key,
                             uint32_t level, uint32_t g, uint64_t *u)
{
    const uint32_t ext = level + 1 + ctx->n_p;
    const dim3 grid((ctx->n + kThreads - 1) / kThreads, ext), block(kThreads);
    // digits (nd rows of ext), key rows (nd x 2 x ext), two outputs of ext rows
    prof_begin(ctx, K_KEYIP, 8.0 * ctx->n * ext * (3.0 * nd + 2.0));
    hipLaunchKernelGGL(k_key_ip, grid, block, 0, ctx->stream, digits, key, u, nd, ext, level, ctx->n_q,
                       ctx->n_primes(), g, ctx->d_mod, ctx->log_n);
    prof_end(ctx, K_KEYIP);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status ks_moddown(ckks_ctx *ctx, uint64_t *u, uint32_t polys, uint32_t level, const uint64_t *add0,
                       uint32_t add0_g, const uint64_t *add1, uint64_t *out, uint64_t *work)
{
    const uint32_t K = ctx->n_p, ext = level + 1 + K, L = level + 1;
    const size_t N = ctx->n;
    // INTT of the P rows of every polynomial, in place
    LimbMap pm = limb_range(ctx->n_q, K);
    CK_TRY(launch_ntt_strided(ctx, u + (size_t)L * N, polys, ext, pm, true));
    const ConvDev *cd;
    CK_TRY(ctx_conv(ctx, (int)level, -1, &cd));
    CK_TRY(launch_conv(ctx, cd, u + (size_t)L * N, ext, work, L, L, 0, polys));
    CK_TRY(launch_ntt(ctx, work, polys * L, limb_range(0, L), false));
    const dim3 grid((ctx->n + kThreads - 1) / kThreads, L, polys), block(kThreads);
    const double adds = (add0 ? 1.0 : 0.0) + (add1 ? 1.0 : 0.0);
    prof_begin(ctx, K_MODDOWN, 8.0 * ctx->n * L * (3.0 * polys + adds));
    hipLaunchKernelGGL(k_moddown_finish, grid, block, 0, ctx->stream, out, u, work, add0, add0_g, add1, ext, level,
                       ctx->d_pinv, ctx->d_mod, ctx->log_n);
    prof_end(ctx, K_MODDOWN);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}
