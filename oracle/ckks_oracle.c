/*
 * Plain CPU oracle for the RNS-CKKS arithmetic under the packed
 * ciphertext x plaintext projection.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark do.  It shares no code, headers or tables with the HIP
 * path.
 *
 * Every modular operation is written the obvious way: a 128-bit product
 * followed by the C `%` operator.  Transforms are the textbook iterative
 * forms.  The paper (Background, "The CKKS Computation Model") names the
 * primitives (Encode, Add, PCMult, Mult, Rot, KeySwitch, Rescale) but leaves
 * their internals to the CKKS literature; the definitions used here are the
 * standard RNS-CKKS ones (Cheon-Kim-Kim-Song 2017; Cheon-Han-Kim-Kim-Song
 * 2018 for the RNS form; Han-Ki 2020 for hybrid key switching).
 *
 * Build: gcc -O2 -fPIC -shared -fopenmp -ffp-contract=off (see build.py).
 */
#define _GNU_SOURCE /* sincos */
#include <math.h>
#include <omp.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

static uint64_t mulm(uint64_t a, uint64_t b, uint64_t q)
{
    return (uint64_t)(((u128)a * (u128)b) % q);
}
static uint64_t addm(uint64_t a, uint64_t b, uint64_t q)
{
    return (uint64_t)(((u128)a + (u128)b) % q);
}
static uint64_t subm(uint64_t a, uint64_t b, uint64_t q)
{
    return (uint64_t)(((u128)a + (u128)q - (u128)(b % q)) % q);
}
static uint64_t powm(uint64_t b, uint64_t e, uint64_t q)
{
    uint64_t r = 1 % q;
    b %= q;
    while (e) {
        if (e & 1) r = mulm(r, b, q);
        b = mulm(b, b, q);
        e >>= 1;
    }
    return r;
}
/* The threads the parallel loops below use, and a way to change them: the benchmark times the oracle with all
 * host threads and with one. */
int or_threads(void) { return omp_get_max_threads(); }
void or_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }

/* q is prime, so a^(q-2) is the inverse (Fermat). */
static uint64_t invm(uint64_t a, uint64_t q) { return powm(a, q - 2, q); }

static uint32_t brev(uint32_t x, int bits)
{
    uint32_t r = 0;
    for (int i = 0; i < bits; i++) {
        r = (r << 1) | (x & 1u);
        x >>= 1;
    }
    return r;
}
static int ilog2(int64_t n)
{
    int l = 0;
    while ((1LL << l) < n) l++;
    return l;
}

/* tw[k] = root^brev(k) for k < n (powers built by repeated multiplication). */
static uint64_t *root_powers_brev(uint64_t root, int64_t n, int logn, uint64_t q)
{
    uint64_t *pw = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)n);
    uint64_t *tw = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)n);
    pw[0] = 1 % q;
    for (int64_t e = 1; e < n; e++) pw[e] = mulm(pw[e - 1], root, q);
    for (int64_t k = 0; k < n; k++) tw[k] = pw[brev((uint32_t)k, logn)];
    free(pw);
    return tw;
}

/* ------------------------------------------------------------------------ */
/* Negacyclic NTT.                                                           */
/* Output index j holds a(psi^(2*brev(j)+1)) mod q: evaluations at the odd   */
/* powers of a primitive 2N-th root psi, in bit-reversed order.  This is the */
/* textbook Cooley-Tukey transform with psi folded into the twiddles         */
/* (Longa-Naehrig 2016): stage with m groups uses psi^brev(m+i).             */
/* ------------------------------------------------------------------------ */
void or_ntt(uint64_t *a, int64_t rows, int64_t n, uint64_t q, uint64_t psi)
{
    int logn = ilog2(n);
    uint64_t *tw = root_powers_brev(psi, n, logn, q);
#pragma omp parallel for schedule(dynamic)
    for (int64_t r = 0; r < rows; r++) {
        uint64_t *x = a + r * n;
        for (int64_t m = 1, t = n / 2; m < n; m *= 2, t /= 2) {
            for (int64_t i = 0; i < m; i++) {
                uint64_t w = tw[m + i];
                for (int64_t j = 2 * i * t; j < 2 * i * t + t; j++) {
                    uint64_t u = x[j] % q;
                    uint64_t v = mulm(x[j + t], w, q);
                    x[j] = addm(u, v, q);
                    x[j + t] = subm(u, v, q);
                }
            }
        }
    }
    free(tw);
}

/* Exact inverse of or_ntt: Gentleman-Sande stages with psi^-brev(m+i), then
 * multiplication by N^-1 mod q. */
void or_intt(uint64_t *a, int64_t rows, int64_t n, uint64_t q, uint64_t psi)
{
    int logn = ilog2(n);
    uint64_t psi_inv = invm(psi, q);
    uint64_t n_inv = invm((uint64_t)(n % (int64_t)q), q);
    uint64_t *tw = root_powers_brev(psi_inv, n, logn, q);
#pragma omp parallel for schedule(dynamic)
    for (int64_t r = 0; r < rows; r++) {
        uint64_t *x = a + r * n;
        for (int64_t m = n / 2, t = 1; m >= 1; m /= 2, t *= 2) {
            for (int64_t i = 0; i < m; i++) {
                uint64_t w = tw[m + i];
                for (int64_t j = 2 * i * t; j < 2 * i * t + t; j++) {
                    uint64_t u = x[j] % q, v = x[j + t] % q;
                    x[j] = addm(u, v, q);
                    x[j + t] = mulm(subm(u, v, q), w, q);
                }
            }
        }
        for (int64_t j = 0; j < n; j++) x[j] = mulm(x[j], n_inv, q);
    }
    free(tw);
}

/* The same transforms over rows that each carry their own prime and root
 * (row r: qs[r], psis[r]); rows run in parallel. */
void or_ntt_rows(uint64_t *a, int64_t rows, int64_t n, const uint64_t *qs, const uint64_t *psis, int inverse)
{
#pragma omp parallel for schedule(dynamic)
    for (int64_t r = 0; r < rows; r++) {
        if (inverse)
            or_intt(a + r * n, 1, n, qs[r], psis[r]);
        else
            or_ntt(a + r * n, 1, n, qs[r], psis[r]);
    }
}

/* ------------------------------------------------------------------------ */
/* Element-wise arithmetic mod q over rows of a [rows][n] array whose row r  */
/* uses modulus qs[r].                                                       */
/* ------------------------------------------------------------------------ */
void or_mul(const uint64_t *a, const uint64_t *b, uint64_t *out, int64_t rows, int64_t n,
            const uint64_t *qs)
{
#pragma omp parallel for
    for (int64_t r = 0; r < rows; r++)
        for (int64_t j = 0; j < n; j++)
            out[r * n + j] = mulm(a[r * n + j] % qs[r], b[r * n + j] % qs[r], qs[r]);
}
void or_add(const uint64_t *a, const uint64_t *b, uint64_t *out, int64_t rows, int64_t n,
            const uint64_t *qs)
{
#pragma omp parallel for
    for (int64_t r = 0; r < rows; r++)
        for (int64_t j = 0; j < n; j++) out[r * n + j] = addm(a[r * n + j], b[r * n + j], qs[r]);
}
void or_sub(const uint64_t *a, const uint64_t *b, uint64_t *out, int64_t rows, int64_t n,
            const uint64_t *qs)
{
#pragma omp parallel for
    for (int64_t r = 0; r < rows; r++)
        for (int64_t j = 0; j < n; j++) out[r * n + j] = subm(a[r * n + j], b[r * n + j], qs[r]);
}
/* out[r][j] = a[r][j] * c[r] mod qs[r] (c: one scalar per row). */
void or_mul_scalar(const uint64_t *a, const uint64_t *c, uint64_t *out, int64_t rows, int64_t n,
                   const uint64_t *qs)
{
#pragma omp parallel for
    for (int64_t r = 0; r < rows; r++)
        for (int64_t j = 0; j < n; j++) out[r * n + j] = mulm(a[r * n + j] % qs[r], c[r] % qs[r], qs[r]);
}
/* Signed integers into residues: out[r][j] = v[j] mod qs[r] in [0, qs[r]). */
void or_reduce_i64(const int64_t *v, uint64_t *out, int64_t rows, int64_t n, const uint64_t *qs)
{
#pragma omp parallel for
    for (int64_t r = 0; r < rows; r++) {
        uint64_t q = qs[r];
        for (int64_t j = 0; j < n; j++) {
            int64_t x = v[j];
            uint64_t mag = x < 0 ? (uint64_t)(-(x + 1)) + 1u : (uint64_t)x;
            uint64_t m = mag % q;
            out[r * n + j] = (x < 0 && m) ? q - m : m;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Fast basis conversion (Cheon-Han-Kim-Kim-Song 2018, the approximate form  */
/* without overflow correction), with centred digits:                        */
/*   y_i = [a_i * Qhat_i^-1]_{q_i} taken in (-q_i/2, q_i/2] (q_i odd),       */
/*   Conv(a)_t = sum_{i in I} y_i * [Qhat_i]_t  (mod t).                     */
/* The integer sum_i y_i Qhat_i is congruent to a modulo Q_I and has zero    */
/* mean over uniform inputs, which keeps the key-switching error centred.    */
/* in: [ni][n] coefficient residues mod qin[i]; out: [nt][n] mod qt[t].      */
/* qhat_inv[i] = Qhat_i^-1 mod q_i; qhat_mod_t[i*nt + t] = Qhat_i mod qt[t]. */
/* ------------------------------------------------------------------------ */
void or_conv(const uint64_t *in, const uint64_t *qin, int64_t ni, uint64_t *out, const uint64_t *qt,
             int64_t nt, int64_t n, const uint64_t *qhat_inv, const uint64_t *qhat_mod_t)
{
#pragma omp parallel for
    for (int64_t t = 0; t < nt; t++) {
        for (int64_t j = 0; j < n; j++) {
            u128 acc = 0;
            for (int64_t i = 0; i < ni; i++) {
                uint64_t y = mulm(in[i * n + j] % qin[i], qhat_inv[i], qin[i]);
                uint64_t qh = qhat_mod_t[i * nt + t] % qt[t];
                if (y > qin[i] / 2) {
                    /* y stands for the negative value -(q_i - y) */
                    uint64_t m = mulm((qin[i] - y) % qt[t], qh, qt[t]);
                    acc += m ? qt[t] - m : 0;
                } else {
                    acc += (u128)mulm(y % qt[t], qh, qt[t]);
                }
            }
            out[t * n + j] = (uint64_t)(acc % qt[t]);
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Encode, fp64 stage: the rounded integer coefficient vector               */
/*   m_i = round(delta * (2/N) * Re sum_{j<N/2} z_j * zeta^(-i*e_j)),        */
/*   zeta = exp(i*pi/N), e_j = 5^j mod 2N, i < N,                            */
/* rounding half away from zero.  Conjugate-symmetric extension of the slot  */
/* vector through the canonical embedding (CKKS 2017, Section 3).            */
/*                                                                           */
/* Evaluation order (fixed, because the rounding of a near-tie depends on    */
/* it):  the exponents e_j are exactly the residues 1 mod 4 of Z_2N, so with */
/* e_j = 4s+1 the sum becomes zeta^-k * Y_k where Y is the length-M=N/2      */
/* inverse-direction DFT of y_s = z_j; m_k = round(c*Re v_k) and             */
/* m_{k+M} = round(c*Im v_k) with c = delta*2/N.  Y is computed by the       */
/* radix-2 decimation-in-time FFT from bit-reversed input:                   */
/*   for len = 2, 4, ..., M: w_k = omega^(-k*M/len),                         */
/*     t = w_k * a[b+k+len/2];  a[b+k+len/2] = a[b+k] - t;  a[b+k] += t      */
/* with omega^-e = (cos(2*pi*e/M), -sin(2*pi*e/M)), zeta^-k = (cos(pi*k/N),  */
/* -sin(pi*k/N)), and a complex product computed as                          */
/*   (ar*br - ai*bi, ar*bi + ai*br) without fused multiply-add.              */
/* The cosine and sine of an angle are the two outputs of one call to the C  */
/* library's sincos(): it can differ from separate sin() and cos() calls in  */
/* the last bit, and compilers merge or split such calls at will, so the     */
/* call is named explicitly.                                                 */
/* ------------------------------------------------------------------------ */
static void cmul(double ar, double ai, double br, double bi, double *cr, double *ci)
{
    double p1 = ar * br, p2 = ai * bi, p3 = ar * bi, p4 = ai * br;
    *cr = p1 - p2;
    *ci = p3 + p4;
}

static void encode_fft(const double *zr, const double *zi, int64_t n, double delta, double *x_out);

void or_encode_round(const double *zr, const double *zi, int64_t n, double delta, int64_t *m_out)
{
    double *x = (double *)malloc(sizeof(double) * (size_t)n);
    encode_fft(zr, zi, n, delta, x);
    for (int64_t i = 0; i < n; i++) m_out[i] = (int64_t)round(x[i]);
    free(x);
}

/* The scaled, unrounded values c * Re v_k, c * Im v_k whose rounding gives m. */
void or_encode_unrounded(const double *zr, const double *zi, int64_t n, double delta, double *x_out)
{
    encode_fft(zr, zi, n, delta, x_out);
}

static void encode_fft(const double *zr, const double *zi, int64_t n, double delta, double *x_out)
{
    int64_t M = n / 2, two_n = 2 * n;
    int logm = ilog2(M);
    double *ar = (double *)malloc(sizeof(double) * (size_t)M);
    double *ai = (double *)malloc(sizeof(double) * (size_t)M);
    /* slot j sits at FFT input position s(j) = (5^j mod 2N - 1)/4, stored bit-reversed */
    int64_t e = 1;
    for (int64_t j = 0; j < M; j++) {
        int64_t s = (e - 1) / 4;
        uint32_t pos = brev((uint32_t)s, logm);
        ar[pos] = zr[j];
        ai[pos] = zi ? zi[j] : 0.0;
        e = (e * 5) % two_n;
    }
    for (int64_t len = 2; len <= M; len *= 2) {
        int64_t half = len / 2, step = M / len;
        for (int64_t b = 0; b < M; b += len) {
            for (int64_t k = 0; k < half; k++) {
                double ang = 2.0 * M_PI * (double)(k * step) / (double)M;
                double sn, cs;
                sincos(ang, &sn, &cs);
                double wr = cs, wi = -sn;
                double tr, ti;
                cmul(wr, wi, ar[b + k + half], ai[b + k + half], &tr, &ti);
                double ur = ar[b + k], ui = ai[b + k];
                ar[b + k] = ur + tr;
                ai[b + k] = ui + ti;
                ar[b + k + half] = ur - tr;
                ai[b + k + half] = ui - ti;
            }
        }
    }
    double c = delta * (2.0 / (double)n);
    for (int64_t k = 0; k < M; k++) {
        double ang = M_PI * (double)k / (double)n;
        double sn, cs;
        sincos(ang, &sn, &cs);
        double tr = cs, ti = -sn;
        double vr, vi;
        cmul(tr, ti, ar[k], ai[k], &vr, &vi);
        x_out[k] = c * vr;
        x_out[k + M] = c * vi;
    }
    free(ar);
    free(ai);
}

/* Definitional O(N^2) encode in long double, for pinning or_encode_round:
 * x_i = delta*(2/N)*Re sum_j z_j zeta^(-i e_j) before rounding.  Returns the
 * unrounded values; the caller rounds and measures distance to ties. */
void or_encode_def(const double *zr, const double *zi, int64_t n, double delta, long double *x_out)
{
    int64_t M = n / 2, two_n = 2 * n;
    int64_t *ex = (int64_t *)malloc(sizeof(int64_t) * (size_t)M);
    int64_t e = 1;
    for (int64_t j = 0; j < M; j++) {
        ex[j] = e;
        e = (e * 5) % two_n;
    }
    const long double pi = 3.141592653589793238462643383279502884L;
#pragma omp parallel for
    for (int64_t i = 0; i < n; i++) {
        long double acc = 0.0L;
        for (int64_t j = 0; j < M; j++) {
            int64_t ph = (i * ex[j]) % two_n; /* zeta^(-i e_j) = exp(-i*pi*ph/N) */
            long double ang = pi * (long double)ph / (long double)n;
            acc += (long double)zr[j] * cosl(ang) + (long double)(zi ? zi[j] : 0.0) * sinl(ang);
        }
        x_out[i] = (long double)delta * 2.0L / (long double)n * acc;
    }
    free(ex);
}
/* long double is not a ctypes-friendly type everywhere: give a double view of
 * the rounded value and its signed distance to the nearest half-integer. */
void or_encode_def_round(const double *zr, const double *zi, int64_t n, double delta, int64_t *m_out,
                         double *tie_dist)
{
    long double *x = (long double *)malloc(sizeof(long double) * (size_t)n);
    or_encode_def(zr, zi, n, delta, x);
    for (int64_t i = 0; i < n; i++) {
        long double r = roundl(x[i]);
        m_out[i] = (int64_t)r;
        long double frac = x[i] - floorl(x[i]);
        tie_dist[i] = (double)fabsl(frac - 0.5L);
    }
    free(x);
}

/* ------------------------------------------------------------------------ */
/* Seed-expanded switching keys.                                            */
/* A key's uniform half a_j need not be stored: it is a deterministic       */
/* function of a 128-bit seed.  The generator is Philox-4x64-10 (Salmon,   */
/* Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",    */
/* SC 2011): ten rounds of two 64x64 -> 128-bit products with the constants */
/* M0, M1, the key bumped by the Weyl constants W0, W1 between rounds.      */
/* ------------------------------------------------------------------------ */
void or_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3], k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; r++) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const u128 p0 = (u128)M0 * x0, p1 = (u128)M1 * x2;
        const uint64_t y0 = (uint64_t)(p1 >> 64) ^ x1 ^ k0, y1 = (uint64_t)p1;
        const uint64_t y2 = (uint64_t)(p0 >> 64) ^ x3 ^ k1, y3 = (uint64_t)p0;
        x0 = y0;
        x1 = y1;
        x2 = y2;
        x3 = y3;
    }
    out[0] = x0;
    out[1] = x1;
    out[2] = x2;
    out[3] = x3;
}

/* The uniform half of a seed-expanded key: out[j][k][n] for digit j < dnum, prime index k < n_primes (modulus
 * qs[k]) and NTT-domain position n < N.  With b the bit length of q: attempt t = 0, 1, ... draws the block
 * Philox-4x64-10(counter (n, k, j / 4, t), key seed) and takes its word j mod 4, w; the residue is w >> (64 - b)
 * if that is below q (rejection sampling: uniform on [0, q)), else the next attempt; after 64 rejections (each
 * has probability 1 - q/2^b < 1/2) the residue is w mod q. */
void or_expand_key_a(const uint64_t seed[2], int64_t dnum, const uint64_t *qs, int64_t n_primes, int64_t n,
                     uint64_t *out)
{
#pragma omp parallel for collapse(2)
    for (int64_t j = 0; j < dnum; j++)
        for (int64_t k = 0; k < n_primes; k++) {
            const uint64_t q = qs[k];
            int b = 0;
            while (b < 64 && (q >> b) != 0) b++;
            for (int64_t i = 0; i < n; i++) {
                uint64_t blk[4], v = 0;
                for (uint64_t t = 0; t < 64; t++) {
                    const uint64_t ctr[4] = {(uint64_t)i, (uint64_t)k, (uint64_t)(j / 4), t};
                    or_philox4x64_10(ctr, seed, blk);
                    const uint64_t w = blk[j % 4];
                    const uint64_t x = w >> (64 - b);
                    if (x < q) {
                        v = x;
                        break;
                    }
                    if (t == 63) v = w % q;
                }
                out[(j * n_primes + k) * n + i] = v;
            }
        }
}
