// One attention block's ciphertext work in the token-major layout s = t*D + f (T tokens, D features per
// ciphertext, heads of hd features): the scores Q K^T as ciphertext products with rotation sums, and the
// weighted sums of values that consume them.  The paper's C-Delta attention layout (Section "C--Delta
// Attention Layout and Computation"; Section "Linear-Computation Performance", Table ccmm-performance) has
// QK^T produce the scores directly on diagonals S_Delta and PV consume P_Delta without repacking, but gives no
// construction; the one below is this library's own, in that spirit: score delta of token t pairs it with
// token (t + delta) mod T.
//
// Scores.  Query ciphertext c holds D/hd heads (slot t*D + h*hd + d = Q[t, h, d]); its key ciphertext holds
// one key head repeated in every head position.  With the left rotation (Rot_k x)[s] = x[s + k]:
//   P_delta = Relin(Rot_{-delta}(Q) x Rot_{delta (D-1)}(K'))                                 0 <= delta < T
//   out     = Rescale(Rescale( sum_k Rot_k( U_k ) )),  U_k = sum_delta M_{(delta + k) mod hd} * P_delta  0 <= k < hd
// and slot t*D + h*hd + delta of out holds sum_d Q[t, h, d] K[(t + delta) mod T, d] (zero for delta >= T).
// The masks M_c (1 on head position c) are slot vectors of period D, so their plaintexts are constant on
// runs of T consecutive NTT positions, with values m[c] on a run.  At one NTT position the sums over delta are
// then a cyclic correlation of the ciphertext values x[delta] with m: U_k = sum_delta m[(delta + k) mod hd]
// x[delta] = z[-k], z = x (*) m_r (cyclic convolution of length hd, m_r[v] = m[-v]), evaluated exactly mod
// q_l as INTT(NTT(x) NTT(m_r)) with a cyclic NTT along delta (root psi^(2N/n)) — O(hd log hd) per position
// instead of hd T products.
//
// Weighted sums.  Scores P in that layout, a value ciphertext V' with one value head in every position:
//   R_delta = Rot_{delta D}(V'),  C_j = Rescale( sum_delta M_{delta - j} * R_delta )   (0 <= delta - j < hd)
//   out     = Rescale(Relin( sum_j Rot_j(P) x C_j ))                                   -hd < j < T
// so that out[t*D + h*hd + d] = sum_delta P[t, h, delta] V[(t + delta) mod T, d].  The C_j depend only on the
// value ciphertext and are shared by every score ciphertext that uses it; the products are summed before
// the single relinearisation.  C_j = z[j mod 2hd] for the same correlation at length 2hd with m zero past hd:
// delta - j spans T + hd - 1 <= 2hd values, so no two of them meet modulo 2hd.
#include <algorithm>
#include <vector>

#include "ckks_internal.h"
#include "ntt_core.h"
#include "ops.h"

namespace {

constexpr int kThreads = 256;
constexpr uint32_t kRotChunk = 32;  // outputs rotated (or rescaled) per batch

// U[c][f] = 1 if f = c (mod hd), else 0; c < hd, f < D
__global__ __launch_bounds__(kThreads) void k_attn_masks(double *U, uint32_t D, uint32_t hd)
{
    const uint32_t i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= D * hd) return;
    const uint32_t c = i / D, f = i % D;
    U[i] = (f & (hd - 1)) == c ? 1.0 : 0.0;
}

// Cyclic NTT of length n = 2^LOGN along the first index of s ([n][P] doubles in LDS, |values| < 2q): the
// Cooley-Tukey loop with natural-order input and bit-reversed output, group i of stage m taking om[m + i] =
// w_(2m)^brev_(log m)(i) (w_(2m) a primitive 2m-th root of unity).  Stages run in pairs (m, 2m) with four points
// per thread (one LDS round trip and one barrier per pair), an odd last stage alone.  Every butterfly keeps its
// values below 2q.
template <int LOGN, int P, int NT>
__device__ __forceinline__ void corr_fwd(double *s, const double *om, const nttc::Ar<true> &ar)
{
    constexpr int n = 1 << LOGN;
#pragma unroll
    for (int st = 0; st + 1 < LOGN; st += 2) {
        // stage m (stride t) on (j, j + t), (j + t/2, j + 3t/2); stage 2m (stride t/2) on (j, j + t/2), (j + t, j + 3t/2)
        const int m = 1 << st, lt = LOGN - 1 - st, t = 1 << lt, h = t >> 1;
        for (int b = threadIdx.x; b < (n / 4) * P; b += NT) {
            const int p = b % P, bi = b / P, i = bi >> (lt - 1), j = (i << (lt + 1)) + (bi & (h - 1));
            double x0 = s[j * P + p], x1 = s[(j + h) * P + p], x2 = s[(j + t) * P + p], x3 = s[(j + t + h) * P + p];
            const double w = om[m + i];
            ar.ct(x0, x2, w);
            ar.ct(x1, x3, w);
            ar.ct(x0, x1, om[2 * m + 2 * i]);
            ar.ct(x2, x3, om[2 * m + 2 * i + 1]);
            s[j * P + p] = x0;
            s[(j + h) * P + p] = x1;
            s[(j + t) * P + p] = x2;
            s[(j + t + h) * P + p] = x3;
        }
        __syncthreads();
    }
    if (LOGN & 1) {
        constexpr int m = n / 2;
        for (int b = threadIdx.x; b < (n / 2) * P; b += NT) {
            const int p = b % P, i = b / P, j = 2 * i;
            double X = s[j * P + p], Y = s[(j + 1) * P + p];
            ar.ct(X, Y, om[m + i]);
            s[j * P + p] = X;
            s[(j + 1) * P + p] = Y;
        }
        __syncthreads();
    }
}

// Its inverse without the 1/n (Gentleman-Sande, bit-reversed input, natural output, omi[m + i] = om[m + i]^-1):
// stages m = n/2 .. 1, an odd first stage alone, then pairs (m, m/2) with four points per thread.
template <int LOGN, int P, int NT>
__device__ __forceinline__ void corr_inv(double *s, const double *omi, const nttc::Ar<true> &ar)
{
    constexpr int n = 1 << LOGN;
    if (LOGN & 1) {
        constexpr int m = n / 2;
        for (int b = threadIdx.x; b < (n / 2) * P; b += NT) {
            const int p = b % P, i = b / P, j = 2 * i;
            double X = s[j * P + p], Y = s[(j + 1) * P + p];
            ar.gs(X, Y, omi[m + i]);
            s[j * P + p] = X;
            s[(j + 1) * P + p] = Y;
        }
        __syncthreads();
    }
#pragma unroll
    for (int st = LOGN - 1 - (LOGN & 1); st >= 1; st -= 2) {
        // stage m (stride t) on (a, a + t), (a + 2t, a + 3t); stage m/2 (stride 2t) on (a, a + 2t), (a + t, a + 3t)
        const int m = 1 << st, lt = LOGN - 1 - st, t = 1 << lt;
        for (int b = threadIdx.x; b < (n / 4) * P; b += NT) {
            const int p = b % P, bi = b / P, i2 = bi >> lt, a = (i2 << (lt + 2)) + (bi & (t - 1));
            double x0 = s[a * P + p], x1 = s[(a + t) * P + p], x2 = s[(a + 2 * t) * P + p],
                   x3 = s[(a + 3 * t) * P + p];
            ar.gs(x0, x1, omi[m + 2 * i2]);
            ar.gs(x2, x3, omi[m + 2 * i2 + 1]);
            const double w = omi[m / 2 + i2];
            ar.gs(x0, x2, w);
            ar.gs(x1, x3, w);
            s[a * P + p] = x0;
            s[(a + t) * P + p] = x1;
            s[(a + 2 * t) * P + p] = x2;
            s[(a + 3 * t) * P + p] = x3;
        }
        __syncthreads();
    }
}

// Twiddles of the cyclic NTT of length n for limbs l < L: om[l][m + i] = psi^e, e = N brev_(log m)(i) / m < N
// (psi^e = twf[brev(e)], the ring's table), omi the inverses from the inverse table.
__global__ __launch_bounds__(kThreads) void k_attn_tw(double *om, double *omi, uint32_t n, uint32_t L,
                                                      const double *__restrict__ twf, const double *__restrict__ itwf,
                                                      uint32_t log_n)
{
    const uint32_t i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= L * n) return;
    const uint32_t l = i / n, k = i % n;
    double w = 1.0, wi = 1.0;
    if (k > 0) {
        const uint32_t logm = 31 - __clz(k), ii = k - (1u << logm);
        const uint32_t br = logm ? __brev(ii) >> (32 - logm) : 0;
        const uint32_t e = (br << log_n) >> logm;
        if (e) {
            const uint32_t idx = __brev(e) >> (32 - log_n);
            w = twf[((size_t)l << log_n) + idx];
            wi = itwf[((size_t)l << log_n) + idx];
        }
    }
    om[i] = w;
    omi[i] = wi;
}

// The transformed masks of one (limb l, run): Mh[l][run][f] = NTT(m_r)[f] / n, m_r[v] = m[(n - v) mod n] with
// m[c] = MQ[l][run][c] for c < hd and 0 for hd <= c < n.  One block per (l, run).
template <int LOGN>
__global__ __launch_bounds__(kThreads) void k_attn_mhat(double *Mh, const double *__restrict__ MQ, uint32_t hd,
                                                        uint32_t D2, const double *__restrict__ Om,
                                                        const ModQ *__restrict__ mods)
{
    constexpr int n = 1 << LOGN;
    __shared__ double s[n], om[n];
    const uint32_t bid = blockIdx.x, l = bid / D2;
    const nttc::Ar<true> ar(mods[l]);
    for (int i = threadIdx.x; i < n; i += kThreads) {
        om[i] = Om[(size_t)l * n + i];
        const uint32_t c = (uint32_t)(n - i) & (n - 1);
        s[i] = c < hd ? MQ[(size_t)bid * hd + c] : 0.0;
    }
    __syncthreads();
    corr_fwd<LOGN, 1, kThreads>(s, om, ar);
    const double q = mods[l].qd;
    const double ninv = q - (q - 1.0) / (double)n;  // n divides q - 1
    for (int f = threadIdx.x; f < n; f += kThreads) Mh[(size_t)bid * n + f] = (double)ar.to_canon(ar.mul(s[f], ninv));
}

// z = x (*) m_r at P consecutive positions of one (limb, polynomial): x[delta] is position p of input ciphertext
// delta < T (x + delta ctw, [2][L][N] each; zero for T <= delta < n), Mh the transformed masks of each position's
// run (p >> logT).  Output e < nout is z[(sgn e + off) mod n], written canonical to out + e ctw.
template <int LOGN, int P>
__global__ __launch_bounds__(kThreads) void k_attn_corr(uint64_t *out, const uint64_t *__restrict__ x, uint32_t T,
                                                        uint32_t nout, int sgn, int off, size_t ctw, uint32_t L,
                                                        uint32_t log_n, uint32_t logT, uint32_t D2,
                                                        const double *__restrict__ Om, const double *__restrict__ Omi,
                                                        const double *__restrict__ Mh, const ModQ *__restrict__ mods)
{
    constexpr int n = 1 << LOGN;
    __shared__ double s[n * P];
    __shared__ double om[n], omi[n];
    const uint32_t groups = (1u << log_n) / P;
    const uint32_t pg = blockIdx.x % groups, rest = blockIdx.x / groups;
    const uint32_t poly = rest & 1, l = rest >> 1;
    const uint32_t p0 = pg * P;
    const nttc::Ar<true> ar(mods[l]);
    for (int i = threadIdx.x; i < n; i += kThreads) {
        om[i] = Om[(size_t)l * n + i];
        omi[i] = Omi[(size_t)l * n + i];
    }
    const size_t row = (((size_t)poly * L + l) << log_n) + p0;
    for (int i = threadIdx.x; i < n * P; i += kThreads) {
        const uint32_t d = i / P, p = i % P;
        s[i] = d < T ? (double)x[(size_t)d * ctw + row + p] : 0.0;
    }
    __syncthreads();
    corr_fwd<LOGN, P, kThreads>(s, om, ar);
    for (int i = threadIdx.x; i < n * P; i += kThreads) {
        const uint32_t f = i / P, p = i % P, run = (p0 + p) >> logT;
        s[i] = ar.mul(s[i], Mh[((size_t)l * D2 + run) * n + f]);
    }
    __syncthreads();
    corr_inv<LOGN, P, kThreads>(s, omi, ar);
    for (int i = threadIdx.x; i < (int)nout * P; i += kThreads) {
        const uint32_t e = i / P, p = i % P;
        const uint32_t f = (uint32_t)(sgn * (int)e + off) & (n - 1);
        out[(size_t)e * ctw + row + p] = ar.to_canon(s[f * P + p]);
    }
}

// out[w] = (accumulate ? out[w] : 0) + sum_{r < count} src[r * stride + w] mod q, w < 2 L N (one ciphertext).
__global__ __launch_bounds__(kThreads) void k_sum_cts(uint64_t *out, const uint64_t *__restrict__ src, uint32_t count,
                                                      size_t stride, uint32_t L, uint32_t log_n, int accumulate,
                                                      const ModQ *__restrict__ mods)
{
    const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    const size_t total = (size_t)2 * L << log_n;
    if (i >= total) return;
    const uint64_t q = mods[(i >> log_n) % L].q;
    uint64_t s = accumulate ? out[i] : 0;
    for (uint32_t r = 0; r < count; r++) s = addmod(s, src[(size_t)r * stride + i], q);
    out[i] = s;
}

// d ([3][L][N]) = sum_{r < count} E_r x C_r: d0 += e0 c0, d1 += e0 c1 + e1 c0, d2 += e1 c1, the sums held in 128
// bits and reduced once: the attention calls take primes below 2^50 only, so each product is below 2^100 and
// count <= 2^16 (2^17 products in d1) keeps every sum below 2^117.  E_r at E + r * 2 L N ([2][L][N]); C_r at
// C + r * 2 Lc N ([2][Lc][N], Lc >= L, its first L limbs used).
__global__ __launch_bounds__(kThreads) void k_tensor_acc(uint64_t *d, const uint64_t *__restrict__ E,
                                                         const uint64_t *__restrict__ C, uint32_t count, uint32_t L,
                                                         uint32_t Lc, uint32_t log_n, const ModQ *__restrict__ mods)
{
    const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    const size_t total = (size_t)L << log_n;
    if (i >= total) return;
    const ModQ m = mods[i >> log_n];
    const size_t ew = total, cw = (size_t)Lc << log_n;
    acc128 a0{0, 0}, a1{0, 0}, a2{0, 0};
    for (uint32_t r = 0; r < count; r++) {
        const uint64_t *e = E + (size_t)r * 2 * ew + i, *c = C + (size_t)r * 2 * cw + i;
        const uint64_t e0 = e[0], e1 = e[ew], c0 = c[0], c1 = c[cw];
        mac(a0, e0, c0);
        mac(a1, e0, c1);
        mac(a1, e1, c0);
        mac(a2, e1, c1);
    }
    d[i] = reduce128(a0, m);
    d[ew + i] = reduce128(a1, m);
    d[2 * ew + i] = reduce128(a2, m);
}

uint32_t log2u(uint32_t v)
{
    uint32_t r = 0;
    while ((1u << r) < v) r++;
    return r;
}

inline dim3 grid_of(size_t total) { return dim3((unsigned)((total + kThreads - 1) / kThreads)); }

ckks_status launch_masks(ckks_ctx *ctx, double *U, double *MQ, uint32_t D, uint32_t hd, double delta, uint32_t L)
{
    hipLaunchKernelGGL(k_attn_masks, grid_of((size_t)D * hd), dim3(kThreads), 0, ctx->stream, U, D, hd);
    HIP_TRY(hipGetLastError());
    return launch_enc_vectors(ctx, U, D, hd, delta, L, MQ);
}

// positions per correlation block: 32 (n <= 128: 34 KB of LDS, four blocks per CU) or 16 (n = 256)
constexpr int corr_positions(uint32_t logn) { return logn >= 8 ? 16 : 32; }

// twiddles and transformed masks for the correlation of length n over L limbs: Om, Omi [L][n]; Mh [L][D2][n]
ckks_status launch_corr_tables(ckks_ctx *ctx, uint32_t logn, uint32_t L, uint32_t D2, uint32_t hd, const double *MQ,
                               double *Om, double *Omi, double *Mh)
{
    const uint32_t n = 1u << logn;
    hipLaunchKernelGGL(k_attn_tw, grid_of((size_t)L * n), dim3(kThreads), 0, ctx->stream, Om, Omi, n, L,
                       (const double *)ctx->d_twf, (const double *)ctx->d_itwf, ctx->log_n);
    HIP_TRY(hipGetLastError());
    if (logn == 7)
        hipLaunchKernelGGL(k_attn_mhat<7>, dim3(L * D2), dim3(kThreads), 0, ctx->stream, Mh, MQ, hd, D2, Om, ctx->d_mod);
    else if (logn == 8)
        hipLaunchKernelGGL(k_attn_mhat<8>, dim3(L * D2), dim3(kThreads), 0, ctx->stream, Mh, MQ, hd, D2, Om, ctx->d_mod);
    else if (logn == 6)
        hipLaunchKernelGGL(k_attn_mhat<6>, dim3(L * D2), dim3(kThreads), 0, ctx->stream, Mh, MQ, hd, D2, Om, ctx->d_mod);
    else if (logn == 5)
        hipLaunchKernelGGL(k_attn_mhat<5>, dim3(L * D2), dim3(kThreads), 0, ctx->stream, Mh, MQ, hd, D2, Om, ctx->d_mod);
    else if (logn == 4)
        hipLaunchKernelGGL(k_attn_mhat<4>, dim3(L * D2), dim3(kThreads), 0, ctx->stream, Mh, MQ, hd, D2, Om, ctx->d_mod);
    else
        return set_error(CKKS_EUNSUPPORTED, "attention: correlation length 2^%u outside [16, 256]", logn);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

// out[e] (e < nout, stride ctw) = z[(sgn e + off) mod n] of the T inputs x (stride ctw), L limbs
ckks_status launch_corr(ckks_ctx *ctx, uint64_t *out, const uint64_t *x, uint32_t T, uint32_t nout, int sgn, int off,
                        uint32_t L, uint32_t logn, uint32_t logT, uint32_t D2, const double *Om, const double *Omi,
                        const double *Mh)
{
    const size_t ctw = 2 * (size_t)L * ctx->n;
    const uint32_t n = 1u << logn;
    const uint32_t P = (uint32_t)corr_positions(logn);
    const dim3 grid(L * 2 * (uint32_t)(ctx->n / P));
    const double res = 2.0 * L * ctx->n;
    // the inputs once, the outputs once; two transforms and a product per position
    prof_begin(ctx, K_ATTN_CORR, 8.0 * res * (T + nout), res * (n * logn * 11.0 + 8.0 * n));
#define CK_CORR(LG)                                                                                                \
    hipLaunchKernelGGL((k_attn_corr<LG, corr_positions(LG)>), grid, dim3(kThreads), 0, ctx->stream, out, x, T, nout, \
                       sgn, off, ctw, L, ctx->log_n, logT, D2, Om, Omi, Mh, ctx->d_mod)
    switch (logn) {
    case 4: CK_CORR(4); break;
    case 5: CK_CORR(5); break;
    case 6: CK_CORR(6); break;
    case 7: CK_CORR(7); break;
    case 8: CK_CORR(8); break;
    default: prof_end(ctx, K_ATTN_CORR); return set_error(CKKS_EUNSUPPORTED, "attention: correlation length %u", n);
    }
#undef CK_CORR
    prof_end(ctx, K_ATTN_CORR);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_sum_cts(ckks_ctx *ctx, uint64_t *out, const uint64_t *src, uint32_t count, size_t stride,
                           uint32_t L, bool accumulate)
{
    if (!count && accumulate) return CKKS_OK;
    const size_t total = (size_t)2 * L * ctx->n;
    prof_begin(ctx, K_ELEM, 8.0 * total * (count + 1 + (accumulate ? 1 : 0)));
    hipLaunchKernelGGL(k_sum_cts, grid_of(total), dim3(kThreads), 0, ctx->stream, out, src, count, stride, L,
                       ctx->log_n, (int)accumulate, ctx->d_mod);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_tensor_acc(ckks_ctx *ctx, uint64_t *d, const uint64_t *E, const uint64_t *C, uint32_t count,
                              uint32_t L, uint32_t Lc)
{
    const size_t total = (size_t)L * ctx->n;
    CK_REQUIRE(count <= 65536u && ntt_uses_f64(ctx, L), CKKS_EUNSUPPORTED,
               "attention: %u products summed exactly need at most 2^16 terms and primes below 2^50", count);
    prof_begin(ctx, K_ELEM, 8.0 * total * (4.0 * count + 3.0));
    hipLaunchKernelGGL(k_tensor_acc, grid_of(total), dim3(kThreads), 0, ctx->stream, d, E, C, count, L, Lc,
                       ctx->log_n, ctx->d_mod);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

// Shape checks shared by both calls: T tokens (a power of two, at most 128), head dimension hd (a power of
// two with max(T, 16) <= hd <= 128, dividing D: the correlations have length hd and 2hd <= 256), D <= 256
// features (the periodic encode's limit).
ckks_status attn_check_shape(const ckks_ctx *ctx, const ckks_attn_shape *shape, const char *what, uint32_t *Dout,
                             uint32_t *logTout)
{
    CK_REQUIRE(shape, CKKS_EINVAL, "%s: null shape", what);
    const uint32_t T = shape->tokens, hd = shape->head_dim, slots = (uint32_t)(ctx->n / 2);
    CK_REQUIRE(T >= 2 && T <= 128 && (T & (T - 1)) == 0 && slots % T == 0, CKKS_EUNSUPPORTED,
               "%s: %u tokens (a power of two in [2, 128] dividing %u slots)", what, T, slots);
    const uint32_t D = slots / T;
    CK_REQUIRE(D <= 256, CKKS_EUNSUPPORTED, "%s: %u features per ciphertext (at most 256)", what, D);
    CK_REQUIRE(hd >= T && hd >= 16 && hd <= 128 && hd <= D && (hd & (hd - 1)) == 0, CKKS_EINVAL,
               "%s: head dimension %u (a power of two with max(%u, 16) <= hd <= min(%u, 128))", what, hd, T, D);
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "%s: the context has no special primes", what);
    *Dout = D;
    *logTout = log2u(T);
    return CKKS_OK;
}

// Scratch of the scores call for inputs of L limbs (words)
struct ScoreScratch {
    uint32_t Jt, logn;
    size_t u_w, mq_w, tw_w, mh_w, b_w, a_w, d_w, pr_w, ub_w, rot_w, tot_w, ua_w, work_w, total;
};

ScoreScratch score_scratch(const ckks_ctx *ctx, uint32_t L, uint32_t D, uint32_t T, uint32_t hd)
{
    ScoreScratch s{};
    const size_t N = ctx->n, ctw = 2 * (size_t)L * N;
    const uint32_t level = L - 1;
    s.Jt = kRotChunk;
    s.logn = log2u(hd);
    s.u_w = (size_t)hd * D;
    s.mq_w = (size_t)L * 2 * D * hd;
    s.tw_w = (size_t)2 * L * hd;
    s.mh_w = (size_t)L * 2 * D * hd;
    s.b_w = s.a_w = s.pr_w = (size_t)T * ctw;
    s.d_w = (size_t)T * 3 * L * N;
    s.ub_w = (size_t)hd * ctw;
    s.rot_w = (size_t)s.Jt * ctw;
    s.tot_w = ctw;
    s.ua_w = (size_t)2 * (L + ctx->n_p) * N;  // the outer sum over Q u P (lazy ModDown)
    s.work_w = std::max({ks_scratch_words(ctx, level, ks_rot_batch(T - 1)),
                         ks_scratch_words(ctx, level, ks_rot_batch(T), T),
                         ks_scratch_words(ctx, level, ks_rot_batch(s.Jt), s.Jt), (size_t)2 * (1 + level) * N});
    s.total = s.u_w + s.mq_w + s.tw_w + s.mh_w + s.b_w + s.a_w + s.d_w + s.pr_w + s.ub_w + s.rot_w + s.tot_w +
              s.ua_w + s.work_w;
    return s;
}

// Scratch of the weighted-sum call for scores of Lp limbs and values of Lv limbs (words)
struct ApplyScratch {
    uint32_t Jt, nj, logn;
    size_t u_w, mq_w, tw_w, mh_w, r_w, cb_w, ctmp_w, c_w, e_w, d_w, o_w, work_w, total;
};

ApplyScratch apply_scratch(const ckks_ctx *ctx, uint32_t Lp, uint32_t Lv, uint32_t D, uint32_t T, uint32_t hd)
{
    ApplyScratch s{};
    const size_t N = ctx->n;
    const uint32_t lv = Lv - 1, lp = Lp - 1;
    s.Jt = kRotChunk;
    s.nj = hd + T - 1;
    s.logn = log2u(2 * hd);
    s.u_w = (size_t)hd * D;
    s.mq_w = (size_t)Lv * 2 * D * hd;
    s.tw_w = (size_t)2 * Lv * 2 * hd;
    s.mh_w = (size_t)Lv * 2 * D * 2 * hd;
    s.r_w = (size_t)T * 2 * Lv * N;
    s.cb_w = (size_t)s.nj * 2 * Lv * N;
    s.ctmp_w = (size_t)s.Jt * 2 * (Lv - 1) * N;
    s.c_w = s.e_w = (size_t)s.nj * 2 * Lp * N;
    s.d_w = (size_t)3 * Lp * N;
    s.o_w = (size_t)2 * Lp * N;
    const size_t ext = Lp + ctx->n_p, nd = n_digits(ctx, lp);
    const size_t relin_w = (nd * ext + ctx->alpha) * N + 2 * ext * N + 2 * (size_t)Lp * N;
    s.work_w = std::max({ks_scratch_words(ctx, lv, ks_rot_batch(T - 1)),
                         ks_scratch_words(ctx, lp, ks_rot_batch(s.nj - 1)), (size_t)2 * s.Jt * (1 + lv) * N,
                         relin_w, (size_t)2 * (1 + lp) * N});
    s.total = s.u_w + s.mq_w + s.tw_w + s.mh_w + s.r_w + s.cb_w + s.ctmp_w + s.c_w + s.e_w + s.d_w + s.o_w +
              s.work_w;
    return s;
}

struct KeyFinder {
    const int32_t *steps;
    const uint64_t *const *keys;
    uint32_t n;
    const uint64_t *operator()(int32_t st) const
    {
        for (uint32_t r = 0; r < n; r++)
            if (steps[r] == st) return keys[r];
        return nullptr;
    }
};

ckks_status check_cts(const ckks_buf *b, uint32_t count, uint32_t L, const char *what, const char *name)
{
    for (uint32_t i = 0; i < count; i++) {
        CK_REQUIRE(b[i].data && b[i].n_polys == 2, CKKS_EINVAL, "%s: %s %u is not a ciphertext", what, name, i);
        CK_REQUIRE(b[i].n_limbs == L, CKKS_ELEVEL, "%s: %s %u has %u limbs, expected %u", what, name, i,
                   b[i].n_limbs, L);
        CK_REQUIRE(b[i].scale == b[0].scale, CKKS_ESCALE, "%s: %s scales differ", what, name);
    }
    return CKKS_OK;
}

}  // namespace

size_t attn_scores_workspace_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t tokens, uint32_t head_dim)
{
    const ckks_attn_shape sh{tokens, head_dim};
    uint32_t D, logT;
    if (attn_check_shape(ctx, &sh, "attention_scores", &D, &logT) != CKKS_OK || L < 3 || L > ctx->n_q) {
        clear_error();
        return SIZE_MAX;
    }
    return score_scratch(ctx, L, D, tokens, head_dim).total * 8;
}

size_t attn_apply_workspace_bytes(const ckks_ctx *ctx, uint32_t Lp, uint32_t Lv, uint32_t tokens, uint32_t head_dim)
{
    const ckks_attn_shape sh{tokens, head_dim};
    uint32_t D, logT;
    if (attn_check_shape(ctx, &sh, "attention_apply", &D, &logT) != CKKS_OK || Lp < 2 || Lp + 1 > Lv ||
        Lv > ctx->n_q) {
        clear_error();
        return SIZE_MAX;
    }
    return apply_scratch(ctx, Lp, Lv, D, tokens, head_dim).total * 8;
}

extern "C" ckks_status ckks_attention_scores(ckks_ctx *ctx, const ckks_buf *q, uint32_t n_q, const ckks_buf *k,
                                             uint32_t n_k, const uint32_t *k_of_q, const ckks_attn_shape *shape,
                                             const uint64_t *rlk, const int32_t *key_steps,
                                             const uint64_t *const *keys, uint32_t n_keys, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx && q && k && k_of_q && rlk && out && (keys || !n_keys), CKKS_EINVAL,
               "attention_scores: null argument");
    CK_REQUIRE(n_q >= 1 && n_k >= 1, CKKS_EINVAL, "attention_scores: no ciphertexts");
    uint32_t D, logT;
    CK_TRY(attn_check_shape(ctx, shape, "attention_scores", &D, &logT));
    const uint32_t T = shape->tokens, hd = shape->head_dim;
    const uint32_t L = q[0].n_limbs, level = L - 1;
    CK_REQUIRE(L >= 3 && L <= ctx->n_q, CKKS_ELEVEL, "attention_scores: inputs need 3..%u limbs", ctx->n_q);
    CK_REQUIRE(ntt_uses_f64(ctx, L), CKKS_EUNSUPPORTED, "attention_scores: needs primes below 2^50");
    CK_TRY(check_cts(q, n_q, L, "attention_scores", "query"));
    CK_TRY(check_cts(k, n_k, L, "attention_scores", "key"));
    for (uint32_t c = 0; c < n_q; c++) {
        CK_REQUIRE(k_of_q[c] < n_k, CKKS_EINVAL, "attention_scores: query %u names key %u of %u", c, k_of_q[c], n_k);
        CK_REQUIRE(out[c].data && out[c].n_polys == 2 && out[c].n_limbs == L - 2, CKKS_EINVAL,
                   "attention_scores: output %u must be a ciphertext with %u limbs", c, L - 2);
    }
    const KeyFinder find{key_steps, keys, n_keys};
    std::vector<int32_t> qsteps, ksteps, osteps;
    std::vector<const uint64_t *> qkeys, kkeys, okeys;
    for (uint32_t d = 1; d < T; d++) {
        qsteps.push_back(-(int32_t)d);
        ksteps.push_back((int32_t)(d * (D - 1)));
    }
    for (uint32_t kk = 1; kk < hd; kk++) osteps.push_back((int32_t)kk);
    for (auto *pr : {&qsteps, &ksteps, &osteps}) {
        auto &dst = pr == &qsteps ? qkeys : (pr == &ksteps ? kkeys : okeys);
        for (int32_t st : *pr) {
            const uint64_t *kp = find(st);
            CK_REQUIRE(kp, CKKS_ENOKEY, "attention_scores: no key for step %d", st);
            dst.push_back(kp);
        }
    }

    const size_t N = ctx->n, ctw = 2 * (size_t)L * N;
    const ScoreScratch ss = score_scratch(ctx, L, D, T, hd);
    void *w;
    CK_TRY(ctx_scratch(ctx, ss.total * 8, &w));
    double *U = (double *)w;
    double *MQ = U + ss.u_w;
    double *Om = MQ + ss.mq_w, *Omi = Om + ss.tw_w / 2;
    double *Mh = Om + ss.tw_w;
    uint64_t *B = (uint64_t *)(Mh + ss.mh_w);  // [T][2][L][N] rotated keys
    uint64_t *A = B + ss.b_w;                  // [T][2][L][N] rotated queries
    uint64_t *Dt = A + ss.a_w;                 // [T][3][L][N] products
    uint64_t *Pr = Dt + ss.d_w;                // [T][2][L][N] relinearised products P_delta
    uint64_t *Ub = Pr + ss.pr_w;               // [hd][2][L][N] U_k
    uint64_t *rot = Ub + ss.ub_w;              // [Jt][2][L][N]
    uint64_t *tot = rot + ss.rot_w;
    uint64_t *uacc = tot + ss.tot_w;           // [2][L+K][N]
    uint64_t *work = uacc + ss.ua_w;

    // the masks at scale q_level (they multiply the products at the inputs' level), and their correlation form
    CK_TRY(launch_masks(ctx, U, MQ, D, hd, (double)ctx->primes[level], L));
    CK_TRY(launch_corr_tables(ctx, ss.logn, L, 2 * D, hd, MQ, Om, Omi, Mh));
    // queries grouped by key: each key's rotations are computed once
    std::vector<uint32_t> order(n_q);
    for (uint32_t c = 0; c < n_q; c++) order[c] = c;
    std::stable_sort(order.begin(), order.end(), [&](uint32_t a, uint32_t b) { return k_of_q[a] < k_of_q[b]; });
    std::vector<uint64_t *> outs(std::max(T, ss.Jt));
    uint32_t cur_k = UINT32_MAX;
    for (uint32_t c : order) {
        const uint32_t kk = k_of_q[c];
        if (kk != cur_k) {
            HIP_TRY(hipMemcpyAsync(B, k[kk].data, ctw * 8, hipMemcpyDeviceToDevice, ctx->stream));
            for (uint32_t d = 1; d < T; d++) outs[d - 1] = B + (size_t)d * ctw;
            CK_TRY(rotate_core(ctx, k[kk].data, level, ksteps.data(), kkeys.data(), T - 1, outs.data(), work));
            cur_k = kk;
        }
        // 1. Rot_{-delta}(Q), hoisted
        HIP_TRY(hipMemcpyAsync(A, q[c].data, ctw * 8, hipMemcpyDeviceToDevice, ctx->stream));
        for (uint32_t d = 1; d < T; d++) outs[d - 1] = A + (size_t)d * ctw;
        CK_TRY(rotate_core(ctx, q[c].data, level, qsteps.data(), qkeys.data(), T - 1, outs.data(), work));
        // 2. products, relinearised in one batch (key switching with sigma = identity and the relinearisation
        //    key: (d0 + u0, u1), then d1 added)
        CK_TRY(launch_tensor_batch(ctx, Dt, Dt + L * N, Dt + 2 * L * N, 3 * L * N, A, ctw, B, ctw, T, L));
        {
            const uint32_t ext = L + ctx->n_p, nd = n_digits(ctx, level);
            const size_t dig_ct = (size_t)nd * ext * N;
            uint64_t *digits = work;
            uint64_t *rw = digits + (size_t)T * (dig_ct + (size_t)ctx->alpha * N);
            CK_TRY(ks_modup_batch(ctx, Dt + 2 * (size_t)L * N, 3 * (size_t)L * N, T, level, digits));
            const uint32_t bs = ks_rot_batch(T);
            std::vector<uint32_t> g(T, 1u);
            std::vector<const uint64_t *> c0s(T), digs(T), rk(T, rlk);
            std::vector<uint64_t *> po(T);
            for (uint32_t d = 0; d < T; d++) {
                c0s[d] = Dt + (size_t)d * 3 * L * N;
                digs[d] = digits + (size_t)d * dig_ct;
                po[d] = Pr + (size_t)d * ctw;
            }
            for (uint32_t r0 = 0; r0 < T; r0 += bs) {
                const uint32_t cnt = std::min(bs, T - r0);
                CK_TRY(ks_rotate_batch(ctx, level, cnt, c0s.data() + r0, digs.data() + r0, g.data() + r0,
                                       rk.data() + r0, po.data() + r0, rw));
            }
            CK_TRY(launch_binary_batch(ctx, Pr + (size_t)L * N, ctw, Pr + (size_t)L * N, ctw, Dt + (size_t)L * N,
                                       3 * (size_t)L * N, T, L, limb_range(0, L), EW_ADD));
        }
        // 3. U_k = sum_delta M_{(delta + k) mod hd} P_delta = z[-k mod hd] for every k, then each rotated by k
        //    (in chunks) and summed
        CK_TRY(launch_corr(ctx, Ub, Pr, T, hd, -1, 0, L, ss.logn, logT, 2 * D, Om, Omi, Mh));
        if (ctx->lazy_moddown) {
            // the hd - 1 key-switching sums accumulated over Q u P, one ModDown, U_0 added in it
            for (uint32_t k0 = 1; k0 < hd; k0 += ss.Jt) {
                const uint32_t cnt = std::min(ss.Jt, hd - k0);
                CK_TRY(rotate_each_lazy(ctx, Ub + (size_t)k0 * ctw, ctw, cnt, level, osteps.data() + (k0 - 1),
                                        okeys.data() + (k0 - 1), uacc, k0 > 1, work));
            }
            CK_TRY(ks_moddown(ctx, uacc, 2, level, Ub, 1, Ub + (size_t)L * N, tot, work));
        } else {
            CK_TRY(launch_sum_cts(ctx, tot, Ub, 1, ctw, L, false));
            for (uint32_t k0 = 1; k0 < hd; k0 += ss.Jt) {
                const uint32_t cnt = std::min(ss.Jt, hd - k0);
                for (uint32_t r = 0; r < cnt; r++) outs[r] = rot + (size_t)r * ctw;
                CK_TRY(rotate_each(ctx, Ub + (size_t)k0 * ctw, ctw, cnt, level, osteps.data() + (k0 - 1),
                                   okeys.data() + (k0 - 1), outs.data(), work));
                CK_TRY(launch_sum_cts(ctx, tot, rot, cnt, ctw, L, true));
            }
        }
        // 4. the two rescales (by q_level, the masks' scale, and by q_(level-1))
        CK_TRY(rescale_core(ctx, tot, level, rot, work));
        CK_TRY(rescale_core(ctx, rot, level - 1, out[c].data, work));
        out[c].scale = q[c].scale * k[kk].scale / (double)ctx->primes[level - 1];
    }
    return CKKS_OK;
}

extern "C" ckks_status ckks_attention_apply(ckks_ctx *ctx, const ckks_buf *p, uint32_t n_p, const ckks_buf *v,
                                            uint32_t n_v, const uint32_t *v_of_p, const ckks_attn_shape *shape,
                                            const uint64_t *rlk, const int32_t *key_steps,
                                            const uint64_t *const *keys, uint32_t n_keys, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx && p && v && v_of_p && rlk && out && (keys || !n_keys), CKKS_EINVAL,
               "attention_apply: null argument");
    CK_REQUIRE(n_p >= 1 && n_v >= 1, CKKS_EINVAL, "attention_apply: no ciphertexts");
    uint32_t D, logT;
    CK_TRY(attn_check_shape(ctx, shape, "attention_apply", &D, &logT));
    const uint32_t T = shape->tokens, hd = shape->head_dim;
    const uint32_t Lp = p[0].n_limbs, Lv = v[0].n_limbs, lp = Lp - 1, lv = Lv - 1;
    CK_REQUIRE(Lp >= 2 && Lp + 1 <= Lv && Lv <= ctx->n_q, CKKS_ELEVEL,
               "attention_apply: scores need at least 2 limbs and fewer than the values (%u and %u given)", Lp, Lv);
    CK_REQUIRE(ntt_uses_f64(ctx, Lv), CKKS_EUNSUPPORTED, "attention_apply: needs primes below 2^50");
    CK_TRY(check_cts(p, n_p, Lp, "attention_apply", "score"));
    CK_TRY(check_cts(v, n_v, Lv, "attention_apply", "value"));
    for (uint32_t c = 0; c < n_p; c++) {
        CK_REQUIRE(v_of_p[c] < n_v, CKKS_EINVAL, "attention_apply: scores %u name value %u of %u", c, v_of_p[c],
                   n_v);
        CK_REQUIRE(out[c].data && out[c].n_polys == 2 && out[c].n_limbs == Lp - 1, CKKS_EINVAL,
                   "attention_apply: output %u must be a ciphertext with %u limbs", c, Lp - 1);
    }
    const KeyFinder find{key_steps, keys, n_keys};
    std::vector<int32_t> vsteps, psteps;
    std::vector<const uint64_t *> vkeys, pkeys;
    for (uint32_t d = 1; d < T; d++) vsteps.push_back((int32_t)(d * D));
    for (int32_t j = -(int32_t)hd + 1; j < (int32_t)T; j++)
        if (j) psteps.push_back(j);
    for (int32_t st : vsteps) {
        const uint64_t *kp = find(st);
        CK_REQUIRE(kp, CKKS_ENOKEY, "attention_apply: no key for step %d", st);
        vkeys.push_back(kp);
    }
    for (int32_t st : psteps) {
        const uint64_t *kp = find(st);
        CK_REQUIRE(kp, CKKS_ENOKEY, "attention_apply: no key for step %d", st);
        pkeys.push_back(kp);
    }

    const size_t N = ctx->n, ctwv = 2 * (size_t)Lv * N, ctwp = 2 * (size_t)Lp * N;
    const ApplyScratch ss = apply_scratch(ctx, Lp, Lv, D, T, hd);
    void *w;
    CK_TRY(ctx_scratch(ctx, ss.total * 8, &w));
    double *U = (double *)w;
    double *MQ = U + ss.u_w;
    double *Om = MQ + ss.mq_w, *Omi = Om + ss.tw_w / 2;
    double *Mh = Om + ss.tw_w;
    uint64_t *R = (uint64_t *)(Mh + ss.mh_w);  // [T][2][Lv][N]
    uint64_t *Cb = R + ss.r_w;                 // [nj][2][Lv][N] C_j before the rescale
    uint64_t *ctmp = Cb + ss.cb_w;             // [Jt][2][Lv-1][N]
    uint64_t *C = ctmp + ss.ctmp_w;            // [nj][2][Lp][N], index j + hd - 1
    uint64_t *E = C + ss.c_w;                  // [nj][2][Lp][N]
    uint64_t *Dacc = E + ss.e_w;               // [3][Lp][N]
    uint64_t *O = Dacc + ss.d_w;               // [2][Lp][N]
    uint64_t *work = O + ss.o_w;

    // masks at scale q_(level of the values): C_j is rescaled by that prime
    CK_TRY(launch_masks(ctx, U, MQ, D, hd, (double)ctx->primes[lv], Lv));
    CK_TRY(launch_corr_tables(ctx, ss.logn, Lv, 2 * D, hd, MQ, Om, Omi, Mh));
    std::vector<uint32_t> order(n_p);
    for (uint32_t c = 0; c < n_p; c++) order[c] = c;
    std::stable_sort(order.begin(), order.end(), [&](uint32_t a, uint32_t b) { return v_of_p[a] < v_of_p[b]; });
    std::vector<uint64_t *> outs(std::max(T, ss.nj));
    uint32_t cur_v = UINT32_MAX;
    for (uint32_t c : order) {
        const uint32_t vv = v_of_p[c];
        if (vv != cur_v) {
            // 1. R_delta = Rot_{delta D}(V'), hoisted
            HIP_TRY(hipMemcpyAsync(R, v[vv].data, ctwv * 8, hipMemcpyDeviceToDevice, ctx->stream));
            for (uint32_t d = 1; d < T; d++) outs[d - 1] = R + (size_t)d * ctwv;
            CK_TRY(rotate_core(ctx, v[vv].data, lv, vsteps.data(), vkeys.data(), T - 1, outs.data(), work));
            // 2. C_j (index e = j + hd - 1) = z[j mod 2hd], rescaled in chunks and kept on the scores' limbs
            CK_TRY(launch_corr(ctx, Cb, R, T, ss.nj, 1, -(int)(hd - 1), Lv, ss.logn, logT, 2 * D, Om, Omi, Mh));
            for (uint32_t e0 = 0; e0 < ss.nj; e0 += ss.Jt) {
                const uint32_t cnt = std::min(ss.Jt, ss.nj - e0);
                uint64_t *dst = C + (size_t)e0 * ctwp;
                if (Lp == Lv - 1) {
                    CK_TRY(rescale_many(ctx, Cb + (size_t)e0 * ctwv, cnt, lv, dst, work));
                } else {
                    CK_TRY(rescale_many(ctx, Cb + (size_t)e0 * ctwv, cnt, lv, ctmp, work));
                    CK_TRY(launch_copy_rows(ctx, dst, (size_t)Lp * N, nullptr, 0, ctmp, (size_t)(Lv - 1) * N,
                                            (size_t)Lp * N, 2 * cnt));
                }
            }
            cur_v = vv;
        }
        // 3. Rot_j(P), hoisted (E index j + hd - 1; j = 0 is P itself)
        HIP_TRY(hipMemcpyAsync(E + (size_t)(hd - 1) * ctwp, p[c].data, ctwp * 8, hipMemcpyDeviceToDevice,
                               ctx->stream));
        for (uint32_t r = 0, e = 0; e < ss.nj; e++)
            if (e != hd - 1) outs[r++] = E + (size_t)e * ctwp;
        CK_TRY(rotate_core(ctx, p[c].data, lp, psteps.data(), pkeys.data(), ss.nj - 1, outs.data(), work));
        // 4. sum_j Rot_j(P) x C_j, one relinearisation, the final rescale
        CK_TRY(launch_tensor_acc(ctx, Dacc, E, C, ss.nj, Lp, Lp));
        {
            const uint32_t ext = Lp + ctx->n_p, nd = n_digits(ctx, lp);
            uint64_t *digits = work;
            uint64_t *u = digits + ((size_t)nd * ext + ctx->alpha) * N;
            uint64_t *cw = u + 2 * (size_t)ext * N;
            CK_TRY(ks_modup(ctx, Dacc + 2 * (size_t)Lp * N, lp, digits));
            CK_TRY(ks_inner_product(ctx, digits, nd, rlk, lp, 1, u));
            CK_TRY(ks_moddown(ctx, u, 2, lp, Dacc, 1, Dacc + (size_t)Lp * N, O, cw));
        }
        CK_TRY(rescale_core(ctx, O, lp, out[c].data, work));
        out[c].scale = p[c].scale * v[vv].scale / (double)ctx->primes[lp];
    }
    return CKKS_OK;
}
