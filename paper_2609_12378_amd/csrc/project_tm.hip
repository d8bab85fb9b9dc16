// The packed projection Y = X W in the token-major layout s = t*D + f: input ciphertext i holds features
// [iD, (i+1)D) of all T = N/2D tokens, output j features [jD, (j+1)D).
//
// A left rotation by k moves feature o + k of a token to feature o only while o + k < D; the entries of the
// cyclic diagonal D_k(A_{j,i})[o] = A[o, (o + k) mod D] (A = W^T) that wrap past D need the rotation by k - D
// instead.  Splitting each diagonal into U_k (no wrap) and V_k (wrap) and factoring out the giant steps as in
// the feature-major case (Section "Matrix Representations and Linear Computation in CKKS", Eq.
// slot-diagonal-matvec, with baby-step/giant-step reuse):
//   out_j = Rescale( sum_g Rot_{n1 g}( sum_{i,b} U_{j,i,g,b} * Rot_b(x_i) + V_{j,i,g,b} * Rot_{b-D}(x_i) ) ),
// U / V the vectors U_k / V_k (k = n1 g + b) shifted right by n1 g, the same for every token.
//
// Why this layout is cheap to encode: a slot vector of period D (a power of two) is fixed by X -> X^a for
// every a = 1 mod 4D, so its encoding is m'(X^T) with m' the encoding of one period in the ring of degree 2D,
// and its NTT value at (bit-reversed) index x is Q[x >> log2 T], Q the 2D-point negacyclic NTT of m' with
// psi^T, whose twiddles psi^(T brev_9(e)) = psi^(brev_16(e)) are the first 2D entries of the ring's table.
// A weight plaintext therefore costs one D-point FFT and one 2D-point NTT per limb instead of an N-point
// encode, and in the multiply-accumulate every run of T consecutive ciphertext values meets one scalar.
//
// The D-point FFT is the encode's own evaluation (radix-2 decimation in time from bit-reversed input,
// butterfly t = w a[hi], complex products without fused multiply-add) at M' = D: its twiddles and twist
// factors are the ring's tables at stride T (the angles 2 pi e T / (D T) and pi k T / (2 D T) differ from
// 2 pi e / D and pi k / 2D by exact powers of two), and the scale is Delta * (2 / 2D), so the rounded
// coefficients are the ones the degree-2D encode gives.
#pragma clang fp contract(off)
#include <vector>

#include "ckks_internal.h"
#include "ntt_core.h"
#include "ops.h"

namespace {

constexpr int kThreads = 256;
constexpr int kPE = 8;        // plaintexts per encode block: 8 consecutive doubles per table row (64 B)
constexpr int kMaxD = 256;    // features per ciphertext handled by the encode kernel
constexpr int kJT = 32;       // output ciphertexts per vector-ALU multiply-accumulate tile
constexpr int kMaxJtMfma = 32; // and per matrix-core one (64 outputs need 452 VGPRs, one wave per SIMD: slower)

__device__ __forceinline__ double2 cmul(double2 a, double2 b)
{
    const double p1 = a.x * b.x, p2 = a.y * b.y, p3 = a.x * b.y, p4 = a.y * b.x;
    return make_double2(p1 - p2, p3 + p4);
}

struct TmArgs {
    const double *Wd;   // W's cyclic diagonals [jb][i][k][o]
    const double *U;    // or explicit period vectors: plaintext pt's D values at U[pt D ..] (then Wd is unused)
    uint32_t D, logD, n_in, n1g, bcount;
    uint32_t j0, jc;    // first output of the tile, outputs in the tile
    uint32_t pb0, P;    // first (input, baby step) pair of the sub-batch, pairs in it
    uint32_t npt;       // plaintexts in the sub-batch: P * 2 * jc, index (p * 2 + uv) * jc + jj
};

// Encode kPE periodic weight plaintexts per block and transform them: Q[l][x][pt] (x < 2D) holds the
// canonical residue of plaintext pt's NTT values x*T .. x*T + T - 1 modulo q_l, as a double.  512 threads.
// For 2D = 512 and 256 the transform runs on the register-resident 8-residue stages: for 512 points the first
// stage (pairs j, j + 256, twiddle Psi[1]) is applied while the values are loaded, leaving two 256-point
// sub-transforms with bases 2 and 3 (group g of their stage S takes Psi[(2 + i) 2^S + g]); every stage
// reduces, so all values stay below 2q.  Other sizes use plain LDS stages.
__global__ __launch_bounds__(512) void k_enc_periodic(TmArgs a, const double2 *__restrict__ fft_w,
                                                      const double2 *__restrict__ twist, uint32_t T, double c,
                                                      uint32_t L, const ModQ *__restrict__ mods,
                                                      const double *__restrict__ twf, uint32_t log_n, double *Q)
{
    constexpr uint32_t kBT = 512;
    __shared__ double2 buf[kPE * kMaxD];        // FFT, then the transform's outputs (kPE x 2D doubles)
    __shared__ int64_t mq[kPE * 2 * kMaxD];     // rounded coefficients m'
    __shared__ double tws[2][256];
    __shared__ double tr[2 * kPE][nttc::kTr8];
    const uint32_t D = a.D, logD = a.logD, D2 = 2 * D;
    const uint32_t pt0 = blockIdx.x * kPE;
    // 1. one period of each plaintext's slot vector, at its bit-reversed FFT position
    for (uint32_t e = threadIdx.x; e < kPE * D; e += kBT) {
        const uint32_t p = e / D, j = e % D, pt = pt0 + p;
        double v = 0.0;
        if (pt < a.npt && a.U) {
            v = a.U[(size_t)pt * D + j];
        } else if (pt < a.npt) {
            const uint32_t jj = pt % a.jc, uv = (pt / a.jc) & 1, pr = a.pb0 + pt / (2 * a.jc);
            const uint32_t i = pr / a.bcount, b = pr % a.bcount, k = a.n1g + b;
            const uint32_t o = (j + D - a.n1g % D) % D;   // feature before the giant-step shift
            const bool wraps = o + k >= D;
            if (wraps == (uv == 1))
                v = a.Wd[(((size_t)(a.j0 + jj) * a.n_in + i) * D + k) * D + o];
        }
        // slot j sits at FFT position brev((5^j mod 4D - 1) / 4)
        uint32_t e5 = 1, base = 5, ex = j;
        while (ex) {
            if (ex & 1) e5 = (e5 * base) & (4 * D - 1);
            base = (base * base) & (4 * D - 1);
            ex >>= 1;
        }
        const uint32_t s = (e5 - 1) >> 2;
        const uint32_t pos = logD ? __brev(s) >> (32 - logD) : 0;
        buf[p * D + pos] = make_double2(v, 0.0);
    }
    __syncthreads();
    // 2. radix-2 stages len = 2 .. D
    for (uint32_t len = 2; len <= D; len <<= 1) {
        const uint32_t half = len >> 1, step = D / len;
        for (uint32_t e = threadIdx.x; e < kPE * (D / 2); e += kBT) {
            const uint32_t p = e / (D / 2), bf = e % (D / 2);
            const uint32_t blk = bf / half, k = bf % half;
            double2 *row = buf + p * D + blk * len;
            const double2 w = fft_w[(size_t)k * step * T];
            const double2 t = cmul(w, row[k + half]);
            const double2 lo = row[k];
            row[k + half] = make_double2(lo.x - t.x, lo.y - t.y);
            row[k] = make_double2(lo.x + t.x, lo.y + t.y);
        }
        __syncthreads();
    }
    // 3. twist, scale and round: m'[k] = round(c Re v_k), m'[k + D] = round(c Im v_k)
    for (uint32_t e = threadIdx.x; e < kPE * D; e += kBT) {
        const uint32_t p = e / D, k = e % D;
        const double2 v = cmul(twist[(size_t)k * T], buf[p * D + k]);
        mq[p * D2 + k] = (int64_t)round(c * v.x);
        mq[p * D2 + k + D] = (int64_t)round(c * v.y);
    }
    double *xs = (double *)buf;  // kPE rows of 2D doubles
    const bool regs = D2 == 512 || D2 == 256;
    const uint32_t nsub = D2 / 256;
    // 4. per limb: the 2D-point negacyclic NTT (Cooley-Tukey, group i of stage m takes Psi[m + i])
    for (uint32_t l = 0; l < L; l++) {
        const ModQ md = mods[l];
        const nttc::Ar<true> ar(md);
        const double *tw = twf + ((size_t)l << log_n);
        __syncthreads();
        if (regs) {
            for (uint32_t e = threadIdx.x; e < nsub * 255; e += kBT) {
                const uint32_t si = e / 255, ee = e % 255 + 1, m = 1u << (31 - __clz(ee));
                tws[si][ee] = tw[(size_t)(nsub == 2 ? 2 + si : 1) * m + (ee - m)];
            }
            __syncthreads();
            const uint32_t sub = threadIdx.x >> 5, t = threadIdx.x & 31;
            const uint32_t p = sub / nsub, si = sub % nsub;
            const bool live = p < (uint32_t)kPE;
            double x[nttc::kE8];
            if (nsub == 2) {
                const double w0 = tw[1];
#pragma unroll
                for (int k = 0; k < nttc::kE8; k++) {
                    const uint32_t u = nttc::u8<0>(t, k);
                    double xo = 0.0;
                    if (live) {
                        const double X = ar.from_i64(mq[p * D2 + u], md), Y = ar.from_i64(mq[p * D2 + u + 256], md);
                        const double r = ar.mul(Y, w0);
                        xo = si == 0 ? X + r : X - r;
                    }
                    x[k] = xo;
                }
            } else {
#pragma unroll
                for (int k = 0; k < nttc::kE8; k++)
                    x[k] = live ? ar.from_i64(mq[p * D2 + nttc::u8<0>(t, k)], md) : 0.0;
            }
            nttc::fwd8_256<0xFFu>(x, tws[si], tr[sub], t, ar);
            if (live) {
#pragma unroll
                for (int k = 0; k < nttc::kE8; k++) xs[p * D2 + 256 * si + nttc::u8<2>(t, k)] = x[k];
            }
            __syncthreads();
        } else {
            for (uint32_t e = threadIdx.x; e < kPE * D2; e += kBT) xs[e] = ar.from_i64(mq[e], md);
            __syncthreads();
            for (uint32_t m = 1, t = D; m < D2; m <<= 1, t >>= 1) {
                for (uint32_t e = threadIdx.x; e < kPE * D; e += kBT) {
                    const uint32_t p = e / D, bf = e % D;
                    const uint32_t g = bf / t, j = bf % t;
                    double *row = xs + p * D2 + 2 * g * t + j;
                    double x0 = row[0], x1 = row[t];
                    ar.ct(x0, x1, tw[m + g]);
                    row[0] = x0;
                    row[t] = x1;
                }
                __syncthreads();
            }
        }
        // rows of Q: for each x, kPE consecutive plaintexts
        for (uint32_t e = threadIdx.x; e < kPE * D2; e += kBT) {
            const uint32_t p = e % kPE, x = e / kPE, pt = pt0 + p;
            if (pt < a.npt) Q[((size_t)l * D2 + x) * a.npt + pt] = (double)ar.to_canon(xs[p * D2 + x]);
        }
    }
}

// Multiply-accumulate of one sub-batch: block (limb l, 128 positions) holds, per thread (polynomial, position),
// the tile's jc accumulators and runs over the sub-batch's pairs:
//   acc_jj += Q_U[jj][pair] * xr[pair] + Q_V[jj][pair] * xw[pair]   (mod q_l),
// the Q values of a position being those of its run x = pos >> log2 T.  With T >= 128 (UNIF) the block lies in
// one run, so its Q values are the same for every lane and are read with scalar loads.  Products (|x| < q,
// 0 <= Q < q) are below 0.875 q, and the sum is range-reduced after every pair (at most 0.5 q + 1.75 q): every
// value is an exact integer below 2^53.  acc ([jc][2][L][N], canonical) is written, or added to when
// `accumulate`.
template <int JT, bool UNIF>
__global__ __launch_bounds__(kThreads) void k_mac_tm(uint64_t *acc, const double *__restrict__ x2,
                                                     const double *__restrict__ Q, TmArgs a, uint32_t n1, uint32_t L,
                                                     uint32_t logT, uint32_t log_n, int accumulate,
                                                     const ModQ *__restrict__ mods)
{
    const uint32_t blocks_per_limb = 1u << (log_n - 7);
    const uint32_t l = blockIdx.x / blocks_per_limb, pb = blockIdx.x % blocks_per_limb;
    const uint32_t poly = threadIdx.x >> 7, pos = (pb << 7) + (threadIdx.x & 127);
    const nttc::Ar<true> ar(mods[l]);
    const uint32_t x = UNIF ? (pb << 7) >> logT : pos >> logT, D2 = 2 * a.D;
    const size_t n = (size_t)1 << log_n, ctw = 2 * (size_t)L * n;
    const double *qrow = Q + ((size_t)l * D2 + x) * a.npt;
    double s[JT];
#pragma unroll
    for (int jj = 0; jj < JT; jj++) s[jj] = 0.0;
    const size_t off = ((size_t)poly * L + l) * n + pos;
    for (uint32_t p = 0; p < a.P; p++) {
        const uint32_t pr = a.pb0 + p, i = pr / a.bcount, b = pr % a.bcount;
        const double *xp = x2 + (size_t)(i * n1 + b) * 2 * ctw + off;
        const double xr = xp[0], xw = xp[ctw];
        const double *qu = qrow + (size_t)p * 2 * a.jc, *qv = qu + a.jc;
#pragma unroll
        for (int jj = 0; jj < JT; jj++) {
            if (jj < (int)a.jc) s[jj] = ar.red(s[jj] + ar.mul(xr, qu[jj]) + ar.mul(xw, qv[jj]));
        }
    }
    const uint64_t q = mods[l].q;
#pragma unroll
    for (int jj = 0; jj < JT; jj++) {
        if (jj < (int)a.jc) {
            uint64_t *dst = acc + (size_t)jj * ctw + off;
            uint64_t r = ar.to_canon(s[jj]);
            if (accumulate) r = addmod(r, *dst, q);
            *dst = r;
        }
    }
}

// ---- the multiply-accumulate on the matrix cores ----------------------------------------------------------
//
// Per (limb l, run x) the sub-batch's sum is a dense product: acc[jj][c] = sum_kappa Q[jj][kappa] X[kappa][c]
// (kappa = 2 pair + uv over the sub-batch, c a position of the run in one polynomial), over residues below
// 2^50.  Each residue is written in seven balanced base-256 digits (v = sum_a d_a 256^a, d_a in [-128, 127]),
// so that with C_s = sum_{a + b = s} sum_kappa Qd_a Xd_b (13 groups, each a sum of int8 x int8 products that
// v_mfma_i32_16x16x64_i8 accumulates exactly in int32 while K <= 4096: |C_s| < 7 * 4096 * 2^14 < 2^31)
//   sum_kappa Q X = sum_s 256^s C_s   (an integer identity, reduced mod q_l in the epilogue).
// The ciphertext digits are laid out once per projection as Xd[digit][l][poly N + pos][kappa] (kappa
// contiguous, 16 bytes per MFMA lane); the plaintext digits of a 64-kappa block are formed in LDS from Q.
// Operand layouts (checked on the hardware): A 16x64, lane i holds row i % 16, bytes k = 16 (i / 16) + 0..15;
// B 64x16, lane i holds column i % 16, the same k; C 16x16, lane i holds column i % 16, rows 4 (i / 16) + r.
typedef int v4i __attribute__((ext_vector_type(4)));
constexpr int kDig = 7, kGroups = 2 * kDig - 1, kKB = 64, kRowW = 20;

__device__ __forceinline__ void digits7(uint64_t v, int8_t *d, size_t stride)
{
#pragma unroll
    for (int a = 0; a < kDig; a++) {
        int t = (int)(v & 255u);
        v >>= 8;
        if (t >= 128) {
            t -= 256;
            v += 1;
        }
        d[(size_t)a * stride] = (int8_t)t;
    }
}

// x2 ([n_in][n1][xr, xw][2][L][N] canonical) -> Xd[a][l][poly N + pos][kappa], kappa = 2 (i n1 + b) + uv < kt
// (rows padded to kt_pad bytes with zeros).  Block: (l, 64 columns, 64 kappa), staged through LDS.
__global__ __launch_bounds__(kThreads) void k_xdigits(const uint64_t *__restrict__ x2, int8_t *Xd, uint32_t L,
                                                      uint32_t log_n, uint32_t kt, uint32_t kt_pad)
{
    __shared__ uint64_t tile[64][65];
    const uint32_t cols = 2u << log_n, cblocks = cols / 64, kblocks = kt_pad / 64;
    const uint32_t kb = blockIdx.x % kblocks, rest = blockIdx.x / kblocks;
    const uint32_t cb = rest % cblocks, l = rest / cblocks;
    const size_t n = (size_t)1 << log_n, ctw = 2 * (size_t)L * n;
    const uint32_t c0 = cb * 64, k0 = kb * 64;
    // all 16 loads of a thread issued before any is stored (one memory wait per thread, not sixteen)
    const uint32_t cc_r = threadIdx.x % 64, c = c0 + cc_r;
    const uint32_t poly = c >> log_n, pos = c & ((1u << log_n) - 1);
    const uint64_t *src = x2 + ((size_t)poly * L + l) * n + pos;
    uint64_t vals[64 * 64 / kThreads];
#pragma unroll
    for (int i = 0; i < 64 * 64 / kThreads; i++) {
        const uint32_t kappa = k0 + threadIdx.x / 64 + (kThreads / 64) * i;
        vals[i] = kappa < kt ? src[(size_t)kappa * ctw] : 0;
    }
#pragma unroll
    for (int i = 0; i < 64 * 64 / kThreads; i++) tile[threadIdx.x / 64 + (kThreads / 64) * i][cc_r] = vals[i];
    __syncthreads();
    // each thread writes 16 consecutive kappa of one column: one 16-byte store per digit plane (kt_pad, k0 and the
    // 16-kappa offset are multiples of 16, and Xd is 16-byte aligned)
    const size_t plane = (size_t)L * cols * kt_pad;
    static_assert(kThreads == 256, "64 columns x 4 groups of 16 kappa");
    const uint32_t cc = threadIdx.x >> 2, kq = (threadIdx.x & 3u) << 4;
    uint32_t w[kDig][4] = {};
#pragma unroll
    for (int i = 0; i < 16; i++) {
        uint64_t v = tile[kq + i][cc];
#pragma unroll
        for (int a = 0; a < kDig; a++) {
            int t = (int)(v & 255u);
            v >>= 8;
            if (t >= 128) {
                t -= 256;
                v += 1;
            }
            w[a][i >> 2] |= (uint32_t)(uint8_t)t << (8 * (i & 3));
        }
    }
    int8_t *dst = Xd + ((size_t)l * cols + c0 + cc) * kt_pad + k0 + kq;
#pragma unroll
    for (int a = 0; a < kDig; a++)
        *(uint4 *)(dst + (size_t)a * plane) = make_uint4(w[a][0], w[a][1], w[a][2], w[a][3]);
}

// Block (limb l, run x, polynomial, part): NW waves, wave w holds 16 positions of the run (x T + 16 (part NW + w)
// + 0..15) of the polynomial and the tile's jc <= 16 MT outputs (MT 16-row MFMA tiles).  Q ([L][2D][npt],
// npt = K jc, kappa-major) gives the plaintext digits of each 64-kappa block (rows jj >= jc and kappa >= K are
// zero); Xd the ciphertext digits from kappa_base on (16-byte aligned, rows padded so a block never reads past
// them).
template <int NW, int MT>
__global__ __launch_bounds__(64 * NW) void k_mac_tm_mfma(uint64_t *acc, const int8_t *__restrict__ Xd,
                                                           const double *__restrict__ Q, uint32_t jc, uint32_t K,
                                                           uint32_t kappa_base, uint32_t kt_pad, uint32_t D2,
                                                           uint32_t L, uint32_t logT, uint32_t log_n,
                                                           int accumulate, const ModQ *__restrict__ mods)
{
    constexpr int R = 16 * MT;
    // plaintext digits of the 64-kappa block: row jj of digit a holds 64 bytes, padded to 80 so that both the
    // packed 4-byte writes (lanes along jj) and the 16-byte MFMA reads spread over the banks
    __shared__ __attribute__((aligned(16))) uint32_t A[kDig][R][kRowW];
    const uint32_t parts = (1u << (logT - 4)) / NW;
    uint32_t bid = blockIdx.x;
    const uint32_t part = bid % parts;
    bid /= parts;
    const uint32_t poly = bid & 1, x = (bid >> 1) % D2, l = (bid >> 1) / D2;
    const uint32_t lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint32_t pos = (x << logT) + 16 * (part * NW + w) + (lane & 15);
    const size_t n = (size_t)1 << log_n, cols = 2 * n;
    const size_t plane = (size_t)L * cols * kt_pad;
    const int8_t *xb = Xd + ((size_t)l * cols + (size_t)poly * n + pos) * kt_pad + kappa_base + 16 * (lane >> 4);
    const double *qx = Q + ((size_t)l * D2 + x) * (size_t)K * jc;
    v4i c[MT][kGroups];
#pragma unroll
    for (int m = 0; m < MT; m++)
#pragma unroll
        for (int g = 0; g < kGroups; g++) c[m][g] = v4i{0, 0, 0, 0};
    // software pipeline: the next block's ciphertext digits and plaintext values are loaded into registers
    // while the current block's products run
    constexpr int QPT = (R * (kKB / 4) + 64 * NW - 1) / (64 * NW);  // packed table entries per thread
    auto load_q = [&](uint32_t k0, double (&qv)[QPT][4]) {
#pragma unroll
        for (int i = 0; i < QPT; i++) {
            const uint32_t e = threadIdx.x + i * 64 * NW, jj = e % R, k4 = e / R;
#pragma unroll
            for (int t = 0; t < 4; t++) {
                const uint32_t kappa = k0 + 4 * k4 + t;
                qv[i][t] = (e < R * (kKB / 4) && jj < jc && kappa < K) ? qx[(size_t)kappa * jc + jj] : 0.0;
            }
        }
    };
    v4i bn[kDig];
    double qn[QPT][4];
#pragma unroll
    for (int d = 0; d < kDig; d++) bn[d] = *(const v4i *)(xb + (size_t)d * plane);
    load_q(0, qn);
    for (uint32_t k0 = 0; k0 < K; k0 += kKB) {
        v4i b[kDig];
        double qc[QPT][4];
#pragma unroll
        for (int d = 0; d < kDig; d++) b[d] = bn[d];
#pragma unroll
        for (int i = 0; i < QPT; i++)
#pragma unroll
            for (int t = 0; t < 4; t++) qc[i][t] = qn[i][t];
        if (k0 + kKB < K) {
#pragma unroll
            for (int d = 0; d < kDig; d++) bn[d] = *(const v4i *)(xb + (size_t)d * plane + k0 + kKB);
            load_q(k0 + kKB, qn);
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < QPT; i++) {
            const uint32_t e = threadIdx.x + i * 64 * NW, jj = e % R, k4 = e / R;
            if (e < R * (kKB / 4)) {
                uint32_t packed[kDig] = {0, 0, 0, 0, 0, 0, 0};
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    int8_t d[kDig];
                    digits7((uint64_t)qc[i][t], d, 1);
#pragma unroll
                    for (int a = 0; a < kDig; a++) packed[a] |= (uint32_t)(uint8_t)d[a] << (8 * t);
                }
#pragma unroll
                for (int a = 0; a < kDig; a++) A[a][jj][k4] = packed[a];
            }
        }
        __syncthreads();
#pragma unroll
        for (int m = 0; m < MT; m++) {
#pragma unroll
            for (int a = 0; a < kDig; a++) {
                const v4i av = *(const v4i *)&A[a][16 * m + (lane & 15)][4 * (lane >> 4)];
#pragma unroll
                for (int d = 0; d < kDig; d++)
                    c[m][a + d] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, b[d], c[m][a + d], 0, 0, 0);
            }
        }
    }
    // epilogue: sum_s 256^s C_s mod q_l, canonical, added to the stored sums when accumulating
    const ModQ md = mods[l];
    const nttc::Ar<true> ar(md);
    double w256[kGroups];
    w256[0] = 1.0;
#pragma unroll
    for (int g = 1; g < kGroups; g++) w256[g] = (double)ar.to_canon(ar.mul(w256[g - 1], 256.0));
    const size_t ctw = 2 * (size_t)L * n;
#pragma unroll
    for (int m = 0; m < MT; m++) {
#pragma unroll
        for (int r = 0; r < 4; r++) {
            const uint32_t jj = 16 * m + 4 * (lane >> 4) + r;
            double sum = 0.0;
#pragma unroll
            for (int g = 0; g < kGroups; g++) {
                sum += ar.mul((double)c[m][g][r], w256[g]);
                if ((g & 3) == 3) sum = ar.red(sum);
            }
            if (jj < jc) {
                uint64_t *dst = acc + (size_t)jj * ctw + ((size_t)poly * L + l) * n + pos;
                uint64_t v = ar.to_canon(sum);
                if (accumulate) v = addmod(v, *dst, md.q);
                *dst = v;
            }
        }
    }
}

struct TmScratch {
    uint32_t Jt, Pb;
    bool mfma;             // the multiply-accumulate runs on the matrix cores
    uint32_t kt, kt_pad;   // kappa count (2 n_in n1) and the padded digit-row length in bytes
    size_t x2_w, acc_w, tot_w, rot_w, q_w, ks_w, wd_w, xd_w, ua_w, total;
};

TmScratch tm_scratch(const ckks_ctx *ctx, uint32_t L, uint32_t D, uint32_t d_in, uint32_t d_out, uint32_t n1)
{
    TmScratch ts{};
    const uint32_t level = L - 1, n_in = d_in / D, n_out = d_out / D;
    const size_t N = ctx->n, ctw = 2 * (size_t)L * N;
    const uint32_t T = (uint32_t)(N / (2 * D));
    // the matrix-core path needs runs of 16..128 positions (a 16-column tile inside one run, at most 8 tiles per
    // block) and every giant step over the same n1 baby steps (D a multiple of n1)
    ts.mfma = T >= 16 && T <= 128 && D % n1 == 0;
    // output tiles of at most kJT (vector ALU) or kMaxJtMfma (matrix cores), balanced
    const uint32_t jmax = ts.mfma ? kMaxJtMfma : kJT;
    const uint32_t tiles = (n_out + jmax - 1) / jmax;
    ts.Jt = (n_out + tiles - 1) / tiles;
    // pairs per sub-batch: the tile's weight tables within 2 GiB, a multiple of 8 (16-byte aligned digit rows),
    // at most 2048 (int32 digit sums stay exact)
    const size_t per_pair = (size_t)2 * ts.Jt * L * 2 * D * sizeof(double);
    const uint32_t maxpairs = n_in * n1;
    uint32_t Pb = (uint32_t)std::min<size_t>(2048, std::max<size_t>(8, ((size_t)1 << 31) / per_pair));
    if (ctx->proj_max_pairs) Pb = std::min(Pb, std::max<uint32_t>(8, ctx->proj_max_pairs));
    Pb &= ~7u;
    ts.Pb = std::min(Pb, maxpairs);
    ts.kt = 2 * n_in * n1;
    ts.kt_pad = ((ts.kt + 63) & ~63u) + 64;
    ts.x2_w = (size_t)n_in * n1 * 2 * ctw;
    ts.acc_w = ts.tot_w = ts.rot_w = (size_t)ts.Jt * ctw;
    ts.q_w = (size_t)ts.Pb * 2 * ts.Jt * L * 2 * D;
    ts.ks_w = std::max(ks_scratch_words(ctx, level, ks_rot_batch(2 * n1 - 1)),
                       ks_scratch_words(ctx, level, ks_rot_batch(ts.Jt), ts.Jt));
    ts.wd_w = (size_t)d_in * d_out;
    ts.xd_w = ts.mfma ? ((size_t)kDig * L * 2 * N * ts.kt_pad + 7) / 8 : 0;
    ts.ua_w = ctx->lazy_moddown ? (size_t)ts.Jt * 2 * (L + ctx->n_p) * N : 0;
    ts.total = ts.x2_w + ts.acc_w + ts.tot_w + ts.rot_w + ts.q_w + ts.ks_w + ts.wd_w + ts.xd_w + ts.ua_w;
    return ts;
}

ckks_status launch_mac_tm_mfma(ckks_ctx *ctx, uint64_t *acc, const int8_t *Xd, const double *Q, const TmArgs &a,
                               uint32_t kt_pad, uint32_t L, uint32_t logT, bool accumulate)
{
    return launch_mac_mfma(ctx, acc, Xd, Q, a.jc, 2 * a.P, 2 * a.pb0, kt_pad, 2 * a.D, L, logT, accumulate);
}

ckks_status launch_mac_tm(ckks_ctx *ctx, uint64_t *acc, const double *x2, const double *Q, const TmArgs &a,
                          uint32_t n1, uint32_t L, uint32_t logT, bool accumulate)
{
    const uint32_t blocks = L << (ctx->log_n - 7);
    const double res = (double)a.jc * 2 * L * ctx->n;
    // the pairs' two ciphertexts once, the accumulators once (read when accumulating) and written
    prof_begin(ctx, K_MAC_TM, 8.0 * (double)a.P * 2 * 2 * L * ctx->n + 8.0 * res * (accumulate ? 2 : 1),
               res * a.P * 2 * 8.0);
    const bool unif = logT >= 7;
#define CK_MAC_TM(J, U)                                                                                          \
    hipLaunchKernelGGL((k_mac_tm<J, U>), dim3(blocks), dim3(kThreads), 0, ctx->stream, acc, x2, Q, a, n1, L, logT, \
                       ctx->log_n, (int)accumulate, ctx->d_mod)
    if (a.jc <= 8) {
        if (unif) CK_MAC_TM(8, true); else CK_MAC_TM(8, false);
    } else if (a.jc <= 16) {
        if (unif) CK_MAC_TM(16, true); else CK_MAC_TM(16, false);
    } else {
        if (unif) CK_MAC_TM(kJT, true); else CK_MAC_TM(kJT, false);
    }
#undef CK_MAC_TM
    prof_end(ctx, K_MAC_TM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_enc_periodic(ckks_ctx *ctx, const TmArgs &a, double delta, uint32_t L, double *Q)
{
    const uint32_t T = (uint32_t)(ctx->n / (2 * a.D));
    const double c = delta * (2.0 / (double)(2 * a.D));
    const double pts = (double)a.npt;
    // W's diagonals in, the tables out; FFT and transforms (D/2 log D + L D log 2D butterflies per plaintext)
    prof_begin(ctx, K_ENC_TM, 8.0 * pts * a.D + 8.0 * pts * L * 2 * a.D,
               pts * (a.D / 2.0 * a.logD * 10.0 + L * (double)a.D * (a.logD + 1) * kOpsButterflyF64));
    hipLaunchKernelGGL(k_enc_periodic, dim3((a.npt + kPE - 1) / kPE), dim3(512), 0, ctx->stream, a,
                       (const double2 *)ctx->d_fft_w, (const double2 *)ctx->d_fft_twist, T, c, L, ctx->d_mod,
                       ctx->d_twf, ctx->log_n, Q);
    prof_end(ctx, K_ENC_TM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status tm_check_shape(const ckks_ctx *ctx, uint32_t L, uint32_t T, uint32_t d_in, uint32_t d_out, uint32_t n1,
                           uint32_t *Dout)
{
    const uint32_t slots = ctx->n / 2;
    CK_REQUIRE(T >= 1 && slots % T == 0, CKKS_EINVAL, "linear_project_tm: %u tokens do not divide %u slots", T,
               slots);
    const uint32_t D = slots / T;
    CK_REQUIRE(D >= 4 && D <= (uint32_t)kMaxD && (D & (D - 1)) == 0 && T >= 2, CKKS_EUNSUPPORTED,
               "linear_project_tm: %u features per ciphertext (a power of two in [4, %d], at least 2 tokens)", D,
               kMaxD);
    CK_REQUIRE(d_in > 0 && d_out > 0 && d_in % D == 0 && d_out % D == 0, CKKS_EINVAL,
               "linear_project_tm: d_in %u and d_out %u must be positive multiples of %u", d_in, d_out, D);
    CK_REQUIRE(n1 >= 1 && n1 <= D, CKKS_EINVAL, "linear_project_tm: n1 %u outside [1, %u]", n1, D);
    CK_REQUIRE(L >= 2 && L <= ctx->n_q, CKKS_ELEVEL, "linear_project_tm: inputs need 2..%u limbs", ctx->n_q);
    CK_REQUIRE(ntt_uses_f64(ctx, L), CKKS_EUNSUPPORTED, "linear_project_tm: needs primes below 2^50");
    CK_REQUIRE(ctx->log_n >= 8, CKKS_EUNSUPPORTED, "linear_project_tm: needs N >= 256");
    *Dout = D;
    return CKKS_OK;
}

}  // namespace

uint32_t mac_kt_pad(uint32_t kt) { return ((kt + 63) & ~63u) + 64; }

size_t mac_digit_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t kt_pad)
{
    return (size_t)kDig * L * 2 * ctx->n * kt_pad;
}

uint32_t mac_max_outputs() { return kMaxJtMfma; }

ckks_status launch_xdigits(ckks_ctx *ctx, const uint64_t *x2, int8_t *Xd, uint32_t L, uint32_t kt, uint32_t kt_pad)
{
    const uint32_t blocks = L * (uint32_t)((2 * ctx->n) / 64) * (kt_pad / 64);
    prof_begin(ctx, K_ELEM, 8.0 * kt * 2 * L * ctx->n + (double)kDig * kt_pad * 2 * L * ctx->n);
    hipLaunchKernelGGL(k_xdigits, dim3(blocks), dim3(kThreads), 0, ctx->stream, x2, Xd, L, ctx->log_n, kt, kt_pad);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_mac_mfma(ckks_ctx *ctx, uint64_t *acc, const int8_t *Xd, const double *Q, uint32_t jc, uint32_t K,
                            uint32_t kbase, uint32_t kt_pad, uint32_t D2, uint32_t L, uint32_t logT, bool accumulate)
{
    const uint32_t tiles16 = 1u << (logT - 4);
    CK_REQUIRE(jc >= 1 && jc <= (uint32_t)kMaxJtMfma && kbase % 16 == 0 && K >= 1 && K <= 4096 && logT >= 4 &&
                   logT <= 7 && kbase + ((K + 63) & ~63u) <= kt_pad,
               CKKS_EINVAL, "matrix-core multiply-accumulate: unsupported tile (jc %u, kappa base %u, K %u, T %u)",
               jc, kbase, K, 1u << logT);
    const double res = (double)jc * 2 * L * ctx->n;
    // the digits of the K ciphertexts once per launch, the tables once, the accumulators
    prof_begin(ctx, K_MAC_TM, (double)kDig * K * 2 * L * ctx->n + 8.0 * (double)K * jc * L * D2 +
                                  8.0 * res * (accumulate ? 2 : 1),
               0.0);
#define CK_MFMA(NWV, MTV)                                                                                          \
    hipLaunchKernelGGL((k_mac_tm_mfma<NWV, MTV>), dim3(L * D2 * 2 * (tiles16 / NWV)), dim3(64 * NWV), 0,           \
                       ctx->stream, acc, Xd, Q, jc, K, kbase, kt_pad, D2, L, logT, ctx->log_n, (int)accumulate,     \
                       ctx->d_mod)
    switch (tiles16) {
    case 1: CK_MFMA(1, 2); break;
    case 2: CK_MFMA(2, 2); break;
    case 4: CK_MFMA(4, 2); break;
    default: CK_MFMA(8, 2); break;
    }
#undef CK_MFMA
    prof_end(ctx, K_MAC_TM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_enc_vectors(ckks_ctx *ctx, const double *U, uint32_t D, uint32_t count, double delta, uint32_t L,
                               double *Q)
{
    CK_REQUIRE(D >= 4 && D <= (uint32_t)kMaxD && (D & (D - 1)) == 0 && 2 * D <= ctx->n && count >= 1, CKKS_EINVAL,
               "periodic encode: period %u outside [4, %d] or not a power of two", D, kMaxD);
    TmArgs a{};
    a.U = U;
    a.D = D;
    while ((1u << a.logD) < D) a.logD++;
    a.jc = 1;
    a.bcount = 1;
    a.npt = count;
    return launch_enc_periodic(ctx, a, delta, L, Q);
}

size_t proj_tm_workspace_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t tokens, uint32_t d_in, uint32_t d_out,
                               uint32_t n1)
{
    uint32_t D;
    if (tm_check_shape(ctx, L, tokens, d_in, d_out, n1, &D) != CKKS_OK) {
        clear_error();
        return SIZE_MAX;
    }
    return tm_scratch(ctx, L, D, d_in, d_out, n1).total * 8;
}

extern "C" ckks_status ckks_linear_project_tm(ckks_ctx *ctx, const ckks_buf *in, const double *W,
                                              const ckks_proj_shape *shape, const int32_t *key_steps,
                                              const uint64_t *const *keys, uint32_t n_keys, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx && in && W && shape && out, CKKS_EINVAL, "linear_project_tm: null argument");
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "linear_project_tm: the context has no special primes");
    const uint32_t T = shape->tokens, n1 = shape->n1;
    const uint32_t L = in[0].n_limbs, level = L - 1;
    uint32_t D;
    CK_TRY(tm_check_shape(ctx, L, T, shape->d_in, shape->d_out, n1, &D));
    const uint32_t n_in = shape->d_in / D, n_out = shape->d_out / D, n2 = (D + n1 - 1) / n1;
    for (uint32_t i = 0; i < n_in; i++) {
        CK_REQUIRE(in[i].data && in[i].n_polys == 2, CKKS_EINVAL, "linear_project_tm: input %u is not a ciphertext",
                   i);
        CK_REQUIRE(in[i].n_limbs == L, CKKS_ELEVEL, "linear_project_tm: input %u has %u limbs, expected %u", i,
                   in[i].n_limbs, L);
        CK_REQUIRE(in[i].scale == in[0].scale, CKKS_ESCALE, "linear_project_tm: input scales differ");
    }
    for (uint32_t j = 0; j < n_out; j++)
        CK_REQUIRE(out[j].data && out[j].n_polys == 2 && out[j].n_limbs == level, CKKS_EINVAL,
                   "linear_project_tm: output %u must be a ciphertext with %u limbs", j, level);
    auto find_key = [&](int32_t st) -> const uint64_t * {
        for (uint32_t r = 0; r < n_keys; r++)
            if (key_steps[r] == st) return keys[r];
        return nullptr;
    };
    // baby steps b (0 < b < n1) then the wrapped ones b - D (0 <= b < n1), all hoisted from one ModUp
    std::vector<int32_t> bsteps;
    std::vector<const uint64_t *> bkeys;
    for (uint32_t b = 1; b < n1; b++) bsteps.push_back((int32_t)b);
    for (uint32_t b = 0; b < n1; b++) bsteps.push_back((int32_t)b - (int32_t)D);
    for (int32_t st : bsteps) {
        const uint64_t *k = find_key(st);
        CK_REQUIRE(k, CKKS_ENOKEY, "linear_project_tm: no key for step %d", st);
        bkeys.push_back(k);
    }
    std::vector<const uint64_t *> gkeys(n2, nullptr);
    for (uint32_t g = 1; g < n2; g++) {
        gkeys[g] = find_key((int32_t)(n1 * g));
        CK_REQUIRE(gkeys[g], CKKS_ENOKEY, "linear_project_tm: no key for giant step %u", n1 * g);
    }

    const size_t N = ctx->n, ctw = 2 * (size_t)L * N;
    const TmScratch ts = tm_scratch(ctx, L, D, shape->d_in, shape->d_out, n1);
    void *w;
    CK_TRY(ctx_scratch(ctx, ts.total * 8, &w));
    uint64_t *x2 = (uint64_t *)w;  // [n_in][n1][xr, xw][2][L][N]
    uint64_t *acc = x2 + ts.x2_w;
    uint64_t *tot = acc + ts.acc_w;
    uint64_t *rot = tot + ts.tot_w;
    double *Q = (double *)(rot + ts.rot_w);
    uint64_t *ksw = (uint64_t *)(Q + ts.q_w);
    double *Wd = (double *)(ksw + ts.ks_w);
    int8_t *Xd = (int8_t *)(Wd + ts.wd_w);
    uint64_t *uacc = (uint64_t *)(Wd + ts.wd_w) + ts.xd_w;  // [Jt][2][L + K][N] when the ModDown is lazy
    const bool lazy = ctx->lazy_moddown;
    CK_TRY(launch_diag_layout(ctx, Wd, W, D, n_in, shape->d_out));

    // 1. Rot_b(x_i) and Rot_{b-D}(x_i), hoisted per input
    for (uint32_t i = 0; i < n_in; i++) {
        uint64_t *xi = x2 + (size_t)i * n1 * 2 * ctw;
        HIP_TRY(hipMemcpyAsync(xi, in[i].data, ctw * 8, hipMemcpyDeviceToDevice, ctx->stream));
        std::vector<uint64_t *> outs;
        for (uint32_t b = 1; b < n1; b++) outs.push_back(xi + (size_t)b * 2 * ctw);
        for (uint32_t b = 0; b < n1; b++) outs.push_back(xi + ((size_t)b * 2 + 1) * ctw);
        CK_TRY(rotate_core(ctx, in[i].data, level, bsteps.data(), bkeys.data(), (uint32_t)bsteps.size(),
                           outs.data(), ksw));
    }
    if (ts.mfma)
        CK_TRY(launch_xdigits(ctx, x2, Xd, L, ts.kt, ts.kt_pad));
    else
        CK_TRY(launch_to_f64(ctx, x2, ts.x2_w));

    // 2./3. tiles of output ciphertexts, giant steps, sub-batches of pairs
    const double delta_w = (double)ctx->primes[level];
    uint32_t logT = 0;
    while ((1u << logT) < T) logT++;
    uint32_t logD = 0;
    while ((1u << logD) < D) logD++;
    for (uint32_t j0 = 0; j0 < n_out; j0 += ts.Jt) {
        const uint32_t jc = std::min(ts.Jt, n_out - j0);
        for (uint32_t g = 0; g < n2; g++) {
            const uint32_t bcount = std::min(n1, D - n1 * g);
            const uint32_t pairs = n_in * bcount;
            const uint32_t nsub = (pairs + ts.Pb - 1) / ts.Pb;
            for (uint32_t sb = 0, pb0 = 0; sb < nsub; sb++) {
                // sub-batches of Pb pairs (a multiple of 8), the last one shorter
                TmArgs a{};
                a.Wd = Wd;
                a.D = D;
                a.logD = logD;
                a.n_in = n_in;
                a.n1g = n1 * g;
                a.bcount = bcount;
                a.j0 = j0;
                a.jc = jc;
                a.pb0 = pb0;
                a.P = std::min(ts.Pb, pairs - pb0);
                a.npt = a.P * 2 * jc;
                CK_TRY(launch_enc_periodic(ctx, a, delta_w, L, Q));
                if (ts.mfma)
                    CK_TRY(launch_mac_tm_mfma(ctx, acc, Xd, Q, a, ts.kt_pad, L, logT, pb0 > 0));
                else
                    CK_TRY(launch_mac_tm(ctx, acc, (const double *)x2, Q, a, n1, L, logT, pb0 > 0));
                pb0 += a.P;
            }
            if (g == 0) {
                HIP_TRY(hipMemcpyAsync(tot, acc, jc * ctw * 8, hipMemcpyDeviceToDevice, ctx->stream));
            } else if (lazy) {
                CK_TRY(rotate_many_lazy(ctx, acc, ctw, jc, level, (int32_t)(n1 * g), gkeys[g], uacc, g > 1, ksw));
            } else {
                std::vector<uint64_t *> outs(jc);
                for (uint32_t jj = 0; jj < jc; jj++) outs[jj] = rot + (size_t)jj * ctw;
                CK_TRY(rotate_many(ctx, acc, ctw, jc, level, (int32_t)(n1 * g), gkeys[g], outs.data(), ksw));
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
