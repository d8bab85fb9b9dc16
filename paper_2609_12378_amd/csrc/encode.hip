// CKKS encoding through the canonical embedding (Cheon-Kim-Kim-Song 2017),
// batched over many slot vectors.
//
// The integer coefficients of Encode_Delta(z) are
//   m_i = round(Delta * (2/N) * Re sum_{j<N/2} z_j zeta^(-i 5^j)),  zeta = e^(i pi/N).
// With M = N/2 the exponents 5^j mod 2N are exactly the residues 1 mod 4, so
// writing 5^j = 4s + 1 turns the sum into v_k = zeta^-k * Y_k, where Y is the
// length-M DFT with omega^(-k s) (omega = e^(2 pi i/M)) of y_s = z_j; then
// m_k = round(c Re v_k), m_{k+M} = round(c Im v_k), c = Delta * 2/N.
//
// Rounding near a half-integer depends on every bit of the fp64 result, so the
// evaluation order is fixed: a radix-2 decimation-in-time FFT from bit-reversed
// input, stages len = 2, 4, ..., M, butterfly t = w * a[hi], a[hi] = a[lo] - t,
// a[lo] = a[lo] + t with w = omega^(-k M/len), complex products formed as
// (ar*br - ai*bi, ar*bi + ai*br) without fused multiply-add, twiddles taken from
// host tables (cos, -sin) of the angles 2 pi e / M and pi k / N.  The schedule
// below (which butterflies run on which thread, in which pass) is free; each
// butterfly's arithmetic is not.
//
// MI355X mapping: pass A runs the first log2(BA) stages on contiguous blocks of
// BA = min(M, 2048) points in LDS; pass B runs the remaining <= 4 stages with
// each thread holding one column of M/BA points in registers, and fuses the
// twist, scaling and rounding.  Slot vectors of the projection are generated
// inside the gather kernel from W's cyclic diagonals, so they never exist in
// memory.
#pragma clang fp contract(off)
#include "ckks_internal.h"
#include "ntt_core.h"
#include "ops.h"

namespace {

constexpr int kThreads = 256;
constexpr int kLogBA = 11;  // pass-A block: 2048 complex = 32 KiB of LDS

__device__ __forceinline__ double2 cmul(double2 a, double2 b)
{
    const double p1 = a.x * b.x, p2 = a.y * b.y, p3 = a.x * b.y, p4 = a.y * b.x;
    return make_double2(p1 - p2, p3 + p4);
}

// slot value j of plaintext p of the batch
__device__ __forceinline__ double2 slot_value(const SlotSource &s, uint32_t p, uint32_t j, uint32_t M)
{
    if (s.W == nullptr) {
        const double re = s.re[(size_t)p * M + j];
        const double im = s.im ? s.im[(size_t)p * M + j] : 0.0;
        return make_double2(re, im);
    }
    // feature-major slot j = f*T + t holds D_{n1 g + b}(A_{jb,i})[(f - n1 g) mod D] with
    // A = W^T, A_{jb,i}[o][c] = W[i D + c][jb D + o], D_k(A)[o] = A[o][(o + k) mod D]
    const uint32_t D = s.feats;
    const uint32_t jb = s.j0 + p / s.pairs;
    const uint32_t pair = s.ib0 + p % s.pairs;
    const uint32_t i = pair / s.bcount, b = pair % s.bcount;
    const uint32_t f = j / s.tokens;
    const uint32_t o = (f + D - s.n1g % D) % D;
    const uint32_t c = (o + s.n1g + b) % D;
    return make_double2(s.W[(size_t)(i * D + c) * s.d_out + (size_t)jb * D + o], 0.0);
}

__device__ __forceinline__ void round_out(int64_t *m, size_t base, uint32_t k, uint32_t M, double2 y, double2 tw,
                                          double c)
{
    const double2 v = cmul(tw, y);
    m[base + k] = (int64_t)round(c * v.x);
    m[base + k + M] = (int64_t)round(c * v.y);
}

// Pass A: stages len = 2 .. 2^logb on contiguous blocks of 2^logb points.
// Input: from `a` (bit-reversed order), or, when `gather` is set, straight from
// the slot source through slot_of_pos (FFT position -> slot index).
// mode 0: write complex back; mode 1: final pass, twist/round into m.
__global__ __launch_bounds__(kThreads) void k_fft_a(double2 *a, const double2 *__restrict__ w, uint32_t logm,
                                                     uint32_t logb, int mode, const double2 *__restrict__ twist,
                                                     double c, int64_t *m, int gather, SlotSource ss,
                                                     const uint32_t *__restrict__ slot_of_pos)
{
    extern __shared__ double2 sh[];
    const uint32_t M = 1u << logm, B = 1u << logb;
    const uint32_t blocks_per = M >> logb;
    const uint32_t p = blockIdx.x / blocks_per, blk = blockIdx.x % blocks_per;
    double2 *src = a + (size_t)p * M + (size_t)blk * B;
    if (gather) {
        for (uint32_t x = threadIdx.x; x < B; x += kThreads)
            sh[x] = slot_value(ss, p, slot_of_pos[(size_t)blk * B + x], M);
    } else {
        for (uint32_t x = threadIdx.x; x < B; x += kThreads) sh[x] = src[x];
    }
    __syncthreads();
    for (uint32_t ls = 1; ls <= logb; ls++) {
        const uint32_t half = 1u << (ls - 1);
        const uint32_t step = M >> ls;  // twiddle exponent multiplier M/len
        for (uint32_t bf = threadIdx.x; bf < B / 2; bf += kThreads) {
            const uint32_t k = bf & (half - 1);
            const uint32_t lo = ((bf >> (ls - 1)) << ls) + k, hi = lo + half;
            const double2 t = cmul(w[k * step], sh[hi]);
            const double2 u = sh[lo];
            sh[lo] = make_double2(u.x + t.x, u.y + t.y);
            sh[hi] = make_double2(u.x - t.x, u.y - t.y);
        }
        __syncthreads();
    }
    if (mode == 0) {
        for (uint32_t x = threadIdx.x; x < B; x += kThreads) src[x] = sh[x];
    } else {
        for (uint32_t x = threadIdx.x; x < B; x += kThreads) round_out(m, (size_t)p * 2 * M, x, M, sh[x], twist[x], c);
    }
}

// Pass A for 2048-point blocks from the projection's diagonal layout, with the
// butterflies three stages at a time in registers: 256 threads hold 8 points
// each, in four layouts whose register bits are the position bits of the
// stages they run (L1: bits 0-2, stages 1-3; L2: bits 3-5; L3: bits 6-8; L4:
// bits 9, 10 and 0, stages 10-11); three LDS transposes with XOR swizzles
// (conflict-free for all six access patterns) connect them.  Each butterfly is
// the same arithmetic as in k_fft_a, so the results are identical.  The
// plaintext's D weights are read once (one contiguous diagonal of Wd) into LDS
// and spread over the block's positions through feat_of_pos.
template <int LAY>
__device__ __forceinline__ uint32_t posA(uint32_t t, int r)
{
    if (LAY == 1) return (t << 3) | (uint32_t)r;
    if (LAY == 2) return ((t >> 3) << 6) | ((uint32_t)r << 3) | (t & 7u);
    if (LAY == 3) return ((t >> 6) << 9) | ((uint32_t)r << 6) | (t & 63u);
    return ((uint32_t)(r >> 1) << 9) | (t << 1) | (uint32_t)(r & 1);
}
__device__ __forceinline__ uint32_t swz_a(uint32_t x) { return x ^ ((x >> 3) & 15u); }
__device__ __forceinline__ uint32_t swz_b(uint32_t x) { return x ^ ((x >> 1) & 15u); }

// wc: the stage-by-stage twiddle table, wc[2^(LS-1) + k] = w[k * M / 2^LS] (32 KiB, cache-resident)
template <int LAY, int LS>
__device__ __forceinline__ void fft8_stage(double2 (&v)[8], const double2 *__restrict__ wc, uint32_t t)
{
    constexpr uint32_t half = 1u << (LS - 1);
    constexpr int xb = LS - 1;
    constexpr int rb = LAY == 1 ? xb : LAY == 2 ? xb - 3 : LAY == 3 ? xb - 6 : xb - 8;
    static_assert(rb >= 0 && rb < 3 && (LAY != 4 || xb >= 9), "stage not in this layout");
#pragma unroll
    for (int r = 0; r < 8; r++) {
        if (r & (1 << rb)) continue;
        const uint32_t k = posA<LAY>(t, r) & (half - 1);
        const double2 tt = cmul(wc[half + k], v[r | (1 << rb)]);
        const double2 u = v[r];
        v[r] = make_double2(u.x + tt.x, u.y + tt.y);
        v[r | (1 << rb)] = make_double2(u.x - tt.x, u.y - tt.y);
    }
}

template <int LA, int LB, bool SWB>
__device__ __forceinline__ void fft8_transpose(double2 (&v)[8], double2 *sh, uint32_t t)
{
#pragma unroll
    for (int r = 0; r < 8; r++) {
        const uint32_t x = posA<LA>(t, r);
        sh[SWB ? swz_b(x) : swz_a(x)] = v[r];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 8; r++) {
        const uint32_t x = posA<LB>(t, r);
        v[r] = sh[SWB ? swz_b(x) : swz_a(x)];
    }
    __syncthreads();
}

__global__ __launch_bounds__(256) void k_fft_a8(double2 *a, const double2 *__restrict__ wc, uint32_t logm, int mode,
                                                const double2 *__restrict__ twist, double c, int64_t *m,
                                                SlotSource ss)
{
    __shared__ double2 sh[2048];
    __shared__ double vals[256];
    const uint32_t M = 1u << logm, blocks_per = M >> 11;
    const uint32_t p = blockIdx.x / blocks_per, blk = blockIdx.x % blocks_per, t = threadIdx.x;
    const uint32_t D = ss.feats;
    const uint32_t jb = ss.j0 + p / ss.pairs, pair = ss.ib0 + p % ss.pairs;
    const uint32_t i = pair / ss.bcount, b = pair % ss.bcount;
    const double *dg = ss.Wd + (((size_t)jb * ss.n_in + i) * D + ss.n1g + b) * D;
    for (uint32_t o = t; o < D; o += 256) vals[o] = dg[o];
    __syncthreads();
    // slot f*T + t' holds diagonal entry (f - n1 g) mod D
    const uint32_t shift = D - ss.n1g % D, mask = D - 1;
    const uint32_t *fp = ss.feat_of_pos + ((size_t)blk << 11);
    double2 v[8];
#pragma unroll
    for (int r = 0; r < 8; r++) v[r] = make_double2(vals[(fp[posA<1>(t, r)] + shift) & mask], 0.0);
    fft8_stage<1, 1>(v, wc, t);
    fft8_stage<1, 2>(v, wc, t);
    fft8_stage<1, 3>(v, wc, t);
    fft8_transpose<1, 2, false>(v, sh, t);
    fft8_stage<2, 4>(v, wc, t);
    fft8_stage<2, 5>(v, wc, t);
    fft8_stage<2, 6>(v, wc, t);
    fft8_transpose<2, 3, false>(v, sh, t);
    fft8_stage<3, 7>(v, wc, t);
    fft8_stage<3, 8>(v, wc, t);
    fft8_stage<3, 9>(v, wc, t);
    fft8_transpose<3, 4, true>(v, sh, t);
    fft8_stage<4, 10>(v, wc, t);
    fft8_stage<4, 11>(v, wc, t);
    if (mode == 0) {
        double2 *dst = a + (size_t)p * M + ((size_t)blk << 11);
#pragma unroll
        for (int r = 0; r < 8; r++) dst[posA<4>(t, r)] = v[r];
    } else {
#pragma unroll
        for (int r = 0; r < 8; r++) {
            const uint32_t x = posA<4>(t, r);
            round_out(m, (size_t)p * 2 * M, x, M, v[r], twist[x], c);
        }
    }
}

// FFT pass B fused with the first NTT pass (N = 2^16: M = 32768 = 16 x 2048, transform columns of 256 points).
// Block (plaintext b, columns c0..c0+15 of the 256 x 256 coefficient matrix, coefficient n = 256 u + c) needs
// pass-B outputs v_k, k = 256 u' + c (u' < 128; m_n = round(c Re v_n) for n < M and m_{n+M} = round(c Im v_n)),
// i.e. pass-B columns c' = k mod 2048 = 256 (u' mod 8) + c at depths h = u' / 8.  Its 512 threads compute those
// 128 pass-B columns (four threads per column, two stages in registers, an LDS exchange, two more), round into an
// int64 tile in LDS, and run the 8-residue column transform of every limb from that tile (as ntt_col8_from_i64).
// The pass-B butterflies, twist and rounding are the same arithmetic as in k_fft_b, so the coefficients are the
// same integers, and they never go to HBM.
__global__ __launch_bounds__(512) void ntt_col8_from_fft(const double2 *__restrict__ work, uint64_t *out,
                                                         uint32_t limbs, const ModQ *__restrict__ mods,
                                                         const double *__restrict__ twf,
                                                         const double2 *__restrict__ fw,
                                                         const double2 *__restrict__ twist, double cs,
                                                         int64_t small)
{
    using nttc::kE8;
    constexpr uint32_t log_n = 16, M = 1u << 15, MT_PITCH = 17;
    __shared__ double tws[2][256];
    __shared__ double tr[16][nttc::kTr8];  // also the pass-B exchange buffer (2048 double2 with padding)
    __shared__ int64_t mt[256 * MT_PITCH];
    const uint32_t b = blockIdx.x >> 4, c0 = (blockIdx.x & 15u) << 4, tid = threadIdx.x;
    // ---- pass B for columns c' = 256 w8 + c0 + cc, ci = 16 w8 + cc, depths h = 4 qq + j
    {
        const uint32_t ci = tid >> 2, qq = tid & 3u, cc = ci & 15u, w8 = ci >> 4;
        const uint32_t cp = (w8 << 8) + c0 + cc;
        const double2 *src = work + ((size_t)b << 15);
        double2 x[4];
#pragma unroll
        for (int j = 0; j < 4; j++) x[j] = src[((4 * qq + j) << 11) + cp];
        // stages 1, 2 (pairs h, h + 1 and h, h + 2: h's low bits are j's)
#pragma unroll
        for (int st = 1; st <= 2; st++) {
            const uint32_t half = 1u << (st - 1), step = M >> (11 + st);
#pragma unroll
            for (int j = 0; j < 4; j++) {
                if (j & half) continue;
                const uint32_t h = 4 * qq + j;
                const uint32_t k = (h & (half - 1)) * 2048 + cp;
                const double2 t = cmul(fw[k * step], x[j + half]);
                const double2 u = x[j];
                x[j] = make_double2(u.x + t.x, u.y + t.y);
                x[j + half] = make_double2(u.x - t.x, u.y - t.y);
            }
        }
        double2 *ex = (double2 *)&tr[0][0];  // [16 depths][128 columns + 1]
#pragma unroll
        for (int j = 0; j < 4; j++) ex[(4 * qq + j) * 129 + ci] = x[j];
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 4; j++) x[j] = ex[(qq + 4 * j) * 129 + ci];
        // stages 3, 4: now h = qq + 4 j, so h's bits 2, 3 are j's
#pragma unroll
        for (int st = 3; st <= 4; st++) {
            const uint32_t half = 1u << (st - 1), jh = half >> 2, step = M >> (11 + st);
#pragma unroll
            for (int j = 0; j < 4; j++) {
                if (j & jh) continue;
                const uint32_t h = qq + 4 * j;
                const uint32_t k = (h & (half - 1)) * 2048 + cp;
                const double2 t = cmul(fw[k * step], x[j + jh]);
                const double2 u = x[j];
                x[j] = make_double2(u.x + t.x, u.y + t.y);
                x[j + jh] = make_double2(u.x - t.x, u.y - t.y);
            }
        }
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const uint32_t h = qq + 4 * j, k = (h << 11) + cp, u = (h << 3) + w8;
            const double2 v = cmul(twist[k], x[j]);
            mt[u * MT_PITCH + cc] = (int64_t)round(cs * v.x);
            mt[(u + 128) * MT_PITCH + cc] = (int64_t)round(cs * v.y);
        }
    }
    if (tid < 255) tws[0][tid + 1] = twf[tid + 1];
    __syncthreads();
    // ---- column transforms (as ntt_col8_from_i64, coefficients from the tile)
    const uint32_t col = tid & 15u, t = tid >> 4;
    const size_t coff = c0 + col;
    double vd[kE8];
    bool big = false, wide = false;
#pragma unroll
    for (int k = 0; k < kE8; k++) {
        const int64_t v = mt[nttc::u8<0>(t, k) * MT_PITCH + col];
        big |= v > (1ll << 52) || v < -(1ll << 52);
        wide |= v > small || v < -small;
        vd[k] = (double)v;
    }
    // every coefficient of the wave below every limb's q/2 (weights at the usual scales): its range reduction is
    // the identity, so the wave skips it for all limbs
    const bool reduce = __any(wide);
    for (uint32_t l = 0; l < limbs; l++) {
        const ModQ md = mods[l];
        const nttc::Ar<true> ar(md);
        double wnext = 0.0;
        if (l + 1 < limbs && tid < 255) wnext = twf[((size_t)(l + 1) << log_n) + tid + 1];
        double x[kE8];
        if (!reduce) {
#pragma unroll
            for (int k = 0; k < kE8; k++) x[k] = vd[k];
        } else if (!big) {
#pragma unroll
            for (int k = 0; k < kE8; k++) x[k] = ar.red(vd[k]);
        } else {
#pragma unroll
            for (int k = 0; k < kE8; k++) x[k] = ar.from_i64(mt[nttc::u8<0>(t, k) * MT_PITCH + col], md);
        }
        const double *tw = tws[l & 1];
        double *trc = tr[col];
        nttc::fwd8_stage<0, 0, (nttc::kColMask8 >> 0) & 1>(x, tw, t, ar);
        nttc::fwd8_stage<0, 1, (nttc::kColMask8 >> 1) & 1>(x, tw, t, ar);
        nttc::fwd8_stage<0, 2, (nttc::kColMask8 >> 2) & 1>(x, tw, t, ar);
#pragma unroll
        for (int k = 0; k < kE8; k++) trc[nttc::pad_ac(nttc::u8<0>(t, k))] = x[k];
        __syncthreads();
        if (l + 1 < limbs && tid < 255) tws[(l + 1) & 1][tid + 1] = wnext;
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
        for (int k = 0; k < kE8; k++) nttc::st_stream(dst + (size_t)nttc::u8<2>(t, k) * 256, nttc::Ar<true>::to_raw(x[k]));
    }
}

// feat_of_pos[x] = slot index at FFT position x, divided by the token count
__global__ __launch_bounds__(kThreads) void k_feat_of_pos(uint32_t *out, const uint32_t *__restrict__ slot_of_pos,
                                                          uint32_t M, uint32_t tokens)
{
    const uint32_t x = blockIdx.x * kThreads + threadIdx.x;
    if (x < M) out[x] = slot_of_pos[x] / tokens;
}

// Pass B: stages len = 2^(logb+1) .. M; thread owns column c (points h*B + c, h < 2^HB).
template <int HB>
__global__ __launch_bounds__(kThreads) void k_fft_b(double2 *a, const double2 *__restrict__ w, uint32_t logm,
                                                     uint32_t logb, int mode, const double2 *__restrict__ twist,
                                                     double c, int64_t *m)
{
    const uint32_t M = 1u << logm, B = 1u << logb;
    const uint32_t cols_blocks = B / kThreads;
    const uint32_t p = blockIdx.x / cols_blocks;
    const uint32_t col = (blockIdx.x % cols_blocks) * kThreads + threadIdx.x;
    double2 *src = a + (size_t)p * M;
    double2 x[1 << HB];
#pragma unroll
    for (int h = 0; h < (1 << HB); h++) x[h] = src[(size_t)h * B + col];
#pragma unroll
    for (int s = 1; s <= HB; s++) {
        const int half = 1 << (s - 1);
        const uint32_t step = M >> (logb + s);  // M / len
#pragma unroll
        for (int h = 0; h < (1 << HB); h++) {
            if (h & half) continue;
            const uint32_t k = (uint32_t)(h & (half - 1)) * B + col;  // position inside the len-block
            const double2 t = cmul(w[k * step], x[h + half]);
            const double2 u = x[h];
            x[h] = make_double2(u.x + t.x, u.y + t.y);
            x[h + half] = make_double2(u.x - t.x, u.y - t.y);
        }
    }
    if (mode == 0) {
#pragma unroll
        for (int h = 0; h < (1 << HB); h++) src[(size_t)h * B + col] = x[h];
    } else {
#pragma unroll
        for (int h = 0; h < (1 << HB); h++) {
            const uint32_t k = (uint32_t)h * B + col;
            round_out(m, (size_t)p * 2 * M, k, M, x[h], twist[k], c);
        }
    }
}

// m (int64 [batch][N]) -> residues [batch][limbs][N]
__global__ __launch_bounds__(kThreads) void k_to_rns(uint64_t *out, const int64_t *m, uint32_t limbs, uint32_t log_n,
                                                      const ModQ *__restrict__ mods)
{
    const uint32_t n = 1u << log_n;
    const uint32_t col = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t p = blockIdx.y;
    if (col >= n) return;
    const int64_t v = m[((size_t)p << log_n) + col];
    const bool neg = v < 0;
    const uint64_t mag = neg ? (uint64_t)(-(v + 1)) + 1u : (uint64_t)v;
    for (uint32_t l = 0; l < limbs; l++) {
        const ModQ md = mods[l];
        uint64_t r = csub(mag - mulhi64(mag, md.one_s) * md.q, md.q);
        if (neg && r) r = md.q - r;
        out[(((size_t)p * limbs + l) << log_n) + col] = r;
    }
}

// Decode, step 1: centred CRT lift of limbs 0 (and 1) of the coefficient form,
// scaled by 1/Delta, twisted by zeta^-i and conjugated, into bit-reversed FFT
// order: the inverse-direction FFT of conj((m_i + i m_{i+M}) zeta^i) is the
// conjugate of the decoding sum.
__global__ __launch_bounds__(kThreads) void k_decode_in(double2 *a, const uint64_t *coef, uint32_t limbs,
                                                         uint32_t log_n, const ModQ *__restrict__ mods,
                                                         const double2 *__restrict__ twist, double inv_scale,
                                                         uint64_t q0inv, uint64_t q0inv_s)
{
    const uint32_t n = 1u << log_n, M = n / 2, logm = log_n - 1;
    const uint32_t i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= M) return;
    const uint64_t q0 = mods[0].q;
    double v[2];
    for (int h = 0; h < 2; h++) {
        const uint32_t idx = i + h * M;
        const uint64_t x0 = coef[idx];
        double val;
        if (limbs == 1) {
            val = x0 > q0 / 2 ? -(double)(q0 - x0) : (double)x0;
        } else {
            const uint64_t q1 = mods[1].q;
            const uint64_t x1 = coef[n + idx];
            const uint64_t d = shoup(submod(x1, csub(x0, q1), q1), q0inv, q0inv_s, q1);
            const unsigned __int128 Q = (unsigned __int128)q0 * q1;
            const unsigned __int128 x = (unsigned __int128)q0 * d + x0;  // in [0, q0 q1)
            const bool neg = x > Q / 2;
            const unsigned __int128 mag = neg ? Q - x : x;
            const double dv = (double)(uint64_t)(mag >> 64) * 18446744073709551616.0 + (double)(uint64_t)mag;
            val = neg ? -dv : dv;
        }
        v[h] = val * inv_scale;
    }
    a[__brev(i) >> (32 - logm)] = cmul(twist[i], make_double2(v[0], -v[1]));
}

// Decode, step 3: slot j = conj(Y[s(j)]), s(j) the natural index whose bit reversal is pos[j]
__global__ __launch_bounds__(kThreads) void k_decode_out(const double2 *y, const uint32_t *__restrict__ pos,
                                                          uint32_t logm, double *re, double *im)
{
    const uint32_t M = 1u << logm;
    const uint32_t j = blockIdx.x * kThreads + threadIdx.x;
    if (j >= M) return;
    const double2 v = y[__brev(pos[j]) >> (32 - logm)];
    re[j] = v.x;
    im[j] = -v.y;
}

}  // namespace

size_t enc_work_bytes(const ckks_ctx *ctx, uint32_t batch) { return (size_t)batch * (ctx->n / 2) * sizeof(double2); }

ckks_status fft_passes(ckks_ctx *ctx, double2 *work, uint32_t batch, int mode, double c, int64_t *m,
                       const SlotSource *gather, bool pass_a_only = false)
{
    const uint32_t logm = ctx->log_n - 1, M = 1u << logm;
    const uint32_t logb = logm < (uint32_t)kLogBA ? logm : (uint32_t)kLogBA;
    const uint32_t B = 1u << logb;
    const bool single = logb == logm;
    const double bytes = 32.0 * batch * M;  // read and write every complex point (or its two integers)
    // with the gather fused, pass A reads the D distinct weights of each plaintext (or the explicit slots)
    const double bytes_a = gather ? batch * (16.0 * M + (gather->W ? 8.0 * gather->feats
                                                                    : (gather->im ? 16.0 : 8.0) * M))
                                  : bytes;
    SlotSource none;
    prof_begin(ctx, K_FFT_A, bytes_a);
    if (gather && gather->Wd && logb == (uint32_t)kLogBA) {
        hipLaunchKernelGGL(k_fft_a8, dim3(batch * (M >> logb)), dim3(256), 0, ctx->stream, work, ctx->d_fft_wc, logm,
                           single ? mode : 0, ctx->d_fft_twist, c, m, *gather);
    } else {
        hipLaunchKernelGGL(k_fft_a, dim3(batch * (M >> logb)), dim3(kThreads), B * sizeof(double2), ctx->stream,
                           work, ctx->d_fft_w, logm, logb, single ? mode : 0, ctx->d_fft_twist, c, m, gather ? 1 : 0,
                           gather ? *gather : none, ctx->d_pos_slot);
    }
    prof_end(ctx, K_FFT_A);
    if (!single && !pass_a_only) {
        const uint32_t hb = logm - logb;
        const dim3 grid(batch * (B / kThreads));
        prof_begin(ctx, K_FFT_B, bytes);
        switch (hb) {
        case 1: hipLaunchKernelGGL(k_fft_b<1>, grid, dim3(kThreads), 0, ctx->stream, work, ctx->d_fft_w, logm, logb,
                                   mode, ctx->d_fft_twist, c, m); break;
        case 2: hipLaunchKernelGGL(k_fft_b<2>, grid, dim3(kThreads), 0, ctx->stream, work, ctx->d_fft_w, logm, logb,
                                   mode, ctx->d_fft_twist, c, m); break;
        case 3: hipLaunchKernelGGL(k_fft_b<3>, grid, dim3(kThreads), 0, ctx->stream, work, ctx->d_fft_w, logm, logb,
                                   mode, ctx->d_fft_twist, c, m); break;
        case 4: hipLaunchKernelGGL(k_fft_b<4>, grid, dim3(kThreads), 0, ctx->stream, work, ctx->d_fft_w, logm, logb,
                                   mode, ctx->d_fft_twist, c, m); break;
        default: prof_end(ctx, K_FFT_B); return set_error(CKKS_EUNSUPPORTED, "fft: unsupported size");
        }
        prof_end(ctx, K_FFT_B);
    }
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status enc_coeffs(ckks_ctx *ctx, const SlotSource &src, uint32_t batch, double scale, double2 *work,
                       int64_t *m_out)
{
    if (!batch) return CKKS_OK;
    return fft_passes(ctx, work, batch, 1, scale * (2.0 / (double)ctx->n), m_out, &src);
}

bool enc_fused_ok(const ckks_ctx *ctx, uint32_t limbs) { return ctx->log_n == 16 && ntt_uses_f64(ctx, limbs); }

ckks_status enc_ntt_first_pass(ckks_ctx *ctx, const SlotSource &src, uint32_t batch, double scale, double2 *work,
                               uint32_t limbs, uint64_t *out)
{
    if (!batch) return CKKS_OK;
    CK_REQUIRE(enc_fused_ok(ctx, limbs), CKKS_EINVAL, "encode: the fused first pass needs N = 2^16 and fp64 primes");
    const double c = scale * (2.0 / (double)ctx->n);
    CK_TRY(fft_passes(ctx, work, batch, 0, c, nullptr, &src, true));
    // pass B's work array once, the limbs' first-pass rows
    const double res = (double)batch * limbs * ctx->n;
    prof_begin(ctx, K_NTT_FWD_COL, batch * 8.0 * ctx->n * (1 + limbs),
               res * ((2 * kOpsButterflyF64 + 6 * (kOpsButterflyF64 - 3)) / 2 + 3.0));
    hipLaunchKernelGGL(ntt_col8_from_fft, dim3(batch * 16), dim3(512), 0, ctx->stream, work, out, limbs, ctx->d_mod,
                       ctx->d_twf, ctx->d_fft_w, ctx->d_fft_twist, c, identity_reduction_bound(ctx, limbs));
    prof_end(ctx, K_NTT_FWD_COL);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status enc_feat_of_pos(ckks_ctx *ctx, uint32_t tokens, uint32_t *out)
{
    const uint32_t M = ctx->n / 2;
    hipLaunchKernelGGL(k_feat_of_pos, dim3((M + kThreads - 1) / kThreads), dim3(kThreads), 0, ctx->stream, out,
                       ctx->d_pos_slot, M, tokens);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status enc_to_rns(ckks_ctx *ctx, const int64_t *m, uint32_t batch, uint32_t limbs, uint64_t *out)
{
    if (!batch) return CKKS_OK;
    prof_begin(ctx, K_TO_RNS, 8.0 * batch * ctx->n * (1 + limbs));
    hipLaunchKernelGGL(k_to_rns, dim3((ctx->n + kThreads - 1) / kThreads, batch), dim3(kThreads), 0, ctx->stream,
                       out, m, limbs, ctx->log_n, ctx->d_mod);
    prof_end(ctx, K_TO_RNS);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status dec_slots(ckks_ctx *ctx, const uint64_t *coef, uint32_t limbs, double scale, double2 *work, double *re,
                      double *im)
{
    const uint32_t M = ctx->n / 2;
    uint64_t q0inv = 0, q0inv_s = 0;
    if (limbs > 1) {
        const unsigned __int128 q1 = ctx->primes[1];
        // q0^-1 mod q1 by Fermat
        uint64_t b = ctx->primes[0] % ctx->primes[1], e = ctx->primes[1] - 2, r = 1;
        while (e) {
            if (e & 1) r = (uint64_t)((unsigned __int128)r * b % q1);
            b = (uint64_t)((unsigned __int128)b * b % q1);
            e >>= 1;
        }
        q0inv = r;
        q0inv_s = (uint64_t)(((unsigned __int128)r << 64) / q1);
    }
    const dim3 grid((M + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(k_decode_in, grid, dim3(kThreads), 0, ctx->stream, work, coef, limbs > 1 ? 2u : 1u,
                       ctx->log_n, ctx->d_mod, ctx->d_fft_twist, 1.0 / scale, q0inv, q0inv_s);
    HIP_TRY(hipGetLastError());
    CK_TRY(fft_passes(ctx, work, 1, 0, 0.0, nullptr, nullptr));
    hipLaunchKernelGGL(k_decode_out, grid, dim3(kThreads), 0, ctx->stream, work, ctx->d_slot_pos, ctx->log_n - 1, re,
                       im);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}
