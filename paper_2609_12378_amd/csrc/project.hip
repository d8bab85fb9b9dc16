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
//  2. for a tile of J = 8 output blocks and one giant step g, the weight
//     plaintexts of a sub-batch of (i, b) pairs are encoded on the fly from W
//     (slot generation fused into the fp64 FFT -> round -> NTT column pass with
//     the RNS reduction fused in -> NTT row pass) and consumed by the
//     multiply-accumulate kernel, which loads each xrot residue once for all J
//     output blocks and accumulates exactly in 128 bits;
//  3. giant-step rotation of each partial sum at level l, summation, rescale.
// The plaintext scale is q_l, so the rescale returns the input scale exactly.
#include <algorithm>
#include <cstring>
#include <vector>

#include "ckks_internal.h"
#include "ops.h"

ckks_status rotate_core(ckks_ctx *ctx, const uint64_t *c, uint32_t level, const int32_t *steps,
                        const uint64_t *const *keys, uint32_t count, uint64_t *const *outs, uint64_t *work);
ckks_status rescale_core(ckks_ctx *ctx, const uint64_t *c, uint32_t l, uint64_t *out, uint64_t *work);

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

constexpr uint32_t kJ = 8;  // output blocks per tile

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

}  // namespace

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
    const uint32_t maxpairs = n_in * n1;
    // plaintext sub-batch of at most 2 GiB: J output blocks x Pb (i, b) pairs
    const size_t budget = size_t(1) << 31;
    const uint32_t Jt = kJ;
    const uint32_t Pb = std::min<uint32_t>(maxpairs, std::max<uint32_t>(1, (uint32_t)(budget / ((size_t)Jt * L * N * 8))));
    const size_t xrot_w = (size_t)n_in * n1 * ctw;
    const size_t acc_w = (size_t)kJ * ctw, tot_w = (size_t)kJ * ctw, rot_w = ctw;
    const size_t pt_w = (size_t)Jt * Pb * L * N;
    const size_t m_w = (size_t)Jt * Pb * N;                       // int64 coefficients
    const size_t fft_w = (size_t)Jt * Pb * (N / 2) * 2;            // double2 per slot
    const size_t ks_w = ks_scratch_words(ctx, level, ks_rot_batch(n1 > 1 ? n1 - 1 : 1));
    const size_t total = xrot_w + acc_w + tot_w + rot_w + pt_w + m_w + fft_w + ks_w;
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

    // ---- 2./3. tiles of output blocks
    const double delta_w = (double)ctx->primes[level];
    for (uint32_t j0 = 0; j0 < n_out; j0 += Jt) {
        const uint32_t jc = std::min<uint32_t>(Jt, n_out - j0);
        for (uint32_t g = 0; g < n2; g++) {
            const uint32_t bcount = std::min<uint32_t>(n1, D - n1 * g);
            const uint32_t pairs = n_in * bcount;
            for (uint32_t pb0 = 0; pb0 < pairs; pb0 += Pb) {
                const uint32_t P = std::min<uint32_t>(Pb, pairs - pb0);
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
                const uint32_t batch = jc * P;
                CK_TRY(enc_coeffs(ctx, src, batch, delta_w, fft, mint));
                CK_TRY(launch_ntt_from_i64(ctx, mint, pts, batch, L));
                CK_TRY(launch_mac(ctx, acc, pts, xrot, P, jc, pb0, bcount, n1, L, pb0 > 0));
            }
            for (uint32_t jj = 0; jj < jc; jj++) {
                uint64_t *a = acc + (size_t)jj * ctw, *t = tot + (size_t)jj * ctw;
                if (g == 0) {
                    HIP_TRY(hipMemcpyAsync(t, a, ctw * 8, hipMemcpyDeviceToDevice, ctx->stream));
                } else {
                    const int32_t st = (int32_t)(T * n1 * g);
                    const uint64_t *k = gkeys[g];
                    uint64_t *o = rot;
                    CK_TRY(rotate_core(ctx, a, level, &st, &k, 1, &o, ksw));
                    CK_TRY(launch_binary(ctx, t, t, rot, 2 * L, limb_range(0, L), EW_ADD));
                }
            }
        }
        for (uint32_t jj = 0; jj < jc; jj++) {
            CK_TRY(rescale_core(ctx, tot + (size_t)jj * ctw, level, out[j0 + jj].data, rot));
            out[j0 + jj].scale = in[0].scale;
        }
    }
    return CKKS_OK;
}
