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
//   P_delta = Rescale(Relin(Rot_{-delta}(Q) x Rot_{delta (D-1)}(K')))                       0 <= delta < T
//   out     = Rescale( sum_k Rot_k( U_k ) ),  U_k = sum_delta M_{(delta + k) mod hd} * P_delta    0 <= k < hd
// and slot t*D + h*hd + delta of out holds sum_d Q[t, h, d] K[(t + delta) mod T, d] (zero for delta >= T).
// The masks M_c (1 on head position c) are slot vectors of period D, so their plaintexts are constant on
// runs of T consecutive NTT positions; each U_k over all delta is a dense residue contraction per run —
// the token-major projection's matrix-core multiply-accumulate, with a mask table in place of the weights.
//
// Weighted sums.  Scores P in that layout, a value ciphertext V' with one value head in every position:
//   R_delta = Rot_{delta D}(V'),  C_j = Rescale( sum_delta M_{delta - j} * R_delta )   (0 <= delta - j < hd)
//   out     = Rescale(Relin( sum_j Rot_j(P) x C_j ))                                   -hd < j < T
// so that out[t*D + h*hd + d] = sum_delta P[t, h, delta] V[(t + delta) mod T, d].  The C_j depend only on the
// value ciphertext and are shared by every score ciphertext that uses it; the products are summed before
// the single relinearisation.
#include <algorithm>
#include <vector>

#include "ckks_internal.h"
#include "ops.h"

namespace {

constexpr int kThreads = 256;

// U[c][f] = 1 if f = c (mod hd), else 0; c < hd, f < D
__global__ __launch_bounds__(kThreads) void k_attn_masks(double *U, uint32_t D, uint32_t hd)
{
    const uint32_t i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= D * hd) return;
    const uint32_t c = i / D, f = i % D;
    U[i] = (f & (hd - 1)) == c ? 1.0 : 0.0;
}

// The multiply-accumulate table of one output tile: Qt[l][x][kappa][jj] = MQ[l][x][c] with
//   scores (wrap = 1): c = (kappa + o0 + jj) mod hd;
//   sums   (wrap = 0): c = kappa - (o0 + jj) if it lies in [0, hd), else the entry is 0.
// MQ: [L][D2][hd] (the mask plaintexts on each run), Qt: [L][D2][K][jc].
__global__ __launch_bounds__(kThreads) void k_attn_table(double *Qt, const double *__restrict__ MQ, uint32_t L,
                                                         uint32_t D2, uint32_t K, uint32_t jc, uint32_t hd, int o0,
                                                         int wrap)
{
    const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    const size_t total = (size_t)L * D2 * K * jc;
    if (i >= total) return;
    const uint32_t jj = (uint32_t)(i % jc);
    const uint32_t kappa = (uint32_t)((i / jc) % K);
    const size_t lx = i / ((size_t)jc * K);  // l * D2 + x
    double v = 0.0;
    if (wrap) {
        const uint32_t c = (uint32_t)((int)kappa + o0 + (int)jj) & (hd - 1);
        v = MQ[lx * hd + c];
    } else {
        const int c = (int)kappa - (o0 + (int)jj);
        if (c >= 0 && c < (int)hd) v = MQ[lx * hd + (uint32_t)c];
    }
    Qt[i] = v;
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
// bits and reduced once (count <= 2^16 keeps them below 2^128).  E_r at E + r * 2 L N ([2][L][N]); C_r at
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

inline dim3 grid_of(size_t total) { return dim3((unsigned)((total + kThreads - 1) / kThreads)); }

ckks_status launch_masks(ckks_ctx *ctx, double *U, double *MQ, uint32_t D, uint32_t hd, double delta, uint32_t L)
{
    hipLaunchKernelGGL(k_attn_masks, grid_of((size_t)D * hd), dim3(kThreads), 0, ctx->stream, U, D, hd);
    HIP_TRY(hipGetLastError());
    return launch_enc_vectors(ctx, U, D, hd, delta, L, MQ);
}

ckks_status launch_table(ckks_ctx *ctx, double *Qt, const double *MQ, uint32_t L, uint32_t D2, uint32_t K,
                         uint32_t jc, uint32_t hd, int o0, bool wrap)
{
    const size_t total = (size_t)L * D2 * K * jc;
    prof_begin(ctx, K_ELEM, 8.0 * total + 8.0 * (double)L * D2 * hd);
    hipLaunchKernelGGL(k_attn_table, grid_of(total), dim3(kThreads), 0, ctx->stream, Qt, MQ, L, D2, K, jc, hd, o0,
                       (int)wrap);
    prof_end(ctx, K_ELEM);
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
    prof_begin(ctx, K_ELEM, 8.0 * total * (4.0 * count + 3.0));
    hipLaunchKernelGGL(k_tensor_acc, grid_of(total), dim3(kThreads), 0, ctx->stream, d, E, C, count, L, Lc,
                       ctx->log_n, ctx->d_mod);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

// Shape checks shared by both calls: T tokens (a power of two in [16, 128]: the runs of the mask plaintexts
// are T positions long, the matrix-core tile's range), head dimension hd (a power of two, T <= hd <= D,
// dividing D), D <= 256 features (the periodic encode's limit).
ckks_status attn_check_shape(const ckks_ctx *ctx, const ckks_attn_shape *shape, const char *what, uint32_t *Dout,
                             uint32_t *logTout)
{
    CK_REQUIRE(shape, CKKS_EINVAL, "%s: null shape", what);
    const uint32_t T = shape->tokens, hd = shape->head_dim, slots = (uint32_t)(ctx->n / 2);
    CK_REQUIRE(T >= 16 && T <= 128 && (T & (T - 1)) == 0 && slots % T == 0, CKKS_EUNSUPPORTED,
               "%s: %u tokens (a power of two in [16, 128] dividing %u slots)", what, T, slots);
    const uint32_t D = slots / T;
    CK_REQUIRE(D <= 256, CKKS_EUNSUPPORTED, "%s: %u features per ciphertext (at most 256)", what, D);
    CK_REQUIRE(hd >= T && hd <= D && (hd & (hd - 1)) == 0, CKKS_EINVAL,
               "%s: head dimension %u (a power of two with %u <= hd <= %u)", what, hd, T, D);
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "%s: the context has no special primes", what);
    uint32_t logT = 0;
    while ((1u << logT) < T) logT++;
    *Dout = D;
    *logTout = logT;
    return CKKS_OK;
}

// Scratch of the scores call for inputs of L limbs (words)
struct ScoreScratch {
    uint32_t Jt, kt_pad;
    size_t u_w, mq_w, b_w, a_w, d_w, pr_w, xd_w, qt_w, acc_w, rot_w, tot_w, work_w, total;
};

ScoreScratch score_scratch(const ckks_ctx *ctx, uint32_t L, uint32_t D, uint32_t T, uint32_t hd)
{
    ScoreScratch s{};
    const size_t N = ctx->n, ctw = 2 * (size_t)L * N, ctw1 = 2 * (size_t)(L - 1) * N;
    const uint32_t level = L - 1;
    s.Jt = std::min(hd, mac_max_outputs());
    s.kt_pad = mac_kt_pad(T);
    s.u_w = (size_t)hd * D;
    s.mq_w = (size_t)(L - 1) * 2 * D * hd;
    s.b_w = s.a_w = s.pr_w = (size_t)T * ctw;
    s.d_w = (size_t)T * 3 * L * N;
    s.xd_w = (mac_digit_bytes(ctx, L - 1, s.kt_pad) + 7) / 8;
    s.qt_w = (size_t)(L - 1) * 2 * D * T * s.Jt;
    s.acc_w = s.rot_w = (size_t)s.Jt * ctw1;
    s.tot_w = ctw1;
    s.work_w = std::max({ks_scratch_words(ctx, level, ks_rot_batch(T - 1)),
                         ks_scratch_words(ctx, level, ks_rot_batch(T), T),
                         ks_scratch_words(ctx, level - 1, ks_rot_batch(s.Jt), s.Jt),
                         (size_t)2 * T * (1 + level) * N});
    s.total = s.u_w + s.mq_w + s.b_w + s.a_w + s.d_w + s.pr_w + s.xd_w + s.qt_w + s.acc_w + s.rot_w + s.tot_w +
              s.work_w;
    return s;
}

// Scratch of the weighted-sum call for scores of Lp limbs and values of Lv limbs (words)
struct ApplyScratch {
    uint32_t Jt, kt_pad, nj;
    size_t u_w, mq_w, r_w, xd_w, qt_w, cacc_w, ctmp_w, c_w, e_w, d_w, o_w, work_w, total;
};

ApplyScratch apply_scratch(const ckks_ctx *ctx, uint32_t Lp, uint32_t Lv, uint32_t D, uint32_t T, uint32_t hd)
{
    ApplyScratch s{};
    const size_t N = ctx->n;
    const uint32_t lv = Lv - 1, lp = Lp - 1;
    s.Jt = std::min(hd + T - 1, mac_max_outputs());
    s.kt_pad = mac_kt_pad(T);
    s.nj = hd + T - 1;
    s.u_w = (size_t)hd * D;
    s.mq_w = (size_t)Lv * 2 * D * hd;
    s.r_w = (size_t)T * 2 * Lv * N;
    s.xd_w = (mac_digit_bytes(ctx, Lv, s.kt_pad) + 7) / 8;
    s.qt_w = (size_t)Lv * 2 * D * T * s.Jt;
    s.cacc_w = (size_t)s.Jt * 2 * Lv * N;
    s.ctmp_w = (size_t)s.Jt * 2 * (Lv - 1) * N;
    s.c_w = s.e_w = (size_t)s.nj * 2 * Lp * N;
    s.d_w = (size_t)3 * Lp * N;
    s.o_w = (size_t)2 * Lp * N;
    const size_t ext = Lp + ctx->n_p, nd = n_digits(ctx, lp);
    const size_t relin_w = (nd * ext + ctx->alpha) * N + 2 * ext * N + 2 * (size_t)Lp * N;
    s.work_w = std::max({ks_scratch_words(ctx, lv, ks_rot_batch(T - 1)),
                         ks_scratch_words(ctx, lp, ks_rot_batch(s.nj - 1)), (size_t)2 * s.Jt * (1 + lv) * N,
                         relin_w, (size_t)2 * (1 + lp) * N});
    s.total = s.u_w + s.mq_w + s.r_w + s.xd_w + s.qt_w + s.cacc_w + s.ctmp_w + s.c_w + s.e_w + s.d_w + s.o_w +
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

    const size_t N = ctx->n, ctw = 2 * (size_t)L * N, ctw1 = 2 * (size_t)(L - 1) * N;
    const ScoreScratch ss = score_scratch(ctx, L, D, T, hd);
    void *w;
    CK_TRY(ctx_scratch(ctx, ss.total * 8, &w));
    double *U = (double *)w;
    double *MQ = U + ss.u_w;
    uint64_t *B = (uint64_t *)(MQ + ss.mq_w);   // [T][2][L][N] rotated keys
    uint64_t *A = B + ss.b_w;                   // [T][2][L][N] rotated queries, then P_delta ([T][2][L-1][N])
    uint64_t *Dt = A + ss.a_w;                  // [T][3][L][N] products
    uint64_t *Pr = Dt + ss.d_w;                 // [T][2][L][N] relinearised products
    int8_t *Xd = (int8_t *)(Pr + ss.pr_w);
    double *Qt = (double *)((uint64_t *)Xd + ss.xd_w);
    uint64_t *acc = (uint64_t *)(Qt + ss.qt_w);  // [Jt][2][L-1][N]
    uint64_t *rot = acc + ss.acc_w;
    uint64_t *tot = rot + ss.rot_w;
    uint64_t *work = tot + ss.tot_w;

    // the masks at scale q_(level-1): the products are multiplied by them after their first rescale
    CK_TRY(launch_masks(ctx, U, MQ, D, hd, (double)ctx->primes[level - 1], L - 1));
    // queries grouped by key: each key's rotations are computed once
    std::vector<uint32_t> order(n_q);
    for (uint32_t c = 0; c < n_q; c++) order[c] = c;
    std::stable_sort(order.begin(), order.end(), [&](uint32_t a, uint32_t b) { return k_of_q[a] < k_of_q[b]; });
    std::vector<uint64_t *> outs(T);
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
        //    key: (d0 + u0, u1), then d1 added), rescaled
        for (uint32_t d = 0; d < T; d++) {
            uint64_t *dd = Dt + (size_t)d * 3 * L * N;
            CK_TRY(launch_tensor(ctx, dd, dd + L * N, dd + 2 * L * N, A + (size_t)d * ctw, B + (size_t)d * ctw, L));
        }
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
            for (uint32_t d = 0; d < T; d++)
                CK_TRY(launch_binary(ctx, po[d] + (size_t)L * N, po[d] + (size_t)L * N, c0s[d] + (size_t)L * N, L,
                                     limb_range(0, L), EW_ADD));
        }
        uint64_t *Pd = A;  // [T][2][L-1][N]
        CK_TRY(rescale_many(ctx, Pr, T, level, Pd, work));
        // 3. U_k = sum_delta M_{(delta + k) mod hd} P_delta on the matrix cores, tiles of Jt values of k; each
        //    tile rotated by its k and summed
        CK_TRY(launch_xdigits(ctx, Pd, Xd, L - 1, T, ss.kt_pad));
        for (uint32_t k0 = 0; k0 < hd; k0 += ss.Jt) {
            const uint32_t jc = std::min(ss.Jt, hd - k0);
            CK_TRY(launch_table(ctx, Qt, MQ, L - 1, 2 * D, T, jc, hd, (int)k0, true));
            CK_TRY(launch_mac_mfma(ctx, acc, Xd, Qt, jc, T, 0, ss.kt_pad, 2 * D, L - 1, logT, false));
            const uint32_t first = k0 == 0 ? 1 : 0;  // k = 0 needs no rotation
            std::vector<uint64_t *> ro(jc);
            for (uint32_t jj = 0; jj < jc; jj++) ro[jj] = rot + (size_t)jj * ctw1;
            CK_TRY(rotate_each(ctx, acc + (size_t)first * ctw1, ctw1, jc - first, level - 1,
                               osteps.data() + (k0 + first - 1), okeys.data() + (k0 + first - 1), ro.data(), work));
            if (k0 == 0) CK_TRY(launch_sum_cts(ctx, tot, acc, 1, ctw1, L - 1, false));
            CK_TRY(launch_sum_cts(ctx, tot, rot, jc - first, ctw1, L - 1, true));
        }
        // 4. the final rescale
        CK_TRY(rescale_core(ctx, tot, level - 1, out[c].data, work));
        out[c].scale = q[c].scale * k[kk].scale / (double)ctx->primes[level];
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
    uint64_t *R = (uint64_t *)(MQ + ss.mq_w);    // [T][2][Lv][N]
    int8_t *Xd = (int8_t *)(R + ss.r_w);
    double *Qt = (double *)((uint64_t *)Xd + ss.xd_w);
    uint64_t *cacc = (uint64_t *)(Qt + ss.qt_w);  // [Jt][2][Lv][N]
    uint64_t *ctmp = cacc + ss.cacc_w;            // [Jt][2][Lv-1][N]
    uint64_t *C = ctmp + ss.ctmp_w;               // [nj][2][Lp][N], index j + hd - 1
    uint64_t *E = C + ss.c_w;                     // [nj][2][Lp][N]
    uint64_t *Dacc = E + ss.e_w;                  // [3][Lp][N]
    uint64_t *O = Dacc + ss.d_w;                  // [2][Lp][N]
    uint64_t *work = O + ss.o_w;

    // masks at scale q_(level of the values): C_j is rescaled by that prime
    CK_TRY(launch_masks(ctx, U, MQ, D, hd, (double)ctx->primes[lv], Lv));
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
            // 2. C_j on the matrix cores in tiles of Jt values of j, rescaled, kept on the scores' limbs
            CK_TRY(launch_xdigits(ctx, R, Xd, Lv, T, ss.kt_pad));
            for (uint32_t j0 = 0; j0 < ss.nj; j0 += ss.Jt) {
                const uint32_t jc = std::min(ss.Jt, ss.nj - j0);
                const int o0 = (int)j0 - (int)hd + 1;
                CK_TRY(launch_table(ctx, Qt, MQ, Lv, 2 * D, T, jc, hd, o0, false));
                CK_TRY(launch_mac_mfma(ctx, cacc, Xd, Qt, jc, T, 0, ss.kt_pad, 2 * D, Lv, logT, false));
                uint64_t *dst = C + (size_t)j0 * ctwp;
                if (Lp == Lv - 1) {
                    CK_TRY(rescale_many(ctx, cacc, jc, lv, dst, work));
                } else {
                    CK_TRY(rescale_many(ctx, cacc, jc, lv, ctmp, work));
                    HIP_TRY(hipMemcpy2DAsync(dst, (size_t)Lp * N * 8, ctmp, (size_t)(Lv - 1) * N * 8,
                                             (size_t)Lp * N * 8, 2 * jc, hipMemcpyDeviceToDevice, ctx->stream));
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
