// C ABI: encoding, encryption, key generation and the homomorphic operations.
// Every call validates its arguments on the host before the first launch.
#include <cmath>
#include <cstring>
#include <vector>

#include "ckks_internal.h"
#include "ops.h"

namespace {

ckks_status check_buf(const ckks_ctx *ctx, const ckks_buf *b, uint32_t polys, const char *what)
{
    CK_REQUIRE(b, CKKS_EINVAL, "%s: null buffer", what);
    CK_REQUIRE(b->data, CKKS_EINVAL, "%s: null data pointer", what);
    CK_REQUIRE(b->n_polys == polys, CKKS_EINVAL, "%s: expected %u polynomials, got %u", what, polys, b->n_polys);
    CK_REQUIRE(b->n_limbs >= 1 && b->n_limbs <= ctx->n_q, CKKS_ELEVEL, "%s: %u limbs outside [1, %u]", what,
               b->n_limbs, ctx->n_q);
    return CKKS_OK;
}

size_t words(const ckks_ctx *ctx, size_t rows) { return rows << ctx->log_n; }

}  // namespace

// Workspace bytes of one call of `op` (ckks_op) with the given shape; SIZE_MAX for an unknown op or shape.
// Every call below takes exactly this many bytes from the context's arena.
size_t op_workspace_bytes(const ckks_ctx *ctx, int op, const uint32_t *shape)
{
    const size_t N = ctx->n;
    const uint32_t a = shape ? shape[0] : 0;
    switch (op) {
    case CKKS_OP_NONE: return 0;
    case CKKS_OP_ENCODE: return enc_work_bytes(ctx, 1) + N * sizeof(int64_t);
    case CKKS_OP_DECODE:
        if (a < 1 || a > ctx->n_q) return SIZE_MAX;
        return words(ctx, a > 1 ? 2 : 1) * 8 + enc_work_bytes(ctx, 1);
    case CKKS_OP_ENCRYPT:
        if (a < 1 || a > ctx->n_q) return SIZE_MAX;
        return words(ctx, 2 * (size_t)a) * 8;
    case CKKS_OP_DECRYPT:
        if (a < 1 || a > ctx->n_q) return SIZE_MAX;
        return words(ctx, a) * 8;
    case CKKS_OP_KEYGEN: return words(ctx, (3 + (size_t)ctx->dnum) * ctx->n_primes()) * 8;
    case CKKS_OP_RESCALE:
        if (a < 2 || a > ctx->n_q) return SIZE_MAX;
        return words(ctx, 2 + 2 * (size_t)(a - 1)) * 8;
    case CKKS_OP_ROTATE: {
        const uint32_t count = shape ? shape[1] : 0;
        if (a < 1 || a > ctx->n_q || count < 1) return SIZE_MAX;
        return ks_scratch_words(ctx, a - 1, ks_rot_batch(count)) * 8;
    }
    case CKKS_OP_MUL_RELIN:
        if (a < 1 || a > ctx->n_q) return SIZE_MAX;
        return (3 * (size_t)a * N + ks_scratch_words(ctx, a - 1, 1)) * 8;
    case CKKS_OP_MODUP:
        if (!shape || a >= ctx->n_q) return SIZE_MAX;
        return ((size_t)n_digits(ctx, a) * (a + 1 + ctx->n_p) + ctx->alpha) * N * 8;
    case CKKS_OP_MODDOWN:
        if (!shape || a >= ctx->n_q) return SIZE_MAX;
        return ((size_t)(a + 1 + ctx->n_p) + (a + 1)) * N * 8;
    case CKKS_OP_LINEAR_PROJECT:
        if (!shape) return SIZE_MAX;
        return proj_workspace_bytes(ctx, shape[0], shape[1], shape[2], shape[3], shape[4]);
    case CKKS_OP_LINEAR_PROJECT_TM:
        if (!shape) return SIZE_MAX;
        return proj_tm_workspace_bytes(ctx, shape[0], shape[1], shape[2], shape[3], shape[4]);
    case CKKS_OP_ATTN_SCORES:
        if (!shape) return SIZE_MAX;
        return attn_scores_workspace_bytes(ctx, shape[0], shape[1], shape[2]);
    case CKKS_OP_ATTN_APPLY:
        if (!shape) return SIZE_MAX;
        return attn_apply_workspace_bytes(ctx, shape[0], shape[1], shape[2], shape[3]);
    default: return SIZE_MAX;
    }
}

// rotations of one ciphertext sharing a single ModUp (used by the API and the projection),
// processed in batches of ks_rot_batch(count).  work: ks_scratch_words(level, ks_rot_batch(count)) words
ckks_status rotate_core(ckks_ctx *ctx, const uint64_t *c, uint32_t level, const int32_t *steps,
                        const uint64_t *const *keys, uint32_t count, uint64_t *const *outs, uint64_t *work,
                        const uint64_t *seeds)
{
    if (!count) return CKKS_OK;
    const uint32_t L = level + 1, ext = L + ctx->n_p, nd = n_digits(ctx, level);
    const size_t N = ctx->n;
    uint64_t *digits = work;
    uint64_t *rw = digits + ((size_t)nd * ext + ctx->alpha) * N;
    CK_TRY(ks_modup(ctx, c + (size_t)L * N, level, digits));
    const uint32_t bs = ks_rot_batch(count);
    std::vector<uint32_t> g(count);
    for (uint32_t r = 0; r < count; r++) g[r] = ckks_galois_elt(ctx, steps[r]);
    std::vector<const uint64_t *> c0s(count, c), digs(count, digits);
    for (uint32_t r0 = 0; r0 < count; r0 += bs) {
        const uint32_t cnt = count - r0 < bs ? count - r0 : bs;
        CK_TRY(ks_rotate_batch(ctx, level, cnt, c0s.data() + r0, digs.data() + r0, g.data() + r0, keys + r0,
                               outs + r0, rw, seeds ? seeds + 2 * (size_t)r0 : nullptr));
    }
    return CKKS_OK;
}

// The same rotation (steps, key) of `count` ciphertexts: ciphertext r at cs + r * stride (words, [2][level+1][N]),
// output r at outs[r]; one batched ModUp, key switching in batches of up to 32.
// work: ks_scratch_words(ctx, level, ks_rot_batch(count), count) words
ckks_status rotate_many(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                        int32_t steps, const uint64_t *key, uint64_t *const *outs, uint64_t *work)
{
    if (!count) return CKKS_OK;
    const uint32_t L = level + 1, ext = L + ctx->n_p, nd = n_digits(ctx, level);
    const size_t N = ctx->n, dig_ct = (size_t)nd * ext * N;
    uint64_t *digits = work;
    uint64_t *rw = digits + (size_t)count * (dig_ct + (size_t)ctx->alpha * N);
    CK_TRY(ks_modup_batch(ctx, cs + (size_t)L * N, stride, count, level, digits));
    const uint32_t bs = ks_rot_batch(count);
    std::vector<uint32_t> g(count, ckks_galois_elt(ctx, steps));
    std::vector<const uint64_t *> keys(count, key), c0s(count), digs(count);
    for (uint32_t r = 0; r < count; r++) {
        c0s[r] = cs + (size_t)r * stride;
        digs[r] = digits + (size_t)r * dig_ct;
    }
    for (uint32_t r0 = 0; r0 < count; r0 += bs) {
        const uint32_t cnt = count - r0 < bs ? count - r0 : bs;
        CK_TRY(ks_rotate_batch(ctx, level, cnt, c0s.data() + r0, digs.data() + r0, g.data() + r0, keys.data() + r0,
                               outs + r0, rw));
    }
    return CKKS_OK;
}

ckks_status rotate_each(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                        const int32_t *steps, const uint64_t *const *keys, uint64_t *const *outs, uint64_t *work)
{
    if (!count) return CKKS_OK;
    const uint32_t L = level + 1, ext = L + ctx->n_p, nd = n_digits(ctx, level);
    const size_t N = ctx->n, dig_ct = (size_t)nd * ext * N;
    uint64_t *digits = work;
    uint64_t *rw = digits + (size_t)count * (dig_ct + (size_t)ctx->alpha * N);
    CK_TRY(ks_modup_batch(ctx, cs + (size_t)L * N, stride, count, level, digits));
    const uint32_t bs = ks_rot_batch(count);
    std::vector<uint32_t> g(count);
    std::vector<const uint64_t *> c0s(count), digs(count);
    for (uint32_t r = 0; r < count; r++) {
        g[r] = ckks_galois_elt(ctx, steps[r]);
        c0s[r] = cs + (size_t)r * stride;
        digs[r] = digits + (size_t)r * dig_ct;
    }
    for (uint32_t r0 = 0; r0 < count; r0 += bs) {
        const uint32_t cnt = count - r0 < bs ? count - r0 : bs;
        CK_TRY(ks_rotate_batch(ctx, level, cnt, c0s.data() + r0, digs.data() + r0, g.data() + r0, keys + r0,
                               outs + r0, rw));
    }
    return CKKS_OK;
}

size_t lazy_work_words(const ckks_ctx *ctx, uint32_t level, uint32_t count)
{
    const size_t ext = level + 1 + ctx->n_p;
    return (size_t)count * ((size_t)n_digits(ctx, level) * ext + ctx->alpha) << ctx->log_n;
}

namespace {

ckks_status rotate_lazy(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                        const int32_t *steps, const uint64_t *const *keys, bool same_step, uint64_t *uacc,
                        bool sum_all, bool accumulate, uint64_t *work)
{
    if (!count) return CKKS_OK;
    const uint32_t L = level + 1, ext = L + ctx->n_p, nd = n_digits(ctx, level);
    const size_t N = ctx->n, dig_ct = (size_t)nd * ext * N;
    CK_TRY(ks_modup_batch(ctx, cs + (size_t)L * N, stride, count, level, work));
    std::vector<uint32_t> g(count);
    std::vector<const uint64_t *> c0s(count), digs(count), ks(count);
    std::vector<uint64_t *> accs(count);
    for (uint32_t r = 0; r < count; r++) {
        g[r] = ckks_galois_elt(ctx, same_step ? steps[0] : steps[r]);
        ks[r] = same_step ? keys[0] : keys[r];
        c0s[r] = cs + (size_t)r * stride;
        digs[r] = work + (size_t)r * dig_ct;
        accs[r] = uacc + (sum_all ? 0 : (size_t)r * 2 * ext * N);
    }
    const uint32_t bs = ks_rot_batch(count);
    for (uint32_t r0 = 0; r0 < count; r0 += bs) {
        const uint32_t cnt = count - r0 < bs ? count - r0 : bs;
        CK_TRY(ks_ip_accumulate(ctx, level, cnt, c0s.data() + r0, digs.data() + r0, g.data() + r0, ks.data() + r0,
                                accs.data() + r0, sum_all, accumulate || (sum_all && r0 > 0)));
    }
    return CKKS_OK;
}

}  // namespace

ckks_status rotate_many_lazy(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                             int32_t steps, const uint64_t *key, uint64_t *uacc, bool accumulate, uint64_t *work)
{
    return rotate_lazy(ctx, cs, stride, count, level, &steps, &key, true, uacc, false, accumulate, work);
}

ckks_status rotate_each_lazy(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                             const int32_t *steps, const uint64_t *const *keys, uint64_t *uacc, bool accumulate,
                             uint64_t *work)
{
    return rotate_lazy(ctx, cs, stride, count, level, steps, keys, false, uacc, true, accumulate, work);
}

ckks_status rescale_many(ckks_ctx *ctx, const uint64_t *c, uint32_t count, uint32_t l, uint64_t *out,
                         uint64_t *work)
{
    if (!count) return CKKS_OK;
    const size_t N = ctx->n;
    const uint32_t polys = 2 * count;
    uint64_t *top = work, *r = top + (size_t)polys * N;
    // the top limb of every polynomial, then the same steps as one rescale over all of them
    CK_TRY(launch_copy_rows(ctx, top, N, nullptr, 0, c + (size_t)l * N, (size_t)(l + 1) * N, N, polys));
    CK_TRY(launch_ntt(ctx, top, polys, limb_range(l, 1), true));
    // the centred top coefficients reduced modulo q_0..q_(l-1) inside the forward transform's first pass
    CK_TRY(launch_rescale_centre(ctx, top, polys, l));
    CK_TRY(launch_ntt_from_i64(ctx, (const int64_t *)top, r, polys, l));
    return launch_rescale_finish(ctx, out, c, r, polys, l);
}

// c ([2][l+1][N]) -> out ([2][l][N]) = round(c / q_l); work: (2 + 2l) N words
ckks_status rescale_core(ckks_ctx *ctx, const uint64_t *c, uint32_t l, uint64_t *out, uint64_t *work)
{
    const size_t N = ctx->n;
    uint64_t *top = work, *r = top + 2 * N;
    for (int k = 0; k < 2; k++)
        HIP_TRY(hipMemcpyAsync(top + k * N, c + ((size_t)k * (l + 1) + l) * N, N * 8, hipMemcpyDeviceToDevice,
                               ctx->stream));
    CK_TRY(launch_ntt(ctx, top, 2, limb_range(l, 1), true));
    CK_TRY(launch_rescale_centre(ctx, top, 2, l));
    CK_TRY(launch_ntt_from_i64(ctx, (const int64_t *)top, r, 2, l));
    return launch_rescale_finish(ctx, out, c, r, 2, l);
}

extern "C" {

ckks_status ckks_encode(ckks_ctx *ctx, const double *re, const double *im, double scale, uint32_t n_limbs,
                        ckks_buf *pt)
{
    clear_error();
    CK_REQUIRE(ctx && re, CKKS_EINVAL, "encode: null argument");
    CK_REQUIRE(pt && pt->data && pt->n_polys == 1, CKKS_EINVAL, "encode: output must be one polynomial");
    CK_REQUIRE(n_limbs >= 1 && n_limbs <= ctx->n_q && pt->n_limbs == n_limbs, CKKS_ELEVEL,
               "encode: limbs %u (buffer %u) outside [1, %u]", n_limbs, pt->n_limbs, ctx->n_q);
    CK_REQUIRE(scale > 0 && std::isfinite(scale), CKKS_EINVAL, "encode: scale must be positive");
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_ENCODE, nullptr), &w));
    double2 *work = (double2 *)w;
    int64_t *m = (int64_t *)((char *)w + enc_work_bytes(ctx, 1));
    SlotSource src;
    src.re = re;
    src.im = im;
    CK_TRY(enc_coeffs(ctx, src, 1, scale, work, m));
    CK_TRY(launch_ntt_from_i64(ctx, m, pt->data, 1, n_limbs));
    pt->scale = scale;
    return CKKS_OK;
}

ckks_status ckks_decode(ckks_ctx *ctx, const ckks_buf *pt, double *re, double *im)
{
    clear_error();
    CK_REQUIRE(ctx && re && im, CKKS_EINVAL, "decode: null argument");
    CK_TRY(check_buf(ctx, pt, 1, "decode"));
    CK_REQUIRE(pt->scale > 0, CKKS_ESCALE, "decode: scale must be positive");
    const uint32_t lim = pt->n_limbs > 1 ? 2 : 1;
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_DECODE, &pt->n_limbs), &w));
    uint64_t *coef = (uint64_t *)w;
    double2 *work = (double2 *)(coef + words(ctx, lim));
    HIP_TRY(hipMemcpyAsync(coef, pt->data, words(ctx, lim) * 8, hipMemcpyDeviceToDevice, ctx->stream));
    CK_TRY(launch_ntt(ctx, coef, lim, limb_range(0, lim), true));
    return dec_slots(ctx, coef, lim, pt->scale, work, re, im);
}

ckks_status ckks_encrypt_sk(ckks_ctx *ctx, const int8_t *s, const ckks_buf *pt, const uint64_t *a, const int32_t *e,
                            ckks_buf *ct)
{
    clear_error();
    CK_REQUIRE(ctx && s && a && e, CKKS_EINVAL, "encrypt: null argument");
    CK_TRY(check_buf(ctx, pt, 1, "encrypt (plaintext)"));
    CK_TRY(check_buf(ctx, ct, 2, "encrypt (ciphertext)"));
    CK_REQUIRE(ct->n_limbs == pt->n_limbs, CKKS_ELEVEL, "encrypt: limb counts differ");
    const uint32_t L = pt->n_limbs;
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_ENCRYPT, &L), &w));
    uint64_t *sn = (uint64_t *)w, *en = sn + words(ctx, L);
    const LimbMap map = limb_range(0, L);
    CK_TRY(launch_expand_i8(ctx, sn, s, map));
    CK_TRY(launch_expand_i32(ctx, en, e, map));
    CK_TRY(launch_ntt(ctx, sn, 2 * L, map, false));
    CK_TRY(launch_encrypt(ctx, ct->data, ct->data + words(ctx, L), a, sn, en, pt->data, map));
    ct->scale = pt->scale;
    return CKKS_OK;
}

ckks_status ckks_decrypt(ckks_ctx *ctx, const int8_t *s, const ckks_buf *ct, ckks_buf *pt)
{
    clear_error();
    CK_REQUIRE(ctx && s, CKKS_EINVAL, "decrypt: null argument");
    CK_TRY(check_buf(ctx, ct, 2, "decrypt (ciphertext)"));
    CK_TRY(check_buf(ctx, pt, 1, "decrypt (plaintext)"));
    CK_REQUIRE(ct->n_limbs == pt->n_limbs, CKKS_ELEVEL, "decrypt: limb counts differ");
    const uint32_t L = ct->n_limbs;
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_DECRYPT, &L), &w));
    uint64_t *sn = (uint64_t *)w;
    const LimbMap map = limb_range(0, L);
    CK_TRY(launch_expand_i8(ctx, sn, s, map));
    CK_TRY(launch_ntt(ctx, sn, L, map, false));
    CK_TRY(launch_binary(ctx, sn, ct->data + words(ctx, L), sn, L, map, EW_MUL));
    CK_TRY(launch_binary(ctx, pt->data, ct->data, sn, L, map, EW_ADD));
    pt->scale = ct->scale;
    return CKKS_OK;
}

// key: [dnum][2][R][N] (b and a), or with b_only the b halves [dnum][R][N] of a seed-expanded key
static ckks_status keygen_common(ckks_ctx *ctx, const int8_t *s, uint32_t g, bool relin, const uint64_t *a,
                                 const int32_t *e, uint64_t *key, bool b_only = false, uint64_t *w_given = nullptr)
{
    CK_REQUIRE(ctx && s && a && e && key, CKKS_EINVAL, "keygen: null argument");
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "keygen: the context has no special primes");
    CK_REQUIRE(relin || (g & 1u), CKKS_EINVAL, "keygen: Galois element %u is even", g);
    const uint32_t R = ctx->n_primes();
    const size_t rows = R;
    void *w = w_given;
    if (!w) CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_KEYGEN, nullptr), &w));
    uint64_t *sn = (uint64_t *)w, *t = sn + words(ctx, rows), *en = t + words(ctx, rows);
    const LimbMap all = limb_range(0, R);
    CK_TRY(launch_expand_i8(ctx, sn, s, all));
    CK_TRY(launch_ntt(ctx, sn, R, all, false));
    if (relin) CK_TRY(launch_binary(ctx, t, sn, sn, R, all, EW_MUL));
    else CK_TRY(launch_automorph(ctx, sn, t, R, g));
    for (uint32_t j = 0; j < ctx->dnum; j++) {
        CK_TRY(launch_expand_i32(ctx, en, e + (size_t)j * ctx->n, all));
        CK_TRY(launch_ntt(ctx, en, R, all, false));
        uint64_t *kb = key + (size_t)j * (b_only ? 1 : 2) * words(ctx, rows);
        const uint32_t lo = digit_lo(ctx, j);
        uint32_t hi = lo + ctx->alpha;
        if (hi > ctx->n_q) hi = ctx->n_q;
        CK_TRY(launch_keygen_digit(ctx, kb, b_only ? nullptr : kb + words(ctx, rows), a + (size_t)j * words(ctx, rows),
                                   sn, en, t, lo, hi));
    }
    return CKKS_OK;
}

ckks_status ckks_keygen_galois(ckks_ctx *ctx, const int8_t *s, uint32_t g, const uint64_t *a, const int32_t *e,
                               uint64_t *key)
{
    clear_error();
    CK_REQUIRE(ctx, CKKS_EINVAL, "keygen: null context");
    CK_REQUIRE(g < 2 * ctx->n, CKKS_EINVAL, "keygen: Galois element %u >= 2N", g);
    return keygen_common(ctx, s, g, false, a, e, key);
}

ckks_status ckks_keygen_relin(ckks_ctx *ctx, const int8_t *s, const uint64_t *a, const int32_t *e, uint64_t *key)
{
    clear_error();
    return keygen_common(ctx, s, 1, true, a, e, key);
}

ckks_status ckks_expand_key_a(ckks_ctx *ctx, const uint64_t *seed, uint64_t *a)
{
    clear_error();
    CK_REQUIRE(ctx && seed && a, CKKS_EINVAL, "expand_key_a: null argument");
    return launch_expand_key_a(ctx, seed[0], seed[1], a);
}

ckks_status ckks_keygen_galois_seeded(ckks_ctx *ctx, const int8_t *s, uint32_t g, const uint64_t *seed,
                                      const int32_t *e, uint64_t *key_b)
{
    clear_error();
    CK_REQUIRE(ctx && seed, CKKS_EINVAL, "keygen (seeded): null argument");
    CK_REQUIRE(g < 2 * ctx->n, CKKS_EINVAL, "keygen: Galois element %u >= 2N", g);
    // scratch: the key generation's own rows, then the expanded a half
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_KEYGEN, nullptr), &w));
    uint64_t *a = (uint64_t *)w + words(ctx, 3 * (size_t)ctx->n_primes());
    CK_TRY(launch_expand_key_a(ctx, seed[0], seed[1], a));
    return keygen_common(ctx, s, g, false, a, e, key_b, true, (uint64_t *)w);
}

ckks_status ckks_add(ckks_ctx *ctx, const ckks_buf *a, const ckks_buf *b, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx, CKKS_EINVAL, "add: null context");
    CK_TRY(check_buf(ctx, a, 2, "add (a)"));
    CK_TRY(check_buf(ctx, b, 2, "add (b)"));
    CK_TRY(check_buf(ctx, out, 2, "add (out)"));
    CK_REQUIRE(a->n_limbs == b->n_limbs && out->n_limbs == a->n_limbs, CKKS_ELEVEL, "add: limb counts differ");
    CK_REQUIRE(a->scale == b->scale, CKKS_ESCALE, "add: scales differ (%g vs %g)", a->scale, b->scale);
    const LimbMap map = limb_range(0, a->n_limbs);
    CK_TRY(launch_binary(ctx, out->data, a->data, b->data, 2 * a->n_limbs, map, EW_ADD));
    out->scale = a->scale;
    return CKKS_OK;
}

ckks_status ckks_mul_plain(ckks_ctx *ctx, const ckks_buf *ct, const ckks_buf *pt, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx, CKKS_EINVAL, "mul_plain: null context");
    CK_TRY(check_buf(ctx, ct, 2, "mul_plain (ciphertext)"));
    CK_TRY(check_buf(ctx, pt, 1, "mul_plain (plaintext)"));
    CK_TRY(check_buf(ctx, out, 2, "mul_plain (out)"));
    CK_REQUIRE(pt->n_limbs >= ct->n_limbs && out->n_limbs == ct->n_limbs, CKKS_ELEVEL,
               "mul_plain: plaintext has fewer limbs than the ciphertext");
    CK_TRY(launch_mul_plain(ctx, out->data, ct->data, pt->data, 2, ct->n_limbs));
    out->scale = ct->scale * pt->scale;
    return CKKS_OK;
}

ckks_status ckks_rescale(ckks_ctx *ctx, const ckks_buf *in, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx, CKKS_EINVAL, "rescale: null context");
    CK_TRY(check_buf(ctx, in, 2, "rescale (in)"));
    CK_TRY(check_buf(ctx, out, 2, "rescale (out)"));
    CK_REQUIRE(in->n_limbs >= 2, CKKS_ELEVEL, "rescale: needs at least two limbs");
    CK_REQUIRE(out->n_limbs == in->n_limbs - 1, CKKS_ELEVEL, "rescale: output must have one limb fewer");
    const uint32_t l = in->n_limbs - 1;
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_RESCALE, &in->n_limbs), &w));
    CK_TRY(rescale_core(ctx, in->data, l, out->data, (uint64_t *)w));
    out->scale = in->scale / (double)ctx->primes[l];
    return CKKS_OK;
}

static ckks_status rotate_hoisted_api(ckks_ctx *ctx, const ckks_buf *in, const int32_t *steps, uint32_t count,
                                      const uint64_t *const *keys, const uint64_t *seeds, ckks_buf *outs)
{
    CK_REQUIRE(ctx, CKKS_EINVAL, "rotate: null context");
    CK_TRY(check_buf(ctx, in, 2, "rotate (in)"));
    if (count == 0) return CKKS_OK;
    CK_REQUIRE(steps && keys && outs, CKKS_EINVAL, "rotate: null argument");
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "rotate: the context has no special primes");
    std::vector<uint64_t *> op(count);
    for (uint32_t r = 0; r < count; r++) {
        CK_TRY(check_buf(ctx, &outs[r], 2, "rotate (out)"));
        CK_REQUIRE(outs[r].n_limbs == in->n_limbs, CKKS_ELEVEL, "rotate: output %u has the wrong limb count", r);
        CK_REQUIRE(keys[r], CKKS_ENOKEY, "rotate: no key for step %d", steps[r]);
        CK_REQUIRE(outs[r].data != in->data, CKKS_EINVAL, "rotate: output %u aliases the input", r);
        op[r] = outs[r].data;
    }
    const uint32_t level = in->n_limbs - 1;
    void *w;
    const uint32_t shp[2] = {in->n_limbs, count};
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_ROTATE, shp), &w));
    CK_TRY(rotate_core(ctx, in->data, level, steps, keys, count, op.data(), (uint64_t *)w, seeds));
    for (uint32_t r = 0; r < count; r++) outs[r].scale = in->scale;
    return CKKS_OK;
}

ckks_status ckks_rotate_hoisted(ckks_ctx *ctx, const ckks_buf *in, const int32_t *steps, uint32_t count,
                                const uint64_t *const *keys, ckks_buf *outs)
{
    clear_error();
    return rotate_hoisted_api(ctx, in, steps, count, keys, nullptr, outs);
}

ckks_status ckks_rotate_hoisted_seeded(ckks_ctx *ctx, const ckks_buf *in, const int32_t *steps, uint32_t count,
                                       const uint64_t *const *key_b, const uint64_t *seeds, ckks_buf *outs)
{
    clear_error();
    CK_REQUIRE(count == 0 || seeds, CKKS_EINVAL, "rotate (seeded): null seeds");
    return rotate_hoisted_api(ctx, in, steps, count, key_b, seeds, outs);
}

ckks_status ckks_rotate(ckks_ctx *ctx, const ckks_buf *in, int32_t steps, const uint64_t *key, ckks_buf *out)
{
    const uint64_t *keys[1] = {key};
    return ckks_rotate_hoisted(ctx, in, &steps, 1, keys, out);
}

ckks_status ckks_mul_relin(ckks_ctx *ctx, const ckks_buf *a, const ckks_buf *b, const uint64_t *rlk, ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx && rlk, CKKS_EINVAL, "mul_relin: null argument");
    CK_TRY(check_buf(ctx, a, 2, "mul_relin (a)"));
    CK_TRY(check_buf(ctx, b, 2, "mul_relin (b)"));
    CK_TRY(check_buf(ctx, out, 2, "mul_relin (out)"));
    CK_REQUIRE(a->n_limbs == b->n_limbs && out->n_limbs == a->n_limbs, CKKS_ELEVEL, "mul_relin: limb counts differ");
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "mul_relin: the context has no special primes");
    const uint32_t L = a->n_limbs, level = L - 1;
    const uint32_t ext = L + ctx->n_p, nd = n_digits(ctx, level);
    const size_t N = ctx->n;
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_MUL_RELIN, &L), &w));
    uint64_t *d0 = (uint64_t *)w, *d1 = d0 + L * N, *d2 = d1 + L * N;
    uint64_t *digits = d2 + L * N;
    uint64_t *u = digits + ((size_t)nd * ext + ctx->alpha) * N;
    uint64_t *cw = u + 2 * (size_t)ext * N;
    CK_TRY(launch_tensor(ctx, d0, d1, d2, a->data, b->data, L));
    CK_TRY(ks_modup(ctx, d2, level, digits));
    CK_TRY(ks_inner_product(ctx, digits, nd, rlk, level, 1, u));
    CK_TRY(ks_moddown(ctx, u, 2, level, d0, 1, d1, out->data, cw));
    out->scale = a->scale * b->scale;
    return CKKS_OK;
}

ckks_status ckks_modup(ckks_ctx *ctx, const uint64_t *c, uint32_t level, uint64_t *digits)
{
    clear_error();
    CK_REQUIRE(ctx && c && digits, CKKS_EINVAL, "modup: null argument");
    CK_REQUIRE(level < ctx->n_q, CKKS_ELEVEL, "modup: level %u >= n_q", level);
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "modup: the context has no special primes");
    const uint32_t ext = level + 1 + ctx->n_p, nd = n_digits(ctx, level);
    const size_t N = ctx->n;
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_MODUP, &level), &w));
    CK_TRY(ks_modup(ctx, c, level, (uint64_t *)w));
    HIP_TRY(hipMemcpyAsync(digits, w, (size_t)nd * ext * N * 8, hipMemcpyDeviceToDevice, ctx->stream));
    return CKKS_OK;
}

ckks_status ckks_moddown(ckks_ctx *ctx, const uint64_t *x, uint32_t level, uint64_t *out)
{
    clear_error();
    CK_REQUIRE(ctx && x && out, CKKS_EINVAL, "moddown: null argument");
    CK_REQUIRE(level < ctx->n_q, CKKS_ELEVEL, "moddown: level %u >= n_q", level);
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "moddown: the context has no special primes");
    const uint32_t ext = level + 1 + ctx->n_p;
    const size_t N = ctx->n;
    void *w;
    CK_TRY(ctx_scratch(ctx, op_workspace_bytes(ctx, CKKS_OP_MODDOWN, &level), &w));
    uint64_t *u = (uint64_t *)w, *cw = u + (size_t)ext * N;
    HIP_TRY(hipMemcpyAsync(u, x, (size_t)ext * N * 8, hipMemcpyDeviceToDevice, ctx->stream));
    return ks_moddown(ctx, u, 1, level, nullptr, 1, nullptr, out, cw);
}

ckks_status ckks_automorph(ckks_ctx *ctx, const uint64_t *in, uint32_t rows, uint32_t g, uint64_t *out)
{
    clear_error();
    CK_REQUIRE(ctx && in && out, CKKS_EINVAL, "automorph: null argument");
    CK_REQUIRE((g & 1u) && g < 2 * ctx->n, CKKS_EINVAL, "automorph: Galois element %u must be odd and < 2N", g);
    CK_REQUIRE(in != out, CKKS_EINVAL, "automorph: output aliases input");
    return launch_automorph(ctx, in, out, rows, g);
}

}  // extern "C"
