// Launchers of the element-wise, structural, key-switching, encoding and
// projection kernels (definitions in ops.hip, keyswitch.hip, encode.hip,
// project.hip).
#pragma once
#include "ckks_internal.h"

enum { EW_ADD = 0, EW_SUB = 1, EW_MUL = 2 };

ckks_status launch_binary(ckks_ctx *ctx, uint64_t *out, const uint64_t *a, const uint64_t *b, uint32_t rows,
                          const LimbMap &map, int op);
ckks_status launch_mul_plain(ckks_ctx *ctx, uint64_t *out, const uint64_t *ct, const uint64_t *pt, uint32_t polys,
                             uint32_t limbs);
ckks_status launch_tensor(ckks_ctx *ctx, uint64_t *d0, uint64_t *d1, uint64_t *d2, const uint64_t *a,
                          const uint64_t *b, uint32_t limbs);
// `count` independent entries in one launch (at most 65535), each pointer advanced by its own stride in words
ckks_status launch_binary_batch(ckks_ctx *ctx, uint64_t *out, size_t out_stride, const uint64_t *a,
                                size_t a_stride, const uint64_t *b, size_t b_stride, uint32_t count, uint32_t rows,
                                const LimbMap &map, int op);
ckks_status launch_tensor_batch(ckks_ctx *ctx, uint64_t *d0, uint64_t *d1, uint64_t *d2, size_t d_stride,
                                const uint64_t *a, size_t a_stride, const uint64_t *b, size_t b_stride,
                                uint32_t count, uint32_t limbs);
ckks_status launch_expand_i8(ckks_ctx *ctx, uint64_t *out, const int8_t *v, const LimbMap &map);
ckks_status launch_expand_i32(ckks_ctx *ctx, uint64_t *out, const int32_t *v, const LimbMap &map);
ckks_status launch_encrypt(ckks_ctx *ctx, uint64_t *c0, uint64_t *c1, const uint64_t *a, const uint64_t *s,
                           const uint64_t *e, const uint64_t *m, const LimbMap &map);
ckks_status launch_keygen_digit(ckks_ctx *ctx, uint64_t *b_out, uint64_t *a_out, const uint64_t *a,
                                const uint64_t *s, const uint64_t *e, const uint64_t *t, uint32_t dig_lo,
                                uint32_t dig_hi);
// count entries of `words` contiguous words: entry b at src + b src_stride copied to dst_a + b a_stride and, when
// dst_b is not null, to dst_b + b b_stride (strides in words; 16-byte accesses where every pointer and stride
// allows them); count <= 65535
ckks_status launch_copy_rows(ckks_ctx *ctx, uint64_t *dst_a, size_t a_stride, uint64_t *dst_b, size_t b_stride,
                             const uint64_t *src, size_t src_stride, size_t words, uint32_t count);
// top ([polys][N], canonical mod q_l) to centred int64 in place
ckks_status launch_rescale_centre(ckks_ctx *ctx, uint64_t *top, uint32_t polys, uint32_t l);
ckks_status launch_rescale_finish(ckks_ctx *ctx, uint64_t *out, const uint64_t *c, const uint64_t *r,
                                  uint32_t polys, uint32_t l);

// key switching (keyswitch.hip)
// digits: [nd][level+1+K][N] from c ([level+1][N]); the buffer must hold alpha more rows
// after the digits (staging for the INTT of a digit's limbs)
ckks_status ks_modup(ckks_ctx *ctx, const uint64_t *c, uint32_t level, uint64_t *digits);
// ModUp of `count` ciphertexts at once: c1 of ciphertext r at c1 + r * in_stride (words); digits: [count][nd][ext][N]
// followed by count * alpha staging rows
ckks_status ks_modup_batch(ckks_ctx *ctx, const uint64_t *c1, size_t in_stride, uint32_t count, uint32_t level,
                           uint64_t *digits);
// (u0, u1) = sum_j sigma_g(d_j) (b_j, a_j); g = 1 for no automorphism; u: [2][level+1+K][N]
ckks_status ks_inner_product(ckks_ctx *ctx, const uint64_t *digits, uint32_t nd, const uint64_t *key,
                             uint32_t level, uint32_t g, uint64_t *u);
// out_k = (u_k - Conv(INTT([u_k]_P))) P^-1 (+ add_k), k < polys; u ([polys][level+1+K][N]) is clobbered.
// add0/add1: [level+1][N] or null, add0 read through the automorphism add0_g (1 = none);
// out: [polys][level+1][N]; work: [polys][level+1][N]
ckks_status ks_moddown(ckks_ctx *ctx, uint64_t *u, uint32_t polys, uint32_t level, const uint64_t *add0,
                       uint32_t add0_g, const uint64_t *add1, uint64_t *out, uint64_t *work);
// scratch words for rotations at `level` processed `batch` at a time (see rotate_core)
size_t ks_scratch_words(const ckks_ctx *ctx, uint32_t level, uint32_t batch, uint32_t n_ct = 1);
// rotations per batched launch for `count` requested rotations
uint32_t ks_rot_batch(uint32_t count);
// the a half [dnum][n_q + n_p][N] of the seed-expanded key with seed (s0, s1) (philox.h)
ckks_status launch_expand_key_a(ckks_ctx *ctx, uint64_t s0, uint64_t s1, uint64_t *a);
// `count` (<= 32) rotations: rotation r applies the automorphism g[r] with key keys[r] to the ciphertext whose
// c0 is c0s[r] and whose ModUp digits are digs[r] (hoisted rotations of one ciphertext share both): key inner
// product, ModDown and the sigma_{g_r}(c0) addition, each stage one launch for all r.
// work: count * (2 ext + 2 (level+1)) N words.  seeds (nullable, [count][2]): seed-expanded keys, keys[r] then holds
// the b half [dnum][n_q + n_p][N] and the a half comes from seeds[2r], seeds[2r + 1] (philox.h)
ckks_status ks_rotate_batch(ckks_ctx *ctx, uint32_t level, uint32_t count, const uint64_t *const *c0s,
                            const uint64_t *const *digs, const uint32_t *g, const uint64_t *const *keys,
                            uint64_t *const *outs, uint64_t *work, const uint64_t *seeds = nullptr);

// lazy ModDown: accs[r] (or accs[0] for all r when sum_all; [2][level+1+K][N]) (+)= the key inner product of
// rotation r over Q_level u P plus P * sigma_{g_r}(c0_r) on the q rows; count <= 32.  ks_moddown of the accumulator
// then gives the sum of the rotations.
ckks_status ks_ip_accumulate(ckks_ctx *ctx, uint32_t level, uint32_t count, const uint64_t *const *c0s,
                             const uint64_t *const *digs, const uint32_t *g, const uint64_t *const *keys,
                             uint64_t *const *accs, bool sum_all, bool accumulate);

// encoding (encode.hip)
struct SlotSource {
    // explicit slots: re/im [batch][N/2] (im may be null)
    const double *re = nullptr, *im = nullptr;
    // or the projection's weight plaintexts, generated from W (d_in x d_out, row-major):
    // plaintext p of the batch is (output block j0 + p / pairs, pair ib0 + p % pairs), where
    // pair = i * bcount + b names input block i and baby step b of giant step g (n1g = n1 * g)
    const double *W = nullptr;
    uint32_t d_out = 0, tokens = 0, feats = 0;
    uint32_t n1g = 0, bcount = 0;
    uint32_t j0 = 0, ib0 = 0, pairs = 1;
    // optional, for feats <= 256 and N >= 2^12: W re-laid as its cyclic diagonals,
    // Wd[((jb * n_in + i) * D + k) * D + o] = D_k(A_{jb,i})[o], and feat_of_pos[x] = (slot at FFT position x) / tokens
    const double *Wd = nullptr;
    const uint32_t *feat_of_pos = nullptr;
    uint32_t n_in = 0;
};
// m_out: [batch][N] int64 rounded coefficients; work: [batch][N/2] double2
ckks_status enc_coeffs(ckks_ctx *ctx, const SlotSource &src, uint32_t batch, double scale, double2 *work,
                       int64_t *m_out);
// encoding of a projection sub-batch fused with the first NTT pass (N = 2^16, fp64 primes 0..limbs-1):
// FFT pass A into work, then pass B, twist, rounding and the column transforms of every limb in one kernel;
// out: [batch][limbs][N] in the inter-pass form of launch_ntt_col_i64
bool enc_fused_ok(const ckks_ctx *ctx, uint32_t limbs);
// bound below which the fp64 range reduction modulo every prime q_0 .. q_{limbs-1} is the identity
int64_t identity_reduction_bound(const ckks_ctx *ctx, uint32_t limbs);
ckks_status enc_ntt_first_pass(ckks_ctx *ctx, const SlotSource &src, uint32_t batch, double scale, double2 *work,
                               uint32_t limbs, uint64_t *out);
// out[x] = (slot index held at FFT position x) / tokens, x < N/2
ckks_status enc_feat_of_pos(ckks_ctx *ctx, uint32_t tokens, uint32_t *out);
// residues of m ([batch][N]) into out ([batch][limbs][N]), primes 0..limbs-1
ckks_status enc_to_rns(ckks_ctx *ctx, const int64_t *m, uint32_t batch, uint32_t limbs, uint64_t *out);
size_t enc_work_bytes(const ckks_ctx *ctx, uint32_t batch);
size_t proj_workspace_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t tokens, uint32_t d_in, uint32_t d_out,
                            uint32_t n1);
size_t proj_tm_workspace_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t tokens, uint32_t d_in, uint32_t d_out,
                               uint32_t n1);
size_t attn_scores_workspace_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t tokens, uint32_t head_dim);
size_t attn_apply_workspace_bytes(const ckks_ctx *ctx, uint32_t Lp, uint32_t Lv, uint32_t tokens, uint32_t head_dim);

// projection helpers (project.hip): W's cyclic diagonals Wd[((jb * n_in + i) * D + k) * D + o] =
// W[(i D + (k + o) mod D) * d_out + jb D + o]; canonical residues -> the same integers as doubles, in place
ckks_status launch_diag_layout(ckks_ctx *ctx, double *Wd, const double *W, uint32_t D, uint32_t n_in,
                               uint32_t d_out);
ckks_status launch_to_f64(ckks_ctx *ctx, uint64_t *v, size_t words);

// ciphertext-level steps shared by the API calls and the projections (api_ops.hip)
// rotations of one ciphertext sharing a single ModUp; work: ks_scratch_words(level, ks_rot_batch(count))
ckks_status rotate_core(ckks_ctx *ctx, const uint64_t *c, uint32_t level, const int32_t *steps,
                        const uint64_t *const *keys, uint32_t count, uint64_t *const *outs, uint64_t *work,
                        const uint64_t *seeds = nullptr);
// rescale of one ciphertext at level l; work: (2 + 2 l) N words
ckks_status rescale_core(ckks_ctx *ctx, const uint64_t *c, uint32_t l, uint64_t *out, uint64_t *work);
// `count` ciphertexts (at cs + r * stride) rotated by the same step; work: ks_scratch_words(level,
// ks_rot_batch(count), count)
ckks_status rotate_many(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                        int32_t steps, const uint64_t *key, uint64_t *const *outs, uint64_t *work);
// `count` ciphertexts (at cs + r * stride) each rotated by its own step with its own key; one batched ModUp.
// work: ks_scratch_words(ctx, level, ks_rot_batch(count), count) words
ckks_status rotate_each(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                        const int32_t *steps, const uint64_t *const *keys, uint64_t *const *outs, uint64_t *work);
// rescale of `count` contiguous ciphertexts c ([count][2][l+1][N]) into out ([count][2][l][N]);
// work: 2 count (1 + l) N words
ckks_status rescale_many(ckks_ctx *ctx, const uint64_t *c, uint32_t count, uint32_t l, uint64_t *out,
                         uint64_t *work);

// matrix-core multiply-accumulate over residues (project_tm.hip): acc[jj] (+)= sum_kappa Q[kappa][jj] x_kappa for
// jj < jc and the K ciphertexts kappa_base .. kappa_base + K - 1 of a digit layout Xd, per limb l and run x of
// 2^logT positions: Q is [L][D2][K][jc] canonical residues as doubles (D2 runs), acc [jc][2][L][N] canonical.
uint32_t mac_kt_pad(uint32_t kt);
size_t mac_digit_bytes(const ckks_ctx *ctx, uint32_t L, uint32_t kt_pad);
uint32_t mac_max_outputs();
// x2 ([kt][2][L][N] canonical) -> Xd, the digit layout of kt ciphertexts (mac_digit_bytes bytes)
ckks_status launch_xdigits(ckks_ctx *ctx, const uint64_t *x2, int8_t *Xd, uint32_t L, uint32_t kt, uint32_t kt_pad);
ckks_status launch_mac_mfma(ckks_ctx *ctx, uint64_t *acc, const int8_t *Xd, const double *Q, uint32_t jc, uint32_t K,
                            uint32_t kbase, uint32_t kt_pad, uint32_t D2, uint32_t L, uint32_t logT, bool accumulate);
// periodic plaintexts of `count` explicit period vectors U ([count][D]) at scale delta: Q[l][x][pt] (x < 2D) holds
// plaintext pt's NTT values on run x (positions x N/2D ..) modulo q_l, l < L, as doubles
ckks_status launch_enc_vectors(ckks_ctx *ctx, const double *U, uint32_t D, uint32_t count, double delta, uint32_t L,
                               double *Q);

// Lazy sums of rotations (one ModDown per output).  rotate_many_lazy: ciphertext r (at cs + r * stride) rotated by
// `steps` is added to accumulator uacc + r * 2 ext N; rotate_each_lazy: ciphertext r rotated by steps[r], all
// added to the one accumulator uacc.  accumulate = false starts the accumulators.
// work: count * (nd ext + alpha) N words (the ModUp digits)
ckks_status rotate_many_lazy(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                             int32_t steps, const uint64_t *key, uint64_t *uacc, bool accumulate, uint64_t *work);
ckks_status rotate_each_lazy(ckks_ctx *ctx, const uint64_t *cs, size_t stride, uint32_t count, uint32_t level,
                             const int32_t *steps, const uint64_t *const *keys, uint64_t *uacc, bool accumulate,
                             uint64_t *work);
size_t lazy_work_words(const ckks_ctx *ctx, uint32_t level, uint32_t count);

// decode: coef = coefficient form of limbs 0..min(limbs,2)-1 ([limbs][N]); writes N/2 slots
ckks_status dec_slots(ckks_ctx *ctx, const uint64_t *coef, uint32_t limbs, double scale, double2 *work, double *re,
                      double *im);
