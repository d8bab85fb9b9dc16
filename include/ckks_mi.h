/*
 * ckks_mi.h -- C ABI of libckks_mi.so: RNS-CKKS arithmetic under the packed
 * ciphertext x plaintext linear projection, on one AMD Instinct MI355X (gfx950).
 *
 * The paper (Background, "The CKKS Computation Model") uses the primitives
 * Encode, Add, PCMult, Mult, Rot_k, KeySwitch and Rescale; its projections
 * evaluate Ax = sum_k D_k(A) * rho^k(x) over slot vectors (Section "Matrix
 * Representations and Linear Computation in CKKS", Eq. slot-diagonal-matvec)
 * with baby-step/giant-step reuse of rotations.  The calls below are those
 * primitives plus the projection itself.  Internals follow the standard RNS
 * form of CKKS with hybrid key switching.
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory.  Every pointer named dev_* or held in a ckks_buf is device memory
 *   owned by the caller.  The library owns only its context tables and a
 *   grow-only scratch arena inside the context.  Nothing is freed behind the
 *   caller's back.
 * Layout.  A polynomial is a [limbs][N] array of uint64 residues, limb-major;
 *   limb k of a ciphertext or plaintext is reduced modulo q_k and stored in
 *   the NTT domain: index j holds a(psi_k^(2*brev(j)+1)) mod q_k, where psi_k
 *   is the context's primitive 2N-th root for q_k (ckks_ctx_tables).  Every
 *   stored residue is canonical, in [0, q_k).  A ciphertext is [2][limbs][N]
 *   (c0 then c1); its level is limbs - 1.
 * Streams.  Calls are asynchronous on the context's HIP stream and validate
 *   all arguments on the host before the first launch.  Calls that return
 *   data to the host say so.
 * Errors.  Every call returns a ckks_status; on failure nothing has been
 *   launched unless the status is CKKS_EHIP, and ckks_last_error() describes
 *   the problem (thread-local, valid until the next call on the thread).  No
 *   C++ exception crosses this boundary.
 * Threads.  A context may be used by one host thread at a time.
 */
#ifndef CKKS_MI_H
#define CKKS_MI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ckks_ctx ckks_ctx;

typedef enum {
    CKKS_OK = 0,
    CKKS_EINVAL = -1,      /* bad argument: null pointer, shape, range */
    CKKS_ELEVEL = -2,      /* operand levels do not match or level too low */
    CKKS_ESCALE = -3,      /* operand scales differ where they must be equal */
    CKKS_ENOKEY = -4,      /* no switching key given for a requested rotation */
    CKKS_EHIP = -5,        /* a HIP runtime call failed */
    CKKS_ENOMEM = -6,      /* device or host allocation failed */
    CKKS_EUNSUPPORTED = -7 /* parameters outside what the kernels support */
} ckks_status;

/* Scheme parameters.  N = 2^log_n with 4 <= log_n <= 16.  The modulus chain
 * is q_0..q_{n_q-1}; P = p_0 * ... * p_{n_p-1} are the special primes of
 * hybrid key switching with dnum digits of alpha = ceil(n_q/dnum) limbs
 * (digit j holds q-limbs [j*alpha, min((j+1)*alpha, n_q))).
 * Primes: if q (resp. p) is NULL they are generated: the largest primes
 * below 2^q_bits that are 1 mod 2N, in descending order; q takes the first
 * n_q of that list and p the next n_p of the list for p_bits (skipping any
 * prime already in q).  Every prime must be 1 mod 2N and below 2^62; explicit
 * primes are checked. */
typedef struct {
    uint32_t log_n, n_q, n_p, dnum;
    const uint64_t *q; /* host, n_q entries, or NULL */
    const uint64_t *p; /* host, n_p entries, or NULL */
    uint32_t q_bits, p_bits;
} ckks_params;

/* A plaintext (n_polys = 1) or ciphertext (n_polys = 2): data is
 * [n_polys][n_limbs][N] uint64 on the device, NTT domain, limb k mod q_k. */
typedef struct {
    uint64_t *data;
    uint32_t n_polys, n_limbs;
    double scale;
} ckks_buf;

/* ---- context ------------------------------------------------------------ */

/* Create a context on the current HIP device: generates or checks primes,
 * finds psi_k (x^((q-1)/2N) for the smallest x >= 2 with psi^N = -1), and
 * uploads twiddle, Shoup-companion, FFT and basis-conversion tables (the
 * latter for ModUp and ModDown at every level).
 * hip_stream: the hipStream_t all calls are enqueued on (NULL = default).
 * CKKS_EUNSUPPORTED also when dnum + 1 products of residues below the largest
 * prime exceed an exact 128-bit sum (the integer key inner products): with
 * 62-bit primes dnum is at most 15, below 2^60 at most 255. */
ckks_status ckks_ctx_create(const ckks_params *params, void *hip_stream, ckks_ctx **out);
void ckks_ctx_destroy(ckks_ctx *ctx);
ckks_status ckks_ctx_set_stream(ckks_ctx *ctx, void *hip_stream);
/* Arithmetic of the number-theoretic transforms.  mode 0 (default): fp64
 * butterflies (exact integer-valued doubles with an FMA error term) for every
 * launch whose primes are all below 2^50, 64-bit integer Shoup butterflies
 * otherwise; mode 1: integer Shoup butterflies everywhere.  Both produce
 * identical canonical residues. */
ckks_status ckks_ctx_set_ntt_arith(ckks_ctx *ctx, int mode);
/* Upper bound on the (input ciphertext, baby step) pairs whose weight
 * plaintexts ckks_linear_project encodes and accumulates per launch (0, the
 * default: as many as fit a 24 GiB staging buffer).  Smaller values use less
 * scratch memory and more launches; results are identical for every value. */
ckks_status ckks_ctx_set_proj_batch(ckks_ctx *ctx, uint32_t max_pairs);
/* Lazy ModDown (on = 1; off, the default, = 0): the giant-step rotations of
 * ckks_linear_project and ckks_linear_project_tm and the outer rotation sum of
 * ckks_attention_scores sum their key-switching inner products over Q u P
 * (with P * sigma(c0)) and divide by P once per output instead of once per
 * rotation (the lazy ModDown of a sum of key switches, e.g. Bossuat et al.
 * 2021).  The division rounds once instead of per rotation, so sums before the
 * final rescale differ by small integers per coefficient (at most n_p times
 * half the number of rotations); the outputs, after it, agree with the eager
 * ones except where such a difference crosses a rounding boundary.  Scratch
 * sizes (ckks_workspace_bytes) depend on this setting. */
ckks_status ckks_ctx_set_lazy_moddown(ckks_ctx *ctx, int on);
/* Host copies of the primes q (n_q), p (n_p) and psi (n_q + n_p, q first);
 * any pointer may be NULL. */
ckks_status ckks_ctx_tables(const ckks_ctx *ctx, uint64_t *q, uint64_t *p, uint64_t *psi);

/* Workspace.  Calls that need device scratch memory take it from the
 * context's arena, which the library grows with hipMalloc on demand.  A
 * caller that cannot have the library allocate (graph capture, pooled
 * allocators) hands it a workspace instead: ckks_set_workspace(ctx, dev,
 * bytes) makes dev[0, bytes) (device memory, 256-byte aligned, owned by the
 * caller, which keeps it alive until the context is destroyed or another
 * workspace is set) the arena; the library frees its own arena and never
 * allocates scratch again (every table, including each level's
 * basis-conversion constants, is built by ckks_ctx_create), and a call that
 * needs more than `bytes` fails with CKKS_ENOMEM before any launch.  ckks_set_workspace(ctx, NULL, 0)
 * returns to library-managed scratch.  It synchronizes the context stream
 * first (work in flight may still use the old arena).  All calls on one
 * context share the workspace, so they must be ordered on its stream.
 *
 * ckks_workspace_bytes returns the bytes one call of `op` takes, for the
 * shape given as shape[] (unused entries may be omitted; shape may be NULL
 * where noted), or SIZE_MAX for an unknown op or invalid shape.  The figure
 * for CKKS_OP_LINEAR_PROJECT depends on ckks_ctx_set_proj_batch, and the
 * figures of the projections and the attention scores on
 * ckks_ctx_set_lazy_moddown. */
typedef enum {
    CKKS_OP_NONE = 0,           /* ntt, intt, add, mul_plain, automorph: no workspace */
    CKKS_OP_ENCODE = 1,         /* shape unused */
    CKKS_OP_DECODE = 2,         /* shape[0] = limbs of the plaintext */
    CKKS_OP_ENCRYPT = 3,        /* shape[0] = limbs */
    CKKS_OP_DECRYPT = 4,        /* shape[0] = limbs */
    CKKS_OP_KEYGEN = 5,         /* Galois, relinearisation and seeded keys; shape unused */
    CKKS_OP_RESCALE = 6,        /* shape[0] = limbs of the input */
    CKKS_OP_ROTATE = 7,         /* shape[0] = limbs, shape[1] = rotations of one hoisted call (1: ckks_rotate) */
    CKKS_OP_MUL_RELIN = 8,      /* shape[0] = limbs */
    CKKS_OP_MODUP = 9,          /* shape[0] = level */
    CKKS_OP_MODDOWN = 10,       /* shape[0] = level */
    CKKS_OP_LINEAR_PROJECT = 11, /* shape = {limbs of the inputs, tokens, d_in, d_out, n1} */
    CKKS_OP_LINEAR_PROJECT_TM = 12, /* the same shape */
    CKKS_OP_ATTN_SCORES = 13,   /* shape = {limbs of the inputs, tokens, head_dim} */
    CKKS_OP_ATTN_APPLY = 14     /* shape = {limbs of the scores, limbs of the values, tokens, head_dim} */
} ckks_op;
size_t ckks_workspace_bytes(const ckks_ctx *ctx, int op, const uint32_t *shape);
ckks_status ckks_set_workspace(ckks_ctx *ctx, void *dev, size_t bytes);
/* Galois element 5^steps mod 2N of a left slot rotation by steps (any sign). */
uint32_t ckks_galois_elt(const ckks_ctx *ctx, int32_t steps);
const char *ckks_last_error(void);

/* ---- number-theoretic transforms --------------------------------------- */

/* In-place negacyclic NTT / inverse NTT of dev[batch][n_limbs][N]; row limb k
 * uses prime index limb0 + k of the combined list (q_0..q_{n_q-1},
 * p_0..p_{n_p-1}).  Input and output residues are canonical. */
ckks_status ckks_ntt(ckks_ctx *ctx, uint64_t *dev, uint32_t batch, uint32_t limb0, uint32_t n_limbs);
ckks_status ckks_intt(ckks_ctx *ctx, uint64_t *dev, uint32_t batch, uint32_t limb0, uint32_t n_limbs);

/* ---- encoding ------------------------------------------------------------ */

/* Encode N/2 complex slots (dev_re, dev_im: fp64 device arrays; dev_im may
 * be NULL for real slots) at scale `scale` into pt_out (n_polys = 1, n_limbs
 * limbs, NTT domain).  The integer coefficients are
 *   m_i = round(scale * (2/N) * Re sum_j z_j zeta^(-i 5^j)), zeta = e^(i pi/N),
 * rounding half away from zero, evaluated in fp64 by the radix-2 FFT whose
 * operation order the library fixes (canonical embedding of CKKS).  Every
 * |m_i| must stay below 2^63, which scale * (2/N) * sum_j |z_j| < 2^63
 * guarantees; beyond that the coefficients are unspecified (no error is
 * reported: the slots are not read on the host). */
ckks_status ckks_encode(ckks_ctx *ctx, const double *dev_re, const double *dev_im, double scale,
                        uint32_t n_limbs, ckks_buf *pt_out);
/* Decode pt (n_polys = 1) at pt->scale into N/2 slots written to the device
 * arrays dev_re/dev_im.  Uses the centred lift of limbs 0 and 1 (limb 0
 * alone if the plaintext has one limb), so |m| must be below q_0*q_1/2. */
ckks_status ckks_decode(ckks_ctx *ctx, const ckks_buf *pt, double *dev_re, double *dev_im);

/* ---- encryption (test path) ---------------------------------------------- */

/* Secret-key encryption ct = (-a*s + e + m, a) over the limbs of pt.
 * dev_s: int8 [N] ternary secret (coefficients); dev_a: uint64 [limbs][N]
 * uniform residues, NTT domain; dev_e: int32 [N] error coefficients. */
ckks_status ckks_encrypt_sk(ckks_ctx *ctx, const int8_t *dev_s, const ckks_buf *pt, const uint64_t *dev_a,
                            const int32_t *dev_e, ckks_buf *ct_out);
/* pt = c0 + c1*s over the ciphertext's limbs; pt_out->scale = ct->scale. */
ckks_status ckks_decrypt(ckks_ctx *ctx, const int8_t *dev_s, const ckks_buf *ct, ckks_buf *pt_out);

/* Switching keys, [dnum][2][n_q + n_p][N] uint64 (key_j = (b_j, a_j)):
 *   b_j = -a_j*s + e_j + [P]_{q_i} * t * [i in digit j]  on q-limbs,
 *   b_j = -a_j*s + e_j                                    on p-limbs,
 * with t = sigma_g(s) for a Galois key and t = s^2 for the relinearisation
 * key.  dev_a: [dnum][n_q+n_p][N] NTT domain; dev_e: int32 [dnum][N]. */
ckks_status ckks_keygen_galois(ckks_ctx *ctx, const int8_t *dev_s, uint32_t galois_elt, const uint64_t *dev_a,
                               const int32_t *dev_e, uint64_t *dev_key);
ckks_status ckks_keygen_relin(ckks_ctx *ctx, const int8_t *dev_s, const uint64_t *dev_a, const int32_t *dev_e,
                              uint64_t *dev_key);

/* Seed-expanded switching keys.  The uniform half a_j of a key need not be
 * stored: a seeded key is its b half [dnum][n_q + n_p][N] plus a 128-bit seed
 * (two uint64 words, host memory) from which a is regenerated where it is
 * needed, which halves the key bytes a key switch streams from HBM (the key
 * format of the paper's Background, "The CKKS Computation Model", KeySwitch,
 * with a compressed a half).  Residue n (NTT-domain position) of prime index k
 * (q_0..q_{n_q-1}, then p_0..) in digit j: over the attempts t = 0, 1, ..., the
 * word j mod 4 of the Philox-4x64-10 block (Salmon, Moraes, Dror and Shaw, SC
 * 2011) of counter (n, k, j / 4, t) under the key `seed`, w, gives the
 * candidate w >> (64 - b), b the bit length of the modulus; the first candidate
 * below the modulus is the residue, and after 64 rejections it is w mod the
 * modulus.
 *
 * ckks_expand_key_a writes that a half, [dnum][n_q + n_p][N], to dev_a.
 * ckks_keygen_galois_seeded writes the b half of the Galois key for galois_elt
 * whose a half is the seed's (b_j as in ckks_keygen_galois) to dev_key_b,
 * [dnum][n_q + n_p][N]; scratch as CKKS_OP_KEYGEN.
 * ckks_rotate_hoisted_seeded is ckks_rotate_hoisted with seeded keys:
 * dev_key_b[r] is the b half and seeds[2r], seeds[2r + 1] (host) the seed of
 * rotation r's key; the results equal ckks_rotate_hoisted's with the keys
 * (b, ckks_expand_key_a(seed)) bit for bit.  Errors as for the unseeded calls. */
ckks_status ckks_expand_key_a(ckks_ctx *ctx, const uint64_t *seed, uint64_t *dev_a);
ckks_status ckks_keygen_galois_seeded(ckks_ctx *ctx, const int8_t *dev_s, uint32_t galois_elt, const uint64_t *seed,
                                      const int32_t *dev_e, uint64_t *dev_key_b);
ckks_status ckks_rotate_hoisted_seeded(ckks_ctx *ctx, const ckks_buf *in, const int32_t *steps, uint32_t count,
                                       const uint64_t *const *dev_key_b, const uint64_t *seeds, ckks_buf *outs);

/* ---- homomorphic operations ---------------------------------------------- */

/* Add: equal limbs and bit-identical scales required (CKKS_ELEVEL/ESCALE). */
ckks_status ckks_add(ckks_ctx *ctx, const ckks_buf *a, const ckks_buf *b, ckks_buf *out);
/* PCMult: ct * pt slot-wise; pt needs at least ct's limbs; scale multiplies. */
ckks_status ckks_mul_plain(ckks_ctx *ctx, const ckks_buf *ct, const ckks_buf *pt, ckks_buf *out);
/* Mult + relinearisation: tensor (a0b0, a0b1+a1b0, a1b1), then key switch of
 * a1b1 with dev_rlk; scale multiplies. */
ckks_status ckks_mul_relin(ckks_ctx *ctx, const ckks_buf *a, const ckks_buf *b, const uint64_t *dev_rlk,
                           ckks_buf *out);
/* Rescale: c_i' = (c_i - [centred c_l mod q_l]) * q_l^-1 mod q_i, i < l,
 * i.e. round(c / q_l); out has one limb fewer and scale / q_l. */
ckks_status ckks_rescale(ckks_ctx *ctx, const ckks_buf *in, ckks_buf *out);
/* Rot_steps: left rotation of the slot vector, (rho^k x)_i = x_{i+k}.  The
 * key must be the Galois key for ckks_galois_elt(steps).  out may not alias in. */
ckks_status ckks_rotate(ckks_ctx *ctx, const ckks_buf *in, int32_t steps, const uint64_t *dev_key, ckks_buf *out);
/* count rotations of one ciphertext sharing a single ModUp of c1 (hoisting).
 * Result r equals ckks_rotate(in, steps[r], dev_keys[r]) bit for bit. */
ckks_status ckks_rotate_hoisted(ckks_ctx *ctx, const ckks_buf *in, const int32_t *steps, uint32_t count,
                                const uint64_t *const *dev_keys, ckks_buf *outs);

/* Allocation-free rotation, for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  The operation, arguments and errors are those of ckks_rotate,
 * and the output equals ckks_rotate's bit for bit; this call takes nothing
 * from the context's arena or workspace and calls no allocating routine.
 * Its scratch is a static device buffer of 128 MiB that each device the
 * library runs on holds until the process ends (located when a context is
 * created on that device).  A rotation whose scratch,
 * ckks_workspace_bytes(ctx, CKKS_OP_ROTATE, {limbs, 1}), exceeds 128 MiB fails
 * with CKKS_ENOMEM before any launch (at N = 2^16: up to 256 rows of N words,
 * e.g. 24 + 8 limbs with dnum 3 at every level).  All calls on one device
 * share the buffer, which keeps the last call's contents: calls that overlap
 * on one device (several streams, contexts or threads) race, so the caller
 * orders them.  The library's event profiler does not record this call. */
ckks_status ckks_rotate_noalloc(ckks_ctx *ctx, const ckks_buf *in, int32_t steps, const uint64_t *dev_key,
                                ckks_buf *out);

/* ---- key-switching stages (exposed for per-stage checks) ----------------- */

/* ModUp of dev_c ([level+1][N], NTT domain): for each digit j meeting
 * [0, level], INTT of its limbs, fast basis conversion to the other q-limbs
 * and P (centred digits, uncorrected), NTT.  dev_digits: [n_digits][level+1+n_p][N]
 * (q-limbs 0..level then p-limbs); n_digits = digits with a limb <= level. */
ckks_status ckks_modup(ckks_ctx *ctx, const uint64_t *dev_c, uint32_t level, uint64_t *dev_digits);
/* ModDown of dev_x ([level+1+n_p][N]): (x - NTT(Conv_{P->Q}(INTT([x]_P)))) * P^-1. */
ckks_status ckks_moddown(ckks_ctx *ctx, const uint64_t *dev_x, uint32_t level, uint64_t *dev_out);
/* NTT-domain automorphism sigma_g of rows of N: out[j] = in[j'] with
 * 2 brev(j') + 1 = (2 brev(j) + 1) g mod 2N.  g odd.  out may not alias in. */
ckks_status ckks_automorph(ckks_ctx *ctx, const uint64_t *dev_in, uint32_t rows, uint32_t galois_elt,
                           uint64_t *dev_out);

/* ---- the projection ------------------------------------------------------ */

/* Feature-major packed projection Y = X W (X: tokens x d_in, W: d_in x d_out
 * row-major fp64 on the device).  Slot f*tokens + t of input ciphertext i
 * holds X[t, i*D + f], D = N/2/tokens features per ciphertext; output
 * ciphertext j holds Y[t, j*D + o] at slot o*tokens + t.  With A = W^T and
 * the cyclic diagonals D_k(A_{j,i})[o] = A_{j,i}[o, (o+k) mod D]:
 *   out_j = Rescale( sum_{g<n2} Rot_{T n1 g}( sum_{i,b<n1} pt_{j,i,g,b} * Rot_{T b}(x_i) ) )
 * where pt_{j,i,g,b} encodes at scale q_level the slot vector
 *   p[f*T + t] = D_{n1 g + b}(A_{j,i})[(f - n1 g) mod D],  n2 = ceil(D/n1).
 * Weight plaintexts are encoded on the fly from W (as ckks_encode: their
 * coefficients must stay below 2^63, which q_level * max|W| < 2^63 guarantees
 * since each diagonal holds D distinct weights repeated over T tokens and
 * (2/N) * (N/2) = 1; beyond that they are unspecified).  Keys: key_steps[r] ->
 * dev_keys[r]; steps T*b (0 < b < n1) and T*n1*g (0 < g < n2) must be present.
 * in: d_in/D ciphertexts, all with the same n_limbs = level + 1 >= 2 and the
 * same scale; out: d_out/D ciphertexts with n_limbs = level (the rescale
 * drops q_level) whose scale is set to the input scale (the plaintext scale
 * q_level cancels exactly in the rescale).  Scratch comes from the context's
 * arena or workspace (ckks_workspace_bytes, CKKS_OP_LINEAR_PROJECT). */
typedef struct {
    uint32_t tokens, d_in, d_out, n1;
} ckks_proj_shape;
ckks_status ckks_linear_project(ckks_ctx *ctx, const ckks_buf *in, const double *dev_W, const ckks_proj_shape *shape,
                                const int32_t *key_steps, const uint64_t *const *dev_keys, uint32_t n_keys,
                                ckks_buf *out);

/* The same projection in the token-major layout: slot t*D + f of input
 * ciphertext i holds X[t, i*D + f] (D = N/2/tokens features, a power of two
 * in [4, 256]); output j holds Y[t, j*D + o] at slot t*D + o.  A left
 * rotation by k then moves feature o + k of the same token to feature o only
 * while o + k < D, so each cyclic diagonal is split into the entries that do
 * not wrap (U, multiplying Rot_b(x_i)) and those that do (V, multiplying
 * Rot_{b-D}(x_i)):
 *   out_j = Rescale( sum_g Rot_{n1 g}( sum_{i,b<n1} U_{j,i,g,b} * Rot_b(x_i)
 *                                              + V_{j,i,g,b} * Rot_{b-D}(x_i) ) )
 * with U_{j,i,g,b}[t*D + o] = A_{j,i}[o', o' + k] if o' + k < D (else 0) and
 * V_{j,i,g,b}[t*D + o] = A_{j,i}[o', o' + k - D] if o' + k >= D (else 0),
 * k = n1 g + b, o' = (o - n1 g) mod D.  Every weight plaintext is periodic
 * in the slots (period D), so it is encoded as m'(X^(N/2D)) with m' the
 * encoding of one period at ring degree 2D (the encode's own rounding rule).
 * Keys: steps b (0 < b < n1), b - D (0 <= b < n1) and n1 g (0 < g < n2).
 * Needs every prime below 2^50.  Arguments, scales and errors as for
 * ckks_linear_project; scratch: ckks_workspace_bytes with
 * CKKS_OP_LINEAR_PROJECT_TM. */
ckks_status ckks_linear_project_tm(ckks_ctx *ctx, const ckks_buf *in, const double *dev_W,
                                   const ckks_proj_shape *shape, const int32_t *key_steps,
                                   const uint64_t *const *dev_keys, uint32_t n_keys, ckks_buf *out);

/* ---- attention block (token-major layout) --------------------------------- */

/* Shape of the attention calls: `tokens` tokens per ciphertext (T, a power of
 * two in [16, 128]) and heads of `head_dim` features (hd, a power of two with
 * T <= hd <= D, where D = N/2/T <= 256 features per ciphertext).  Slot
 * t*D + h*hd + d of a ciphertext holds feature d of head h of token t. */
typedef struct {
    uint32_t tokens, head_dim;
} ckks_attn_shape;

/* Attention scores on token diagonals (the scores S_Delta that QK^T produces
 * in the paper's C-Delta layout, Section "C--Delta Attention Layout and
 * Computation" and Table ccmm-performance; the paper gives no construction,
 * this one is QK^T as Mult plus rotation sums).  q: n_q query ciphertexts
 * (D/hd heads each); k: n_k key ciphertexts, each holding one key head
 * repeated in every head position (slot t*D + h*hd + d = K[t, d] for all h);
 * query c uses key k_of_q[c].  Output c holds, at slot t*D + h*hd + delta,
 *   S[t, h, delta] = sum_d Q[t, h, d] K[(t + delta) mod T, d]   (delta < T)
 * and 0 for T <= delta < hd, computed as
 *   P_delta = Relin(Rot_{-delta}(Q) x Rot_{delta(D-1)}(K'))
 *   out = Rescale(Rescale(sum_{k<hd} Rot_k(sum_delta M_{(delta+k) mod hd} * P_delta)))
 * with M_c the 0/1 mask of head position c, a periodic plaintext at scale
 * q_level.  Inputs: n_limbs = level + 1 >= 3, equal within q and within k,
 * equal scales within each; out[c]: n_limbs = level - 1, scale set to
 * scale(q) scale(k) / q_(level-1).  Keys (Galois, key_steps[r] -> dev_keys[r]):
 * steps -delta and delta (D-1) for 0 < delta < T, and 1 .. hd-1; dev_rlk: the
 * relinearisation key.  All device memory is the caller's; scratch from the
 * arena or workspace (CKKS_OP_ATTN_SCORES).  Errors: CKKS_EINVAL (shapes,
 * k_of_q out of range, output descriptors), CKKS_EUNSUPPORTED (token count,
 * primes of 50 bits or more, no special primes), CKKS_ELEVEL, CKKS_ESCALE,
 * CKKS_ENOKEY; all checked before any launch. */
ckks_status ckks_attention_scores(ckks_ctx *ctx, const ckks_buf *q, uint32_t n_q, const ckks_buf *k, uint32_t n_k,
                                  const uint32_t *k_of_q, const ckks_attn_shape *shape, const uint64_t *dev_rlk,
                                  const int32_t *key_steps, const uint64_t *const *dev_keys, uint32_t n_keys,
                                  ckks_buf *out);

/* Weighted sums of values consuming scores in the layout ckks_attention_scores
 * writes (the paper's PV consuming P_Delta, same sections).  p: n_p score
 * ciphertexts (slot t*D + h*hd + delta = P[t, h, delta] for delta < T; the
 * positions delta >= T are not read); v: n_v value ciphertexts, each holding
 * one value head repeated in every head position; scores c use value
 * v_of_p[c].  Output c holds, at slot t*D + h*hd + d,
 *   O[t, h, d] = sum_{delta<T} P[t, h, delta] V[(t + delta) mod T, d]
 * computed as C_j = Rescale(sum_delta M_{delta-j} * Rot_{delta D}(V')) over
 * 0 <= delta - j < hd (masks at scale q_(level of v), C_j then kept on the
 * scores' limbs) and out = Rescale(Relin(sum_{-hd<j<T} Rot_j(P) x C_j)).
 * The scores' level must be below the values': 2 <= p.n_limbs < v.n_limbs;
 * out[c]: n_limbs = p.n_limbs - 1, scale set to scale(p) scale(v) / q_(level
 * of p).  Keys: steps delta D (0 < delta < T) and j (-hd < j < T, j != 0);
 * dev_rlk as above; scratch: CKKS_OP_ATTN_APPLY; errors as above. */
ckks_status ckks_attention_apply(ckks_ctx *ctx, const ckks_buf *p, uint32_t n_p, const ckks_buf *v, uint32_t n_v,
                                 const uint32_t *v_of_p, const ckks_attn_shape *shape, const uint64_t *dev_rlk,
                                 const int32_t *key_steps, const uint64_t *const *dev_keys, uint32_t n_keys,
                                 ckks_buf *out);

/* ---- measurement helpers ------------------------------------------------- */

/* Per-kernel timing with HIP events on the context stream.  While enabled,
 * every kernel launch is bracketed by two events and tagged with its
 * algorithmic HBM bytes (each input and output word once; cache-resident
 * tables excluded) and its nominal VALU lane instructions (the kernel's
 * arithmetic model: 11 per fp64 butterfly, 37 per integer one, plus the
 * stated extra work; 0 where no model is given).  ckks_profile_read
 * synchronizes and returns, for the kernel named `kernel`, the summed
 * milliseconds, launch count, bytes and VALU instructions (any output pointer
 * may be NULL).  ckks_profile_name(i) enumerates the kernel names (NULL past
 * the last). */
ckks_status ckks_profile_enable(ckks_ctx *ctx, int on);
ckks_status ckks_profile_read(ckks_ctx *ctx, const char *kernel, double *total_ms, uint64_t *launches,
                              double *bytes, double *valu_ops);
ckks_status ckks_profile_reset(ckks_ctx *ctx);
const char *ckks_profile_name(int i);
/* A plain device copy of `bytes` bytes (multiple of 16, at most 8 TiB) on the context
 * stream, for calibrating HBM counters and achievable bandwidth: one 16-byte word per
 * thread with nontemporal loads and stores, the fastest copy shape measured on gfx950. */
ckks_status ckks_calib_copy(ckks_ctx *ctx, void *dev_dst, const void *dev_src, size_t bytes);
/* Modular-multiply throughput probe: `iters` dependent-chain multiplications
 * per lane on `lanes` lanes, mode 0 = integer Shoup (64-bit, built from 32-bit
 * multiplies), mode 1 = fp64 fused-multiply-add reduction.  Writes one value
 * per lane to dev_out (uint64 [lanes]) so the work cannot be elided. */
ckks_status ckks_calib_modmul(ckks_ctx *ctx, uint64_t *dev_out, uint32_t lanes, uint32_t iters, int mode);

#ifdef __cplusplus
}
#endif
#endif /* CKKS_MI_H */
