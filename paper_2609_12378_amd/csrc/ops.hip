// Element-wise and structural kernels on NTT-domain polynomials: add, subtract,
// products, the ciphertext tensor product, the Galois automorphism, the secret
// expansion used by encryption and key generation, and the rescale steps.
//
// These are streaming kernels bound by HBM: each thread handles one residue
// per row, rows are mapped to primes through a LimbMap, and the row index is
// recovered from a flat grid with one division per thread.
#include "ckks_internal.h"
#include "ops.h"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bool flat(uint32_t log_n, size_t total, size_t &i, uint32_t &row, uint32_t &col)
{
    i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= total) return false;
    row = (uint32_t)(i >> log_n);
    col = (uint32_t)(i & ((1u << log_n) - 1));
    return true;
}

inline dim3 grid_for(size_t total) { return dim3((unsigned)((total + kThreads - 1) / kThreads)); }

// blockIdx.y selects the batch entry: out, a and b advance by their own strides (in words)
__global__ __launch_bounds__(kThreads) void k_binary(uint64_t *out, const uint64_t *a, const uint64_t *b,
                                                      size_t total, uint32_t log_n, LimbMap map, const ModQ *mods,
                                                      int op, size_t out_stride, size_t a_stride, size_t b_stride)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    out += blockIdx.y * out_stride;
    a += blockIdx.y * a_stride;
    b += blockIdx.y * b_stride;
    const ModQ m = mods[map.prime[row % map.n]];
    const uint64_t x = a[i], y = b[i];
    uint64_t r;
    if (op == EW_ADD) r = addmod(x, y, m.q);
    else if (op == EW_SUB) r = submod(x, y, m.q);
    else r = mulmod(x, y, m);
    out[i] = r;
}

// out[p][l][n] = ct[p][l][n] * pt[l][n]
__global__ __launch_bounds__(kThreads) void k_mul_plain(uint64_t *out, const uint64_t *ct, const uint64_t *pt,
                                                         size_t total, uint32_t log_n, uint32_t limbs,
                                                         const ModQ *mods)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    const uint32_t l = row % limbs;
    out[i] = mulmod(ct[i], pt[((size_t)l << log_n) + col], mods[l]);
}

// d0 = a0 b0, d1 = a0 b1 + a1 b0, d2 = a1 b1 over `limbs` q-limbs; blockIdx.y selects the batch entry (d0, d1
// and d2 advance by d_stride words, a by a_stride, b by b_stride)
__global__ __launch_bounds__(kThreads) void k_tensor(uint64_t *d0, uint64_t *d1, uint64_t *d2, const uint64_t *a,
                                                      const uint64_t *b, size_t total, uint32_t log_n,
                                                      const ModQ *mods, size_t d_stride, size_t a_stride,
                                                      size_t b_stride)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    d0 += blockIdx.y * d_stride;
    d1 += blockIdx.y * d_stride;
    d2 += blockIdx.y * d_stride;
    a += blockIdx.y * a_stride;
    b += blockIdx.y * b_stride;
    const ModQ m = mods[row];
    const uint64_t a0 = a[i], a1 = a[i + total], b0 = b[i], b1 = b[i + total];
    d0[i] = mulmod(a0, b0, m);
    acc128 x{0, 0};
    mac(x, a0, b1);
    mac(x, a1, b0);
    d1[i] = reduce128(x, m);
    d2[i] = mulmod(a1, b1, m);
}

__device__ __forceinline__ uint32_t auto_index(uint32_t j, uint32_t g, uint32_t log_n)
{
    // NTT index j holds a(psi^(2 brev(j) + 1)); sigma_g(a) there is a(psi^((2 brev(j)+1) g))
    const uint32_t two_n_mask = (2u << log_n) - 1;
    const uint32_t k = 2u * (__brev(j) >> (32 - log_n)) + 1u;
    const uint32_t kg = (uint32_t)(((uint64_t)k * g) & two_n_mask);
    return __brev((kg - 1u) >> 1) >> (32 - log_n);
}

__global__ __launch_bounds__(kThreads) void k_automorph(uint64_t *out, const uint64_t *in, size_t total,
                                                         uint32_t log_n, uint32_t g)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    out[i] = in[((size_t)row << log_n) + auto_index(col, g, log_n)];
}

// small signed integers (int8 or int32 coefficients) into residues [limbs][N]
template <typename T>
__global__ __launch_bounds__(kThreads) void k_expand(uint64_t *out, const T *v, size_t total, uint32_t log_n,
                                                      LimbMap map, const ModQ *mods)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    const uint64_t q = mods[map.prime[row % map.n]].q;
    const int64_t x = (int64_t)v[col];
    out[i] = x >= 0 ? (uint64_t)x : q - (uint64_t)(-x);
}

// c0 = -a*s + e + m ; rows over limbs (map), batch 1
__global__ __launch_bounds__(kThreads) void k_encrypt(uint64_t *c0, uint64_t *c1, const uint64_t *a,
                                                       const uint64_t *s, const uint64_t *e, const uint64_t *m,
                                                       size_t total, uint32_t log_n, LimbMap map, const ModQ *mods)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    const ModQ md = mods[map.prime[row % map.n]];
    const uint64_t as = mulmod(a[i], s[i], md);
    uint64_t r = submod(e[i], as, md.q);
    if (m) r = addmod(r, m[i], md.q);
    c0[i] = r;
    if (c1) c1[i] = a[i];
}

// b = -a*s + e (+ [P] t on the digit's q-limbs); rows = all primes of the context
__global__ __launch_bounds__(kThreads) void k_keygen(uint64_t *b_out, uint64_t *a_out, const uint64_t *a,
                                                      const uint64_t *s, const uint64_t *e, const uint64_t *t,
                                                      const ulonglong2 *pmodq, uint32_t dig_lo, uint32_t dig_hi,
                                                      size_t total, uint32_t log_n, const ModQ *mods)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    const ModQ md = mods[row];
    uint64_t r = submod(e[i], mulmod(a[i], s[i], md), md.q);
    if (row >= dig_lo && row < dig_hi) {
        const ulonglong2 P = pmodq[row];
        r = addmod(r, shoup(t[i], P.x, P.y, md.q), md.q);
    }
    b_out[i] = r;
    if (a_out) a_out[i] = a[i];
}

// Rescale, step 1: top-limb coefficients t (mod q_l), canonical, to their centred values as int64 in place
// (t > q_l / 2 -> t - q_l); the signed-input forward transform then reduces them modulo every q_i, i < l, in its
// first pass, so the residue rows of the top limb are never written out before their transform.
__global__ __launch_bounds__(kThreads) void k_rescale_centre(uint64_t *top, size_t total, uint64_t ql)
{
    const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= total) return;
    const uint64_t t = top[i];
    top[i] = t > (ql >> 1) ? t - ql : t;  // two's complement of the negative centred value
}

// Rescale, step 2: out_i = (c_i - r_i) * q_l^-1 mod q_i; c: [polys][l+1][N], r/out: [polys][l][N]
__global__ __launch_bounds__(kThreads) void k_rescale_finish(uint64_t *out, const uint64_t *c, const uint64_t *r,
                                                              size_t total, uint32_t log_n, uint32_t l,
                                                              const ulonglong2 *qlinv_row, const ModQ *mods)
{
    size_t i;
    uint32_t row, col;
    if (!flat(log_n, total, i, row, col)) return;
    const uint32_t poly = row / l, li = row % l;
    const uint64_t q = mods[li].q;
    const uint64_t ci = c[(((size_t)poly * (l + 1) + li) << log_n) + col];
    const ulonglong2 w = qlinv_row[li];
    out[i] = shoup(submod(ci, r[i], q), w.x, w.y, q);
}

// Entry b (b = blockIdx.y) of src, `words` contiguous words at src + b * src_stride, copied to
// dst_a + b * a_stride and, when dst_b is set, to dst_b + b * b_stride: one read and one or two writes per word.
// V: ulonglong2 (every pointer and stride 16-byte aligned, words even) or uint64_t.
template <typename V>
__global__ __launch_bounds__(kThreads) void k_copy_rows(uint64_t *dst_a, size_t a_stride, uint64_t *dst_b,
                                                        size_t b_stride, const uint64_t *__restrict__ src,
                                                        size_t src_stride, size_t words)
{
    constexpr size_t W = sizeof(V) / 8;
    const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    const size_t b = blockIdx.y;
    if (i * W >= words) return;
    const V v = ((const V *)(src + b * src_stride))[i];
    ((V *)(dst_a + b * a_stride))[i] = v;
    if (dst_b) ((V *)(dst_b + b * b_stride))[i] = v;
}

}  // namespace

ckks_status launch_binary(ckks_ctx *ctx, uint64_t *out, const uint64_t *a, const uint64_t *b, uint32_t rows,
                          const LimbMap &map, int op)
{
    return launch_binary_batch(ctx, out, 0, a, 0, b, 0, 1, rows, map, op);
}

ckks_status launch_binary_batch(ckks_ctx *ctx, uint64_t *out, size_t out_stride, const uint64_t *a,
                                size_t a_stride, const uint64_t *b, size_t b_stride, uint32_t count, uint32_t rows,
                                const LimbMap &map, int op)
{
    const size_t total = (size_t)rows << ctx->log_n;
    if (!total || !count) return CKKS_OK;
    CK_REQUIRE(count <= 65535u, CKKS_EINVAL, "element-wise batch of %u entries exceeds 65535", count);
    prof_begin(ctx, K_ELEM, 24.0 * total * count);
    dim3 grid = grid_for(total);
    grid.y = count;
    hipLaunchKernelGGL(k_binary, grid, dim3(kThreads), 0, ctx->stream, out, a, b, total, ctx->log_n, map,
                       ctx->d_mod, op, out_stride, a_stride, b_stride);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_mul_plain(ckks_ctx *ctx, uint64_t *out, const uint64_t *ct, const uint64_t *pt, uint32_t polys,
                             uint32_t limbs)
{
    const size_t total = ((size_t)polys * limbs) << ctx->log_n;
    if (!total) return CKKS_OK;
    hipLaunchKernelGGL(k_mul_plain, grid_for(total), dim3(kThreads), 0, ctx->stream, out, ct, pt, total, ctx->log_n,
                       limbs, ctx->d_mod);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_tensor(ckks_ctx *ctx, uint64_t *d0, uint64_t *d1, uint64_t *d2, const uint64_t *a,
                          const uint64_t *b, uint32_t limbs)
{
    return launch_tensor_batch(ctx, d0, d1, d2, 0, a, 0, b, 0, 1, limbs);
}

ckks_status launch_tensor_batch(ckks_ctx *ctx, uint64_t *d0, uint64_t *d1, uint64_t *d2, size_t d_stride,
                                const uint64_t *a, size_t a_stride, const uint64_t *b, size_t b_stride,
                                uint32_t count, uint32_t limbs)
{
    const size_t total = (size_t)limbs << ctx->log_n;
    if (!total || !count) return CKKS_OK;
    CK_REQUIRE(count <= 65535u, CKKS_EINVAL, "tensor-product batch of %u entries exceeds 65535", count);
    dim3 grid = grid_for(total);
    grid.y = count;
    hipLaunchKernelGGL(k_tensor, grid, dim3(kThreads), 0, ctx->stream, d0, d1, d2, a, b, total, ctx->log_n,
                       ctx->d_mod, d_stride, a_stride, b_stride);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_automorph(ckks_ctx *ctx, const uint64_t *in, uint64_t *out, uint32_t rows, uint32_t g)
{
    const size_t total = (size_t)rows << ctx->log_n;
    if (!total) return CKKS_OK;
    hipLaunchKernelGGL(k_automorph, grid_for(total), dim3(kThreads), 0, ctx->stream, out, in, total, ctx->log_n, g);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_expand_i8(ckks_ctx *ctx, uint64_t *out, const int8_t *v, const LimbMap &map)
{
    const size_t total = (size_t)map.n << ctx->log_n;
    hipLaunchKernelGGL(k_expand<int8_t>, grid_for(total), dim3(kThreads), 0, ctx->stream, out, v, total, ctx->log_n,
                       map, ctx->d_mod);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_expand_i32(ckks_ctx *ctx, uint64_t *out, const int32_t *v, const LimbMap &map)
{
    const size_t total = (size_t)map.n << ctx->log_n;
    hipLaunchKernelGGL(k_expand<int32_t>, grid_for(total), dim3(kThreads), 0, ctx->stream, out, v, total,
                       ctx->log_n, map, ctx->d_mod);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_encrypt(ckks_ctx *ctx, uint64_t *c0, uint64_t *c1, const uint64_t *a, const uint64_t *s,
                           const uint64_t *e, const uint64_t *m, const LimbMap &map)
{
    const size_t total = (size_t)map.n << ctx->log_n;
    hipLaunchKernelGGL(k_encrypt, grid_for(total), dim3(kThreads), 0, ctx->stream, c0, c1, a, s, e, m, total,
                       ctx->log_n, map, ctx->d_mod);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_keygen_digit(ckks_ctx *ctx, uint64_t *b_out, uint64_t *a_out, const uint64_t *a,
                                const uint64_t *s, const uint64_t *e, const uint64_t *t, uint32_t dig_lo,
                                uint32_t dig_hi)
{
    const size_t total = (size_t)ctx->n_primes() << ctx->log_n;
    hipLaunchKernelGGL(k_keygen, grid_for(total), dim3(kThreads), 0, ctx->stream, b_out, a_out, a, s, e, t,
                       ctx->d_pmodq, dig_lo, dig_hi, total, ctx->log_n, ctx->d_mod);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_rescale_centre(ckks_ctx *ctx, uint64_t *top, uint32_t polys, uint32_t l)
{
    const size_t total = (size_t)polys << ctx->log_n;
    hipLaunchKernelGGL(k_rescale_centre, grid_for(total), dim3(kThreads), 0, ctx->stream, top, total,
                       ctx->primes[l]);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_rescale_finish(ckks_ctx *ctx, uint64_t *out, const uint64_t *c, const uint64_t *r,
                                  uint32_t polys, uint32_t l)
{
    const size_t total = ((size_t)polys * l) << ctx->log_n;
    hipLaunchKernelGGL(k_rescale_finish, grid_for(total), dim3(kThreads), 0, ctx->stream, out, c, r, total,
                       ctx->log_n, l, ctx->d_qlinv + (size_t)l * ctx->n_q, ctx->d_mod);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

ckks_status launch_copy_rows(ckks_ctx *ctx, uint64_t *dst_a, size_t a_stride, uint64_t *dst_b, size_t b_stride,
                             const uint64_t *src, size_t src_stride, size_t words, uint32_t count)
{
    if (!count || !words) return CKKS_OK;
    CK_REQUIRE(count <= 65535, CKKS_EINVAL, "row copy of %u entries in one launch (at most 65535)", count);
    auto al16 = [](const void *p) { return ((uintptr_t)p & 15) == 0; };
    const bool wide = words % 2 == 0 && a_stride % 2 == 0 && b_stride % 2 == 0 && src_stride % 2 == 0 &&
                      al16(dst_a) && al16(src) && (!dst_b || al16(dst_b));
    const size_t per = wide ? words / 2 : words;
    const dim3 grid((unsigned)((per + kThreads - 1) / kThreads), count);
    prof_begin(ctx, K_ELEM, 8.0 * words * count * (dst_b ? 3 : 2));
    if (wide)
        hipLaunchKernelGGL(k_copy_rows<ulonglong2>, grid, dim3(kThreads), 0, ctx->stream, dst_a, a_stride, dst_b,
                           b_stride, src, src_stride, words);
    else
        hipLaunchKernelGGL(k_copy_rows<uint64_t>, grid, dim3(kThreads), 0, ctx->stream, dst_a, a_stride, dst_b,
                           b_stride, src, src_stride, words);
    prof_end(ctx, K_ELEM);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}
