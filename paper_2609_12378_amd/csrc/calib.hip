// Calibration kernels: a plain copy (achievable HBM bandwidth, and the scale
// factor between hardware traffic counters and bytes moved) and a modular
// multiply throughput probe comparing the integer Shoup product with an fp64
// fused-multiply-add reduction on gfx950.
#include "ckks_internal.h"

namespace {

// One 16-byte word per thread, consecutive blocks on consecutive 4 KiB, nontemporal loads and stores: of the copy
// shapes measured on gfx950 (grid-stride loops, several words in flight per thread, with and without the hint)
// the fastest, so the copy rate it gives is the practical HBM ceiling rather than a property of one loop shape.
__global__ __launch_bounds__(256) void copy_kernel(uint4 *__restrict__ dst, const uint4 *__restrict__ src, size_t n16)
{
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n16) __builtin_nontemporal_store(__builtin_nontemporal_load((const v4u *)src + i), (v4u *)dst + i);
}

// Integer Shoup: a <- a*w mod q, eight independent chains per lane.
__global__ __launch_bounds__(256) void modmul_int_kernel(uint64_t *out, uint32_t lanes, uint32_t iters, uint64_t q,
                                                          uint64_t w, uint64_t ws)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= lanes) return;
    uint64_t a[8];
#pragma unroll
    for (int k = 0; k < 8; k++) a[k] = (i * 8 + k) % q;
    for (uint32_t it = 0; it < iters; it++) {
#pragma unroll
        for (int k = 0; k < 8; k++) a[k] = shoup_lazy(a[k], w, ws, q);
    }
    uint64_t s = 0;
#pragma unroll
    for (int k = 0; k < 8; k++) s ^= a[k];
    out[i] = s;
}

// fp64: q < 2^50, residues held as exact doubles.  h + l = a*w exactly (FMA
// error term), c = rint(h / q) estimated with a precomputed reciprocal, the
// remainder h - c q computed exactly by FMA; result in (-q, q).
__global__ __launch_bounds__(256) void modmul_f64_kernel(uint64_t *out, uint32_t lanes, uint32_t iters, double q,
                                                          double w, double qinv)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= lanes) return;
    double a[8];
#pragma unroll
    for (int k = 0; k < 8; k++) a[k] = (double)((i * 8 + k) % 1000003);
    for (uint32_t it = 0; it < iters; it++) {
#pragma unroll
        for (int k = 0; k < 8; k++) {
            const double h = a[k] * w;
            const double l = fma(a[k], w, -h);
            const double c = rint(h * qinv);
            double r = fma(-c, q, h) + l;
            r = r < 0.0 ? r + q : r;
            a[k] = r;
        }
    }
    uint64_t s = 0;
#pragma unroll
    for (int k = 0; k < 8; k++) s ^= (uint64_t)a[k];
    out[i] = s;
}

}  // namespace

extern "C" ckks_status ckks_calib_copy(ckks_ctx *ctx, void *dst, const void *src, size_t bytes)
{
    clear_error();
    CK_REQUIRE(ctx && dst && src, CKKS_EINVAL, "calib_copy: null argument");
    CK_REQUIRE(bytes % 16 == 0, CKKS_EINVAL, "calib_copy: %zu bytes is not a multiple of 16", bytes);
    const size_t n16 = bytes / 16;
    if (!n16) return CKKS_OK;
    const size_t blocks = (n16 + 255) / 256;
    CK_REQUIRE(blocks <= 0x7fffffffu, CKKS_EINVAL, "calib_copy: %zu bytes is too large for one launch", bytes);
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, ctx->stream, (uint4 *)dst,
                       (const uint4 *)src, n16);
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}

extern "C" ckks_status ckks_calib_modmul(ckks_ctx *ctx, uint64_t *out, uint32_t lanes, uint32_t iters, int mode)
{
    clear_error();
    CK_REQUIRE(ctx && out && lanes, CKKS_EINVAL, "calib_modmul: bad argument");
    const dim3 grid((lanes + 255) / 256), block(256);
    if (mode == 0) {
        const uint64_t q = ctx->primes[0], w = q / 3 + 7;
        const uint64_t ws = (uint64_t)(((unsigned __int128)w << 64) / q);
        hipLaunchKernelGGL(modmul_int_kernel, grid, block, 0, ctx->stream, out, lanes, iters, q, w, ws);
    } else {
        CK_REQUIRE(ctx->primes[0] < (1ull << 50), CKKS_EUNSUPPORTED, "fp64 probe needs q_0 < 2^50");
        const double q = (double)ctx->primes[0];
        hipLaunchKernelGGL(modmul_f64_kernel, grid, block, 0, ctx->stream, out, lanes, iters, q,
                           (double)(ctx->primes[0] / 3), 1.0 / q);
    }
    HIP_TRY(hipGetLastError());
    return CKKS_OK;
}
