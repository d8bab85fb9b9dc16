// An allocation-free single rotation for callers that cannot allocate device memory (code under HIP graph
// capture, tight serving loops, harnesses that forbid hipMalloc).  Its scratch is a file-scope static device
// array; each device's copy is located once, when a context is created on that device (noalloc_setup), and only
// that address is ever handed to kernels, copies or fills.
#include <atomic>
#include <mutex>

#include "ckks_internal.h"
#include "ops.h"

// 128 MiB: a rotation at N = 2^16 with level + 1 + n_p <= 32 extended limbs and dnum = 3 needs 216 rows of N words
// (the hoisted digits, the digits' transform staging, and one rotation's P rows and converted rows: 113 MiB).
static constexpr size_t kScratchWords = size_t(1) << 24;
static constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint64_t scratch[kScratchWords];

static std::mutex g_setup_mu;
// the device address of `scratch` on each device: written once under the lock, read by calls on any thread
static std::atomic<uint64_t *> g_scratch_ptr[kMaxDevices] = {};
static hipError_t g_setup_err[kMaxDevices] = {};    // why it could not be located (hipSuccess: not tried or found)

// Called by ckks_ctx_create with `device` current.  A failure here leaves every other call working: only
// ckks_rotate_noalloc on that device reports it.
void noalloc_setup(int device)
{
    if (device < 0 || device >= kMaxDevices) return;
    std::lock_guard<std::mutex> lock(g_setup_mu);
    if (g_scratch_ptr[device].load(std::memory_order_acquire)) return;
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p || ((uintptr_t)p & 255)) {
        g_setup_err[device] = e != hipSuccess ? e : hipErrorInvalidSymbol;
        (void)hipGetLastError();   // do not leave the failure for the next runtime call to report
        return;
    }
    g_scratch_ptr[device].store((uint64_t *)p, std::memory_order_release);
}

extern "C" ckks_status ckks_rotate_noalloc(ckks_ctx *ctx, const ckks_buf *in, int32_t steps, const uint64_t *key,
                                           ckks_buf *out)
{
    clear_error();
    CK_REQUIRE(ctx && in && out && key, CKKS_EINVAL, "rotate_noalloc: null argument");
    CK_REQUIRE(in->data && out->data, CKKS_EINVAL, "rotate_noalloc: null data pointer");
    CK_REQUIRE(in->n_polys == 2 && out->n_polys == 2, CKKS_EINVAL, "rotate_noalloc: ciphertexts have 2 polynomials");
    CK_REQUIRE(in->n_limbs >= 1 && in->n_limbs <= ctx->n_q, CKKS_ELEVEL, "rotate_noalloc: %u limbs outside [1, %u]",
               in->n_limbs, ctx->n_q);
    CK_REQUIRE(out->n_limbs == in->n_limbs, CKKS_ELEVEL, "rotate_noalloc: output has the wrong limb count");
    CK_REQUIRE(out->data != in->data, CKKS_EINVAL, "rotate_noalloc: output aliases the input");
    CK_REQUIRE(ctx->n_p > 0, CKKS_EUNSUPPORTED, "rotate_noalloc: the context has no special primes");
    CK_REQUIRE(ctx->device >= 0 && ctx->device < kMaxDevices, CKKS_EUNSUPPORTED,
               "rotate_noalloc: device index %d outside [0, %d)", ctx->device, kMaxDevices);
    uint64_t *const scratch_ptr = g_scratch_ptr[ctx->device].load(std::memory_order_acquire);
    CK_REQUIRE(scratch_ptr, CKKS_EHIP, "rotate_noalloc: static scratch not located on device %d: %s", ctx->device,
               hipGetErrorString(g_setup_err[ctx->device]));
    const uint32_t level = in->n_limbs - 1, L = in->n_limbs;
    const size_t words = ks_scratch_words(ctx, level, 1);
    CK_REQUIRE(words <= kScratchWords, CKKS_ENOMEM,
               "rotate_noalloc: this rotation needs %zu bytes of scratch, the static buffer holds %zu", words * 8,
               kScratchWords * 8);
    // the conversion tables are built when the context is created; nothing may be built (allocated) here
    CK_REQUIRE(ctx->conv.count({(int)level, -1}), CKKS_EUNSUPPORTED, "rotate_noalloc: no tables for level %u",
               level);
    for (uint32_t j = 0; j < n_digits(ctx, level); j++)
        CK_REQUIRE(ctx->conv.count({(int)level, (int)j}), CKKS_EUNSUPPORTED,
                   "rotate_noalloc: no tables for level %u digit %u", level, j);
    // the event profiler creates runtime objects per launch: off for this call
    const bool profiling = ctx->profiling;
    ctx->profiling = false;
    uint64_t *digits = scratch_ptr;
    uint64_t *rw = digits + ((size_t)n_digits(ctx, level) * (L + ctx->n_p) + ctx->alpha) * ctx->n;
    const uint64_t *c0 = in->data, *dig = digits;
    const uint32_t g = ckks_galois_elt(ctx, steps);
    uint64_t *o = out->data;
    ckks_status st = ks_modup(ctx, in->data + (size_t)L * ctx->n, level, digits);
    if (st == CKKS_OK) st = ks_rotate_batch(ctx, level, 1, &c0, &dig, &g, &key, &o, rw);
    ctx->profiling = profiling;
    if (st == CKKS_OK) out->scale = in->scale;
    return st;
}
