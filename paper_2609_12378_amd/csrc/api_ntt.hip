// C ABI: number-theoretic transforms.
#include "ckks_internal.h"

static ckks_status ntt_common(ckks_ctx *ctx, uint64_t *dev, uint32_t batch, uint32_t limb0, uint32_t n_limbs,
                              bool inverse)
{
    clear_error();
    CK_REQUIRE(ctx, CKKS_EINVAL, "null context");
    if (batch == 0 || n_limbs == 0) return CKKS_OK;
    CK_REQUIRE(dev, CKKS_EINVAL, "null data pointer");
    CK_REQUIRE((uint64_t)limb0 + n_limbs <= ctx->n_primes(), CKKS_EINVAL,
               "limbs [%u, %u) exceed the %u primes of the context", limb0, limb0 + n_limbs, ctx->n_primes());
    CK_REQUIRE(n_limbs <= (uint32_t)kMaxLimbMap, CKKS_EUNSUPPORTED, "at most %d limbs per call", kMaxLimbMap);
    return launch_ntt(ctx, dev, batch * n_limbs, limb_range(limb0, n_limbs), inverse);
}

extern "C" ckks_status ckks_ntt(ckks_ctx *ctx, uint64_t *dev, uint32_t batch, uint32_t limb0, uint32_t n_limbs)
{
    return ntt_common(ctx, dev, batch, limb0, n_limbs, false);
}

extern "C" ckks_status ckks_intt(ckks_ctx *ctx, uint64_t *dev, uint32_t batch, uint32_t limb0, uint32_t n_limbs)
{
    return ntt_common(ctx, dev, batch, limb0, n_limbs, true);
}
