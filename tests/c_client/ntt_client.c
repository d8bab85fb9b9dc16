/* A C client of libckks_mi.so that uses neither Python nor torch: the HIP runtime for device memory and the
 * library's C ABI for the transforms.  It creates a context (N = 2^8, three 36-bit primes), transforms seeded
 * residues, compares every output with the transform's definition evaluated here in 128-bit integer arithmetic,
 *     A[j] = sum_i a_i * psi^((2 brev(j) + 1) i) mod q,
 * (the layout the header states: index j holds a(psi^(2 brev(j) + 1))), and checks that the inverse returns the
 * input.  Exit status 0 with "ntt_client: ok" on success, 1 on a mismatch, 2 when no context can be created
 * (no GPU), 3 on a HIP runtime error. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ckks_mi.h"

enum { LOG_N = 8, N = 1 << LOG_N, LIMBS = 3, BATCH = 2 };

static uint64_t mulmod(uint64_t a, uint64_t b, uint64_t q) { return (uint64_t)((unsigned __int128)a * b % q); }

static uint64_t powmod(uint64_t b, uint64_t e, uint64_t q)
{
    uint64_t r = 1 % q;
    for (b %= q; e; e >>= 1, b = mulmod(b, b, q))
        if (e & 1) r = mulmod(r, b, q);
    return r;
}

static uint32_t brev(uint32_t j, int bits)
{
    uint32_t r = 0;
    for (int i = 0; i < bits; i++) r |= ((j >> i) & 1u) << (bits - 1 - i);
    return r;
}

static uint64_t splitmix(uint64_t *s)
{
    uint64_t z = (*s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

#define HIP_OK(call)                                                                    \
    do {                                                                                \
        hipError_t e_ = (call);                                                         \
        if (e_ != hipSuccess) {                                                         \
            fprintf(stderr, "ntt_client: %s failed: %s\n", #call, hipGetErrorString(e_)); \
            return 3;                                                                   \
        }                                                                               \
    } while (0)

int main(void)
{
    ckks_params prm;
    memset(&prm, 0, sizeof prm);
    prm.log_n = LOG_N;
    prm.n_q = LIMBS;
    prm.n_p = 0;
    prm.dnum = 1;
    prm.q_bits = 36;
    ckks_ctx *ctx = NULL;
    if (ckks_ctx_create(&prm, NULL, &ctx) != CKKS_OK) {
        fprintf(stderr, "ntt_client: no context: %s\n", ckks_last_error());
        return 2;
    }
    uint64_t q[LIMBS], psi[LIMBS];
    if (ckks_ctx_tables(ctx, q, NULL, psi) != CKKS_OK) {
        fprintf(stderr, "ntt_client: tables: %s\n", ckks_last_error());
        return 1;
    }
    static uint64_t a[BATCH][LIMBS][N], got[BATCH][LIMBS][N];
    uint64_t seed = 20260;
    for (int b = 0; b < BATCH; b++)
        for (int k = 0; k < LIMBS; k++)
            for (int i = 0; i < N; i++) a[b][k][i] = splitmix(&seed) % q[k];
    uint64_t *dev = NULL;
    HIP_OK(hipMalloc((void **)&dev, sizeof a));
    HIP_OK(hipMemcpy(dev, a, sizeof a, hipMemcpyHostToDevice));
    if (ckks_ntt(ctx, dev, BATCH, 0, LIMBS) != CKKS_OK) {
        fprintf(stderr, "ntt_client: ntt: %s\n", ckks_last_error());
        return 1;
    }
    HIP_OK(hipMemcpy(got, dev, sizeof got, hipMemcpyDeviceToHost));   /* synchronizes with the null stream */
    for (int b = 0; b < BATCH; b++)
        for (int k = 0; k < LIMBS; k++)
            for (int j = 0; j < N; j++) {
                const uint64_t root = powmod(psi[k], 2 * (uint64_t)brev((uint32_t)j, LOG_N) + 1, q[k]);
                uint64_t want = 0, w = 1;
                for (int i = 0; i < N; i++) {
                    want = (want + mulmod(a[b][k][i], w, q[k])) % q[k];
                    w = mulmod(w, root, q[k]);
                }
                if (got[b][k][j] != want) {
                    fprintf(stderr, "ntt_client: NTT[%d][%d][%d] = %llu, definition %llu\n", b, k, j,
                            (unsigned long long)got[b][k][j], (unsigned long long)want);
                    return 1;
                }
            }
    if (ckks_intt(ctx, dev, BATCH, 0, LIMBS) != CKKS_OK) {
        fprintf(stderr, "ntt_client: intt: %s\n", ckks_last_error());
        return 1;
    }
    HIP_OK(hipMemcpy(got, dev, sizeof got, hipMemcpyDeviceToHost));
    if (memcmp(got, a, sizeof a) != 0) {
        fprintf(stderr, "ntt_client: the inverse does not return the input\n");
        return 1;
    }
    /* an argument error comes back as a status and a message, never as a crash */
    if (ckks_ntt(ctx, dev, BATCH, LIMBS, 1) == CKKS_OK) {
        fprintf(stderr, "ntt_client: a limb beyond the context was accepted\n");
        return 1;
    }
    HIP_OK(hipFree(dev));
    ckks_ctx_destroy(ctx);
    printf("ntt_client: ok (%d x %d limbs x 2^%d, against the definition)\n", BATCH, LIMBS, LOG_N);
    return 0;
}
