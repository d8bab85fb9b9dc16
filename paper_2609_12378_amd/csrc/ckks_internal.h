// Internal declarations of libckks_mi: the context, error plumbing, kernel launchers.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <string>
#include <utility>
#include <vector>

#include "ckks_mi.h"
#include "modarith.h"

// ---------------------------------------------------------------- errors ----
ckks_status set_error(ckks_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

#define HIP_TRY(expr)                                                                              \
    do {                                                                                           \
        hipError_t e_ = (expr);                                                                    \
        if (e_ != hipSuccess)                                                                      \
            return set_error(CKKS_EHIP, "%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_),     \
                             __FILE__, __LINE__);                                                  \
    } while (0)
#define CK_TRY(expr)                                                                               \
    do {                                                                                           \
        ckks_status s_ = (expr);                                                                   \
        if (s_ != CKKS_OK) return s_;                                                              \
    } while (0)
#define CK_REQUIRE(cond, st, ...)                                                                  \
    do {                                                                                           \
        if (!(cond)) return set_error(st, __VA_ARGS__);                                            \
    } while (0)

// Upper bound on the primes a context holds (n_q + n_p); the row->prime map
// travels to kernels by value.
constexpr int kMaxPrimes = 64;
constexpr int kMaxLimbMap = 96;

// Row r of a [rows][N] launch uses prime index prime[r % n] (r / n is the batch
// index).
struct LimbMap {
    uint32_t n;
    uint8_t prime[kMaxLimbMap];
};

// Device constants of one fast basis conversion, from the primes src[0..ns) to
// dst[0..nt): y_i = [x_i * qhat_inv_i]_{src_i} centred in (-src_i/2, src_i/2],
// out_t = sum_i y_i [Qhat_i]_t.
struct ConvDev {
    int ns = 0, nt = 0;
    uint8_t src[kMaxPrimes];
    uint8_t dst[kMaxPrimes];
    ulonglong2 *d_qhat_inv = nullptr;  // [ns] (value, Shoup companion) mod src_i
    ulonglong2 *d_qhat_mod = nullptr;  // [ns][nt] (value, Shoup companion) mod dst_t
    ulonglong2 *d_neg_q = nullptr;     // [nt] (value, Shoup companion) of [-Q_src]_dst_t
    bool f64 = false;                  // primes below 2^50, sources below twice the targets: fp64 tables set
    double *d_qhat_inv_f = nullptr;    // [ns] the values of d_qhat_inv as doubles
    double *d_qhat_mod_f = nullptr;    // [ns][nt] the values of d_qhat_mod as doubles
};

// Kernels timed by the optional event profiler.  Each launch is bracketed by
// two events and tagged with its algorithmic bytes: the bytes the kernel must
// read and write in HBM at minimum (each input and output word once; twiddle
// and constant tables, which stay cache-resident, are not counted).
enum KClass {
    K_NTT_FWD_COL = 0, K_NTT_FWD_ROW, K_NTT_INV_ROW, K_NTT_INV_COL, K_FFT_A, K_FFT_B, K_GATHER, K_TO_RNS,
    K_MAC, K_KEYIP, K_CONV, K_MODDOWN, K_ELEM, K_ROW_MAC, K_ENC_TM, K_MAC_TM, K_ATTN_CORR, K_NCLASS
};
extern const char *const kKClassNames[K_NCLASS];

struct ckks_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    uint32_t log_n = 0, n = 0, n_q = 0, n_p = 0, dnum = 1, alpha = 1;
    std::vector<uint64_t> primes, psi;   // q_0..q_{n_q-1}, p_0..p_{n_p-1}
    std::vector<ModQ> mods;

    // device tables
    ModQ *d_mod = nullptr;               // [n_primes]
    ulonglong2 *d_tw = nullptr;          // [n_primes][N] (psi^brev(k), Shoup)
    ulonglong2 *d_itw = nullptr;         // [n_primes][N] (psi^-brev(k), Shoup)
    double *d_twf = nullptr;             // [n_primes][N] psi^brev(k) as doubles (primes < 2^50)
    double *d_itwf = nullptr;            // [n_primes][N] psi^-brev(k) as doubles
    bool f64_ok[kMaxPrimes] = {};        // q < 2^50: the fp64 butterflies are exact
    bool int_only = false;               // force the integer Shoup butterflies
    uint32_t proj_max_pairs = 0;         // projection sub-batch limit (0 = by the staging budget)
    bool lazy_moddown = false;           // sums of rotations with one ModDown per output
    uint32_t sum128_terms = 0;           // products of two residues an exact 128-bit sum holds (with a residue)
    double2 *d_fft_w = nullptr;          // [N/4]  omega^-e, omega = exp(2 pi i/(N/2))
    double2 *d_fft_wc = nullptr;         // [2048] stage-by-stage copy for 2048-point blocks (N >= 2^12)
    double2 *d_fft_twist = nullptr;      // [N/2]  zeta^-k, zeta = exp(i pi / N)
    uint32_t *d_slot_pos = nullptr;      // [N/2]  bit-reversed FFT position of slot j
    uint32_t *d_pos_slot = nullptr;      // [N/2]  slot index held at FFT position x (inverse of d_slot_pos)
    std::map<std::pair<int, int>, ConvDev> conv;  // (level, digit) ; digit -1 = ModDown
    ulonglong2 *d_pinv = nullptr;        // [n_q] (P^-1 mod q_i, Shoup)
    ulonglong2 *d_pmodq = nullptr;       // [n_q] ([P]_{q_i}, Shoup)
    ulonglong2 *d_qlinv = nullptr;       // [n_q][n_q] (q_l^-1 mod q_i, Shoup) row l

    // grow-only scratch arena
    void *scratch = nullptr;
    size_t scratch_bytes = 0;
    bool scratch_external = false;  // the arena is a caller's workspace (ckks_set_workspace): never reallocated

    // optional per-kernel event profiling
    bool profiling = false;
    struct ProfRec {
        hipEvent_t a, b;
        double bytes, ops;
    };
    std::vector<ProfRec> prof_events[K_NCLASS];
    double prof_ms[K_NCLASS] = {0};
    double prof_bytes[K_NCLASS] = {0};
    double prof_ops[K_NCLASS] = {0};
    uint64_t prof_count[K_NCLASS] = {0};

    uint32_t n_primes() const { return n_q + n_p; }
};

// scratch of at least `bytes` bytes (256-byte aligned), growing the arena
ckks_status ctx_scratch(ckks_ctx *ctx, size_t bytes, void **out);
// once per device, with that device current: locate the allocation-free calls' static scratch on it
void noalloc_setup(int device);
// workspace bytes of one call of a ckks_op (SIZE_MAX: unknown op or invalid shape)
size_t op_workspace_bytes(const ckks_ctx *ctx, int op, const uint32_t *shape);

// profiler brackets: call prof_begin before a launch and prof_end after;
// bytes = the launch's algorithmic HBM bytes, ops = its nominal VALU lane
// instructions (the arithmetic model of the kernel; 0 where none is stated)
void prof_begin(ckks_ctx *ctx, KClass k, double bytes, double ops = 0.0);
void prof_end(ckks_ctx *ctx, KClass k);

// basis-conversion tables for ModUp of digit j at `level` (dst = other q-limbs
// then P) and ModDown at `level` (digit = -1: src = P, dst = q_0..q_level)
ckks_status ctx_conv(ckks_ctx *ctx, int level, int digit, const ConvDev **out);

// digit helpers
inline uint32_t digit_lo(const ckks_ctx *c, uint32_t j) { return j * c->alpha; }
inline uint32_t digit_hi(const ckks_ctx *c, uint32_t j, uint32_t level)  // exclusive, clipped at level
{
    uint32_t h = (j + 1) * c->alpha;
    if (h > c->n_q) h = c->n_q;
    if (h > level + 1) h = level + 1;
    return h;
}
inline uint32_t n_digits(const ckks_ctx *c, uint32_t level) { return level / c->alpha + 1; }

// ------------------------------------------------------------- launchers ----
// All launchers enqueue on ctx->stream and return CKKS_EHIP on launch failure.
// NTT over rows [batch][map.n][N] of `data` (in place).
ckks_status launch_ntt(ckks_ctx *ctx, uint64_t *data, uint32_t rows, const LimbMap &map, bool inverse);
// NTT of `batch` groups of map.n rows; group b starts at row b * bstride of `data`.
ckks_status launch_ntt_strided(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride, const LimbMap &map,
                               bool inverse);
// forward NTT of signed coefficient rows m[batch][N] into out[batch][limbs][N] (primes 0..limbs-1)
ckks_status launch_ntt_from_i64(ckks_ctx *ctx, const int64_t *m, uint64_t *out, uint32_t batch, uint32_t limbs);
// split of log_n into the column pass (s1 stages, 0 = single pass) and the row pass (s2 stages)
void ntt_split(uint32_t log_n, int *s1, int *s2);
// the transforms over primes 0..limbs-1 use the fp64 butterflies
bool ntt_uses_f64(const ckks_ctx *ctx, uint32_t limbs);
// column pass only of a forward transform (fp64 primes, two-pass sizes); the rows are left as raw doubles
ckks_status launch_ntt_fwd_first_pass(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride,
                                      const LimbMap &map);
// column pass only of an inverse transform whose row pass a fused kernel ran (rows as raw doubles below 2q; fp64
// primes, two-pass sizes): canonical coefficients out
ckks_status launch_ntt_inv_second_pass(ckks_ctx *ctx, uint64_t *data, uint32_t batch, uint32_t bstride,
                                       const LimbMap &map);
// column pass only of launch_ntt_from_i64 (two-pass sizes); the rows stay in the inter-pass form
ckks_status launch_ntt_col_i64(ckks_ctx *ctx, const int64_t *m, uint64_t *out, uint32_t batch, uint32_t limbs);
// nominal VALU instructions of one radix-2 butterfly: fp64 (product with FMA
// error term, quotient estimate and rint, remainder, range reduction of the
// other input, add and subtract) and 64-bit integer Shoup (from the gfx950 ISA)
constexpr double kOpsButterflyF64 = 11.0, kOpsButterflyInt = 37.0;
// identity map for a contiguous range of prime indices
LimbMap limb_range(uint32_t first, uint32_t count);

// element-wise and structural kernels (ops.hip)
ckks_status launch_automorph(ckks_ctx *ctx, const uint64_t *in, uint64_t *out, uint32_t rows, uint32_t g);
