// Host runtime of libckks_mi: parameter generation, precomputed tables, the
// scratch arena, errors and the per-kernel event profiler.
//
// Parameters follow the standard RNS-CKKS set-up: NTT-friendly primes
// q = 1 mod 2N (so Z_q holds a primitive 2N-th root psi and X^N + 1 splits),
// the modulus chain q_0..q_{L-1}, special primes P for hybrid key switching
// with dnum digits.  All host arithmetic is exact (128-bit products).
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "ckks_internal.h"

typedef unsigned __int128 u128;

// ------------------------------------------------------------------ errors --
static thread_local char g_err[512];

ckks_status set_error(ckks_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}
void clear_error() { g_err[0] = 0; }
extern "C" const char *ckks_last_error(void) { return g_err; }

const char *const kKClassNames[K_NCLASS] = {"ntt_fwd_col", "ntt_fwd_row", "ntt_inv_row", "ntt_inv_col", "fft_a",
                                            "fft_b",       "gather",      "to_rns",      "mac",         "key_ip",
                                            "conv",        "moddown",     "elementwise", "ntt_row_mac",
                                            "encode_tm",   "mac_tm",     "attn_corr"};

// --------------------------------------------------------------- host math --
namespace hm {
static uint64_t mul(uint64_t a, uint64_t b, uint64_t q) { return (uint64_t)((u128)a * b % q); }
static uint64_t pw(uint64_t b, uint64_t e, uint64_t q)
{
    uint64_t r = 1;
    b %= q;
    for (; e; e >>= 1) {
        if (e & 1) r = mul(r, b, q);
        b = mul(b, b, q);
    }
    return r;
}
static uint64_t inv(uint64_t a, uint64_t q) { return pw(a % q, q - 2, q); }
static uint64_t shoup(uint64_t w, uint64_t q) { return (uint64_t)(((u128)w << 64) / q); }
static bool is_prime(uint64_t n)
{
    if (n < 2) return false;
    static const uint64_t bases[] = {2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37};
    for (uint64_t p : bases)
        if (n % p == 0) return n == p;
    uint64_t d = n - 1;
    int s = 0;
    while ((d & 1) == 0) {
        d >>= 1;
        s++;
    }
    for (uint64_t a : bases) {
        uint64_t x = pw(a, d, n);
        if (x == 1 || x == n - 1) continue;
        bool comp = true;
        for (int i = 1; i < s && comp; i++) {
            x = mul(x, x, n);
            if (x == n - 1) comp = false;
        }
        if (comp) return false;
    }
    return true;
}
// descending primes below 2^bits that are 1 mod two_n
static std::vector<uint64_t> prime_list(uint32_t bits, uint64_t two_n, size_t count,
                                        const std::vector<uint64_t> &skip)
{
    std::vector<uint64_t> out;
    uint64_t top = (bits >= 64) ? ~0ull : ((1ull << bits) - 1);
    uint64_t c = top / two_n * two_n + 1;
    if (c > top) c -= two_n;
    const uint64_t low = 1ull << (bits - 1);
    while (out.size() < count && c > low) {
        bool used = false;
        for (uint64_t s : skip) used |= (s == c);
        if (!used && is_prime(c)) out.push_back(c);
        c -= two_n;
    }
    return out;
}
static uint32_t brev(uint32_t x, int bits)
{
    uint32_t r = 0;
    for (int i = 0; i < bits; i++) {
        r = (r << 1) | (x & 1u);
        x >>= 1;
    }
    return r;
}
}  // namespace hm

// ----------------------------------------------------------------- context --
static ckks_status upload(void **dst, const void *src, size_t bytes)
{
    HIP_TRY(hipMalloc(dst, bytes));
    HIP_TRY(hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice));
    return CKKS_OK;
}

static ulonglong2 shoup_pair(uint64_t w, uint64_t q) { return make_ulonglong2(w, hm::shoup(w, q)); }

static ckks_status build_tables(ckks_ctx *c)
{
    const uint32_t np = c->n_primes(), n = c->n;
    const uint64_t two_n = 2ull * n;
    c->psi.resize(np);
    c->mods.resize(np);
    std::vector<ulonglong2> tw((size_t)np * n), itw((size_t)np * n);
    std::vector<double> twf((size_t)np * n), itwf((size_t)np * n);
    for (uint32_t k = 0; k < np; k++) {
        const uint64_t q = c->primes[k];
        uint64_t psi = 0;
        for (uint64_t x = 2; x < (1u << 20); x++) {
            uint64_t cand = hm::pw(x, (q - 1) / two_n, q);
            if (hm::pw(cand, n, q) == q - 1) {
                psi = cand;
                break;
            }
        }
        CK_REQUIRE(psi != 0, CKKS_EINVAL, "no primitive 2N-th root of unity modulo %llu", (unsigned long long)q);
        c->psi[k] = psi;
        const uint64_t psi_inv = hm::inv(psi, q);
        std::vector<uint64_t> pw(n), ipw(n);  // psi^e, psi^-e for e < N
        pw[0] = ipw[0] = 1;
        for (uint32_t e = 1; e < n; e++) {
            pw[e] = hm::mul(pw[e - 1], psi, q);
            ipw[e] = hm::mul(ipw[e - 1], psi_inv, q);
        }
        for (uint32_t i = 0; i < n; i++) {
            const uint32_t e = hm::brev(i, (int)c->log_n);
            tw[(size_t)k * n + i] = shoup_pair(pw[e], q);
            itw[(size_t)k * n + i] = shoup_pair(ipw[e], q);
            twf[(size_t)k * n + i] = (double)pw[e];
            itwf[(size_t)k * n + i] = (double)ipw[e];
        }
        c->f64_ok[k] = q < (1ull << 50);
        ModQ &m = c->mods[k];
        m.q = q;
        m.twoq = 2 * q;
        m.r64 = (uint64_t)(((u128)1 << 64) % q);
        m.r64s = hm::shoup(m.r64, q);
        m.one_s = (uint64_t)(((u128)1 << 64) / q);
        m.ninv = hm::inv(n % q, q);
        m.ninvs = hm::shoup(m.ninv, q);
        m.iw1n = hm::mul(ipw[hm::brev(1, (int)c->log_n)], m.ninv, q);
        m.iw1ns = hm::shoup(m.iw1n, q);
        m.qd = (double)q;
        m.qinvd = 1.0 / (double)q;
        m.ninvd = (double)m.ninv;
    }
    CK_TRY(upload((void **)&c->d_tw, tw.data(), tw.size() * sizeof(ulonglong2)));
    CK_TRY(upload((void **)&c->d_itw, itw.data(), itw.size() * sizeof(ulonglong2)));
    CK_TRY(upload((void **)&c->d_twf, twf.data(), twf.size() * sizeof(double)));
    CK_TRY(upload((void **)&c->d_itwf, itwf.data(), itwf.size() * sizeof(double)));
    CK_TRY(upload((void **)&c->d_mod, c->mods.data(), c->mods.size() * sizeof(ModQ)));

    // fp64 tables of the encode/decode FFT.  The expressions are fixed (the
    // rounding of the encoded integers depends on every bit of them):
    //   omega^-e = (cos(2 pi e / M), -sin(2 pi e / M)),  M = N/2,
    //   zeta^-k  = (cos(pi k / N),  -sin(pi k / N)),
    // with cosine and sine taken from one call to the C library's sincos(),
    // named explicitly because it can differ from separate sin()/cos() calls
    // in the last bit and compilers merge or split such calls at will.
    const uint32_t M = n / 2;
    std::vector<double2> w(M / 2 > 0 ? M / 2 : 1), twist(M);
    for (uint32_t e = 0; e < M / 2; e++) {
        const double ang = 2.0 * M_PI * (double)e / (double)M;
        double sn, cs;
        sincos(ang, &sn, &cs);
        w[e] = make_double2(cs, -sn);
    }
    for (uint32_t k = 0; k < M; k++) {
        const double ang = M_PI * (double)k / (double)n;
        double sn, cs;
        sincos(ang, &sn, &cs);
        twist[k] = make_double2(cs, -sn);
    }
    std::vector<uint32_t> pos(M);
    int logm = 0;
    while ((1u << logm) < M) logm++;
    uint64_t e5 = 1;
    for (uint32_t j = 0; j < M; j++) {
        pos[j] = hm::brev((uint32_t)((e5 - 1) / 4), logm);
        e5 = e5 * 5 % two_n;
    }
    CK_TRY(upload((void **)&c->d_fft_w, w.data(), w.size() * sizeof(double2)));
    if (M >= 2048) {
        // the same twiddles, stage by stage for 2048-point blocks: wc[2^(s-1) + k] = w[k * M / 2^s]
        std::vector<double2> wc(2048, make_double2(0.0, 0.0));
        for (uint32_t s = 1; s <= 11; s++)
            for (uint32_t k = 0; k < (1u << (s - 1)); k++) wc[(1u << (s - 1)) + k] = w[(size_t)k * (M >> s)];
        CK_TRY(upload((void **)&c->d_fft_wc, wc.data(), wc.size() * sizeof(double2)));
    }
    CK_TRY(upload((void **)&c->d_fft_twist, twist.data(), twist.size() * sizeof(double2)));
    CK_TRY(upload((void **)&c->d_slot_pos, pos.data(), pos.size() * sizeof(uint32_t)));
    std::vector<uint32_t> inv_pos(M);
    for (uint32_t j = 0; j < M; j++) inv_pos[pos[j]] = j;
    CK_TRY(upload((void **)&c->d_pos_slot, inv_pos.data(), inv_pos.size() * sizeof(uint32_t)));

    // P mod q_i, P^-1 mod q_i, q_l^-1 mod q_i
    std::vector<ulonglong2> pm(c->n_q), pinv(c->n_q), qlinv((size_t)c->n_q * c->n_q);
    for (uint32_t i = 0; i < c->n_q; i++) {
        const uint64_t q = c->primes[i];
        uint64_t P = 1;
        for (uint32_t j = 0; j < c->n_p; j++) P = hm::mul(P, c->primes[c->n_q + j] % q, q);
        pm[i] = shoup_pair(P, q);
        pinv[i] = shoup_pair(hm::inv(P, q), q);
        for (uint32_t l = 0; l < c->n_q; l++)
            qlinv[(size_t)l * c->n_q + i] = shoup_pair(l == i ? 0 : hm::inv(c->primes[l] % q, q), q);
    }
    CK_TRY(upload((void **)&c->d_pmodq, pm.data(), pm.size() * sizeof(ulonglong2)));
    CK_TRY(upload((void **)&c->d_pinv, pinv.data(), pinv.size() * sizeof(ulonglong2)));
    CK_TRY(upload((void **)&c->d_qlinv, qlinv.data(), qlinv.size() * sizeof(ulonglong2)));
    return CKKS_OK;
}

// Conversion constants from src primes to dst primes.
static ckks_status make_conv(ckks_ctx *c, const std::vector<uint32_t> &src, const std::vector<uint32_t> &dst,
                             ConvDev *out)
{
    out->ns = (int)src.size();
    out->nt = (int)dst.size();
    std::vector<ulonglong2> qinv(src.size()), qmod(src.size() * (dst.size() ? dst.size() : 1));
    for (size_t a = 0; a < src.size(); a++) {
        out->src[a] = (uint8_t)src[a];
        const uint64_t qa = c->primes[src[a]];
        uint64_t qhat = 1;  // prod_{b != a} q_b mod q_a
        for (size_t b = 0; b < src.size(); b++)
            if (b != a) qhat = hm::mul(qhat, c->primes[src[b]] % qa, qa);
        qinv[a] = shoup_pair(hm::inv(qhat, qa), qa);
        for (size_t t = 0; t < dst.size(); t++) {
            const uint64_t qt = c->primes[dst[t]];
            uint64_t v = 1;
            for (size_t b = 0; b < src.size(); b++)
                if (b != a) v = hm::mul(v, c->primes[src[b]] % qt, qt);
            qmod[a * dst.size() + t] = shoup_pair(v, qt);
        }
    }
    std::vector<ulonglong2> negq(dst.size() ? dst.size() : 1);
    for (size_t t = 0; t < dst.size(); t++) {
        out->dst[t] = (uint8_t)dst[t];
        const uint64_t qt = c->primes[dst[t]];
        uint64_t v = 1;  // Q_src mod q_t
        for (uint32_t b : src) v = hm::mul(v, c->primes[b] % qt, qt);
        negq[t] = shoup_pair(v ? qt - v : 0, qt);
    }
    CK_TRY(upload((void **)&out->d_qhat_inv, qinv.data(), qinv.size() * sizeof(ulonglong2)));
    CK_TRY(upload((void **)&out->d_qhat_mod, qmod.data(), qmod.size() * sizeof(ulonglong2)));
    CK_TRY(upload((void **)&out->d_neg_q, negq.data(), negq.size() * sizeof(ulonglong2)));
    // fp64 conversion: every prime below 2^50 and every source prime below twice every target prime (so the
    // centred |y_i| < q_t and the sums stay exact)
    out->f64 = true;
    uint64_t max_src = 0, min_dst = ~0ull;
    for (uint32_t v : src) {
        out->f64 = out->f64 && c->f64_ok[v];
        max_src = std::max(max_src, c->primes[v]);
    }
    for (uint32_t v : dst) {
        out->f64 = out->f64 && c->f64_ok[v];
        min_dst = std::min(min_dst, c->primes[v]);
    }
    out->f64 = out->f64 && !dst.empty() && max_src / 2 < min_dst;
    if (out->f64) {
        std::vector<double> fi(qinv.size()), fm(qmod.size());
        for (size_t k = 0; k < qinv.size(); k++) fi[k] = (double)qinv[k].x;
        for (size_t k = 0; k < qmod.size(); k++) fm[k] = (double)qmod[k].x;
        CK_TRY(upload((void **)&out->d_qhat_inv_f, fi.data(), fi.size() * sizeof(double)));
        CK_TRY(upload((void **)&out->d_qhat_mod_f, fm.data(), fm.size() * sizeof(double)));
    }
    return CKKS_OK;
}

ckks_status ctx_conv(ckks_ctx *c, int level, int digit, const ConvDev **out)
{
    auto key = std::make_pair(level, digit);
    auto it = c->conv.find(key);
    if (it != c->conv.end()) {
        *out = &it->second;
        return CKKS_OK;
    }
    std::vector<uint32_t> src, dst;
    if (digit < 0) {
        for (uint32_t j = 0; j < c->n_p; j++) src.push_back(c->n_q + j);
        for (int i = 0; i <= level; i++) dst.push_back((uint32_t)i);
    } else {
        const uint32_t lo = digit_lo(c, (uint32_t)digit), hi = digit_hi(c, (uint32_t)digit, (uint32_t)level);
        for (uint32_t i = lo; i < hi; i++) src.push_back(i);
        for (int i = 0; i <= level; i++)
            if ((uint32_t)i < lo || (uint32_t)i >= hi) dst.push_back((uint32_t)i);
        for (uint32_t j = 0; j < c->n_p; j++) dst.push_back(c->n_q + j);
    }
    ConvDev cd;
    CK_TRY(make_conv(c, src, dst, &cd));
    auto res = c->conv.emplace(key, cd);
    *out = &res.first->second;
    return CKKS_OK;
}

// Every level's basis-conversion tables (ModUp of each digit, ModDown), built when the context is created so that
// no later call allocates them on first use.
static ckks_status build_all_conv(ckks_ctx *c)
{
    if (!c->n_p) return CKKS_OK;
    const ConvDev *cd;
    for (uint32_t level = 0; level < c->n_q; level++) {
        CK_TRY(ctx_conv(c, (int)level, -1, &cd));
        for (uint32_t j = 0; j < n_digits(c, level); j++) CK_TRY(ctx_conv(c, (int)level, (int)j, &cd));
    }
    return CKKS_OK;
}

ckks_status ctx_scratch(ckks_ctx *c, size_t bytes, void **out)
{
    if (bytes == SIZE_MAX) return set_error(CKKS_EINVAL, "workspace size of an invalid shape");
    if (bytes > c->scratch_bytes && c->scratch_external)
        return set_error(CKKS_ENOMEM, "workspace of %zu bytes is too small: this call needs %zu", c->scratch_bytes,
                         bytes);
    if (bytes > c->scratch_bytes) {
        if (c->scratch) {
            HIP_TRY(hipStreamSynchronize(c->stream));
            HIP_TRY(hipFree(c->scratch));
            c->scratch = nullptr;
            c->scratch_bytes = 0;
        }
        const size_t sz = (bytes + 255) & ~(size_t)255;
        hipError_t e = hipMalloc(&c->scratch, sz);
        if (e != hipSuccess) {
            c->scratch = nullptr;
            return set_error(CKKS_ENOMEM, "scratch arena of %zu bytes: %s", sz, hipGetErrorString(e));
        }
        c->scratch_bytes = sz;
    }
    *out = c->scratch;
    return CKKS_OK;
}

void prof_begin(ckks_ctx *c, KClass k, double bytes, double ops)
{
    if (!c->profiling) return;
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) {
        (void)hipEventDestroy(a);
        return;
    }
    (void)hipEventRecord(a, c->stream);
    c->prof_events[k].push_back({a, b, bytes, ops});
}
void prof_end(ckks_ctx *c, KClass k)
{
    if (!c->profiling || c->prof_events[k].empty()) return;
    (void)hipEventRecord(c->prof_events[k].back().b, c->stream);
}

static ckks_status prof_collect(ckks_ctx *c)
{
    for (int k = 0; k < K_NCLASS; k++) {
        for (auto &ev : c->prof_events[k]) {
            HIP_TRY(hipEventSynchronize(ev.b));
            float ms = 0;
            HIP_TRY(hipEventElapsedTime(&ms, ev.a, ev.b));
            c->prof_ms[k] += ms;
            c->prof_bytes[k] += ev.bytes;
            c->prof_ops[k] += ev.ops;
            c->prof_count[k]++;
            (void)hipEventDestroy(ev.a);
            (void)hipEventDestroy(ev.b);
        }
        c->prof_events[k].clear();
    }
    return CKKS_OK;
}

// --------------------------------------------------------------- C ABI ------
extern "C" {

ckks_status ckks_ctx_create(const ckks_params *p, void *stream, ckks_ctx **out)
{
    clear_error();
    CK_REQUIRE(p && out, CKKS_EINVAL, "ctx_create: null argument");
    CK_REQUIRE(p->log_n >= 4 && p->log_n <= 16, CKKS_EUNSUPPORTED, "log_n %u outside [4, 16]", p->log_n);
    CK_REQUIRE(p->n_q >= 1 && p->n_q + p->n_p <= (uint32_t)kMaxPrimes, CKKS_EUNSUPPORTED,
               "n_q + n_p = %u outside [1, %d]", p->n_q + p->n_p, kMaxPrimes);
    CK_REQUIRE(p->dnum >= 1 && p->dnum <= p->n_q, CKKS_EINVAL, "dnum %u outside [1, n_q]", p->dnum);
    ckks_ctx *c = new (std::nothrow) ckks_ctx();
    CK_REQUIRE(c, CKKS_ENOMEM, "ctx_create: out of host memory");
    c->log_n = p->log_n;
    c->n = 1u << p->log_n;
    c->n_q = p->n_q;
    c->n_p = p->n_p;
    c->dnum = p->dnum;
    c->alpha = (p->n_q + p->dnum - 1) / p->dnum;
    c->stream = (hipStream_t)stream;
    const uint64_t two_n = 2ull * c->n;
    ckks_status st = CKKS_OK;
    if (p->q) {
        c->primes.assign(p->q, p->q + p->n_q);
    } else {
        if (p->q_bits < 20 || p->q_bits > 62) st = set_error(CKKS_EUNSUPPORTED, "q_bits %u outside [20, 62]", p->q_bits);
        else c->primes = hm::prime_list(p->q_bits, two_n, p->n_q, {});
    }
    if (st == CKKS_OK && c->primes.size() != p->n_q)
        st = set_error(CKKS_EUNSUPPORTED, "only %zu primes of %u bits are 1 mod 2N", c->primes.size(), p->q_bits);
    if (st == CKKS_OK && p->n_p) {
        std::vector<uint64_t> pp;
        if (p->p) pp.assign(p->p, p->p + p->n_p);
        else {
            const uint32_t pb = p->p_bits ? p->p_bits : p->q_bits;
            if (pb < 20 || pb > 62) st = set_error(CKKS_EUNSUPPORTED, "p_bits %u outside [20, 62]", pb);
            else pp = hm::prime_list(pb, two_n, p->n_p, c->primes);
        }
        if (st == CKKS_OK && pp.size() != p->n_p) st = set_error(CKKS_EUNSUPPORTED, "not enough special primes");
        c->primes.insert(c->primes.end(), pp.begin(), pp.end());
    }
    for (size_t i = 0; st == CKKS_OK && i < c->primes.size(); i++) {
        const uint64_t q = c->primes[i];
        if (q >= (1ull << 62) || q % two_n != 1 || !hm::is_prime(q))
            st = set_error(CKKS_EINVAL, "modulus %llu is not a prime below 2^62 that is 1 mod 2N",
                           (unsigned long long)q);
        for (size_t j = 0; j < i && st == CKKS_OK; j++)
            if (c->primes[j] == q) st = set_error(CKKS_EINVAL, "modulus %llu repeated", (unsigned long long)q);
    }
    if (st == CKKS_OK) {
        hipError_t e = hipGetDevice(&c->device);
        if (e != hipSuccess) st = set_error(CKKS_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    }
    if (st == CKKS_OK) {
        // the integer kernels sum products of two residues exactly in 128 bits: at most sum128_terms of them
        // (each below (q - 1)^2) together with one residue below q, for the largest prime q of the context
        uint64_t qmax = 0;
        for (uint64_t q : c->primes) qmax = q > qmax ? q : qmax;
        const unsigned __int128 sq = (unsigned __int128)(qmax - 1) * (qmax - 1);
        const unsigned __int128 room = ~(unsigned __int128)0 - qmax;
        const unsigned __int128 t = sq ? room / sq : (unsigned __int128)1 << 30;
        c->sum128_terms = t > ((unsigned __int128)1 << 30) ? 1u << 30 : (uint32_t)t;
        // a key inner product sums dnum products (one more for the c0 term of a lazy sum)
        if (c->dnum + 1 > c->sum128_terms)
            st = set_error(CKKS_EUNSUPPORTED, "dnum %u: %u products of residues below 2^%d exceed an exact 128-bit sum",
                           c->dnum, c->dnum + 1, 64 - __builtin_clzll(qmax));
    }
    if (st == CKKS_OK) st = build_tables(c);
    if (st == CKKS_OK) st = build_all_conv(c);
    if (st == CKKS_OK) noalloc_setup(c->device);
    if (st != CKKS_OK) {
        ckks_ctx_destroy(c);
        return st;
    }
    *out = c;
    return CKKS_OK;
}

void ckks_ctx_destroy(ckks_ctx *c)
{
    if (!c) return;
    (void)hipDeviceSynchronize();
    (void)prof_collect(c);
    if (c->scratch_external) c->scratch = nullptr;  // the caller's workspace
    void *ptrs[] = {c->d_mod, c->d_tw, c->d_itw, c->d_twf, c->d_itwf, c->d_fft_w, c->d_fft_wc, c->d_fft_twist, c->d_slot_pos,
                    c->d_pos_slot,
                    c->d_pinv, c->d_pmodq, c->d_qlinv, c->scratch};
    for (void *p : ptrs)
        if (p) (void)hipFree(p);
    for (auto &kv : c->conv) {
        if (kv.second.d_qhat_inv) (void)hipFree(kv.second.d_qhat_inv);
        if (kv.second.d_qhat_mod) (void)hipFree(kv.second.d_qhat_mod);
        if (kv.second.d_neg_q) (void)hipFree(kv.second.d_neg_q);
        if (kv.second.d_qhat_inv_f) (void)hipFree(kv.second.d_qhat_inv_f);
        if (kv.second.d_qhat_mod_f) (void)hipFree(kv.second.d_qhat_mod_f);
    }
    delete c;
}

ckks_status ckks_ctx_set_stream(ckks_ctx *c, void *stream)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "null context");
    c->stream = (hipStream_t)stream;
    return CKKS_OK;
}

ckks_status ckks_ctx_set_ntt_arith(ckks_ctx *c, int mode)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "null context");
    CK_REQUIRE(mode == 0 || mode == 1, CKKS_EINVAL, "ntt arithmetic mode %d is not 0 or 1", mode);
    c->int_only = mode == 1;
    return CKKS_OK;
}

ckks_status ckks_ctx_set_proj_batch(ckks_ctx *c, uint32_t max_pairs)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "null context");
    c->proj_max_pairs = max_pairs;
    return CKKS_OK;
}

ckks_status ckks_ctx_set_lazy_moddown(ckks_ctx *c, int on)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "null context");
    c->lazy_moddown = on != 0;
    return CKKS_OK;
}

ckks_status ckks_ctx_tables(const ckks_ctx *c, uint64_t *q, uint64_t *p, uint64_t *psi)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "null context");
    if (q) memcpy(q, c->primes.data(), c->n_q * sizeof(uint64_t));
    if (p) memcpy(p, c->primes.data() + c->n_q, c->n_p * sizeof(uint64_t));
    if (psi) memcpy(psi, c->psi.data(), c->psi.size() * sizeof(uint64_t));
    return CKKS_OK;
}

size_t ckks_workspace_bytes(const ckks_ctx *c, int op, const uint32_t *shape)
{
    clear_error();
    if (!c) {
        set_error(CKKS_EINVAL, "workspace_bytes: null context");
        return SIZE_MAX;
    }
    const size_t b = op_workspace_bytes(c, op, shape);
    if (b == SIZE_MAX) set_error(CKKS_EINVAL, "workspace_bytes: unknown op %d or invalid shape", op);
    return b;
}

ckks_status ckks_set_workspace(ckks_ctx *c, void *dev, size_t bytes)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "set_workspace: null context");
    CK_REQUIRE((dev == nullptr) == (bytes == 0), CKKS_EINVAL,
               "set_workspace: dev and bytes must be both set or both zero");
    CK_REQUIRE(((uintptr_t)dev & 255) == 0, CKKS_EINVAL, "set_workspace: dev must be 256-byte aligned");
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (c->scratch && !c->scratch_external) HIP_TRY(hipFree(c->scratch));
    c->scratch = dev;
    c->scratch_bytes = bytes;
    c->scratch_external = dev != nullptr;
    return CKKS_OK;
}

uint32_t ckks_galois_elt(const ckks_ctx *c, int32_t steps)
{
    if (!c) return 0;
    const int64_t half = c->n / 2;
    int64_t r = ((int64_t)steps % half + half) % half;
    return (uint32_t)hm::pw(5, (uint64_t)r, 2ull * c->n);
}

ckks_status ckks_profile_enable(ckks_ctx *c, int on)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "null context");
    c->profiling = on != 0;
    return CKKS_OK;
}
ckks_status ckks_profile_reset(ckks_ctx *c)
{
    clear_error();
    CK_REQUIRE(c, CKKS_EINVAL, "null context");
    CK_TRY(prof_collect(c));
    for (int k = 0; k < K_NCLASS; k++) {
        c->prof_ms[k] = 0;
        c->prof_bytes[k] = 0;
        c->prof_ops[k] = 0;
        c->prof_count[k] = 0;
    }
    return CKKS_OK;
}
ckks_status ckks_profile_read(ckks_ctx *c, const char *cls, double *total_ms, uint64_t *launches, double *bytes,
                              double *valu_ops)
{
    clear_error();
    CK_REQUIRE(c && cls, CKKS_EINVAL, "null argument");
    CK_TRY(prof_collect(c));
    for (int k = 0; k < K_NCLASS; k++) {
        if (strcmp(cls, kKClassNames[k]) == 0) {
            if (total_ms) *total_ms = c->prof_ms[k];
            if (launches) *launches = c->prof_count[k];
            if (bytes) *bytes = c->prof_bytes[k];
            if (valu_ops) *valu_ops = c->prof_ops[k];
            return CKKS_OK;
        }
    }
    return set_error(CKKS_EINVAL, "unknown kernel '%s'", cls);
}
const char *ckks_profile_name(int k) { return (k >= 0 && k < K_NCLASS) ? kKClassNames[k] : nullptr; }

}  // extern "C"
