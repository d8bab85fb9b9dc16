"""Plain, slow RNS-CKKS oracle (test infrastructure only).

The paper (Background, "The CKKS Computation Model") uses the CKKS primitives
Encode, Add, PCMult, Mult, Rot_k, KeySwitch and Rescale and delegates their
internals to an external library; its linear projections are the slot-diagonal
matrix-vector identity Ax = sum_k D_k(A) * rho^k(x) with the left rotation
(rho^k x)_i = x_{(i+k) mod D} (Section "Matrix Representations and Linear
Computation in CKKS", Eq. slot-diagonal-matvec), organised with baby-step /
giant-step (BSGS) reuse of rotations.  Everything below the primitive level
follows the standard RNS-CKKS literature:

* CKKS encoding through the canonical embedding (Cheon-Kim-Kim-Song 2017);
* the RNS representation, fast basis conversion and rescaling
  (Cheon-Han-Kim-Kim-Song 2018);
* hybrid key switching with dnum digits and special primes P (Han-Ki 2020);
* the negacyclic NTT with psi folded into the twiddles (Longa-Naehrig 2016).

Where the paper is silent the conventions are fixed here (each is a reading
recorded in the design notes): prime choice, psi, bit-reversed evaluation
order, round-half-away encode, centred uncorrected basis conversion,
centred rescale, sigma applied after ModUp, giant-step rotation before the
rescale, and the feature-major slot map s = f*T + t.

Arrays are numpy uint64 with rows [limb][N]; a ciphertext is [2][limbs][N] in
the NTT domain.  Scalars that need more than 64 bits are Python ints.
"""
import ctypes
import math
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import build as _build

__all__ = [
    "is_prime", "gen_primes", "find_psi", "Ckks", "lib",
]

_LIB = None


def lib():
    """Load (building if missing or stale) the oracle's C library."""
    global _LIB
    if _LIB is None:
        path = _build.build(force=False)
        L = ctypes.CDLL(path)
        u64p = np.ctypeslib.ndpointer(np.uint64, flags="C_CONTIGUOUS")
        i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")
        f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
        i64, u64, f64 = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
        L.or_ntt.argtypes = [u64p, i64, i64, u64, u64]
        L.or_intt.argtypes = [u64p, i64, i64, u64, u64]
        L.or_ntt_rows.argtypes = [u64p, i64, i64, u64p, u64p, ctypes.c_int]
        for name in ("or_mul", "or_add", "or_sub"):
            getattr(L, name).argtypes = [u64p, u64p, u64p, i64, i64, u64p]
        L.or_mul_scalar.argtypes = [u64p, u64p, u64p, i64, i64, u64p]
        L.or_reduce_i64.argtypes = [i64p, u64p, i64, i64, u64p]
        L.or_conv.argtypes = [u64p, u64p, i64, u64p, u64p, i64, i64, u64p, u64p]
        L.or_encode_round.argtypes = [f64p, ctypes.c_void_p, i64, f64, i64p]
        L.or_encode_def_round.argtypes = [f64p, ctypes.c_void_p, i64, f64, i64p, f64p]
        L.or_encode_unrounded.argtypes = [f64p, ctypes.c_void_p, i64, f64, f64p]
        L.or_philox4x64_10.argtypes = [u64p, u64p, u64p]
        L.or_philox4x64_10.restype = None
        L.or_expand_key_a.argtypes = [u64p, i64, u64p, i64, i64, u64p]
        L.or_expand_key_a.restype = None
        L.or_threads.argtypes = []
        L.or_threads.restype = ctypes.c_int
        L.or_set_threads.argtypes = [ctypes.c_int]
        L.or_set_threads.restype = None
        for name in ("or_ntt", "or_intt", "or_ntt_rows", "or_mul", "or_add", "or_sub", "or_mul_scalar",
                     "or_reduce_i64", "or_conv", "or_encode_round", "or_encode_def_round",
                     "or_encode_unrounded"):
            getattr(L, name).restype = None
        _LIB = L
    return _LIB


# ----------------------------------------------------------------------------
# Primes and roots (parameter generation)
# ----------------------------------------------------------------------------

def is_prime(n: int) -> bool:
    """Miller-Rabin with the bases 2..37, deterministic for n < 3.3e24."""
    if n < 2:
        return False
    small = (2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37)
    for p in small:
        if n % p == 0:
            return n == p
    d, s = n - 1, 0
    while d % 2 == 0:
        d //= 2
        s += 1
    for a in small:
        x = pow(a, d, n)
        if x in (1, n - 1):
            continue
        for _ in range(s - 1):
            x = x * x % n
            if x == n - 1:
                break
        else:
            return False
    return True


def gen_primes(bits: int, two_n: int, count: int) -> List[int]:
    """The `count` largest primes below 2^bits that are 1 mod 2N, in descending order."""
    out = []
    c = ((1 << bits) - 1) // two_n * two_n + 1
    if c >= (1 << bits):
        c -= two_n
    while len(out) < count:
        if c < (1 << (bits - 1)):
            raise ValueError("not enough %d-bit primes 1 mod %d" % (bits, two_n))
        if is_prime(c):
            out.append(c)
        c -= two_n
    return out


def find_psi(q: int, two_n: int) -> int:
    """psi = x^((q-1)/2N) mod q for the smallest x >= 2 with psi^N = -1 mod q."""
    assert (q - 1) % two_n == 0
    for x in range(2, 1 << 20):
        psi = pow(x, (q - 1) // two_n, q)
        if pow(psi, two_n // 2, q) == q - 1:
            return psi
    raise ValueError("no primitive 2N-th root found")


def bitrev(x: int, bits: int) -> int:
    return int(format(x, "0%db" % bits)[::-1], 2) if bits else 0


def _u64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.uint64)


class Ckks:
    """The oracle's scheme context: ring degree, modulus chain q_0..q_{L-1}, special primes P.

    Prime index k < n_q is q_k; n_q + j is p_j.  Ciphertext limbs are indexed by
    q-limb 0..level; extended (ModUp) polynomials hold limbs 0..level then p_0..p_{K-1}.
    """

    def __init__(self, log_n: int, q: Sequence[int], p: Sequence[int] = (), dnum: int = 1):
        self.log_n = log_n
        self.n = 1 << log_n
        self.q = [int(x) for x in q]
        self.p = [int(x) for x in p]
        self.n_q, self.n_p = len(self.q), len(self.p)
        self.dnum = dnum
        self.alpha = -(-self.n_q // dnum)
        self.primes = self.q + self.p
        self.psi = [find_psi(x, 2 * self.n) for x in self.primes]
        self.P = math.prod(self.p) if self.p else 1
        self._perm_cache: Dict[int, np.ndarray] = {}

    @classmethod
    def from_bits(cls, log_n: int, bits: int, n_q: int, n_p: int = 0, dnum: int = 1) -> "Ckks":
        pr = gen_primes(bits, 2 << log_n, n_q + n_p)
        return cls(log_n, pr[:n_q], pr[n_q:], dnum)

    # ---------------- index helpers ----------------
    def level_primes(self, level: int) -> List[int]:
        """Prime indices of a ciphertext at `level`: q_0..q_level."""
        return list(range(level + 1))

    def ext_primes(self, level: int) -> List[int]:
        """Prime indices of Q_level union P: q_0..q_level, p_0..p_{K-1}."""
        return list(range(level + 1)) + list(range(self.n_q, self.n_q + self.n_p))

    def mods(self, idx: Sequence[int]) -> np.ndarray:
        return np.array([self.primes[k] for k in idx], dtype=np.uint64)

    def digit_limbs(self, j: int, level: int) -> List[int]:
        """I_j intersected with [0, level]: the q-limbs of digit j available at `level`."""
        return [i for i in range(j * self.alpha, min((j + 1) * self.alpha, self.n_q)) if i <= level]

    def n_digits(self, level: int) -> int:
        return sum(1 for j in range(self.dnum) if self.digit_limbs(j, level))

    # ---------------- transforms ----------------
    def ntt(self, a: np.ndarray, idx: Sequence[int], inverse: bool = False) -> np.ndarray:
        """Forward (or inverse) negacyclic NTT of each row; row r uses prime idx[r]."""
        a = _u64(a).copy()
        lib().or_ntt_rows(a.reshape(-1), len(idx), self.n, self.mods(idx),
                          _u64([self.psi[k] for k in idx]), int(inverse))
        return a

    def intt(self, a: np.ndarray, idx: Sequence[int]) -> np.ndarray:
        return self.ntt(a, idx, inverse=True)

    def ntt_rows_same_prime(self, a: np.ndarray, k: int, inverse: bool = False) -> np.ndarray:
        """Transform every row of a [rows][N] array with prime k (the batched microbench form)."""
        a = _u64(a).copy()
        rows = a.size // self.n
        (lib().or_intt if inverse else lib().or_ntt)(a.reshape(-1), rows, self.n, self.primes[k],
                                                        self.psi[k])
        return a

    # ---------------- element-wise ----------------
    def _ew(self, fn, a, b, idx):
        a, b = _u64(a), _u64(b)
        out = np.empty_like(a)
        L = len(idx)
        fn(a.reshape(-1), b.reshape(-1), out.reshape(-1), L, self.n, self.mods(idx))
        return out

    def mul(self, a, b, idx):
        return self._ew(lib().or_mul, a, b, idx)

    def add(self, a, b, idx):
        return self._ew(lib().or_add, a, b, idx)

    def sub(self, a, b, idx):
        return self._ew(lib().or_sub, a, b, idx)

    def mul_scalar(self, a, consts: Sequence[int], idx):
        a = _u64(a)
        out = np.empty_like(a)
        lib().or_mul_scalar(a.reshape(-1), _u64([c % self.primes[k] for c, k in zip(consts, idx)]),
                            out.reshape(-1), len(idx), self.n, self.mods(idx))
        return out

    def reduce_int(self, v: np.ndarray, idx: Sequence[int]) -> np.ndarray:
        """Signed int64 coefficient vector -> residues [len(idx)][N]."""
        v = np.ascontiguousarray(v, dtype=np.int64)
        out = np.empty((len(idx), self.n), dtype=np.uint64)
        lib().or_reduce_i64(v, out.reshape(-1), len(idx), self.n, self.mods(idx))
        return out

    # ---------------- automorphism (NTT domain) ----------------
    def galois_elt(self, steps: int) -> int:
        """Galois element 5^r mod 2N for a left slot rotation by r (negative r wraps mod N/2)."""
        return pow(5, steps % (self.n // 2), 2 * self.n)

    def auto_perm(self, g: int) -> np.ndarray:
        """perm[j] = j' with 2*brev(j')+1 = (2*brev(j)+1)*g mod 2N: sigma_g(A)[j] = A[perm[j]].

        NTT index j holds the evaluation at psi^(2 brev(j) + 1); sigma_g(a)(X) = a(X^g) evaluated
        there equals a at psi^((2 brev(j) + 1) g)."""
        if g not in self._perm_cache:
            n, lg = self.n, self.log_n
            br = np.array([bitrev(j, lg) for j in range(n)], dtype=np.int64)
            k = ((2 * br + 1) * g) % (2 * n)
            self._perm_cache[g] = br[(k - 1) // 2]
        return self._perm_cache[g]

    def automorph(self, a: np.ndarray, g: int) -> np.ndarray:
        return np.ascontiguousarray(_u64(a)[..., self.auto_perm(g)])

    # ---------------- encode / decode ----------------
    def encode_int(self, zr: np.ndarray, zi: Optional[np.ndarray], delta: float) -> np.ndarray:
        """Rounded integer coefficients of Encode_delta(z) (fp64, fixed evaluation order)."""
        zr = np.ascontiguousarray(zr, dtype=np.float64)
        assert zr.shape == (self.n // 2,)
        m = np.empty(self.n, dtype=np.int64)
        if zi is None:
            lib().or_encode_round(zr, None, self.n, float(delta), m)
        else:
            zi = np.ascontiguousarray(zi, dtype=np.float64)
            lib().or_encode_round(zr, zi.ctypes.data, self.n, float(delta), m)
        return m

    def encode_unrounded(self, zr, zi, delta: float) -> np.ndarray:
        """The fp64 values whose rounding (half away from zero) gives encode_int."""
        zr = np.ascontiguousarray(zr, dtype=np.float64)
        x = np.empty(self.n, dtype=np.float64)
        lib().or_encode_unrounded(zr, None if zi is None else np.ascontiguousarray(zi, dtype=np.float64).ctypes.data,
                                  self.n, float(delta), x)
        return x

    def encode_int_def(self, zr, zi, delta):
        """Definitional O(N^2) encode in long double: (rounded ints, distance of each to a tie)."""
        zr = np.ascontiguousarray(zr, dtype=np.float64)
        m = np.empty(self.n, dtype=np.int64)
        d = np.empty(self.n, dtype=np.float64)
        if zi is None:
            lib().or_encode_def_round(zr, None, self.n, float(delta), m, d)
        else:
            zi = np.ascontiguousarray(zi, dtype=np.float64)
            lib().or_encode_def_round(zr, zi.ctypes.data, self.n, float(delta), m, d)
        return m, d

    def encode(self, zr, zi, delta: float, n_limbs: int) -> np.ndarray:
        """Plaintext in the NTT domain over q_0..q_{n_limbs-1}."""
        idx = list(range(n_limbs))
        return self.ntt(self.reduce_int(self.encode_int(zr, zi, delta), idx), idx)

    def encode_periodic(self, u, delta: float, n_limbs: int) -> np.ndarray:
        """Plaintext (NTT domain, limbs q_0..q_{n_limbs-1}) of the slot vector z[t*D + f] = u[f], period D = len(u).

        A slot vector of period D (a power of two) is fixed by the automorphisms X -> X^a, a = 1 mod 4D, so
        its encoding is a polynomial in X^(N/2D): m(X) = m'(X^(N/2D)) with m' the encoding of the D values u
        in the ring of degree 2D (the same fp64 evaluation and rounding rule as encode, run at degree 2D).
        Zero coefficients stay exactly zero, so the plaintext's NTT values are constant over runs of N/2D
        consecutive (bit-reversed) indices."""
        u = np.ascontiguousarray(u, dtype=np.float64)
        D = u.shape[0]
        assert D >= 1 and D & (D - 1) == 0 and 2 * D <= self.n
        mp = np.empty(2 * D, dtype=np.int64)
        lib().or_encode_round(u, None, 2 * D, float(delta), mp)
        m = np.zeros(self.n, dtype=np.int64)
        m[::self.n // (2 * D)] = mp
        idx = list(range(n_limbs))
        return self.ntt(self.reduce_int(m, idx), idx)

    def lift_centered(self, rows: np.ndarray, idx: Sequence[int]) -> List[int]:
        """Coefficient residues -> the centred integer in (-Q/2, Q/2] by CRT (Python big ints)."""
        mods = [self.primes[k] for k in idx]
        Q = math.prod(mods)
        out = [0] * self.n
        parts = []
        for r, qk in enumerate(mods):
            Qh = Q // qk
            parts.append((Qh, pow(Qh, -1, qk), qk))
        cols = [rows[r].tolist() for r in range(len(mods))]
        for j in range(self.n):
            x = 0
            for r, (Qh, inv, qk) in enumerate(parts):
                x += (cols[r][j] * inv % qk) * Qh
            x %= Q
            out[j] = x - Q if x > Q // 2 else x
        return out

    def decode(self, pt: np.ndarray, scale: float) -> np.ndarray:
        """Slots z_j = scale^-1 * sum_i m_i zeta^(i e_j), m the centred CRT lift of INTT(pt)."""
        L = pt.shape[0]
        idx = list(range(L))
        m = self.lift_centered(self.intt(pt, idx), idx)
        mf = np.array([float(x) for x in m], dtype=np.float64)
        return self.decode_coeffs(mf, scale)

    def decode_coeffs(self, mf: np.ndarray, scale: float) -> np.ndarray:
        n, M = self.n, self.n // 2
        zeta = np.exp(1j * np.pi * np.arange(M) / n)
        # sum_{i<N} m_i zeta^(i(4s+1)) = sum_{i<M} (m_i + i*m_{i+M}) zeta^i omega^(i s), omega = zeta^4
        x = (mf[:M] + 1j * mf[M:]) * zeta
        Y = np.fft.ifft(x) * M
        e = np.array([pow(5, j, 2 * n) for j in range(M)], dtype=np.int64)
        return Y[(e - 1) // 4] / scale

    # ---------------- encryption ----------------
    def secret_ntt(self, s: np.ndarray, idx: Sequence[int]) -> np.ndarray:
        return self.ntt(self.reduce_int(np.asarray(s, dtype=np.int64), idx), idx)

    def encrypt(self, s, pt: np.ndarray, a: np.ndarray, e: np.ndarray) -> np.ndarray:
        """ct = (-a*s + e + m, a) over the limbs of pt (a given in the NTT domain)."""
        L = pt.shape[0]
        idx = list(range(L))
        sn = self.secret_ntt(s, idx)
        en = self.ntt(self.reduce_int(np.asarray(e, dtype=np.int64), idx), idx)
        a = _u64(a)[:L]
        c0 = self.add(self.sub(en, self.mul(a, sn, idx), idx), pt, idx)
        return np.stack([c0, a.copy()])

    def decrypt(self, s, ct: np.ndarray) -> np.ndarray:
        L = ct.shape[1]
        idx = list(range(L))
        sn = self.secret_ntt(s, idx)
        return self.add(ct[0], self.mul(ct[1], sn, idx), idx)

    def _keygen(self, s, target_ntt_all: np.ndarray, a: np.ndarray, e: np.ndarray) -> np.ndarray:
        """Key [dnum][2][n_q+n_p][N]: b_j = -a_j s + e_j + [P]_{q_i} * t * [i in I_j], key_j = (b_j, a_j)."""
        idx = list(range(self.n_q + self.n_p))
        sn = self.secret_ntt(s, idx)
        key = np.empty((self.dnum, 2, len(idx), self.n), dtype=np.uint64)
        for j in range(self.dnum):
            aj = _u64(a[j])
            ej = self.ntt(self.reduce_int(np.asarray(e[j], dtype=np.int64), idx), idx)
            bj = self.sub(ej, self.mul(aj, sn, idx), idx)
            lim = list(range(j * self.alpha, min((j + 1) * self.alpha, self.n_q)))
            if lim:
                gad = self.mul_scalar(target_ntt_all[lim], [self.P % self.q[i] for i in lim], lim)
                bj[lim] = self.add(bj[lim], gad, lim)
            key[j, 0] = bj
            key[j, 1] = aj
        return key

    def keygen_galois(self, s, g: int, a: np.ndarray, e: np.ndarray) -> np.ndarray:
        """Switching key from sigma_g(s) to s."""
        idx = list(range(self.n_q + self.n_p))
        return self._keygen(s, self.automorph(self.secret_ntt(s, idx), g), a, e)

    # ---------------- seed-expanded keys ----------------
    @staticmethod
    def philox(ctr: Sequence[int], key: Sequence[int]) -> List[int]:
        """One Philox-4x64-10 block (Salmon et al., SC 2011) of counter ctr (4 words) under key (2 words)."""
        out = np.empty(4, dtype=np.uint64)
        lib().or_philox4x64_10(_u64(ctr), _u64(key), out)
        return [int(x) for x in out]

    def expand_key_a(self, seed: Sequence[int]) -> np.ndarray:
        """The uniform half [dnum][n_q+n_p][N] (NTT domain) that the 128-bit seed stands for: residue n of prime k in
        digit j is the first w >> (64 - b) below q over the words j mod 4 of the blocks Philox-4x64-10((n, k, j/4, t),
        seed), t = 0, 1, ... (b = bit length of q; after 64 rejections w mod q)."""
        out = np.empty((self.dnum, len(self.primes), self.n), dtype=np.uint64)
        lib().or_expand_key_a(_u64(seed), self.dnum, _u64(self.primes), len(self.primes), self.n, out.reshape(-1))
        return out

    def keygen_galois_seeded(self, s, g: int, seed: Sequence[int], e: np.ndarray) -> np.ndarray:
        """The b half [dnum][n_q+n_p][N] of the Galois key for g whose a half is expand_key_a(seed)."""
        return np.ascontiguousarray(self.keygen_galois(s, g, self.expand_key_a(seed), e)[:, 0])

    def seeded_key(self, b: np.ndarray, seed: Sequence[int]) -> np.ndarray:
        """The full key (b_j, a_j) a seeded key (b half, seed) stands for: the oracle's seeded mode is the plain key
        switching with this key."""
        return np.ascontiguousarray(np.stack([b, self.expand_key_a(seed)], axis=1))

    def keygen_relin(self, s, a: np.ndarray, e: np.ndarray) -> np.ndarray:
        """Switching key from s^2 to s."""
        idx = list(range(self.n_q + self.n_p))
        sn = self.secret_ntt(s, idx)
        return self._keygen(s, self.mul(sn, sn, idx), a, e)

    # ---------------- basis conversion, ModUp, ModDown ----------------
    def conv(self, coef: np.ndarray, src: Sequence[int], dst: Sequence[int]) -> np.ndarray:
        """Fast basis conversion of coefficient rows from primes src to primes dst (centred digits
        y_i in (-q_i/2, q_i/2], no overflow correction): result = x + u * Q_src, x the centred
        representative modulo Q_src and |u| <= len(src) // 2."""
        qs = [self.primes[k] for k in src]
        qt = [self.primes[k] for k in dst]
        Qs = math.prod(qs)
        qhat_inv = [pow(Qs // qi, -1, qi) for qi in qs]
        qhat_t = [(Qs // qi) % t for qi in qs for t in qt]
        out = np.empty((len(dst), self.n), dtype=np.uint64)
        lib().or_conv(_u64(coef).reshape(-1), _u64(qs), len(qs), out.reshape(-1), _u64(qt), len(qt),
                      self.n, _u64(qhat_inv), _u64(qhat_t))
        return out

    def modup(self, c: np.ndarray, level: int) -> np.ndarray:
        """Digits [n_digits][level+1+K][N] (NTT domain) of an NTT-domain polynomial at `level`."""
        ext = self.ext_primes(level)
        nd = self.n_digits(level)
        out = np.empty((nd, len(ext), self.n), dtype=np.uint64)
        for j in range(nd):
            I = self.digit_limbs(j, level)
            coef = self.intt(c[I], I)
            tgt_pos = [r for r, k in enumerate(ext) if k not in I]
            tgt = [ext[r] for r in tgt_pos]
            conv = self.ntt(self.conv(coef, I, tgt), tgt)
            out[j, I] = c[I]
            out[j, tgt_pos] = conv
        return out

    def moddown(self, x: np.ndarray, level: int) -> np.ndarray:
        """[level+1+K][N] over Q_l u P  ->  round-free (x - Conv_{P->Q}([x]_P)) * P^-1 over Q_l."""
        ql = self.level_primes(level)
        pidx = list(range(self.n_q, self.n_q + self.n_p))
        xp = self.intt(x[level + 1:], pidx)
        conv = self.ntt(self.conv(xp, pidx, ql), ql)
        diff = self.sub(x[:level + 1], conv, ql)
        return self.mul_scalar(diff, [pow(self.P % self.q[i], -1, self.q[i]) for i in ql], ql)

    def _key_rows(self, key: np.ndarray, level: int) -> np.ndarray:
        return key[:, :, self.ext_primes(level), :]

    def key_inner(self, digits: np.ndarray, key: np.ndarray, level: int, g: Optional[int]):
        """(u0, u1) = sum_j sigma_g(d_j) * (b_j, a_j) over Q_level u P (g None: no sigma)."""
        ext = self.ext_primes(level)
        kr = self._key_rows(key, level)
        u = [np.zeros((len(ext), self.n), dtype=np.uint64) for _ in range(2)]
        for j in range(digits.shape[0]):
            d = digits[j] if g is None else self.automorph(digits[j], g)
            for k in range(2):
                u[k] = self.add(u[k], self.mul(d, kr[j, k], ext), ext)
        return u

    def keyswitch_digits(self, digits: np.ndarray, key: np.ndarray, level: int, g: Optional[int]):
        """(u0, u1) = sum_j sigma_g(d_j) * (b_j, a_j), then ModDown of each (g None: no sigma)."""
        u = self.key_inner(digits, key, level, g)
        return self.moddown(u[0], level), self.moddown(u[1], level)

    def rotate_sum_lazy(self, cts: Sequence[np.ndarray], steps: Sequence[int], keys: Sequence[np.ndarray]):
        """sum_r Rot_{steps[r]}(cts[r]) with one ModDown: the key-switching inner products of all terms are summed
        over Q_level u P together with P * sigma_r(c0_r) (zero modulo P), and the sum is divided by P once.
        ModDown(x + P y) = ModDown(x) + y exactly, so one term gives the rotation bit for bit; with several
        terms only the rounding of the division differs from summing separately rotated ciphertexts (the lazy
        ModDown across a sum of rotations of the key-switching literature, e.g. Bossuat et al. 2021)."""
        level = self.level_of(cts[0])
        ext = self.ext_primes(level)
        ql = self.level_primes(level)
        u = [np.zeros((len(ext), self.n), dtype=np.uint64) for _ in range(2)]
        pq = [self.P % self.q[i] for i in ql]
        for ct, st, key in zip(cts, steps, keys):
            g = self.galois_elt(st)
            t = self.key_inner(self.modup(ct[1], level), key, level, g)
            c0 = self.mul_scalar(self.automorph(ct[0], g), pq, ql)
            u[0] = self.add(u[0], t[0], ext)
            u[1] = self.add(u[1], t[1], ext)
            u[0][:level + 1] = self.add(u[0][:level + 1], c0, ql)
        return np.stack([self.moddown(u[0], level), self.moddown(u[1], level)])

    # ---------------- ciphertext operations ----------------
    @staticmethod
    def level_of(ct: np.ndarray) -> int:
        return ct.shape[1] - 1

    def ct_add(self, a, b):
        idx = self.level_primes(self.level_of(a))
        return np.stack([self.add(a[0], b[0], idx), self.add(a[1], b[1], idx)])

    def ct_mul_plain(self, ct, pt):
        idx = self.level_primes(self.level_of(ct))
        return np.stack([self.mul(ct[0], pt, idx), self.mul(ct[1], pt, idx)])

    def rescale(self, ct: np.ndarray) -> np.ndarray:
        """Divide by q_l with rounding: t = centred INTT(c_l); c_i' = (c_i - NTT_i(t)) q_l^-1."""
        level = self.level_of(ct)
        ql = self.q[level]
        low = self.level_primes(level - 1)
        out = np.empty((2, level, self.n), dtype=np.uint64)
        for k in range(2):
            t = self.intt(ct[k, level:level + 1], [level])[0].astype(object)
            tc = np.array([int(x) - ql if int(x) > ql // 2 else int(x) for x in t], dtype=np.int64)
            tr = self.ntt(self.reduce_int(tc, low), low)
            diff = self.sub(ct[k, :level], tr, low)
            out[k] = self.mul_scalar(diff, [pow(ql, -1, self.q[i]) for i in low], low)
        return out

    def rotate(self, ct: np.ndarray, steps: int, key: np.ndarray) -> np.ndarray:
        """Left slot rotation by `steps` with the Galois key for g = 5^steps."""
        return self.rotate_hoisted(ct, [steps], [key])[0]

    def rotate_hoisted(self, ct: np.ndarray, steps: Sequence[int], keys: Sequence[np.ndarray]):
        """One ModUp of c1 shared by all rotations; sigma_g acts on the ModUp digits."""
        level = self.level_of(ct)
        idx = self.level_primes(level)
        digits = self.modup(ct[1], level)
        outs = []
        for r, key in zip(steps, keys):
            g = self.galois_elt(r)
            u0, u1 = self.keyswitch_digits(digits, key, level, g)
            outs.append(np.stack([self.add(self.automorph(ct[0], g), u0, idx), u1]))
        return outs

    def tensor(self, a: np.ndarray, b: np.ndarray) -> np.ndarray:
        """(d0, d1, d2) = (a0 b0, a0 b1 + a1 b0, a1 b1): the product decrypting under (1, s, s^2)."""
        idx = self.level_primes(self.level_of(a))
        d0 = self.mul(a[0], b[0], idx)
        d1 = self.add(self.mul(a[0], b[1], idx), self.mul(a[1], b[0], idx), idx)
        d2 = self.mul(a[1], b[1], idx)
        return np.stack([d0, d1, d2])

    def relin(self, d: np.ndarray, rlk: np.ndarray) -> np.ndarray:
        """Key switching of d2 from s^2 to s: (d0 + u0, d1 + u1)."""
        level = d.shape[1] - 1
        idx = self.level_primes(level)
        u0, u1 = self.keyswitch_digits(self.modup(d[2], level), rlk, level, None)
        return np.stack([self.add(d[0], u0, idx), self.add(d[1], u1, idx)])

    def mul_relin(self, a: np.ndarray, b: np.ndarray, rlk: np.ndarray) -> np.ndarray:
        return self.relin(self.tensor(a, b), rlk)

    # ---------------- the projection ----------------
    @staticmethod
    def diag_slot_vector(W: np.ndarray, T: int, D: int, j: int, i: int, n1: int, g: int, b: int) -> np.ndarray:
        """Slots of plaintext (j, i, g, b) in the feature-major layout s = f*T + t:
        p[f*T + t] = D_{n1 g + b}(A_{j,i})[(f - n1 g) mod D] with A = W^T, block
        A_{j,i} = W[iD:(i+1)D, jD:(j+1)D]^T and D_k(A)[o] = A[o, (o + k) mod D]."""
        k = n1 * g + b
        f = np.arange(D)
        o = (f - n1 * g) % D
        vals = W[i * D + (o + k) % D, j * D + o]
        return np.repeat(vals, T)

    @staticmethod
    def periodic_diag_vectors(W: np.ndarray, D: int, j: int, i: int, n1: int, g: int, b: int):
        """One period (D values) of the two plaintexts of (j, i, g, b) in the token-major layout s = t*D + f.

        With A = W^T, A_{j,i} = W[iD:(i+1)D, jD:(j+1)D]^T and k = n1 g + b, the diagonal D_k(A)[o] =
        A[o, (o + k) mod D] splits by whether o + k wraps past D: U_k keeps the entries with o + k < D, V_k
        the others.  A left rotation by k of a token-major ciphertext moves feature o + k of the same token to
        feature o only when o + k < D; the wrapped entries need the rotation by k - D instead, so
            y = sum_k U_k * rho^k(x) + V_k * rho^(k-D)(x).
        The giant step rho^(n1 g) is factored out as in the feature-major case, which rotates both vectors
        right by n1 g: returned are U[o] = U_k[(o - n1 g) mod D] and V[o] = V_k[(o - n1 g) mod D]."""
        k = n1 * g + b
        o = (np.arange(D) - n1 * g) % D
        wraps = o + k >= D
        vals = W[i * D + (o + k) % D, j * D + o]
        return np.where(wraps, 0.0, vals), np.where(wraps, vals, 0.0)

    def linear_project_tm(self, cts: Sequence[np.ndarray], W: np.ndarray, T: int, n1: int,
                          keys: Dict[int, np.ndarray], out_blocks: Optional[Sequence[int]] = None,
                          lazy: bool = False):
        """The projection in the token-major layout s = t*D + f (input i holds features [iD, (i+1)D) of every
        token):
            out_j = Rescale( sum_g Rot_{n1 g}( sum_{i,b} U_{j,i,g,b} * Rot_b(x_i) + V_{j,i,g,b} * Rot_{b-D}(x_i) ) )
        with U, V from periodic_diag_vectors, encoded with encode_periodic at scale q_level.  Keys: steps
        b (0 < b < n1), b - D (0 <= b < n1) and n1 g (0 < g < n2)."""
        level = self.level_of(cts[0])
        D = (self.n // 2) // T
        d_in, d_out = W.shape
        n_in, n_out = d_in // D, d_out // D
        n2 = -(-D // n1)
        delta_w = float(self.q[level])
        xr, xw = [], []
        for i in range(n_in):
            steps = [b for b in range(1, n1)] + [b - D for b in range(n1)]
            rots = self.rotate_hoisted(cts[i], steps, [keys[s] for s in steps])
            xr.append([cts[i]] + rots[:n1 - 1])
            xw.append(rots[n1 - 1:])
        outs = []
        for j in (range(n_out) if out_blocks is None else out_blocks):
            total = None
            for g in range(n2):
                acc = None
                for i in range(n_in):
                    for b in range(n1):
                        if n1 * g + b >= D:
                            continue
                        uu, vv = self.periodic_diag_vectors(W, D, j, i, n1, g, b)
                        for vec, x in ((uu, xr[i][b]), (vv, xw[i][b])):
                            term = self.ct_mul_plain(x, self.encode_periodic(vec, delta_w, level + 1))
                            acc = term if acc is None else self.ct_add(acc, term)
                total = self._giant_step(total, acc, g, n1 * g, keys, lazy)
            outs.append(self.rescale(self._giant_finish(total, lazy)))
        return outs

    # ---------------- the attention block (token-major) ----------------
    @staticmethod
    def attention_mask(D: int, hd: int, c: int) -> np.ndarray:
        """One period (D features) of the mask M_c: 1 at the features f = c mod hd, position c of every head."""
        u = np.zeros(D)
        u[c::hd] = 1.0
        return u

    def attention_scores(self, q_cts: Sequence[np.ndarray], k_cts: Sequence[np.ndarray], k_of_q: Sequence[int],
                         T: int, hd: int, rlk: np.ndarray, keys: Dict[int, np.ndarray], lazy: bool = False):
        """Scores of one attention block in the token-major layout s = t*D + f, heads of hd features.

        Query ciphertext c holds D/hd heads, slot t*D + h*hd + d = Q[t, h, d]; key ciphertext k_of_q[c] holds
        one key head repeated in every head position, K'[t*D + h*hd + d] = K[t, d].  The output holds the
        scores on cyclic token diagonals: slot t*D + h*hd + delta = sum_d Q[t, h, d] K[(t + delta) mod T, d]
        for delta < T, 0 for T <= delta < hd: the scores on token diagonals (the S_Delta of Section "C--Delta
        Attention Layout and Computation", for which the paper gives no construction; this one is QK^T as Mult
        plus rotation sums):
            P_delta = Relin(Rot_{-delta}(Q) x Rot_{delta (D-1)}(K'))                  (0 <= delta < T)
            out     = Rescale(Rescale( sum_k Rot_k( sum_delta M_{(delta + k) mod hd} * P_delta ) ))  (0 <= k < hd)
        With the left rotation (Rot_k x)[s] = x[s + k], slot t*D + h*hd + delta + d of P_delta holds
        Q[t, h, d] K[t + delta, d]; M_c selects head position c, so the term k brings position delta + k of
        P_delta to position delta: the sum over k is the dot product over d, placed at position delta.
        The masks are periodic plaintexts encoded at scale q_level and multiply the products at the inputs' level
        (no rescale in between); the two rescales at the end divide by q_level and q_(level-1), so the output
        scale is scale(Q) scale(K) / q_(level-1).  Keys: -delta and delta (D - 1) (0 < delta < T), k (0 < k < hd).
        With `lazy` the hd - 1 rotations of the outer sum share one ModDown (rotate_sum_lazy)."""
        level = self.level_of(q_cts[0])
        D = (self.n // 2) // T
        assert T <= hd and D % hd == 0 and level >= 2
        masks = [self.encode_periodic(self.attention_mask(D, hd, c), float(self.q[level]), level + 1)
                 for c in range(hd)]
        bcache = {}
        outs = []
        for c, q in enumerate(q_cts):
            kk = k_of_q[c]
            if kk not in bcache:
                st = [d * (D - 1) for d in range(1, T)]
                bcache[kk] = [k_cts[kk]] + self.rotate_hoisted(k_cts[kk], st, [keys[s] for s in st])
            B = bcache[kk]
            st = [-d for d in range(1, T)]
            A = [q] + self.rotate_hoisted(q, st, [keys[s] for s in st])
            P = [self.mul_relin(A[d], B[d], rlk) for d in range(T)]
            total = None
            for k in range(hd):
                U = None
                for d in range(T):
                    term = self.ct_mul_plain(P[d], masks[(d + k) % hd])
                    U = term if U is None else self.ct_add(U, term)
                total = self._giant_step(total, U, k, k, keys, lazy)
            outs.append(self.rescale(self.rescale(self._giant_finish(total, lazy))))
        return outs

    def attention_apply(self, p_cts: Sequence[np.ndarray], v_cts: Sequence[np.ndarray], v_of_p: Sequence[int],
                        T: int, hd: int, rlk: np.ndarray, keys: Dict[int, np.ndarray]):
        """Weighted sums of values consuming scores in the layout attention_scores writes.

        p_cts[c] holds P[t, h, delta] at slot t*D + h*hd + delta (delta < T; the positions delta >= T are not
        read); value ciphertext v_of_p[c] holds one value head repeated in every head position, V'[t*D + h*hd
        + d] = V[t, d].  The output holds O[t, h, d] = sum_delta P[t, h, delta] V[(t + delta) mod T, d] at slot
        t*D + h*hd + d.  Broadcasting position delta over a head is sum_d M_d * Rot_(delta - d)(P); with
        j = delta - d:
            R_delta = Rot_{delta D}(V')                                                (0 <= delta < T)
            C_j     = Rescale( sum_delta M_{delta - j} * R_delta )  over 0 <= delta - j < hd  (-hd < j < T)
            out     = Rescale(Relin( sum_j Rot_j(P) x C_j ))
        C_j is computed at the value ciphertexts' level, rescaled (masks at scale q_(level of V)) and then
        reduced to the scores' limbs (the scores' level must be below the values'); out has scale
        scale(P) scale(V) / q_(level of P).  Keys: delta D (0 < delta < T), j (-hd < j < T, j != 0)."""
        lp, lv = self.level_of(p_cts[0]), self.level_of(v_cts[0])
        D = (self.n // 2) // T
        assert T <= hd and D % hd == 0 and 1 <= lp <= lv - 1
        masks = [self.encode_periodic(self.attention_mask(D, hd, c), float(self.q[lv]), lv + 1) for c in range(hd)]
        js = list(range(-(hd - 1), T))
        ccache = {}
        outs = []
        for c, p in enumerate(p_cts):
            kk = v_of_p[c]
            if kk not in ccache:
                st = [d * D for d in range(1, T)]
                R = [v_cts[kk]] + self.rotate_hoisted(v_cts[kk], st, [keys[s] for s in st])
                C = {}
                for j in js:
                    acc = None
                    for d in range(T):
                        if 0 <= d - j < hd:
                            term = self.ct_mul_plain(R[d], masks[d - j])
                            acc = term if acc is None else self.ct_add(acc, term)
                    C[j] = np.ascontiguousarray(self.rescale(acc)[:, :lp + 1])
                ccache[kk] = C
            C = ccache[kk]
            st = [j for j in js if j != 0]
            E = dict(zip(st, self.rotate_hoisted(p, st, [keys[s] for s in st])))
            E[0] = p
            idx = self.level_primes(lp)
            acc = None
            for j in js:
                d = self.tensor(E[j], C[j])
                acc = d if acc is None else np.stack([self.add(acc[i], d[i], idx) for i in range(3)])
            outs.append(self.rescale(self.relin(acc, rlk)))
        return outs

    def linear_project(self, cts: Sequence[np.ndarray], W: np.ndarray, T: int, n1: int,
                       keys: Dict[int, np.ndarray], out_blocks: Optional[Sequence[int]] = None,
                       lazy: bool = False):
        """out_j = Rescale( sum_g Rot_{T n1 g}( sum_{i,b} pt_{j,i,g,b} * Rot_{T b}(x_i) ) ).

        Plaintext scale is q_level, so the rescale returns the ciphertext scale unchanged.
        `out_blocks` restricts the computation to the listed output ciphertexts; `lazy` sums the giant-step
        rotations with one ModDown (rotate_sum_lazy)."""
        level = self.level_of(cts[0])
        idx = self.level_primes(level)
        D = (self.n // 2) // T
        d_in, d_out = W.shape
        n_in, n_out = d_in // D, d_out // D
        n2 = -(-D // n1)
        delta_w = float(self.q[level])
        xrot = []
        for i in range(n_in):
            steps = [T * b for b in range(1, n1)]
            rots = self.rotate_hoisted(cts[i], steps, [keys[s] for s in steps]) if steps else []
            xrot.append([cts[i]] + rots)
        outs = []
        for j in (range(n_out) if out_blocks is None else out_blocks):
            total = None
            for g in range(n2):
                acc = None
                for i in range(n_in):
                    for b in range(n1):
                        if n1 * g + b >= D:
                            continue
                        z = self.diag_slot_vector(W, T, D, j, i, n1, g, b)
                        pt = self.encode(z, None, delta_w, level + 1)
                        term = self.ct_mul_plain(xrot[i][b], pt)
                        acc = term if acc is None else self.ct_add(acc, term)
                total = self._giant_step(total, acc, g, T * n1 * g, keys, lazy)
            outs.append(self.rescale(self._giant_finish(total, lazy)))
        return outs

    def _giant_step(self, total, acc, g: int, step: int, keys, lazy: bool):
        """Add the giant-step partial sum acc (rotated by step for g > 0) to total; with lazy, total is
        (partial sum of g = 0, [rotated terms]) and the rotations are summed by _giant_finish."""
        if lazy:
            if g == 0:
                return (acc, [], [], [])
            total[1].append(acc)
            total[2].append(step)
            total[3].append(keys[step])
            return total
        if g > 0:
            acc = self.rotate(acc, step, keys[step])
        return acc if total is None else self.ct_add(total, acc)

    def _giant_finish(self, total, lazy: bool):
        if not lazy:
            return total
        base, terms, steps, ks = total
        return self.ct_add(base, self.rotate_sum_lazy(terms, steps, ks)) if terms else base
