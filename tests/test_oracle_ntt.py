"""Pins for the oracle's negacyclic NTT.

* brute force: INTT(NTT(a) * NTT(b)) equals the schoolbook negacyclic product
  a*b mod (X^N + 1, q), computed here with Python integers;
* definition: NTT(a)[j] = sum_i a_i psi^((2 brev(j) + 1) i) mod q, written out
  as an O(N^2) Python loop;
* round trip at the full ring degree 2^16.
The primes are those of the 2^16 chain (1 mod 2^17), which are also 1 mod 2N
for the small N used here.
"""
import numpy as np
import pytest

from oracle import Ckks, find_psi, gen_primes
from workloads import rng, uniform_residues

CHAIN50 = gen_primes(50, 1 << 17, 36)


def bitrev(x, bits):
    r = 0
    for _ in range(bits):
        r = (r << 1) | (x & 1)
        x >>= 1
    return r


def _schoolbook_negacyclic(a, b, q):
    n = len(a)
    out = [0] * n
    for i in range(n):
        for j in range(n):
            k = i + j
            if k < n:
                out[k] += a[i] * b[j]
            else:
                out[k - n] -= a[i] * b[j]
    return [x % q for x in out]


def _ntt_definition(a, q, psi):
    n = len(a)
    lg = n.bit_length() - 1
    return [sum(a[i] * pow(psi, (2 * bitrev(j, lg) + 1) * i, q) for i in range(n)) % q for j in range(n)]


@pytest.mark.parametrize("log_n", [4, 8])
@pytest.mark.parametrize("pi", [0, 17, 35])
def test_ntt_product_is_negacyclic_convolution(log_n, pi):
    q = CHAIN50[pi]
    ck = Ckks(log_n, [q])
    g = rng(2, 1, extra=log_n * 100 + pi)
    a = uniform_residues(g, [q], ck.n)
    b = uniform_residues(g, [q], ck.n)
    A, B = ck.ntt(a, [0]), ck.ntt(b, [0])
    c = ck.intt(ck.mul(A, B, [0]), [0])
    want = _schoolbook_negacyclic([int(x) for x in a[0]], [int(x) for x in b[0]], q)
    assert [int(x) for x in c[0]] == want


@pytest.mark.parametrize("log_n", [2, 4, 6, 8])
def test_ntt_matches_definition(log_n):
    q = CHAIN50[3]
    ck = Ckks(log_n, [q])
    a = uniform_residues(rng(2, 1, extra=7 + log_n), [q], ck.n)
    got = [int(x) for x in ck.ntt(a, [0])[0]]
    assert got == _ntt_definition([int(x) for x in a[0]], q, find_psi(q, 2 * ck.n))


def test_ntt_of_monomials():
    # NTT(X^k)[j] = psi^((2 brev(j)+1) k): a closed form for single coefficients
    q = CHAIN50[5]
    ck = Ckks(10, [q])
    psi = ck.psi[0]
    for k in (0, 1, 513, 1023):
        a = np.zeros((1, ck.n), dtype=np.uint64)
        a[0, k] = 1
        got = ck.ntt(a, [0])[0]
        for j in (0, 1, 2, 511, 1000):
            assert int(got[j]) == pow(psi, (2 * bitrev(j, 10) + 1) * k, q)


def test_round_trip_full_degree():
    ck = Ckks(16, CHAIN50[:3])
    a = uniform_residues(rng(2, 1), ck.q, ck.n)
    A = ck.ntt(a, [0, 1, 2])
    assert not np.array_equal(A, a)
    assert np.array_equal(ck.intt(A, [0, 1, 2]), a)
    assert (A < np.array(ck.q, dtype=np.uint64)[:, None]).all()


def test_batched_same_prime_equals_per_row():
    ck = Ckks(8, CHAIN50[:1])
    a = uniform_residues(rng(2, 1, extra=3), ck.q * 5, ck.n)
    batched = ck.ntt_rows_same_prime(a, 0)
    per_row = np.stack([ck.ntt(a[r:r + 1], [0])[0] for r in range(5)])
    assert np.array_equal(batched, per_row)
    assert np.array_equal(ck.ntt_rows_same_prime(batched, 0, inverse=True), a)


def test_sixty_bit_primes():
    # the integer path accepts primes up to 2^62: pin the oracle there too
    qs = gen_primes(60, 1 << 9, 2)
    ck = Ckks(8, qs)
    g = rng(2, 1, extra=99)
    a = uniform_residues(g, qs, ck.n)
    b = uniform_residues(g, qs, ck.n)
    c = ck.intt(ck.mul(ck.ntt(a, [0, 1]), ck.ntt(b, [0, 1]), [0, 1]), [0, 1])
    for r, q in enumerate(qs):
        assert [int(x) for x in c[r]] == _schoolbook_negacyclic([int(x) for x in a[r]],
                                                                [int(x) for x in b[r]], q)
