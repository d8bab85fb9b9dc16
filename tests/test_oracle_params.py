"""Pins for the oracle's parameter generation: primes and 2N-th roots of unity.

The primes are certified independently of the oracle's Miller-Rabin test:
small lists by exhaustive trial division, and 50-bit primes by a Lucas
certificate built from a full trial-division factorisation of q - 1.
"""
import math

import pytest

from oracle import find_psi, gen_primes, is_prime


def _trial_prime(n):
    if n < 2:
        return False
    f = 2
    while f * f <= n:
        if n % f == 0:
            return False
        f += 1
    return True


def _factor(n):
    fs, f = set(), 2
    while f * f <= n:
        while n % f == 0:
            fs.add(f)
            n //= f
        f += 1 if f == 2 else 2
    if n > 1:
        fs.add(n)
    return fs


def _lucas_certified(q):
    """q is prime iff some a has order exactly q-1 mod q (Lucas); q-1 factored by trial division."""
    fs = _factor(q - 1)
    for a in range(2, 200):
        if pow(a, q - 1, q) != 1:
            return False
        if all(pow(a, (q - 1) // r, q) != 1 for r in fs):
            return True
    return False


def test_small_prime_list_is_exhaustive():
    # 20-bit primes 1 mod 512, every candidate checked by trial division.
    two_n = 512
    got = gen_primes(20, two_n, 12)
    want = [c for c in range((1 << 20) - 1, 1 << 19, -1) if c % two_n == 1 and _trial_prime(c)][:12]
    assert got == want


def test_miller_rabin_against_trial_division():
    for n in range(1, 20000):
        assert is_prime(n) == _trial_prime(n), n
    # strong pseudoprimes to several small bases must be rejected
    for n in (3215031751, 2152302898747, 3474749660383, 341550071728321):
        assert not is_prime(n)


@pytest.mark.parametrize("bits,two_n,count", [(50, 1 << 17, 36), (36, 1 << 13, 6)])
def test_chain_primes_certified(bits, two_n, count):
    ps = gen_primes(bits, two_n, count)
    assert len(set(ps)) == count
    assert ps == sorted(ps, reverse=True)
    for q in ps:
        assert q % two_n == 1
        assert (1 << (bits - 1)) < q < (1 << bits)
        assert _lucas_certified(q), q
    # nothing skipped between consecutive chosen primes (candidates in between are composite)
    for hi, lo in zip(ps, ps[1:]):
        for c in range(lo + two_n, hi, two_n):
            assert not is_prime(c) or c in ps


@pytest.mark.parametrize("bits,two_n", [(50, 1 << 17), (36, 1 << 13), (50, 1 << 9)])
def test_psi_is_primitive_2n_root(bits, two_n):
    for q in gen_primes(bits, 1 << 17 if bits == 50 else two_n, 4):
        psi = find_psi(q, two_n)
        n = two_n // 2
        assert pow(psi, n, q) == q - 1
        assert pow(psi, two_n, q) == 1
        # primitive: order is exactly 2N (2N is a power of two, so psi^N = -1 suffices); and the
        # generator x is the smallest one that works
        for x in range(2, 2 + 50):
            cand = pow(x, (q - 1) // two_n, q)
            if pow(cand, n, q) == q - 1:
                assert cand == psi
                break


def test_chain_prime_sizes_match_paper_setup_alternative():
    # The paper's own chain uses 60/59-bit moduli (Evaluation, experimental setup); the integer
    # path must accept primes up to 2^62, so the generator must also produce those.
    ps = gen_primes(60, 1 << 17, 3)
    assert all(q.bit_length() == 60 and q % (1 << 17) == 1 for q in ps)
    assert math.gcd(*ps) == 1
