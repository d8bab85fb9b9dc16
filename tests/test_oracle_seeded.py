"""Pins for the oracle's seed-expanded switching keys.

* The C Philox-4x64-10 block equals numpy's Philox bit generator (an independent implementation of the same
  published generator) for random keys and counters, carries included.
* The expansion of a seed equals a pure-Python sampler that draws its blocks from numpy's Philox, on a small
  ring whose primes include one just above a power of two (half of its candidates are rejected, so the retry
  path runs) and one with dnum > 4 (a second block index).
* Expanded residues are canonical and uniform (chi-square over 64 buckets, mean), deterministic in the seed, and
  different seeds give different halves.
* A rotation with a seeded key decrypts to the rotated slots within the key-switching bound (Background, "The
  CKKS Computation Model": Rot_k through KeySwitch): the seeded key is a valid switching key.
"""
import numpy as np
import pytest

from oracle import Ckks, gen_primes, is_prime
from workloads import TOY, gaussian_error, rng, ternary_secret, uniform_residues, uniform_slots


def numpy_block(ctr, key):
    """Philox-4x64-10 block of counter ctr from numpy, which increments its 256-bit counter before each block."""
    c = sum(int(x) << (64 * i) for i, x in enumerate(ctr)) - 1
    c %= 1 << 256
    prev = np.array([(c >> (64 * i)) & ((1 << 64) - 1) for i in range(4)], dtype=np.uint64)
    g = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=prev)
    return [int(x) for x in g.random_raw(4)]


def test_philox_matches_numpy():
    g = np.random.default_rng(5)
    for _ in range(20):
        ctr = [int(x) for x in g.integers(0, 1 << 63, 4, dtype=np.uint64)]
        key = [int(x) for x in g.integers(0, 1 << 63, 2, dtype=np.uint64)]
        assert Ckks.philox(ctr, key) == numpy_block(ctr, key)
    # counter words at their limits (numpy's increment carries across words)
    for ctr in ([0, 0, 0, 0], [2 ** 64 - 1, 0, 0, 0], [0, 2 ** 64 - 1, 7, 1], [5, 3, 2 ** 64 - 1, 2 ** 64 - 1]):
        assert Ckks.philox(ctr, [11, 13]) == numpy_block(ctr, [11, 13])


def python_expand(primes, dnum, n, seed):
    out = np.empty((dnum, len(primes), n), dtype=np.uint64)
    for j in range(dnum):
        for k, q in enumerate(primes):
            b = q.bit_length()
            for i in range(n):
                for t in range(64):
                    w = numpy_block([i, k, j // 4, t], seed)[j % 4]
                    if (w >> (64 - b)) < q:
                        out[j, k, i] = w >> (64 - b)
                        break
                else:
                    out[j, k, i] = w % q
    return out


def small_prime_above(p2, two_n):
    c = p2 + 1
    c += (1 - c) % two_n
    while not is_prime(c):
        c += two_n
    return c


def test_expansion_matches_numpy_sampler():
    n = 16
    q_low = small_prime_above(1 << 40, 2 * n)    # just above 2^40: about half the 41-bit candidates are rejected
    qs = gen_primes(36, 2 * n, 2) + [q_low]
    ck = Ckks(4, qs[:2], qs[2:], 1)
    ck.dnum = 6                                  # six digits: block index j // 4 takes two values
    seed = [0x0123456789ABCDEF, 0x0FEDCBA987654321]
    got = ck.expand_key_a(seed)
    assert np.array_equal(got, python_expand(qs, 6, n, seed))
    assert np.all(got[:, 2] < q_low)


def test_expansion_uniform_and_deterministic():
    qs = gen_primes(TOY.q_bits, 2 * TOY.n, TOY.n_q + TOY.n_p)
    ck = Ckks(TOY.log_n, qs[:TOY.n_q], qs[TOY.n_q:], TOY.dnum)
    a = ck.expand_key_a([1, 2])
    assert a.shape == (TOY.dnum, len(qs), ck.n)
    assert np.array_equal(a, ck.expand_key_a([1, 2]))
    assert not np.array_equal(a, ck.expand_key_a([1, 3]))
    for j in range(TOY.dnum):
        for k, q in enumerate(qs):
            row = a[j, k].astype(np.float64)
            assert np.all(a[j, k] < q)
            # 4096 draws: the mean of U[0, q) within 5 standard errors, and chi-square over 64 equal buckets below
            # its 99.99% point (df 63: about 119)
            assert abs(row.mean() / q - 0.5) < 5 * np.sqrt(1 / 12 / row.size)
            counts = np.bincount((row / q * 64).astype(np.int64), minlength=64)
            exp = row.size / 64
            assert np.sum((counts - exp) ** 2 / exp) < 119.0
    # different digits and primes are different streams
    assert not np.array_equal(a[0, 0], a[1, 0]) and not np.array_equal(a[0, 0] % qs[1], a[0, 1])


def test_seeded_key_rotation_decrypts():
    qs = gen_primes(TOY.q_bits, 2 * TOY.n, TOY.n_q + TOY.n_p)
    ck = Ckks(TOY.log_n, qs[:TOY.n_q], qs[TOY.n_q:], TOY.dnum)
    n = ck.n
    s = ternary_secret(rng(1, 3, extra=90), n)
    z = uniform_slots(rng(1, 1, extra=90), n // 2)
    ge = rng(1, 4, extra=90)
    ct = ck.encrypt(s, ck.encode(z, None, 2.0 ** 30, TOY.n_q), uniform_residues(ge, qs[:TOY.n_q], n),
                    gaussian_error(ge, n))
    for r, seed in ((3, [7, 8]), (-5, [9, 10])):
        e = gaussian_error(rng(1, 5, extra=90 + r), (TOY.dnum, n))
        b = ck.keygen_galois_seeded(s, ck.galois_elt(r), seed, e)
        assert b.shape == (TOY.dnum, len(qs), n)
        key = ck.seeded_key(b, seed)
        assert np.array_equal(key, ck.keygen_galois(s, ck.galois_elt(r), ck.expand_key_a(seed), e))
        out = ck.rotate(ct, r, key)
        got = ck.decode(ck.decrypt(s, out), 2.0 ** 30)
        assert np.max(np.abs(got.real - np.roll(z, -r))) < 2.0 ** -12
        assert np.max(np.abs(got.imag)) < 2.0 ** -12
