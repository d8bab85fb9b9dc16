"""Pins for the oracle's encode and decode (canonical embedding, CKKS 2017).

* the fixed-order fp64 FFT encode agrees with the O(N^2) long-double definition,
  except at coefficients whose exact value lies within the fp64 error of a
  rounding tie, and there by exactly one;
* closed forms: constant slots give a constant polynomial; the slots
  zeta^(5^j) give Delta*X; a purely imaginary constant gives a multiple of X^(N/2);
* decode is pinned against its O(N^2) definition written out here, and
  decode(encode(z)) returns z within the rounding bound.
"""
import numpy as np
import pytest

from oracle import Ckks, gen_primes
from workloads import rng, uniform_slots

Q36 = gen_primes(36, 1 << 13, 6)
Q50 = gen_primes(50, 1 << 17, 24)


def _slots(n, seed, cplx=True):
    g = rng(1, 1, extra=seed)
    zr = uniform_slots(g, n // 2)
    zi = uniform_slots(g, n // 2) if cplx else None
    return zr, zi


@pytest.mark.parametrize("log_n,delta_log2", [(5, 20), (8, 30), (12, 30), (12, 50)])
def test_fft_encode_matches_long_double_definition(log_n, delta_log2):
    ck = Ckks(log_n, Q50[:1])
    zr, zi = _slots(ck.n, log_n + delta_log2)
    delta = float(2 ** delta_log2)
    m = ck.encode_int(zr, zi, delta)
    m_def, tie = ck.encode_int_def(zr, zi, delta)
    diff = m - m_def
    # fp64 error bound of the transform: a few units of eps * log2(N) * sum|z| * delta * 2/N
    bound = 8 * log_n * 2.0 ** -53 * delta * 2.0 * np.sqrt(2.0)
    assert np.all(np.abs(diff) <= 1)
    assert np.all(tie[diff != 0] < bound), (tie[diff != 0], bound)
    if delta_log2 <= 30:
        assert np.count_nonzero(diff) == 0


def test_constant_slots_give_constant_polynomial():
    ck = Ckks(12, Q36[:1])
    delta = 2.0 ** 30
    for c in (0.25, -0.7, 1.0):
        zr = np.full(ck.n // 2, c)
        m = ck.encode_int(zr, None, delta)
        assert m[0] == int(np.round(c * delta))
        assert np.count_nonzero(m[1:]) == 0


def test_imaginary_constant_gives_half_degree_monomial():
    # i*c in every slot: m(zeta^(e_j)) = i*c*Delta for all j; X^(N/2) evaluates to
    # zeta^(e_j N/2) = i^(e_j) = i since e_j = 1 mod 4, so m = c*Delta*X^(N/2).
    ck = Ckks(10, Q36[:1])
    delta = 2.0 ** 30
    m = ck.encode_int(np.zeros(ck.n // 2), np.full(ck.n // 2, 0.5), delta)
    want = np.zeros(ck.n, dtype=np.int64)
    want[ck.n // 2] = int(0.5 * delta)
    assert np.array_equal(m, want)


def test_root_slots_give_delta_x():
    ck = Ckks(11, Q36[:1])
    n = ck.n
    e = np.array([pow(5, j, 2 * n) for j in range(n // 2)])
    z = np.exp(1j * np.pi * e / n)
    delta = 2.0 ** 30
    m = ck.encode_int(z.real, z.imag, delta)
    want = np.zeros(n, dtype=np.int64)
    want[1] = int(delta)
    assert np.array_equal(m, want)


@pytest.mark.parametrize("log_n", [4, 7])
def test_decode_matches_definition(log_n):
    ck = Ckks(log_n, Q36[:2])
    n = ck.n
    g = rng(1, 1, extra=500 + log_n)
    m = g.integers(-(1 << 30), 1 << 30, size=n)
    pt = ck.ntt(ck.reduce_int(m, [0, 1]), [0, 1])
    got = ck.decode(pt, 2.0 ** 20)
    zeta = np.exp(1j * np.pi / n)
    e = [pow(5, j, 2 * n) for j in range(n // 2)]
    want = np.array([sum(int(m[i]) * zeta ** (i * e[j]) for i in range(n)) for j in range(n // 2)]) / 2.0 ** 20
    assert np.max(np.abs(got - want)) < 1e-9 * np.max(np.abs(want))


@pytest.mark.parametrize("log_n,bits,delta_log2,limbs", [(12, 36, 30, 4), (16, 50, 40, 3)])
def test_encode_decode_round_trip(log_n, bits, delta_log2, limbs):
    qs = Q36 if bits == 36 else Q50
    ck = Ckks(log_n, qs[:limbs])
    zr, zi = _slots(ck.n, 77)
    delta = float(2 ** delta_log2)
    pt = ck.encode(zr, zi, delta, limbs)
    z = ck.decode(pt, delta)
    # each coefficient moves by at most 1/2; a slot sums N of them: |err| <= N/(2 Delta)
    assert np.max(np.abs(z - (zr + 1j * zi))) <= ck.n / (2 * delta)
    # the NTT-domain plaintext is consistent across limbs: every limb lifts to the same integers
    m = ck.encode_int(zr, zi, delta)
    for k in range(limbs):
        coef = ck.intt(pt[k:k + 1], [k])[0]
        assert np.array_equal(coef, ck.reduce_int(m, [k])[0])


def test_rotation_and_conjugation_on_slots():
    ck = Ckks(8, Q36[:2])
    n = ck.n
    zr, zi = _slots(n, 9)
    z = zr + 1j * zi
    delta = 2.0 ** 25
    pt = ck.encode(zr, zi, delta, 2)
    for k in (1, 3, n // 2 - 1):
        zk = ck.decode(ck.automorph(pt, pow(5, k, 2 * n)), delta)
        assert np.max(np.abs(zk - np.roll(z, -k))) < 1e-5
    zc = ck.decode(ck.automorph(pt, 2 * n - 1), delta)
    assert np.max(np.abs(zc - np.conj(z))) < 1e-5
