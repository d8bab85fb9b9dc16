"""Pins for the oracle's ciphertext operations, by decryption against the slot arithmetic they
stand for (Background, "The CKKS Computation Model": Add, PCMult, Mult, Rot_k, KeySwitch,
Rescale), plus the definitional identity hoisted == one-at-a-time rotation.

Error bounds: a fresh encryption error e (|e_i| <= 19) moves a decoded slot by at
most N*19/Delta.  Key switching adds E = sum_j d_j e_j / P.  The digits d_j come
from the centred basis conversion: each coefficient is Q_j times a sum of alpha
independent values uniform on (-1/2, 1/2), zero mean and variance alpha/12, so
d_j(zeta) has standard deviation Q_j sqrt(alpha N / 12) and e_j(zeta) 3.2 sqrt(N).
Six standard deviations of each give
|E| <= n_digits * (Q_j / P) * 6 sqrt(alpha N / 12) * 6 * 3.2 * sqrt(N) / Delta  (ks_bound).
(Digits in [0, Q_j) instead carry a mean offset of about Q_j (alpha + 1)/2 times
the all-ones polynomial, whose value at zeta^k reaches 2N/pi, and break it.)
"""
import math

import numpy as np
import pytest

from oracle import Ckks, gen_primes
from workloads import (ROLE_DATA, ROLE_ENC, ROLE_KEYS, ROLE_SECRET, gaussian_error, rng,
                       ternary_secret, uniform_residues, uniform_slots)

Q36 = gen_primes(36, 1 << 13, 6)


@pytest.fixture(scope="module")
def toy():
    ck = Ckks(12, Q36[:4], Q36[4:6], 2)
    s = ternary_secret(rng(1, ROLE_SECRET), ck.n)
    return ck, s


def _enc(ck, s, z, delta, seed, level=3):
    pt = ck.encode(z.real, z.imag, delta, level + 1)
    g = rng(1, ROLE_ENC, extra=seed)
    a = uniform_residues(g, ck.q[:level + 1], ck.n)
    e = gaussian_error(g, ck.n)
    return ck.encrypt(s, pt, a, e)


def _keys(ck, s, seed):
    g = rng(1, ROLE_KEYS, extra=seed)
    a = uniform_residues(g, ck.primes, ck.n, lead=(ck.dnum,))
    e = gaussian_error(g, (ck.dnum, ck.n))
    return a, e


def _z(ck, seed):
    g = rng(1, ROLE_DATA, extra=seed)
    return uniform_slots(g, ck.n // 2) + 1j * uniform_slots(g, ck.n // 2)


def ks_bound(ck, level, delta):
    qj = max(math.prod(ck.q[i] for i in ck.digit_limbs(j, level)) for j in range(ck.n_digits(level)))
    return (ck.n_digits(level) * (qj / ck.P) * 6 * math.sqrt(ck.alpha * ck.n / 12) * 6 * 3.2 * math.sqrt(ck.n)
            / delta)


def _dec(ck, s, ct, scale):
    return ck.decode(ck.decrypt(s, ct), scale)


DELTA = 2.0 ** 30


def test_encrypt_decrypt(toy):
    ck, s = toy
    z = _z(ck, 1)
    ct = _enc(ck, s, z, DELTA, 1)
    err = np.max(np.abs(_dec(ck, s, ct, DELTA) - z))
    assert err < ck.n * 20 / DELTA
    # a ciphertext is not its plaintext
    assert not np.array_equal(ct[0], ck.encode(z.real, z.imag, DELTA, 4))


def test_add_and_mul_plain(toy):
    ck, s = toy
    z1, z2 = _z(ck, 2), _z(ck, 3)
    c1, c2 = _enc(ck, s, z1, DELTA, 2), _enc(ck, s, z2, DELTA, 3)
    assert np.max(np.abs(_dec(ck, s, ck.ct_add(c1, c2), DELTA) - (z1 + z2))) < 2 * ck.n * 20 / DELTA
    w = _z(ck, 4)
    pt = ck.encode(w.real, w.imag, float(ck.q[3]), 4)
    prod = ck.rescale(ck.ct_mul_plain(c1, pt))
    assert prod.shape == (2, 3, ck.n)
    assert np.max(np.abs(_dec(ck, s, prod, DELTA) - z1 * w)) < 1e-3


@pytest.mark.parametrize("steps", [1, 5, 16, -3, 1000])
def test_rotate(toy, steps):
    ck, s = toy
    z = _z(ck, 5)
    ct = _enc(ck, s, z, DELTA, 5)
    a, e = _keys(ck, s, 10 + steps)
    key = ck.keygen_galois(s, ck.galois_elt(steps), a, e)
    out = ck.rotate(ct, steps, key)
    assert np.max(np.abs(_dec(ck, s, out, DELTA) - np.roll(z, -steps))) < ks_bound(ck, 3, DELTA)


def test_rotate_at_lower_level_uses_partial_digit(toy):
    ck, s = toy
    z = _z(ck, 6)
    ct = _enc(ck, s, z, DELTA, 6, level=2)  # limbs 0..2: digit 1 holds only q_2
    a, e = _keys(ck, s, 20)
    key = ck.keygen_galois(s, ck.galois_elt(7), a, e)
    assert ck.n_digits(2) == 2 and ck.digit_limbs(1, 2) == [2]
    out = ck.rotate(ct, 7, key)
    assert np.max(np.abs(_dec(ck, s, out, DELTA) - np.roll(z, -7))) < ks_bound(ck, 2, DELTA)


def test_hoisted_equals_single_rotations(toy):
    ck, s = toy
    ct = _enc(ck, s, _z(ck, 7), DELTA, 7)
    steps = [1, 2, 16, 100]
    keys = []
    for r in steps:
        a, e = _keys(ck, s, 30 + r)
        keys.append(ck.keygen_galois(s, ck.galois_elt(r), a, e))
    hoisted = ck.rotate_hoisted(ct, steps, keys)
    for r, k, h in zip(steps, keys, hoisted):
        assert np.array_equal(h, ck.rotate(ct, r, k))


def test_lazy_rotation_sum_single_term_is_the_rotation(toy):
    # ModDown(x + P y) = ModDown(x) + y exactly: one term of the lazy sum is the rotation bit for bit
    ck, s = toy
    for lvl, st in ((3, 5), (2, -3)):
        ct = _enc(ck, s, _z(ck, 40 + lvl), DELTA, 40 + lvl, level=lvl)
        a, e = _keys(ck, s, 41 + lvl)
        key = ck.keygen_galois(s, ck.galois_elt(st), a, e)
        assert np.array_equal(ck.rotate_sum_lazy([ct], [st], [key]), ck.rotate(ct, st, key))


def test_lazy_rotation_sum_decrypts_to_the_sum(toy):
    ck, s = toy
    steps = [1, 7, -16, 300]
    zs = [_z(ck, 50 + i) for i in range(len(steps))]
    cts = [_enc(ck, s, z, DELTA, 50 + i) for i, z in enumerate(zs)]
    keys = []
    for i, r in enumerate(steps):
        a, e = _keys(ck, s, 60 + i)
        keys.append(ck.keygen_galois(s, ck.galois_elt(r), a, e))
    lazy = ck.rotate_sum_lazy(cts, steps, keys)
    want = sum(np.roll(z, -r) for z, r in zip(zs, steps))
    # the encryption errors of four inputs and four key-switching errors, one rounding of the division
    bound = 4 * ck.n * 20 / DELTA + 4 * ks_bound(ck, 3, DELTA)
    assert np.max(np.abs(_dec(ck, s, lazy, DELTA) - want)) < bound
    eager = ck.rotate(cts[0], steps[0], keys[0])
    for ct, r, k in zip(cts[1:], steps[1:], keys[1:]):
        eager = ck.ct_add(eager, ck.rotate(ct, r, k))
    # the two forms differ only in the rounding of the divisions by P
    assert not np.array_equal(lazy, eager)
    assert np.max(np.abs(_dec(ck, s, lazy, DELTA) - _dec(ck, s, eager, DELTA))) < 4 * ks_bound(ck, 3, DELTA)


def test_rotation_composes(toy):
    ck, s = toy
    z = _z(ck, 8)
    ct = _enc(ck, s, z, DELTA, 8)
    ks = {}
    for r in (3, 4, 7):
        a, e = _keys(ck, s, 40 + r)
        ks[r] = ck.keygen_galois(s, ck.galois_elt(r), a, e)
    two = ck.rotate(ck.rotate(ct, 3, ks[3]), 4, ks[4])
    one = ck.rotate(ct, 7, ks[7])
    d2, d1 = _dec(ck, s, two, DELTA), _dec(ck, s, one, DELTA)
    assert np.max(np.abs(d2 - d1)) < 3 * ks_bound(ck, 3, DELTA)
    assert np.max(np.abs(d1 - np.roll(z, -7))) < ks_bound(ck, 3, DELTA)


def test_conjugation_key(toy):
    ck, s = toy
    z = _z(ck, 9)
    ct = _enc(ck, s, z, DELTA, 9)
    a, e = _keys(ck, s, 50)
    g = 2 * ck.n - 1
    key = ck.keygen_galois(s, g, a, e)
    digits = ck.modup(ct[1], 3)
    u0, u1 = ck.keyswitch_digits(digits, key, 3, g)
    out = np.stack([ck.add(ck.automorph(ct[0], g), u0, [0, 1, 2, 3]), u1])
    assert np.max(np.abs(_dec(ck, s, out, DELTA) - np.conj(z))) < ks_bound(ck, 3, DELTA)


def test_mul_relin_and_rescale(toy):
    ck, s = toy
    z1, z2 = _z(ck, 10), _z(ck, 11)
    c1, c2 = _enc(ck, s, z1, DELTA, 10), _enc(ck, s, z2, DELTA, 11)
    a, e = _keys(ck, s, 60)
    rlk = ck.keygen_relin(s, a, e)
    prod = ck.mul_relin(c1, c2, rlk)
    assert np.max(np.abs(_dec(ck, s, prod, DELTA * DELTA) - z1 * z2)) < 1e-3
    rs = ck.rescale(prod)
    assert np.max(np.abs(_dec(ck, s, rs, DELTA * DELTA / ck.q[3]) - z1 * z2)) < 1e-3
