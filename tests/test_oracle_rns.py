"""Pins for the oracle's RNS machinery, checked with Python big integers:

* CRT lift reproduces the integer it came from;
* fast basis conversion with centred digits equals x + u*Q_I, x the centred
  representative modulo Q_I and |u| <= |I|//2 (Cheon-Han-Kim-Kim-Song 2018), so
  one source limb gives the centred lift itself;
* ModDown(P * c) = c exactly;
* rescale equals round(c / q_l) coefficient by coefficient;
* the NTT-domain automorphism sigma_g(a)(X) = a(X^g) agrees with the
  coefficient-domain substitution X^i -> +-X^(i g mod N), written out here.
"""
import math

import numpy as np
import pytest

from oracle import Ckks, gen_primes
from workloads import rng, uniform_residues

Q50 = gen_primes(50, 1 << 17, 32)


def _ck(log_n=8, n_q=6, n_p=3, dnum=2):
    return Ckks(log_n, Q50[:n_q], Q50[24:24 + n_p], dnum)


def _crt(cols, mods):
    Q = math.prod(mods)
    x = 0
    for r, m in zip(cols, mods):
        Qh = Q // m
        x += int(r) * pow(Qh, -1, m) % m * Qh
    return x % Q


def test_crt_lift_round_trip():
    ck = _ck()
    g = np.random.default_rng(5)
    Q = math.prod(ck.q)
    vals = [int(g.integers(0, 1 << 62)) * int(g.integers(0, 1 << 62)) % Q - Q // 2 for _ in range(ck.n)]
    vals[0], vals[1] = Q // 2, -(Q // 2)
    rows = np.array([[v % q for v in vals] for q in ck.q], dtype=np.uint64)
    assert ck.lift_centered(rows, list(range(ck.n_q))) == vals


@pytest.mark.parametrize("src,dst", [([0, 1, 2], [3, 4, 5, 6, 7, 8]), ([6, 7, 8], [0, 1, 2, 3, 4, 5]),
                                     ([0, 1, 2, 3], [6, 7, 8]), ([4], [0, 1, 6])])
def test_basis_conversion_overflow_form(src, dst):
    ck = _ck()
    a = uniform_residues(rng(3, 1, extra=len(src)), [ck.primes[k] for k in src], ck.n)
    out = ck.conv(a, src, dst)
    qs = [ck.primes[k] for k in src]
    QI = math.prod(qs)
    half = len(src) // 2
    seen = set()
    for j in range(0, ck.n, 3):
        x = _crt([a[r, j] for r in range(len(src))], qs)
        if x > QI // 2:
            x -= QI
        ok = [u for u in range(-half, half + 1)
              if all((x + u * QI) % ck.primes[k] == int(out[r, j]) for r, k in enumerate(dst))]
        assert len(ok) == 1, j
        seen.add(ok[0])
    # the overflow takes both signs once there are two or more digits (it is centred, not one-sided)
    assert min(seen) < 0 < max(seen) if half else seen == {0}


def test_moddown_of_p_multiple_is_exact():
    ck = _ck()
    level = 4
    ext = ck.ext_primes(level)
    c = uniform_residues(rng(3, 2), [ck.primes[k] for k in range(level + 1)], ck.n)
    pc = np.zeros((len(ext), ck.n), dtype=np.uint64)
    pc[:level + 1] = ck.mul_scalar(c, [ck.P % ck.q[i] for i in range(level + 1)], list(range(level + 1)))
    # P*c is 0 modulo every special prime
    assert np.array_equal(ck.moddown(pc, level), c)


def test_moddown_divides_by_p_with_bounded_error():
    ck = _ck(log_n=5)
    level = 3
    ext = ck.ext_primes(level)
    x = uniform_residues(rng(3, 3), [ck.primes[k] for k in ext], ck.n)
    out = ck.moddown(x, level)
    xc = ck.intt(x, ext)
    oc = ck.intt(out, list(range(level + 1)))
    mods_ext = [ck.primes[k] for k in ext]
    mods_q = ck.q[:level + 1]
    Ql = math.prod(mods_q)
    for j in range(ck.n):
        X = _crt(xc[:, j], mods_ext)
        Y = _crt(oc[:, j], mods_q)
        # Y = (X - (x_c + u P)) / P mod Q_l, x_c the centred residue of X mod P and |u| <= K // 2:
        # division rounded to nearest, up to the centred overflow
        P = ck.P
        xc_ = (X + (P - 1) // 2) % P - (P - 1) // 2
        base = (X - xc_) // P
        half = ck.n_p // 2
        assert sum((base - u) % Ql == Y for u in range(-half, half + 1)) == 1, j


def test_rescale_is_rounded_division():
    ck = _ck(log_n=6)
    level = 5
    idx = list(range(level + 1))
    ct = uniform_residues(rng(3, 4), ck.q[:level + 1], ck.n, lead=(2,))
    out = ck.rescale(ct)
    ql = ck.q[level]
    Ql = math.prod(ck.q[:level + 1])
    Qo = math.prod(ck.q[:level])
    for k in range(2):
        cc = ck.intt(ct[k], idx)
        oc = ck.intt(out[k], idx[:-1])
        for j in range(ck.n):
            c = _crt(cc[:, j], ck.q[:level + 1])
            c = c - Ql if c > Ql // 2 else c
            want = (2 * c + ql) // (2 * ql)  # round half up; ties impossible (q odd)
            assert _crt(oc[:, j], ck.q[:level]) == want % Qo


def test_automorphism_matches_coefficient_substitution():
    ck = _ck(log_n=6, n_q=2, n_p=0, dnum=1)
    n = ck.n
    a = uniform_residues(rng(3, 5), ck.q, n)
    for g in (5, 25, 2 * n - 1, pow(5, 7, 2 * n)):
        want = np.zeros_like(a)
        for i in range(n):
            k = (i * g) % (2 * n)
            for r, q in enumerate(ck.q):
                v = int(a[r, i])
                if k < n:
                    want[r, k] = (int(want[r, k]) + v) % q
                else:
                    want[r, k - n] = (int(want[r, k - n]) - v) % q
        got = ck.intt(ck.automorph(ck.ntt(a, [0, 1]), g), [0, 1])
        assert np.array_equal(got, want), g
