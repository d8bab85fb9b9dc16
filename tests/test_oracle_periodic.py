"""Pins for the oracle's token-major (periodic) projection.

* The periodic encode (a D-value period encoded at ring degree 2D and embedded as
  m'(X^(N/2D))) agrees with the O(N^2) long-double definition of the encoding of
  the full periodic slot vector: the coefficients off the multiples of N/2D are
  exactly zero and the others agree except within the fp64 error of a tie.
* Its NTT-domain values are constant over runs of N/2D consecutive indices (the
  structure the GPU path relies on), and decode returns the periodic slots.
* The slot-level identity in the token-major layout s = t*D + f with the wrap
  split U/V (Section "Matrix Representations and Linear Computation in CKKS",
  Eq. slot-diagonal-matvec, with the left rotation rho^k), evaluated with numpy
  rolls on plain slot vectors, equals X @ W for every baby-step size n1; dropping
  the wrapped part breaks it.
* End to end on the toy ring: decrypt(linear_project_tm(Enc(X), W)) is within
  2^-12 of X @ W.
"""
import numpy as np
import pytest

from oracle import Ckks, gen_primes
from workloads import (ROLE_DATA, ROLE_ENC, ROLE_KEYS, ROLE_SECRET, ROLE_WEIGHTS, TOY,
                       gaussian_error, gaussian_weights, rng, ternary_secret, uniform_residues,
                       uniform_slots)

Q50 = gen_primes(50, 1 << 17, 4)


def tm_pack(X, T, D, i):
    """Input ciphertext i of the token-major layout: slot t*D + f holds X[t, i*D + f]."""
    return X[:, i * D:(i + 1) * D].reshape(-1)


@pytest.mark.parametrize("log_n,D,delta_log2", [(6, 8, 20), (8, 16, 30), (8, 64, 30), (10, 4, 30),
                                                (10, 256, 30), (8, 128, 30)])
def test_periodic_encode_matches_definition(log_n, D, delta_log2):
    ck = Ckks(log_n, Q50[:1])
    n, T = ck.n, ck.n // (2 * D)
    u = uniform_slots(rng(8, 1, extra=log_n * 1000 + D), D)
    delta = float(2 ** delta_log2)
    m_def, tie = ck.encode_int_def(np.tile(u, n // (2 * D)), None, delta)
    mp = np.empty(2 * D, dtype=np.int64)
    from oracle.ckks import lib
    lib().or_encode_round(np.ascontiguousarray(u), None, 2 * D, delta, mp)
    off = np.ones(n, dtype=bool)
    off[::T] = False
    assert np.count_nonzero(m_def[off]) == 0
    diff = mp - m_def[::T]
    bound = 8 * np.log2(2 * D) * 2.0 ** -53 * delta * 2.0
    assert np.all(np.abs(diff) <= 1)
    assert np.all(tie[::T][diff != 0] < bound)
    # the plaintext the oracle builds is exactly that sparse polynomial, reduced and transformed
    pt = ck.encode_periodic(u, delta, 1)
    m = np.zeros(n, dtype=np.int64)
    m[::T] = mp
    assert np.array_equal(ck.intt(pt, [0])[0], ck.reduce_int(m, [0])[0])


@pytest.mark.parametrize("log_n,D", [(10, 64), (12, 128), (12, 8)])
def test_periodic_plaintext_is_blockwise_constant_and_decodes(log_n, D):
    ck = Ckks(log_n, Q50[:3])
    T = ck.n // (2 * D)
    u = uniform_slots(rng(8, 2, extra=log_n * 1000 + D), D)
    delta = 2.0 ** 40
    pt = ck.encode_periodic(u, delta, 3)
    for l in range(3):
        blocks = pt[l].reshape(-1, T)
        assert np.all(blocks == blocks[:, :1])
    z = ck.decode(pt, delta)
    assert np.max(np.abs(z.real - np.tile(u, T))) < 1e-9
    assert np.max(np.abs(z.imag)) < 1e-9


def test_periodic_encode_of_zero_is_zero():
    ck = Ckks(8, Q50[:2])
    assert not ck.encode_periodic(np.zeros(16), 2.0 ** 40, 2).any()


def _tm_slots(X, W, T, D, n1, wrap=True):
    n_in, n_out = X.shape[1] // D, W.shape[1] // D
    n2 = -(-D // n1)
    outs = []
    for j in range(n_out):
        total = np.zeros(T * D)
        for gi in range(n2):
            acc = np.zeros(T * D)
            for i in range(n_in):
                x = tm_pack(X, T, D, i)
                for b in range(n1):
                    if n1 * gi + b >= D:
                        continue
                    uu, vv = Ckks.periodic_diag_vectors(W, D, j, i, n1, gi, b)
                    acc += np.tile(uu, T) * np.roll(x, -b)
                    if wrap:
                        acc += np.tile(vv, T) * np.roll(x, -(b - D))
            total += np.roll(acc, -n1 * gi)
        outs.append(total)
    return outs


@pytest.mark.parametrize("T,D,n_in,n_out,n1", [(4, 8, 2, 3, 1), (4, 8, 2, 3, 2), (4, 8, 2, 3, 3),
                                              (4, 8, 2, 3, 8), (2, 16, 1, 2, 4), (8, 4, 3, 1, 2)])
def test_tm_bsgs_slot_identity(T, D, n_in, n_out, n1):
    g = np.random.default_rng(T * 100 + D + n1 + 7)
    X = g.uniform(-1, 1, (T, n_in * D))
    W = g.normal(0, 0.02, (n_in * D, n_out * D))
    Y = X @ W
    for j, y in enumerate(_tm_slots(X, W, T, D, n1)):
        assert np.max(np.abs(y - tm_pack(Y, T, D, j))) < 1e-14
    # the wrapped entries matter: without them the identity fails
    bad = _tm_slots(X, W, T, D, n1, wrap=False)
    assert max(np.max(np.abs(y - tm_pack(Y, T, D, j))) for j, y in enumerate(bad)) > 1e-3


def test_periodic_diag_vectors_split_the_cyclic_diagonal():
    g = np.random.default_rng(11)
    D = 8
    W = g.normal(size=(2 * D, 3 * D))
    A = W.T
    for (j, i, n1, gi, b) in [(0, 0, 8, 0, 0), (2, 1, 8, 0, 5), (1, 0, 2, 3, 1), (0, 1, 4, 1, 3)]:
        k = n1 * gi + b
        uu, vv = Ckks.periodic_diag_vectors(W, D, j, i, n1, gi, b)
        for o in range(D):
            op = (o - n1 * gi) % D
            want = A[j * D + op, i * D + (op + k) % D]
            wraps = op + k >= D
            assert (vv[o] if wraps else uu[o]) == want
            assert (uu[o] if wraps else vv[o]) == 0.0


@pytest.fixture(scope="module")
def toy_tm_projection():
    cfg = TOY
    qs = gen_primes(cfg.q_bits, 2 * cfg.n, cfg.n_q + cfg.n_p)
    ck = Ckks(cfg.log_n, qs[:cfg.n_q], qs[cfg.n_q:], cfg.dnum)
    T, D, n1 = cfg.tokens, cfg.feats, 16
    d_in, d_out = 2 * D, 3 * D
    s = ternary_secret(rng(cfg.index, ROLE_SECRET, extra=9), ck.n)
    X = uniform_slots(rng(cfg.index, ROLE_DATA, extra=9), (T, d_in))
    W = gaussian_weights(rng(cfg.index, ROLE_WEIGHTS, extra=9), (d_in, d_out))
    delta = float(2 ** cfg.scale_log2)
    level = cfg.level
    ge = rng(cfg.index, ROLE_ENC, extra=9)
    cts = []
    for i in range(d_in // D):
        pt = ck.encode(tm_pack(X, T, D, i), None, delta, level + 1)
        cts.append(ck.encrypt(s, pt, uniform_residues(ge, ck.q[:level + 1], ck.n), gaussian_error(ge, ck.n)))
    gk = rng(cfg.index, ROLE_KEYS, extra=9)
    keys = {}
    n2 = -(-D // n1)
    for st in [b for b in range(1, n1)] + [b - D for b in range(n1)] + [n1 * g for g in range(1, n2)]:
        a = uniform_residues(gk, ck.primes, ck.n, lead=(ck.dnum,))
        e = gaussian_error(gk, (ck.dnum, ck.n))
        keys[st] = ck.keygen_galois(s, ck.galois_elt(st), a, e)
    outs = ck.linear_project_tm(cts, W, T, n1, keys, out_blocks=[0, 2])
    lazy = ck.linear_project_tm(cts, W, T, n1, keys, out_blocks=[0], lazy=True)
    return ck, s, X, W, outs, delta, lazy


def test_toy_tm_projection_accuracy(toy_tm_projection):
    ck, s, X, W, outs, delta, _ = toy_tm_projection
    T, D = TOY.tokens, TOY.feats
    Y = X @ W
    for j, ct in zip([0, 2], outs):
        assert ct.shape == (2, TOY.level, ck.n)
        z = ck.decode(ck.decrypt(s, ct), delta)
        err = np.max(np.abs(z.real - tm_pack(Y, T, D, j)))
        assert err <= 2.0 ** -12, err
        assert np.max(np.abs(z.imag)) <= 2.0 ** -12


def test_toy_tm_projection_lazy_giant_steps(toy_tm_projection):
    """The giant-step rotations summed with one ModDown (the division by P rounds once instead of per rotation;
    the final rescale absorbs the difference except near a rounding boundary): the same accuracy."""
    ck, s, X, W, outs, delta, lazy = toy_tm_projection
    T, D = TOY.tokens, TOY.feats
    assert lazy[0].shape == outs[0].shape
    z = ck.decode(ck.decrypt(s, lazy[0]), delta)
    assert np.max(np.abs(z.real - tm_pack(X @ W, T, D, 0))) <= 2.0 ** -12
