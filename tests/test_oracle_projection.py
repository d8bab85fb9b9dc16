"""Pins for the oracle's linear projection.

* The slot-level BSGS identity (Section "Matrix Representations and Linear
  Computation in CKKS", Eq. slot-diagonal-matvec, with the left rotation
  rho^k) in the feature-major layout s = f*T + t, evaluated with numpy rolls
  on plain slot vectors, equals X @ W for every baby-step size n1.
* End to end on the toy ring (N = 2^12, 16 tokens x 128 features, 127
  rotations): decrypt(linear_project(Enc(X), W)) is within 2^-12 of X @ W.
* The same ring with giant steps (n1 = 16, n2 = 8; two inputs, three outputs),
  eager and with the lazy ModDown: every output within 2^-12 of X @ W, so the
  giant-step rotation Rot_{T n1 g} and the plaintexts' shift by n1 g are pinned.
"""
import numpy as np
import pytest

from oracle import Ckks, gen_primes
from workloads import (ROLE_DATA, ROLE_ENC, ROLE_KEYS, ROLE_SECRET, ROLE_WEIGHTS, TOY,
                       gaussian_error, gaussian_weights, rng, ternary_secret, uniform_residues,
                       uniform_slots)


def fm_pack(X, T, D, i):
    """Input ciphertext i of the feature-major layout: slot f*T + t holds X[t, i*D + f]."""
    return X[:, i * D:(i + 1) * D].T.reshape(-1)


@pytest.mark.parametrize("T,D,n_in,n_out,n1", [(4, 8, 2, 3, 1), (4, 8, 2, 3, 2), (4, 8, 2, 3, 3),
                                              (4, 8, 2, 3, 8), (2, 16, 1, 2, 4), (8, 4, 3, 1, 2)])
def test_bsgs_slot_identity(T, D, n_in, n_out, n1):
    g = np.random.default_rng(T * 100 + D + n1)
    X = g.uniform(-1, 1, (T, n_in * D))
    W = g.normal(0, 0.02, (n_in * D, n_out * D))
    n2 = -(-D // n1)
    Y = X @ W
    for j in range(n_out):
        total = np.zeros(T * D)
        for gi in range(n2):
            acc = np.zeros(T * D)
            for i in range(n_in):
                x = fm_pack(X, T, D, i)
                for b in range(n1):
                    if n1 * gi + b >= D:
                        continue
                    p = Ckks.diag_slot_vector(W, T, D, j, i, n1, gi, b)
                    acc += p * np.roll(x, -T * b)          # rho^{T b}: left rotation
            total += np.roll(acc, -T * n1 * gi)
        assert np.max(np.abs(total - fm_pack(Y, T, D, j))) < 1e-14


def test_diag_slot_vector_is_cyclic_diagonal():
    # D_k(A)[o] = A[o, (o+k) mod D] with A_{j,i} = W[iD:(i+1)D, jD:(j+1)D]^T, replicated over tokens
    g = np.random.default_rng(3)
    T, D = 3, 5
    W = g.normal(size=(2 * D, 2 * D))
    A = W.T
    for (j, i, k) in [(0, 0, 0), (1, 0, 3), (0, 1, 4), (1, 1, 2)]:
        p = Ckks.diag_slot_vector(W, T, D, j, i, n1=D, g=0, b=k)
        want = np.repeat([A[j * D + o, i * D + (o + k) % D] for o in range(D)], T)
        assert np.array_equal(p, want)


@pytest.fixture(scope="module")
def toy_projection():
    cfg = TOY
    qs = gen_primes(cfg.q_bits, 2 * cfg.n, cfg.n_q + cfg.n_p)
    ck = Ckks(cfg.log_n, qs[:cfg.n_q], qs[cfg.n_q:], cfg.dnum)
    T, D = cfg.tokens, cfg.feats
    s = ternary_secret(rng(cfg.index, ROLE_SECRET), ck.n)
    X = uniform_slots(rng(cfg.index, ROLE_DATA), (T, cfg.d_in))
    W = gaussian_weights(rng(cfg.index, ROLE_WEIGHTS), (cfg.d_in, cfg.d_out))
    delta = float(2 ** cfg.scale_log2)
    level = cfg.level
    ge = rng(cfg.index, ROLE_ENC)
    cts = []
    for i in range(cfg.d_in // D):
        pt = ck.encode(fm_pack(X, T, D, i), None, delta, level + 1)
        cts.append(ck.encrypt(s, pt, uniform_residues(ge, ck.q[:level + 1], ck.n), gaussian_error(ge, ck.n)))
    gk = rng(cfg.index, ROLE_KEYS)
    keys = {}
    for b in range(1, cfg.n1):
        a = uniform_residues(gk, ck.primes, ck.n, lead=(ck.dnum,))
        e = gaussian_error(gk, (ck.dnum, ck.n))
        keys[T * b] = ck.keygen_galois(s, ck.galois_elt(T * b), a, e)
    outs = ck.linear_project(cts, W, T, cfg.n1, keys)
    return ck, s, X, W, outs, delta


def test_toy_projection_accuracy(toy_projection):
    ck, s, X, W, outs, delta = toy_projection
    T, D = TOY.tokens, TOY.feats
    Y = X @ W
    assert len(outs) == TOY.d_out // D
    for j, ct in enumerate(outs):
        assert ct.shape == (2, TOY.level, ck.n)
        z = ck.decode(ck.decrypt(s, ct), delta)
        err = np.max(np.abs(z.real - fm_pack(Y, T, D, j)))
        assert err <= 2.0 ** -12, err
        assert np.max(np.abs(z.imag)) <= 2.0 ** -12


@pytest.fixture(scope="module")
def toy_bsgs_setup():
    """The toy ring with a baby-step/giant-step split n1 = 16, n2 = 8: two input and three output ciphertexts."""
    cfg = TOY
    qs = gen_primes(cfg.q_bits, 2 * cfg.n, cfg.n_q + cfg.n_p)
    ck = Ckks(cfg.log_n, qs[:cfg.n_q], qs[cfg.n_q:], cfg.dnum)
    T, D, n1, level = cfg.tokens, cfg.feats, 16, cfg.level
    n2 = D // n1
    d_in, d_out = 2 * D, 3 * D
    s = ternary_secret(rng(cfg.index, ROLE_SECRET, extra=7), ck.n)
    X = uniform_slots(rng(cfg.index, ROLE_DATA, extra=7), (T, d_in))
    W = gaussian_weights(rng(cfg.index, ROLE_WEIGHTS, extra=7), (d_in, d_out))
    delta = float(2 ** cfg.scale_log2)
    ge = rng(cfg.index, ROLE_ENC, extra=7)
    cts = []
    for i in range(d_in // D):
        pt = ck.encode(fm_pack(X, T, D, i), None, delta, level + 1)
        cts.append(ck.encrypt(s, pt, uniform_residues(ge, ck.q[:level + 1], ck.n), gaussian_error(ge, ck.n)))
    gk = rng(cfg.index, ROLE_KEYS, extra=7)
    keys = {}
    for st in [T * b for b in range(1, n1)] + [T * n1 * g for g in range(1, n2)]:
        a = uniform_residues(gk, ck.primes, ck.n, lead=(ck.dnum,))
        e = gaussian_error(gk, (ck.dnum, ck.n))
        keys[st] = ck.keygen_galois(s, ck.galois_elt(st), a, e)
    return ck, s, X, W, cts, keys, delta, n1


@pytest.mark.parametrize("lazy", [False, True])
def test_toy_projection_giant_steps(toy_bsgs_setup, lazy):
    """Seven giant-step rotations by T*n1*g per output (Eq. slot-diagonal-matvec with BSGS reuse): a wrong
    giant-step shift, plaintext shift or rotation direction leaves an O(1) error, far above 2^-12."""
    ck, s, X, W, cts, keys, delta, n1 = toy_bsgs_setup
    T, D = TOY.tokens, TOY.feats
    blocks = [1] if lazy else [0, 2]
    outs = ck.linear_project(cts, W, T, n1, keys, out_blocks=blocks, lazy=lazy)
    Y = X @ W
    assert len(outs) == len(blocks)
    for j, ct in zip(blocks, outs):
        assert ct.shape == (2, TOY.level, ck.n)
        z = ck.decode(ck.decrypt(s, ct), delta)
        err = np.max(np.abs(z.real - fm_pack(Y, T, D, j)))
        assert err <= 2.0 ** -12, (lazy, j, err)
        assert np.max(np.abs(z.imag)) <= 2.0 ** -12

