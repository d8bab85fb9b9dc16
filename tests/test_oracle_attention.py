"""Pins for the oracle's attention block (token-major layout s = t*D + f, heads of hd features).

* Slot identities: the construction of attention_scores / attention_apply, evaluated with numpy rolls on
  plain slot vectors, equals the definitions S[t, h, delta] = sum_d Q[t, h, d] K[(t + delta) mod T, d] and
  O[t, h, d] = sum_delta P[t, h, delta] V[(t + delta) mod T, d] for several (T, D, hd), including fewer
  tokens than head features; planted mistakes (no pre-rotation of Q, the mask index delta + j instead of
  delta - j, the wrong key rotation) break them.
* The mask plaintexts decode to their 0/1 slot vectors.
* End to end on a toy ring (N = 2^12, two heads of 64 per ciphertext, 16 tokens): the decrypted oracle
  scores and weighted sums agree with the plain definitions within the bound stated in the test.
"""
import numpy as np
import pytest

from oracle import Ckks, gen_primes
from workloads import ATTN_TOY, gaussian_error, rng, ternary_secret, uniform_residues


def rot(x, k):
    """Left rotation (Rot_k x)[s] = x[s + k]."""
    return np.roll(x, -k)


def pack(M, T, D):
    """Token-major slot vector of a [T][D] array."""
    return M.reshape(T * D)


def scores_def(Q, K, T, D, hd):
    """Q [T][D] (heads of hd), K [T][hd] -> scores in the diagonal layout [T][D]."""
    out = np.zeros((T, D))
    for h in range(D // hd):
        for delta in range(T):
            out[:, h * hd + delta] = np.sum(Q[:, h * hd:(h + 1) * hd] * np.roll(K, -delta, axis=0), axis=1)
    return out


def apply_def(P, V, T, D, hd):
    out = np.zeros((T, D))
    for h in range(D // hd):
        for delta in range(T):
            out[:, h * hd:(h + 1) * hd] += P[:, h * hd + delta:h * hd + delta + 1] * np.roll(V, -delta, axis=0)
    return out


def scores_slots(q, kp, T, D, hd, pre_rotate=True, key_step=None):
    key_step = D - 1 if key_step is None else key_step
    masks = [np.tile(Ckks.attention_mask(D, hd, c), T) for c in range(hd)]
    P = [(rot(q, -d) if pre_rotate else q) * rot(kp, d * key_step) for d in range(T)]
    total = np.zeros(T * D)
    for k in range(hd):
        U = sum(masks[(d + k) % hd] * P[d] for d in range(T))
        total += rot(U, k)
    return total


def apply_slots(p, vp, T, D, hd, sign=-1):
    masks = [np.tile(Ckks.attention_mask(D, hd, c), T) for c in range(hd)]
    R = [rot(vp, d * D) for d in range(T)]
    total = np.zeros(T * D)
    for j in range(-(hd - 1), T):
        C = np.zeros(T * D)
        for d in range(T):
            c = d + sign * j
            if 0 <= c < hd:
                C += masks[c] * R[d]
        total += rot(p, j) * C
    return total


SHAPES = [(4, 8, 4), (4, 8, 8), (2, 16, 8), (8, 8, 8), (4, 16, 8), (8, 16, 16)]


@pytest.mark.parametrize("T,D,hd", SHAPES)
def test_scores_slot_identity(T, D, hd):
    g = np.random.default_rng(T * 1000 + D * 10 + hd)
    Q = g.uniform(-1, 1, (T, D))
    K = g.uniform(-1, 1, (T, hd))
    kp = pack(np.tile(K, (1, D // hd)), T, D)
    want = scores_def(Q, K, T, D, hd)
    got = scores_slots(pack(Q, T, D), kp, T, D, hd).reshape(T, D)
    assert np.max(np.abs(got - want)) < 1e-12
    for h in range(D // hd):
        assert np.all(got[:, h * hd + T:(h + 1) * hd] == 0.0)
    bad = scores_slots(pack(Q, T, D), kp, T, D, hd, pre_rotate=False).reshape(T, D)
    assert np.max(np.abs(bad - want)) > 1e-3
    bad = scores_slots(pack(Q, T, D), kp, T, D, hd, key_step=D).reshape(T, D)
    assert np.max(np.abs(bad - want)) > 1e-3


@pytest.mark.parametrize("T,D,hd", SHAPES)
def test_apply_slot_identity(T, D, hd):
    g = np.random.default_rng(T * 1000 + D * 10 + hd + 5)
    P = np.zeros((T, D))
    for h in range(D // hd):
        P[:, h * hd:h * hd + T] = g.uniform(-1, 1, (T, T))
    # positions delta >= T of the scores are never read
    junk = P.copy()
    for h in range(D // hd):
        junk[:, h * hd + T:(h + 1) * hd] = g.uniform(-1, 1, (T, hd - T))
    V = g.uniform(-1, 1, (T, hd))
    vp = pack(np.tile(V, (1, D // hd)), T, D)
    want = apply_def(P, V, T, D, hd)
    got = apply_slots(pack(junk, T, D), vp, T, D, hd).reshape(T, D)
    assert np.max(np.abs(got - want)) < 1e-12
    bad = apply_slots(pack(junk, T, D), vp, T, D, hd, sign=1).reshape(T, D)
    assert np.max(np.abs(bad - want)) > 1e-3


def test_attention_masks_decode_to_their_slot_vectors():
    qs = gen_primes(50, 2 * 4096, 3)
    ck = Ckks(12, qs)
    T, D, hd = 16, 128, 64
    for c in (0, 5, 63):
        pt = ck.encode_periodic(Ckks.attention_mask(D, hd, c), float(ck.q[1]), 2)
        z = ck.decode(pt, float(ck.q[1]))
        want = np.tile(Ckks.attention_mask(D, hd, c), T)
        assert np.max(np.abs(z.real - want)) < 1e-9
        assert np.max(np.abs(z.imag)) < 1e-9


def attn_keys(ck, s, T, D, hd, gk):
    steps = sorted(set([-d for d in range(1, T)] + [d * (D - 1) for d in range(1, T)] + list(range(1, hd))
                       + [d * D for d in range(1, T)] + [j for j in range(-(hd - 1), T) if j != 0]))
    keys = {}
    for st in steps:
        a = uniform_residues(gk, ck.primes, ck.n, lead=(ck.dnum,))
        e = gaussian_error(gk, (ck.dnum, ck.n))
        keys[st] = ck.keygen_galois(s, ck.galois_elt(st), a, e)
    a = uniform_residues(gk, ck.primes, ck.n, lead=(ck.dnum,))
    e = gaussian_error(gk, (ck.dnum, ck.n))
    rlk = ck.keygen_relin(s, a, e)
    return keys, rlk


@pytest.fixture(scope="module")
def toy_attention():
    cfg = ATTN_TOY
    qs = gen_primes(cfg.q_bits, 2 * cfg.n, cfg.n_q + cfg.n_p)
    ck = Ckks(cfg.log_n, qs[:cfg.n_q], qs[cfg.n_q:], cfg.dnum)
    T, D, hd = cfg.tokens, cfg.feats, cfg.head_dim
    delta = float(2 ** cfg.scale_log2)
    s = ternary_secret(rng(cfg.index, 3), ck.n)
    g = rng(cfg.index, 1)
    Q = g.uniform(-1, 1, (T, D))
    K = g.uniform(-1, 1, (T, hd))
    V = g.uniform(-1, 1, (T, hd))
    ge = rng(cfg.index, 4)

    def enc(x, level):
        pt = ck.encode(x, None, delta, level + 1)
        return ck.encrypt(s, pt, uniform_residues(ge, ck.q[:level + 1], ck.n), gaussian_error(ge, ck.n))

    lv = cfg.level
    q_ct = enc(pack(Q, T, D), lv)
    k_ct = enc(pack(np.tile(K, (1, D // hd)), T, D), lv)
    v_ct = enc(pack(np.tile(V, (1, D // hd)), T, D), lv)
    keys, rlk = attn_keys(ck, s, T, D, hd, rng(cfg.index, 5))
    S = ck.attention_scores([q_ct], [k_ct], [0], T, hd, rlk, keys)[0]
    O = ck.attention_apply([S], [v_ct], [0], T, hd, rlk, keys)[0]
    S_lazy = ck.attention_scores([q_ct], [k_ct], [0], T, hd, rlk, keys, lazy=True)[0]
    return dict(ck=ck, s=s, Q=Q, K=K, V=V, S=S, O=O, S_lazy=S_lazy, delta=delta, T=T, D=D, hd=hd)


def test_toy_attention_scores_accuracy(toy_attention):
    t = toy_attention
    ck, T, D, hd = t["ck"], t["T"], t["D"], t["hd"]
    assert t["S"].shape == (2, ATTN_TOY.level - 1, ck.n)
    scale = t["delta"] * t["delta"] / ck.q[ATTN_TOY.level - 1]
    z = ck.decode(ck.decrypt(t["s"], t["S"]), scale)
    want = scores_def(t["Q"], t["K"], T, D, hd)
    err = np.max(np.abs(z.real.reshape(T, D) - want))
    assert err < 2.0 ** -30, err
    assert np.max(np.abs(z.imag)) < 2.0 ** -30


def test_toy_attention_apply_accuracy(toy_attention):
    t = toy_attention
    ck, T, D, hd = t["ck"], t["T"], t["D"], t["hd"]
    ls = ATTN_TOY.level - 2
    assert t["O"].shape == (2, ls, ck.n)
    s_scale = t["delta"] * t["delta"] / ck.q[ATTN_TOY.level - 1]
    o_scale = s_scale * t["delta"] / ck.q[ls]
    z = ck.decode(ck.decrypt(t["s"], t["O"]), o_scale)
    S = scores_def(t["Q"], t["K"], T, D, hd)
    want = apply_def(S, t["V"], T, D, hd)
    err = np.max(np.abs(z.real.reshape(T, D) - want))
    assert err < 2.0 ** -28, err


def test_toy_attention_scores_lazy_outer_sum(toy_attention):
    """The outer sum's hd - 1 rotations with one ModDown: before the final rescale the sum differs from the eager
    one by a few units per coefficient (the conversion digits' wrap), which the division by q rounds away except
    within a few units of a rounding boundary; the accuracy is the same."""
    t = toy_attention
    ck, T, D, hd = t["ck"], t["T"], t["D"], t["hd"]
    assert t["S_lazy"].shape == t["S"].shape
    scale = t["delta"] * t["delta"] / ck.q[ATTN_TOY.level - 1]
    z = ck.decode(ck.decrypt(t["s"], t["S_lazy"]), scale)
    err = np.max(np.abs(z.real.reshape(T, D) - scores_def(t["Q"], t["K"], T, D, hd)))
    assert err < 2.0 ** -30, err
