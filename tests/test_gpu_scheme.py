"""GPU parity of encoding, encryption, key generation, the homomorphic operations and
each key-switching stage, bit for bit against the oracle on the same seeded inputs.

Two parameter sets: the toy ring (N = 2^12, 4 + 2 limbs of 36-bit primes, dnum 2)
and the key-switching / projection chain at full degree (N = 2^16, 24 + 8 limbs of
50-bit primes, dnum 3) at level 12 (partial second digit) and level 23.
"""
import dataclasses

import numpy as np
import pytest

from gpu_common import require_gpu, say, to_dev, to_host
from oracle import Ckks
from workloads import (KEYSWITCH, TOY, gaussian_error, rng, ternary_secret, uniform_residues,
                       uniform_slots)

pytestmark = pytest.mark.gpu


class Env:
    def __init__(self, cfg, seed):
        require_gpu()
        from paper_2609_12378_amd import Buf, Context
        self.Buf = Buf
        self.cfg = cfg
        self.ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
        self.ck = Ckks(cfg.log_n, self.ctx.q, self.ctx.p, cfg.dnum)
        self.n = self.ctx.n
        self.s = ternary_secret(rng(cfg.index, 3, extra=seed), self.n)
        self.s_dev = to_dev(self.s)
        self.seed = seed

    def slots(self, seed, cplx=True):
        g = rng(self.cfg.index, 1, extra=self.seed * 100 + seed)
        re = uniform_slots(g, self.n // 2)
        im = uniform_slots(g, self.n // 2) if cplx else None
        return re, im

    def encrypt_both(self, seed, limbs, scale):
        re, im = self.slots(seed)
        pt_o = self.ck.encode(re, im, scale, limbs)
        g = rng(self.cfg.index, 4, extra=self.seed * 100 + seed)
        a = uniform_residues(g, self.ctx.q[:limbs], self.n)
        e = gaussian_error(g, self.n)
        ct_o = self.ck.encrypt(self.s, pt_o, a, e)
        pt_g = self.ctx.encode(to_dev(re), to_dev(im), scale, limbs)
        ct_g = self.ctx.encrypt(self.s_dev, pt_g, to_dev(a), to_dev(e))
        return ct_o, ct_g, (re, im)

    def key_randomness(self, seed):
        g = rng(self.cfg.index, 5, extra=self.seed * 100 + seed)
        a = uniform_residues(g, self.ctx.primes, self.n, lead=(self.cfg.dnum,))
        e = gaussian_error(g, (self.cfg.dnum, self.n))
        return a, e

    def galois_keys(self, seed, steps):
        a, e = self.key_randomness(seed)
        g = self.ck.galois_elt(steps)
        assert self.ctx.galois_elt(steps) == g
        return self.ck.keygen_galois(self.s, g, a, e), self.ctx.keygen_galois(self.s_dev, g, to_dev(a), to_dev(e))


@pytest.fixture(scope="module")
def toy():
    return Env(TOY, 1)


@pytest.fixture(scope="module")
def big():
    return Env(KEYSWITCH, 2)


def eq(dev, host):
    got = to_host(dev)
    assert got.shape == host.shape, (got.shape, host.shape)
    bad = np.argwhere(got != host)
    assert bad.size == 0, "first mismatches at %s" % bad[:5].tolist()


@pytest.mark.parametrize("scale_log2,cplx", [(30, True), (30, False), (35, True)])
def test_encode_toy(toy, scale_log2, cplx):
    re, im = toy.slots(10 + scale_log2, cplx)
    scale = float(2 ** scale_log2)
    pt = toy.ctx.encode(to_dev(re), to_dev(im) if cplx else None, scale, 4)
    eq(pt.data[0], toy.ck.encode(re, im, scale, 4))


def test_encode_full_degree_at_projection_scale(big):
    # the projection encodes weights at scale q_12 (about 2^50): many coefficients lie within
    # the fp64 error of a rounding tie, so this checks that the evaluation order matches
    g = rng(4, 2, extra=7)
    re = g.normal(0, 0.02, big.n // 2)
    scale = float(big.ctx.q[12])
    pt = big.ctx.encode(to_dev(re), None, scale, 13)
    eq(pt.data[0], big.ck.encode(re, None, scale, 13))


def test_encode_integer_arithmetic(big):
    # the same plaintexts through the integer Shoup butterflies
    g = rng(4, 2, extra=9)
    scale = float(big.ctx.q[12])
    big.ctx.set_ntt_arith(1)
    try:
        for r in range(4):
            re = np.repeat(g.normal(0, 0.02, 256), 128)
            pt = big.ctx.encode(to_dev(re), None, scale, 13)
            eq(pt.data[0], big.ck.encode(re, None, scale, 13))
    finally:
        big.ctx.set_ntt_arith(0)


def test_encode_large_coefficients(toy):
    # coefficients beyond 2^52 take the exact integer reduction inside the fp64 transform
    re, im = toy.slots(99)
    scale = float(2 ** 61)
    pt = toy.ctx.encode(to_dev(re), to_dev(im), scale, 4)
    eq(pt.data[0], toy.ck.encode(re, im, scale, 4))


def test_encode_large_coefficients_full_degree(big):
    # the same at N = 2^16 (the 8-residue column pass and its exact integer reduction)
    g = rng(4, 2, extra=10)
    re = g.uniform(-1, 1, big.n // 2)
    scale = float(2 ** 61)
    pt = big.ctx.encode(to_dev(re), None, scale, 4)
    want = big.ck.encode(re, None, scale, 4)
    assert np.abs(big.ck.encode_int(re, None, scale)).max() > 2 ** 52
    eq(pt.data[0], want)


def test_encode_many_weight_vectors_full_degree(big):
    # 24 more weight-like vectors at scale q_12: each has tens of coefficients within one ulp
    # of a rounding tie, so any difference in twiddles or operation order shows up here
    g = rng(4, 2, extra=8)
    scale = float(big.ctx.q[12])
    for r in range(24):
        re = np.repeat(g.normal(0, 0.02, 256), 128)
        pt = big.ctx.encode(to_dev(re), None, scale, 2)
        eq(pt.data[0], big.ck.encode(re, None, scale, 2))


def test_decode(toy, big):
    for env, limbs, scale in ((toy, 4, 2.0 ** 30), (toy, 1, 2.0 ** 30), (big, 13, 2.0 ** 40)):
        re, im = env.slots(20)
        pt = env.ctx.encode(to_dev(re), to_dev(im), scale, limbs)
        dre, dim = env.ctx.decode(pt)
        z = to_host(dre) + 1j * to_host(dim)
        assert np.max(np.abs(z - (re + 1j * im))) <= env.n / (2 * scale) + 1e-9


def test_encrypt_decrypt(toy):
    ct_o, ct_g, (re, im) = toy.encrypt_both(1, 4, 2.0 ** 30)
    eq(ct_g.data, ct_o)
    pt_g = toy.ctx.decrypt(toy.s_dev, ct_g)
    eq(pt_g.data[0], toy.ck.decrypt(toy.s, ct_o))


def test_keygen(toy, big):
    for env in (toy, big):
        ko, kg = env.galois_keys(3, 5)
        eq(kg, ko)
    a, e = toy.key_randomness(4)
    eq(toy.ctx.keygen_relin(toy.s_dev, to_dev(a), to_dev(e)), toy.ck.keygen_relin(toy.s, a, e))


def test_add_mul_plain_rescale(toy):
    c1o, c1g, _ = toy.encrypt_both(5, 4, 2.0 ** 30)
    c2o, c2g, _ = toy.encrypt_both(6, 4, 2.0 ** 30)
    eq(toy.ctx.add(c1g, c2g).data, toy.ck.ct_add(c1o, c2o))
    re, im = toy.slots(7)
    pto = toy.ck.encode(re, im, float(toy.ctx.q[3]), 4)
    ptg = toy.ctx.encode(to_dev(re), to_dev(im), float(toy.ctx.q[3]), 4)
    prod_g = toy.ctx.mul_plain(c1g, ptg)
    prod_o = toy.ck.ct_mul_plain(c1o, pto)
    eq(prod_g.data, prod_o)
    eq(toy.ctx.rescale(prod_g).data, toy.ck.rescale(prod_o))


def test_add_rejects_mismatched_scales(toy):
    from paper_2609_12378_amd import CkksError
    _, c1g, _ = toy.encrypt_both(8, 4, 2.0 ** 30)
    _, c2g, _ = toy.encrypt_both(9, 4, 2.0 ** 31)
    with pytest.raises(CkksError, match="scale"):
        toy.ctx.add(c1g, c2g)


@pytest.mark.parametrize("level", [3, 2, 0])
def test_modup_moddown_automorph_toy(toy, level):
    c = uniform_residues(rng(1, 6, extra=level), toy.ctx.q[:level + 1], toy.n)
    eq(toy.ctx.modup(to_dev(c), level), toy.ck.modup(c, level))
    ext = toy.ck.ext_primes(level)
    x = uniform_residues(rng(1, 7, extra=level), [toy.ck.primes[k] for k in ext], toy.n)
    eq(toy.ctx.moddown(to_dev(x), level), toy.ck.moddown(x, level))
    for g in (5, 25, 2 * toy.n - 1):
        eq(toy.ctx.automorph(to_dev(c), g), toy.ck.automorph(c, g))


@pytest.mark.parametrize("level", [12, 23])
def test_modup_moddown_full_degree(big, level):
    say("modup/moddown level", level)
    c = uniform_residues(rng(3, 6, extra=level), big.ctx.q[:level + 1], big.n)
    eq(big.ctx.modup(to_dev(c), level), big.ck.modup(c, level))
    ext = big.ck.ext_primes(level)
    x = uniform_residues(rng(3, 7, extra=level), [big.ck.primes[k] for k in ext], big.n)
    eq(big.ctx.moddown(to_dev(x), level), big.ck.moddown(x, level))


@pytest.mark.parametrize("steps", [1, 7, -2])
def test_rotate_toy(toy, steps):
    cto, ctg, _ = toy.encrypt_both(11, 4, 2.0 ** 30)
    ko, kg = toy.galois_keys(20 + steps, steps)
    eq(toy.ctx.rotate(ctg, steps, kg).data, toy.ck.rotate(cto, steps, ko))


def test_rotate_buffer_off_16_byte_boundary(toy):
    """A ciphertext whose data starts 8 bytes past a 16-byte boundary: ModUp's row copies take their 8-byte form."""
    import torch
    from paper_2609_12378_amd import Buf
    cto, ctg, _ = toy.encrypt_both(17, 4, 2.0 ** 30)
    flat = torch.zeros(ctg.data.numel() + 1, dtype=torch.uint64, device="cuda")
    view = flat[1:].view(ctg.data.shape)
    view.copy_(ctg.data)
    assert view.data_ptr() % 16 == 8
    ko, kg = toy.galois_keys(27, 7)
    eq(toy.ctx.rotate(Buf(view, ctg.scale), 7, kg).data, toy.ck.rotate(cto, 7, ko))


def test_rotate_hoisted_toy_lower_level(toy):
    cto, ctg, _ = toy.encrypt_both(12, 3, 2.0 ** 30)   # level 2: partial second digit
    steps = [1, 2, 16, 100]
    keys = [toy.galois_keys(40 + s, s) for s in steps]
    outs_g = toy.ctx.rotate_hoisted(ctg, steps, [k[1] for k in keys])
    outs_o = toy.ck.rotate_hoisted(cto, steps, [k[0] for k in keys])
    for og, oo in zip(outs_g, outs_o):
        eq(og.data, oo)


def test_rotate_full_degree(big):
    say("rotate full degree")
    cto, ctg, _ = big.encrypt_both(13, 13, 2.0 ** 40)
    ko, kg = big.galois_keys(50, 3)
    eq(big.ctx.rotate(ctg, 3, kg).data, big.ck.rotate(cto, 3, ko))


def test_rotate_hoisted_full_degree_few_special_primes():
    """N = 2^16 with 6 + 3 limbs and dnum 2: the ModDown's fused conversion and first forward pass take 3 source
    limbs (the guarded variant; the benchmark parameters have 8), ModUp digits of 3 limbs, bit for bit."""
    cfg = dataclasses.replace(KEYSWITCH, n_q=6, n_p=3, dnum=2, level=5, batch=3)
    env = Env(cfg, 3)
    say("rotate hoisted, 6 + 3 limbs at N = 2^16")
    cto, ctg, _ = env.encrypt_both(31, 6, 2.0 ** 40)
    steps = [1, 5, -3]
    keys = [env.galois_keys(70 + i, st) for i, st in enumerate(steps)]
    outs_g = env.ctx.rotate_hoisted(ctg, steps, [k[1] for k in keys])
    outs_o = env.ck.rotate_hoisted(cto, steps, [k[0] for k in keys])
    for og, oo in zip(outs_g, outs_o):
        eq(og.data, oo)


def test_rotate_hoisted_full_degree_wide_special_primes():
    """N = 2^16 with 50-bit q primes and 55-bit special primes: the batched ModDown keeps the fp64 finish over the
    q rows but takes the integer transforms and conversion for the P rows (no fp64-exact product there)."""
    require_gpu()
    from paper_2609_12378_amd import Context
    ctx = Context(16, 4, 2, 2, q_bits=50, p_bits=55)
    assert all(p >= 1 << 54 for p in ctx.p)
    ck = Ckks(16, ctx.q, ctx.p, 2)
    n = ctx.n
    s = ternary_secret(rng(3, 3, extra=55), n)
    re = uniform_slots(rng(3, 1, extra=55), n // 2)
    g = rng(3, 4, extra=55)
    a, e = uniform_residues(g, ctx.q, n), gaussian_error(g, n)
    cto = ck.encrypt(s, ck.encode(re, None, 2.0 ** 40, 4), a, e)
    ctg = ctx.encrypt(to_dev(s), ctx.encode(to_dev(re), None, 2.0 ** 40, 4), to_dev(a), to_dev(e))
    steps = [1, -4]
    keys_o, keys_g = [], []
    for i, st in enumerate(steps):
        gk = rng(3, 5, extra=550 + i)
        ka, ke = uniform_residues(gk, ctx.primes, n, lead=(2,)), gaussian_error(gk, (2, n))
        gel = ck.galois_elt(st)
        keys_o.append(ck.keygen_galois(s, gel, ka, ke))
        keys_g.append(ctx.keygen_galois(to_dev(s), gel, to_dev(ka), to_dev(ke)))
    say("rotate hoisted, 55-bit special primes at N = 2^16")
    outs_g = ctx.rotate_hoisted(ctg, steps, keys_g)
    outs_o = ck.rotate_hoisted(cto, steps, keys_o)
    for og, oo in zip(outs_g, outs_o):
        eq(og.data, oo)


def test_keyswitch_benchmark_batch_sampled(big):
    """The key-switching benchmark's own launch: 32 hoisted rotations by 1..32 of one level-23 ciphertext in one
    batch; rotations 1, 17 and 32 against the oracle bit for bit (a hoisted batch equals the same rotations made
    alone, so the oracle computes only those three)."""
    say("keyswitch benchmark batch: 32 hoisted rotations at level 23")
    cto, ctg, _ = big.encrypt_both(90, 24, 2.0 ** 40)
    steps = list(range(1, 33))
    keys_g, keys_o = [], {}
    for st in steps:
        a, e = big.key_randomness(200 + st)
        gel = big.ctx.galois_elt(st)
        keys_g.append(big.ctx.keygen_galois(big.s_dev, gel, to_dev(a), to_dev(e)))
        if st in (1, 17, 32):
            keys_o[st] = big.ck.keygen_galois(big.s, gel, a, e)
    outs_g = big.ctx.rotate_hoisted(ctg, steps, keys_g)
    sample = [1, 17, 32]
    outs_o = big.ck.rotate_hoisted(cto, sample, [keys_o[st] for st in sample])
    for st, oo in zip(sample, outs_o):
        eq(outs_g[st - 1].data, oo)


def test_mul_relin(toy):
    c1o, c1g, _ = toy.encrypt_both(14, 4, 2.0 ** 30)
    c2o, c2g, _ = toy.encrypt_both(15, 4, 2.0 ** 30)
    a, e = toy.key_randomness(60)
    rlk_o = toy.ck.keygen_relin(toy.s, a, e)
    rlk_g = toy.ctx.keygen_relin(toy.s_dev, to_dev(a), to_dev(e))
    eq(toy.ctx.mul_relin(c1g, c2g, rlk_g).data, toy.ck.mul_relin(c1o, c2o, rlk_o))


@pytest.mark.parametrize("limbs", [24, 13])
def test_mul_relin_full_degree(big, limbs):
    """Mult + relinearisation at N = 2^16 (24 + 8 limbs of 50-bit primes, dnum 3): at level 23 (three full digits)
    and level 12 (a partial second digit), bit for bit, and decrypted close to the slot-wise product."""
    say("mul_relin at N = 2^16 with", limbs, "limbs")
    c1o, c1g, (r1, i1) = big.encrypt_both(30 + limbs, limbs, 2.0 ** 40)
    c2o, c2g, (r2, i2) = big.encrypt_both(31 + limbs, limbs, 2.0 ** 40)
    a, e = big.key_randomness(61)
    rlk_o = big.ck.keygen_relin(big.s, a, e)
    rlk_g = big.ctx.keygen_relin(big.s_dev, to_dev(a), to_dev(e))
    out = big.ctx.mul_relin(c1g, c2g, rlk_g)
    eq(out.data, big.ck.mul_relin(c1o, c2o, rlk_o))
    assert out.scale == 2.0 ** 80
    dre, dim = big.ctx.decode(big.ctx.decrypt(big.s_dev, out))
    z = to_host(dre) + 1j * to_host(dim)
    assert np.max(np.abs(z - (r1 + 1j * i1) * (r2 + 1j * i2))) < 2.0 ** -20


def test_decrypted_rotation_is_slot_shift(toy):
    cto, ctg, (re, im) = toy.encrypt_both(16, 4, 2.0 ** 30)
    _, kg = toy.galois_keys(70, 5)
    out = toy.ctx.rotate(ctg, 5, kg)
    dre, dim = toy.ctx.decode(toy.ctx.decrypt(toy.s_dev, out))
    z = to_host(dre) + 1j * to_host(dim)
    assert np.max(np.abs(z - np.roll(re + 1j * im, -5))) < 1e-2


@pytest.mark.parametrize("steps", [0, 2048])
def test_rotate_identity_steps(toy, steps):
    # steps 0 and N/2 (the slot count) both give the Galois element 1: a key switch from s to s (the output
    # differs from the input by the key-switching noise only), bit for bit as the oracle
    cto, ctg, _ = toy.encrypt_both(17, 4, 2.0 ** 30)
    assert toy.ctx.galois_elt(steps) == 1
    ko, kg = toy.galois_keys(80 + steps, steps)
    eq(toy.ctx.rotate(ctg, steps, kg).data, toy.ck.rotate(cto, steps, ko))


def test_lowest_level_operations(toy):
    # one limb: rotation (a single partial digit), relinearised product; two limbs -> one: rescale
    c1o, c1g, _ = toy.encrypt_both(18, 1, 2.0 ** 20)
    c2o, c2g, _ = toy.encrypt_both(19, 1, 2.0 ** 10)
    ko, kg = toy.galois_keys(90, 3)
    eq(toy.ctx.rotate(c1g, 3, kg).data, toy.ck.rotate(c1o, 3, ko))
    a, e = toy.key_randomness(91)
    rlk_o = toy.ck.keygen_relin(toy.s, a, e)
    rlk_g = toy.ctx.keygen_relin(toy.s_dev, to_dev(a), to_dev(e))
    eq(toy.ctx.mul_relin(c1g, c2g, rlk_g).data, toy.ck.mul_relin(c1o, c2o, rlk_o))
    c3o, c3g, _ = toy.encrypt_both(20, 2, 2.0 ** 30)
    eq(toy.ctx.rescale(c3g).data, toy.ck.rescale(c3o))


@pytest.mark.parametrize("count", [33, 40])
def test_rotate_hoisted_beyond_one_batch(toy, count):
    # more rotations than one key-switching launch takes (32): a second, ragged batch
    cto, ctg, _ = toy.encrypt_both(21, 4, 2.0 ** 30)
    steps = [s + 1 for s in range(count)]
    keys = [toy.galois_keys(100 + s, s) for s in steps]
    outs_g = toy.ctx.rotate_hoisted(ctg, steps, [k[1] for k in keys])
    outs_o = toy.ck.rotate_hoisted(cto, steps, [k[0] for k in keys])
    for og, oo in zip(outs_g, outs_o):
        eq(og.data, oo)
