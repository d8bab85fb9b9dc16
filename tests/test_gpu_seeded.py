"""GPU parity of seed-expanded switching keys against the oracle's seeded mode.

A seeded key is its b half plus a 128-bit seed; the a half is Philox-4x64-10 output rejection-sampled per digit,
prime and position, regenerated inside the key-switching kernels.  Against the oracle (whose seeded key is the
plain key (b, expand_key_a(seed))), bit for bit:

* the expanded a half: the toy ring, the key-switching parameters at N = 2^16, and a ring whose last prime lies
  just above 2^40 (about half the candidates rejected: the retry path runs on the device);
* the b half from ckks_keygen_galois_seeded, toy and N = 2^16;
* hoisted rotations with seeded keys: toy (three steps), the key-switching benchmark's 32-rotation batch at level
  23 (rotations 1, 17, 32 compared; the fused P-row inner product and the fused ModDown generate a), and 59/60-bit
  primes at N = 2^13 (the integer inner product over every row).
"""
import numpy as np
import pytest

from gpu_common import require_gpu, say, to_dev, to_host
from oracle import Ckks, is_prime
from workloads import KEYSWITCH, TOY, gaussian_error, rng, ternary_secret, uniform_residues, uniform_slots

pytestmark = pytest.mark.gpu


def eq(dev, host, what=""):
    got = to_host(dev)
    assert got.shape == host.shape, (what, got.shape, host.shape)
    bad = np.argwhere(got != host)
    assert bad.size == 0, "%s: first mismatches at %s" % (what, bad[:5].tolist())


def make(cfg=None, log_n=None, n_q=None, n_p=None, dnum=None, q_bits=None, p_bits=0, q=None, p=None):
    from paper_2609_12378_amd import Context
    if cfg is not None:
        log_n, n_q, n_p, dnum, q_bits = cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, cfg.q_bits
    ctx = Context(log_n, n_q, n_p, dnum, q_bits=q_bits or 50, p_bits=p_bits, q=q, p=p)
    return ctx, Ckks(log_n, ctx.q, ctx.p, dnum)


def test_expand_key_a_matches_oracle():
    require_gpu()
    for cfg in (TOY, KEYSWITCH):
        ctx, ck = make(cfg)
        for seed in ([1, 2], [0xFFFFFFFFFFFFFFFF, 0x8000000000000001]):
            say("expand_key_a", cfg.name, seed)
            eq(ctx.expand_key_a(seed), ck.expand_key_a(seed), "a half")
    # a prime just above 2^40: 41-bit candidates, about half rejected
    two_n = 2 << 12
    c = (1 << 40) + 1
    c += (1 - c) % two_n
    while not is_prime(c):
        c += two_n
    from oracle import gen_primes
    qs = gen_primes(36, two_n, 3) + [c]
    ctx, ck = make(log_n=12, n_q=3, n_p=1, dnum=2, q=qs[:3], p=qs[3:])
    a = ctx.expand_key_a([5, 6])
    eq(a, ck.expand_key_a([5, 6]), "a half with rejections")
    assert np.all(to_host(a)[:, 3] < c)


@pytest.mark.parametrize("cfg", [TOY, KEYSWITCH], ids=["toy", "n16"])
def test_keygen_seeded_matches_oracle(cfg):
    require_gpu()
    ctx, ck = make(cfg)
    n = ctx.n
    s = ternary_secret(rng(cfg.index, 3, extra=80), n)
    e = gaussian_error(rng(cfg.index, 5, extra=80), (cfg.dnum, n))
    g = ck.galois_elt(7)
    say("keygen seeded", cfg.name)
    eq(ctx.keygen_galois_seeded(to_dev(s), g, [11, 12], to_dev(e)), ck.keygen_galois_seeded(s, g, [11, 12], e),
       "b half")


def rotation_case(ctx, ck, cfg_index, limbs, steps, compare, scale=2.0 ** 40, tag=81):
    n = ctx.n
    s = ternary_secret(rng(cfg_index, 3, extra=tag), n)
    re = uniform_slots(rng(cfg_index, 1, extra=tag), n // 2)
    g = rng(cfg_index, 4, extra=tag)
    a, e = uniform_residues(g, ctx.q[:limbs], n), gaussian_error(g, n)
    cto = ck.encrypt(s, ck.encode(re, None, scale, limbs), a, e)
    ctg = ctx.encrypt(to_dev(s), ctx.encode(to_dev(re), None, scale, limbs), to_dev(a), to_dev(e))
    eq(ctg.data, cto, "ciphertext")
    keys_b, seeds, keys_o = [], [], {}
    for i, st in enumerate(steps):
        seed = [1000 + i, 77 * i + 3]
        ke = gaussian_error(rng(cfg_index, 5, extra=tag * 100 + i), (ck.dnum, n))
        gel = ck.galois_elt(st)
        keys_b.append(ctx.keygen_galois_seeded(to_dev(s), gel, seed, to_dev(ke)))
        seeds.append(seed)
        if st in compare:
            keys_o[st] = ck.seeded_key(ck.keygen_galois_seeded(s, gel, seed, ke), seed)
    outs = ctx.rotate_hoisted_seeded(ctg, steps, keys_b, seeds)
    want = ck.rotate_hoisted(cto, compare, [keys_o[st] for st in compare])
    for st, w in zip(compare, want):
        eq(outs[steps.index(st)].data, w, "rotation %d" % st)
        assert outs[steps.index(st)].scale == scale
    # the last rotation decrypts to the rotated slots
    dre, _ = ctx.decode(ctx.decrypt(to_dev(s), outs[-1]))
    return float(np.max(np.abs(to_host(dre) - np.roll(re, -steps[-1]))))


def test_rotate_hoisted_seeded_toy():
    require_gpu()
    ctx, ck = make(TOY)
    err = rotation_case(ctx, ck, TOY.index, TOY.n_q, [1, -2, 5], [1, -2, 5], scale=2.0 ** 30)
    say("toy seeded rotations: decrypted error", err)
    assert err < 2.0 ** -12


def test_rotate_hoisted_seeded_benchmark_batch():
    require_gpu()
    ctx, ck = make(KEYSWITCH)
    say("seeded batch: 32 hoisted rotations at level 23")
    err = rotation_case(ctx, ck, KEYSWITCH.index, KEYSWITCH.level + 1, list(range(1, 33)), [1, 17, 32])
    say("seeded batch: decrypted error", err)
    assert err < 2.0 ** -18


def test_rotate_hoisted_seeded_wide_primes():
    """59-bit q and 60-bit special primes (the paper's sizes) at N = 2^13: every row takes the integer path."""
    require_gpu()
    ctx, ck = make(log_n=13, n_q=5, n_p=2, dnum=3, q_bits=59, p_bits=60)
    assert all(q >= 1 << 58 for q in ctx.q) and all(p >= 1 << 59 for p in ctx.p)
    say("seeded rotations, 59/60-bit primes, N = 2^13")
    err = rotation_case(ctx, ck, 3, 5, [3, -1], [3, -1], scale=2.0 ** 40, tag=82)
    say("wide primes seeded rotations: decrypted error", err)
    assert err < 2.0 ** -12
