"""GPU parity at the paper's modulus sizes (Evaluation, "Experimental Setup": N = 2^16, 60-bit first modulus,
59-bit others, dnum = 5), where every prime is at least 2^50 and the integer (64-bit Shoup) paths run: transforms,
inner products, basis conversions, ModDown and the unfused projection multiply-accumulate.  Bit for bit against
the oracle:

* the NTT and inverse of sampled rows of all 45 primes;
* a hoisted batch of three rotations of a level-36 ciphertext (37 q-limbs + 8 special primes, five digits), two
  compared, and a single rotation at level 12 (three digits, the last partial);
* the projection's parameters on a 256 x 512 slice of the weights at level 12 (31 baby, 7 giant rotations;
  weight plaintexts at scale q_12 of 59 bits), with the lazy ModDown, decrypted within 2^-18 of X @ W.
* mul_relin of two level-12 ciphertexts at scale 2^50 and the rescale after it, decrypted within 2^-20 of the
  slot-wise product.
"""
import numpy as np
import pytest

from gpu_common import require_gpu, say, to_dev, to_host
from oracle import Ckks, gen_primes
from workloads import (KEYSWITCH_PAPER, PROJECTION, fm_pack, gaussian_error, gaussian_weights, paper_chain, rng,
                       ternary_secret, uniform_residues, uniform_slots)

pytestmark = pytest.mark.gpu


def eq(dev, host, what=""):
    got = to_host(dev)
    assert got.shape == host.shape, (what, got.shape, host.shape)
    bad = np.argwhere(got != host)
    assert bad.size == 0, "%s: first mismatches at %s" % (what, bad[:5].tolist())


@pytest.fixture(scope="module")
def env():
    require_gpu()
    from paper_2609_12378_amd import Context
    cfg = KEYSWITCH_PAPER
    q, p = paper_chain(gen_primes(60, 2 * cfg.n, 1 + cfg.n_p), gen_primes(59, 2 * cfg.n, cfg.n_q - 1), cfg.n_q,
                       cfg.n_p)
    assert q[0] >= 1 << 59 and all((1 << 58) <= x < (1 << 59) for x in q[1:]) and all(x >= 1 << 59 for x in p)
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q=q, p=p)
    return cfg, ctx, Ckks(cfg.log_n, q, p, cfg.dnum)


def test_ntt_paper_primes(env):
    cfg, ctx, ck = env
    R = cfg.n_q + cfg.n_p
    a = uniform_residues(rng(cfg.index, 1), ctx.primes, ctx.n)
    t = to_dev(a)
    ctx.ntt(t)
    got = to_host(t)
    for k in (0, 1, 20, 36, 37, 44):
        assert np.array_equal(got[k], ck.ntt(a[k:k + 1], [k])[0]), k
    ctx.intt(t)
    eq(t, a, "round trip")
    assert R == 45


def rotations(env, limbs, steps, compare, tag):
    cfg, ctx, ck = env
    n = ctx.n
    s = ternary_secret(rng(cfg.index, 3, extra=tag), n)
    z = uniform_slots(rng(cfg.index, 1, extra=tag), n // 2)
    g = rng(cfg.index, 4, extra=tag)
    a, e = uniform_residues(g, ctx.q[:limbs], n), gaussian_error(g, n)
    cto = ck.encrypt(s, ck.encode(z, None, 2.0 ** 40, limbs), a, e)
    ctg = ctx.encrypt(to_dev(s), ctx.encode(to_dev(z), None, 2.0 ** 40, limbs), to_dev(a), to_dev(e))
    eq(ctg.data, cto, "ciphertext")
    keys_g, keys_o = [], {}
    for i, st in enumerate(steps):
        gk = rng(cfg.index, 5, extra=tag * 10 + i)
        ka, ke = uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,)), gaussian_error(gk, (cfg.dnum, n))
        gel = ck.galois_elt(st)
        keys_g.append(ctx.keygen_galois(to_dev(s), gel, to_dev(ka), to_dev(ke)))
        if st in compare:
            keys_o[st] = ck.keygen_galois(s, gel, ka, ke)
            eq(keys_g[-1], keys_o[st], "key %d" % st)
    outs = ctx.rotate_hoisted(ctg, steps, keys_g)
    for st, w in zip(compare, ck.rotate_hoisted(cto, compare, [keys_o[st] for st in compare])):
        eq(outs[steps.index(st)].data, w, "rotation %d" % st)
    re, _ = ctx.decode(ctx.decrypt(to_dev(s), outs[-1]))
    return float(np.max(np.abs(to_host(re) - np.roll(z, -steps[-1]))))


def test_rotate_hoisted_paper_params_top_level(env):
    say("paper parameters: 3 hoisted rotations at level 36")
    err = rotations(env, 37, [1, 5, -3], [5, -3], 60)
    say("decrypted error", err)
    assert err < 2.0 ** -18


def test_rotate_paper_params_level12(env):
    say("paper parameters: one rotation at level 12")
    err = rotations(env, 13, [7], [7], 61)
    say("decrypted error", err)
    assert err < 2.0 ** -18


def test_projection_slice_paper_params(env):
    cfg, ctx, ck = env
    proj = PROJECTION
    T, D, n1, level = proj.tokens, proj.feats, proj.n1, proj.level
    n = ctx.n
    n2 = D // n1
    ctx.set_lazy_moddown(True)
    s = ternary_secret(rng(cfg.index, 3, extra=62), n)
    X = uniform_slots(rng(cfg.index, 1, extra=62), (T, 256))
    W = gaussian_weights(rng(cfg.index, 2, extra=62), (256, 512))
    g = rng(cfg.index, 4, extra=62)
    a, e = uniform_residues(g, ctx.q[:level + 1], n), gaussian_error(g, n)
    x = fm_pack(X, T, D, 0)
    cto = ck.encrypt(s, ck.encode(x, None, 2.0 ** 40, level + 1), a, e)
    ctg = ctx.encrypt(to_dev(s), ctx.encode(to_dev(x), None, 2.0 ** 40, level + 1), to_dev(a), to_dev(e))
    keys_g, keys_o = {}, {}
    gk = rng(cfg.index, 5, extra=62)
    for st in [T * b for b in range(1, n1)] + [T * n1 * gg for gg in range(1, n2)]:
        ka, ke = uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,)), gaussian_error(gk, (cfg.dnum, n))
        gel = ck.galois_elt(st)
        keys_o[st] = ck.keygen_galois(s, gel, ka, ke)
        keys_g[st] = ctx.keygen_galois(to_dev(s), gel, to_dev(ka), to_dev(ke))
    say("paper parameters: 256 x 512 projection slice at level 12")
    outs = ctx.linear_project([ctg], to_dev(W), T, n1, keys_g)
    want = ck.linear_project([cto], W, T, n1, keys_o, lazy=True)
    Y = X @ W
    for j in range(2):
        eq(outs[j].data, want[j], "output %d" % j)
        re, _ = ctx.decode(ctx.decrypt(to_dev(s), outs[j]))
        err = float(np.max(np.abs(to_host(re) - fm_pack(Y, T, D, j))))
        say("output", j, "decrypted error", err)
        assert err <= 2.0 ** -18


def test_mul_relin_rescale_paper_params(env):
    """Mult + relinearisation and the rescale that follows it at level 12 of the paper's chain (two digits, the
    second partial): the 128-bit tensor products, the relinearisation's integer key switch and the integer rescale,
    bit for bit, and the decrypted result close to the slot-wise product."""
    cfg, ctx, ck = env
    n, limbs = ctx.n, 13
    say("paper parameters: mul_relin and rescale at level 12")
    s = ternary_secret(rng(cfg.index, 3, extra=63), n)
    cts_o, cts_g, zs = [], [], []
    for k in range(2):
        z = uniform_slots(rng(cfg.index, 1, extra=64 + k), n // 2)
        g = rng(cfg.index, 4, extra=64 + k)
        a, e = uniform_residues(g, ctx.q[:limbs], n), gaussian_error(g, n)
        cts_o.append(ck.encrypt(s, ck.encode(z, None, 2.0 ** 50, limbs), a, e))
        cts_g.append(ctx.encrypt(to_dev(s), ctx.encode(to_dev(z), None, 2.0 ** 50, limbs), to_dev(a), to_dev(e)))
        zs.append(z)
    gk = rng(cfg.index, 5, extra=63)
    ka, ke = uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,)), gaussian_error(gk, (cfg.dnum, n))
    rlk_o = ck.keygen_relin(s, ka, ke)
    rlk_g = ctx.keygen_relin(to_dev(s), to_dev(ka), to_dev(ke))
    eq(rlk_g, rlk_o, "relinearisation key")
    prod_g = ctx.mul_relin(cts_g[0], cts_g[1], rlk_g)
    prod_o = ck.mul_relin(cts_o[0], cts_o[1], rlk_o)
    eq(prod_g.data, prod_o, "mul_relin")
    res_g = ctx.rescale(prod_g)
    eq(res_g.data, ck.rescale(prod_o), "rescale")
    assert abs(res_g.scale / (2.0 ** 100 / float(ctx.q[limbs - 1])) - 1.0) < 1e-15
    re, _ = ctx.decode(ctx.decrypt(to_dev(s), res_g))
    err = float(np.max(np.abs(to_host(re) - zs[0] * zs[1])))
    say("decrypted error", err)
    assert err < 2.0 ** -20
