"""GPU parity of the attention block (scores on token diagonals, weighted sums of values) against the oracle.

Every output ciphertext compared is identical bit for bit to the oracle's, with the same scale, and its
decrypted slots agree with the plain definitions S[t, h, delta] = sum_d Q[t, h, d] K[(t + delta) mod T, d]
and O[t, h, d] = sum_delta S[t, h, delta] V[(t + delta) mod T, d] within the stated bounds:

* toy ring (N = 2^12, 16 tokens, two heads of 64 per ciphertext, inputs at level 5): three query
  ciphertexts on two key and two value ciphertexts, named out of order (the calls group them);
* a ring of degree 2^13 with 32 tokens and four heads of 32 per ciphertext, and the toy ring with 8 tokens
  and four heads of 64 (several mask runs per correlation block);
* a ring of degree 2^13 with 16 tokens and two heads of 128 per ciphertext: the correlation lengths of the
  benchmark (128 and 256), eager and lazy;
* the attention parameters at full degree (N = 2^16, 24 + 8 limbs, 128 tokens, two heads of 128 per
  ciphertext, inputs at level 11, scale 2^50: the launch shapes of the benchmark), two query ciphertexts on
  one key and one value ciphertext: decrypted results against the definitions (the oracle is too slow for
  the 508 keys at this degree);
* argument checks that fail before any launch, and a caller workspace of exactly the reported size.
"""
import dataclasses

import numpy as np
import pytest

from gpu_common import require_gpu, say, to_dev, to_host
from oracle import Ckks
from workloads import (ATTENTION, ATTN_HD128, ATTN_TOY, attention_inputs, gaussian_error, rng, ternary_secret,
                       uniform_residues)

pytestmark = pytest.mark.gpu


def scores_def(Q, K, T, D, hd):
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


def rep(Kh, D, hd):
    """A key or value head repeated in every head position: [T][hd] -> [T][D]."""
    return np.tile(Kh, (1, D // hd))


def gpu_attention(ctx, cfg, inp, kv_of_q, lazy):
    """Encrypt the inputs and generate the keys on the GPU, then run the scores and the weighted sums."""
    n, T, hd, level = ctx.n, cfg.tokens, cfg.head_dim, cfg.level
    D = (n // 2) // T
    delta = float(2 ** cfg.scale_log2)
    s_dev = to_dev(inp.s)
    plain = list(inp.Q) + [rep(K, D, hd) for K in inp.K] + [rep(V, D, hd) for V in inp.V]
    cts = [ctx.encrypt(s_dev, ctx.encode(to_dev(x.reshape(-1)), None, delta, level + 1), to_dev(a), to_dev(e))
           for x, (a, e) in zip(plain, inp.enc)]
    n_q, n_kv = len(inp.Q), len(inp.K)
    q_g, k_g, v_g = cts[:n_q], cts[n_q:n_q + n_kv], cts[n_q + n_kv:]
    keys_g = {st: ctx.keygen_galois(s_dev, ctx.galois_elt(st), to_dev(a), to_dev(e)) for st, (a, e) in inp.keys.items()}
    rlk_g = ctx.keygen_relin(s_dev, to_dev(inp.rlk[0]), to_dev(inp.rlk[1]))
    say("keys ready", len(keys_g))
    ctx.set_lazy_moddown(lazy)
    ctx.profile(True)
    ctx.profile_reset()
    S_g = ctx.attention_scores(q_g, k_g, kv_of_q, T, hd, rlk_g, keys_g)
    moddowns = ctx.profile_read("moddown")[1]
    ctx.profile(False)
    if lazy:
        # the keys' rotations (per key ciphertext used), then per query ciphertext its pre-rotations and the
        # batched relinearisation (batches of 32) and one ModDown for the whole outer sum
        b32 = -(-(T - 1) // 32)
        expect = len(set(kv_of_q)) * b32 + n_q * (b32 + -(-T // 32) + 1)
        assert moddowns == expect, (moddowns, expect)
    O_g = ctx.attention_apply(S_g, v_g, kv_of_q, T, hd, rlk_g, keys_g)
    say("gpu attention done")
    return S_g, O_g, s_dev


def decrypted_errors(ctx, cfg, inp, kv_of_q, S_g, O_g, s_dev):
    """Max decrypted error of the scores and the sums against the plain definitions."""
    T, hd = cfg.tokens, cfg.head_dim
    D = (ctx.n // 2) // T
    errs_s, errs_o = [], []
    for c in range(len(S_g)):
        Sd = scores_def(inp.Q[c], inp.K[kv_of_q[c]], T, D, hd)
        re, _ = ctx.decode(ctx.decrypt(s_dev, S_g[c]))
        errs_s.append(np.max(np.abs(to_host(re).reshape(T, D) - Sd)))
        Od = apply_def(Sd, inp.V[kv_of_q[c]], T, D, hd)
        re, _ = ctx.decode(ctx.decrypt(s_dev, O_g[c]))
        errs_o.append(np.max(np.abs(to_host(re).reshape(T, D) - Od)))
    return max(errs_s), max(errs_o)


def run_parity(cfg, n_q, n_kv, kv_of_q, lazy=False):
    require_gpu()
    from paper_2609_12378_amd import Context
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    ck = Ckks(cfg.log_n, ctx.q, ctx.p, cfg.dnum)
    n, T, hd, level = ctx.n, cfg.tokens, cfg.head_dim, cfg.level
    D = (n // 2) // T
    delta = float(2 ** cfg.scale_log2)
    inp = attention_inputs(cfg, ctx.q, ctx.primes, n_q, n_kv)
    S_g, O_g, s_dev = gpu_attention(ctx, cfg, inp, kv_of_q, lazy)
    plain = list(inp.Q) + [rep(K, D, hd) for K in inp.K] + [rep(V, D, hd) for V in inp.V]
    cts = [ck.encrypt(inp.s, ck.encode(x.reshape(-1), None, delta, level + 1), a, e)
           for x, (a, e) in zip(plain, inp.enc)]
    q_o, k_o, v_o = cts[:n_q], cts[n_q:n_q + n_kv], cts[n_q + n_kv:]
    keys_o = {st: ck.keygen_galois(inp.s, ck.galois_elt(st), a, e) for st, (a, e) in inp.keys.items()}
    rlk_o = ck.keygen_relin(inp.s, *inp.rlk)
    S_o = ck.attention_scores(q_o, k_o, kv_of_q, T, hd, rlk_o, keys_o, lazy=lazy)
    O_o = ck.attention_apply(S_o, v_o, kv_of_q, T, hd, rlk_o, keys_o)
    say("oracle attention done")
    s_scale = delta * delta / ctx.q[level - 1]
    o_scale = s_scale * delta / ctx.q[level - 2]
    for c in range(n_q):
        for got, want, scale, name in ((S_g[c], S_o[c], s_scale, "scores"), (O_g[c], O_o[c], o_scale, "sums")):
            gh = to_host(got.data)
            assert gh.shape == want.shape, name
            bad = np.argwhere(gh != want)
            assert bad.size == 0, "%s %d: first mismatches %s" % (name, c, bad[:5].tolist())
            assert got.scale == scale, (name, got.scale, scale)
    return decrypted_errors(ctx, cfg, inp, kv_of_q, S_g, O_g, s_dev)


def test_toy_attention_parity_grouped():
    es, eo = run_parity(ATTN_TOY, 3, 2, [1, 0, 1])
    say("toy attention max error: scores %.3g, sums %.3g" % (es, eo))
    assert es <= 2.0 ** -30
    assert eo <= 2.0 ** -28


def test_toy_attention_parity_lazy_moddown():
    es, eo = run_parity(ATTN_TOY, 2, 1, [0, 0], lazy=True)
    say("toy attention (lazy ModDown) max error: scores %.3g, sums %.3g" % (es, eo))
    assert es <= 2.0 ** -30
    assert eo <= 2.0 ** -28


def test_attention_parity_ring13_four_heads():
    cfg = dataclasses.replace(ATTN_TOY, name="attn13", log_n=13, tokens=32, head_dim=32)
    es, eo = run_parity(cfg, 1, 1, [0])
    say("N=2^13 attention max error: scores %.3g, sums %.3g" % (es, eo))
    assert es <= 2.0 ** -29
    assert eo <= 2.0 ** -26


def test_attention_parity_eight_tokens():
    # 8 tokens x 256 features (four heads of 64): runs of 8 NTT positions, several per correlation block
    cfg = dataclasses.replace(ATTN_TOY, name="attn8", tokens=8, head_dim=64)
    es, eo = run_parity(cfg, 1, 1, [0])
    say("8-token attention max error: scores %.3g, sums %.3g" % (es, eo))
    assert es <= 2.0 ** -30
    assert eo <= 2.0 ** -28


@pytest.mark.parametrize("mode", ["eager", "lazy"])
def test_attention_parity_bench_correlation_lengths(mode):
    """Heads of 128 with 16 tokens at N = 2^13 (256 features, two heads per ciphertext): the correlations run at
    the benchmark's lengths (128 for the scores, 256 for the weighted sums) with its positions per block.  The
    oracle's outputs for these seeded inputs are stored as SHA-256 digests (with 32 residues per row to locate a
    mismatch) by tests/golden/make_attention_golden.py; both outputs must match them bit for bit, with the
    oracle's scales, eager and with the lazy ModDown of the outer sum."""
    require_gpu()
    import hashlib
    import json
    import os
    from paper_2609_12378_amd import Context
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                           "attention_n13_hd128_outputs.json")) as f:
        golden = json.load(f)
    cfg = ATTN_HD128
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    inp = attention_inputs(cfg, ctx.q, ctx.primes, 1, 1)
    S_g, O_g, s_dev = gpu_attention(ctx, cfg, inp, [0], mode == "lazy")
    pos = golden["positions"]
    for got, name in ((S_g[0], "scores"), (O_g[0], "sums")):
        rec = golden["modes"][mode][name]
        gh = to_host(got.data)
        assert list(gh.shape) == rec["shape"], name
        samples = np.array([gh[c, r, pos] for c in range(gh.shape[0]) for r in range(gh.shape[1])], dtype=np.uint64)
        bad = np.argwhere(samples != np.array(rec["samples"], dtype=np.uint64))
        assert bad.size == 0, "%s: sampled residues differ at (row, sample) %s" % (name, bad[:5].tolist())
        assert hashlib.sha256(np.ascontiguousarray(gh, dtype="<u8").tobytes()).hexdigest() == rec["sha256"], name
        assert got.scale == rec["scale"], (name, got.scale, rec["scale"])
    es, eo = decrypted_errors(ctx, cfg, inp, [0], S_g, O_g, s_dev)
    say("N=2^13, hd=128 attention (%s) max error: scores %.3g, sums %.3g" % (mode, es, eo))
    assert es <= 2.0 ** -28
    assert eo <= 2.0 ** -26


def _dev_keys(ctx, s_dev, steps, seed):
    """Galois and relinearisation keys from device randomness (no oracle at this degree)."""
    import torch
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    n, dnum = ctx.n, ctx.dnum

    def rand_a():
        rows = [torch.randint(0, p, (dnum, 1, n), generator=gen, device="cuda", dtype=torch.int64)
                for p in ctx.primes]
        return torch.cat(rows, dim=1).view(torch.uint64).contiguous()

    def rand_e():
        e = torch.round(torch.randn((dnum, n), generator=gen, device="cuda", dtype=torch.float64) * 3.2)
        return e.clamp(-19, 19).to(torch.int32).contiguous()

    keys = {st: ctx.keygen_galois(s_dev, ctx.galois_elt(st), rand_a(), rand_e()) for st in steps}
    rlk = ctx.keygen_relin(s_dev, rand_a(), rand_e())
    return keys, rlk


def test_attention_full_degree_accuracy():
    require_gpu()
    import torch
    from paper_2609_12378_amd import Context
    cfg = ATTENTION
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    n, T, hd = ctx.n, cfg.tokens, cfg.head_dim
    D = (n // 2) // T
    level = cfg.level - 1  # as the projections leave them
    delta = float(2 ** cfg.scale_log2)
    s_dev = to_dev(ternary_secret(rng(cfg.index, 3, extra=51), n))
    g = rng(cfg.index, 1, extra=51)
    Qs = [g.uniform(-1, 1, (T, D)) for _ in range(2)]
    K = g.uniform(-1, 1, (T, hd))
    V = g.uniform(-1, 1, (T, hd))
    ge = rng(cfg.index, 4, extra=51)

    def enc(x):
        pt = ctx.encode(to_dev(x.reshape(-1)), None, delta, level + 1)
        return ctx.encrypt(s_dev, pt, to_dev(uniform_residues(ge, ctx.q[:level + 1], n)),
                           to_dev(gaussian_error(ge, n)))

    q_g = [enc(Q) for Q in Qs]
    k_g, v_g = enc(rep(K, D, hd)), enc(rep(V, D, hd))
    steps = Context.attention_steps(n // 2, T, hd)
    keys, rlk = _dev_keys(ctx, s_dev, steps, 51)
    say("full-degree keys ready", len(keys))
    S = ctx.attention_scores(q_g, [k_g], [0, 0], T, hd, rlk, keys)
    O = ctx.attention_apply(S, [v_g], [0, 0], T, hd, rlk, keys)
    torch.cuda.synchronize()
    say("full-degree attention done")
    es, eo = [], []
    for c in range(2):
        assert S[c].n_limbs == level - 1 and O[c].n_limbs == level - 2
        Sd = scores_def(Qs[c], K, T, D, hd)
        re, im = ctx.decode(ctx.decrypt(s_dev, S[c]))
        es.append(np.max(np.abs(to_host(re).reshape(T, D) - Sd)))
        assert np.max(np.abs(to_host(im))) <= 2.0 ** -24
        re, _ = ctx.decode(ctx.decrypt(s_dev, O[c]))
        eo.append(np.max(np.abs(to_host(re).reshape(T, D) - apply_def(Sd, V, T, D, hd))))
    say("full-degree attention max error: scores %.3g, sums %.3g" % (max(es), max(eo)))
    assert max(es) <= 2.0 ** -26
    assert max(eo) <= 2.0 ** -23
    del keys, rlk
    torch.cuda.empty_cache()


@pytest.fixture(scope="module")
def toy_env():
    require_gpu()
    from paper_2609_12378_amd import Context
    cfg = ATTN_TOY
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    n, T, hd = ctx.n, cfg.tokens, cfg.head_dim
    D = (n // 2) // T
    s_dev = to_dev(ternary_secret(rng(cfg.index, 3, extra=52), n))
    g = rng(cfg.index, 1, extra=52)
    ge = rng(cfg.index, 4, extra=52)
    L = cfg.level + 1

    def enc(x, limbs):
        pt = ctx.encode(to_dev(x.reshape(-1)), None, 2.0 ** cfg.scale_log2, limbs)
        return ctx.encrypt(s_dev, pt, to_dev(uniform_residues(ge, ctx.q[:limbs], n)), to_dev(gaussian_error(ge, n)))

    q = enc(g.uniform(-1, 1, (T, D)), L)
    k = enc(rep(g.uniform(-1, 1, (T, hd)), D, hd), L)
    v = enc(rep(g.uniform(-1, 1, (T, hd)), D, hd), L)
    gk = rng(cfg.index, 5, extra=52)
    keys = {}
    for st in ctx.attention_steps(n // 2, T, hd):
        keys[st] = ctx.keygen_galois(s_dev, ctx.galois_elt(st),
                                     to_dev(uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,))),
                                     to_dev(gaussian_error(gk, (cfg.dnum, n))))
    rlk = ctx.keygen_relin(s_dev, to_dev(uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,))),
                           to_dev(gaussian_error(gk, (cfg.dnum, n))))
    return dict(ctx=ctx, q=q, k=k, v=v, keys=keys, rlk=rlk, T=T, hd=hd, L=L)


def test_attention_rejects_bad_arguments(toy_env):
    from paper_2609_12378_amd import Buf, CkksError
    t = toy_env
    ctx, q, k, v, keys, rlk, T, hd, L = (t[x] for x in ("ctx", "q", "k", "v", "keys", "rlk", "T", "hd", "L"))
    out = Buf(ctx.zeros(2, L - 2), 1.0)
    with pytest.raises(CkksError, match="tokens"):
        ctx.attention_scores([q], [k], [0], 3, hd, rlk, keys, outs=[out])
    with pytest.raises(CkksError, match="head dimension"):
        ctx.attention_scores([q], [k], [0], T, 8, rlk, keys, outs=[out])
    with pytest.raises(CkksError, match="names key"):
        ctx.attention_scores([q], [k], [1], T, hd, rlk, keys, outs=[out])
    missing = {st: key for st, key in keys.items() if st != 5}
    with pytest.raises(CkksError, match="no key for step 5"):
        ctx.attention_scores([q], [k], [0], T, hd, rlk, missing, outs=[out])
    with pytest.raises(CkksError, match="limbs"):
        ctx.attention_scores([q], [k], [0], T, hd, rlk, keys, outs=[Buf(ctx.zeros(2, L - 1), 1.0)])
    # the scores must sit below the values
    out1 = Buf(ctx.zeros(2, L - 1), 1.0)
    with pytest.raises(CkksError, match="fewer than the values"):
        ctx.attention_apply([q], [v], [0], T, hd, rlk, keys, outs=[out1])
    assert not to_host(out.data).any() and not to_host(out1.data).any()
    with pytest.raises(CkksError):
        ctx.workspace_bytes(ctx.OP_ATTN_SCORES, (L, 3, hd))
    with pytest.raises(CkksError):
        ctx.workspace_bytes(ctx.OP_ATTN_APPLY, (L, L, T, hd))


def test_attention_with_exact_workspace(toy_env):
    import torch
    t = toy_env
    ctx, q, k, v, keys, rlk, T, hd, L = (t[x] for x in ("ctx", "q", "k", "v", "keys", "rlk", "T", "hd", "L"))
    S = ctx.attention_scores([q], [k], [0], T, hd, rlk, keys)
    O = ctx.attention_apply(S, [v], [0], T, hd, rlk, keys)
    want_s, want_o = to_host(S[0].data), to_host(O[0].data)
    nb_s = ctx.workspace_bytes(ctx.OP_ATTN_SCORES, (L, T, hd))
    nb_o = ctx.workspace_bytes(ctx.OP_ATTN_APPLY, (L - 2, L, T, hd))
    say("attention workspace bytes", nb_s, nb_o)
    ctx.set_workspace(torch.empty(nb_s // 8, dtype=torch.uint64, device="cuda"))
    S2 = ctx.attention_scores([q], [k], [0], T, hd, rlk, keys)
    ctx.set_workspace(torch.empty(nb_o // 8, dtype=torch.uint64, device="cuda"))
    O2 = ctx.attention_apply(S2, [v], [0], T, hd, rlk, keys)
    ctx.set_workspace(None)
    assert np.array_equal(to_host(S2[0].data), want_s)
    assert np.array_equal(to_host(O2[0].data), want_o)
