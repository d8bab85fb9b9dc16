"""Caller-owned workspace (ckks_set_workspace / ckks_workspace_bytes).

Every operation that takes scratch memory runs once with the library's own arena
and once with a caller workspace of exactly ckks_workspace_bytes for its shape;
the outputs must agree bit for bit.  A workspace one 256-byte step too small must
fail with CKKS_ENOMEM before any launch (the output buffer keeps its contents),
and clearing the workspace returns to the library's arena.
"""
import numpy as np
import pytest

from gpu_common import require_gpu, say, to_dev, to_host
from workloads import TOY, gaussian_error, gaussian_weights, rng, ternary_secret, uniform_residues, uniform_slots

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    require_gpu()
    import torch
    from paper_2609_12378_amd import Context
    cfg = TOY
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    n = ctx.n
    s = to_dev(ternary_secret(rng(cfg.index, 3, extra=77), n))
    g = rng(cfg.index, 1, extra=77)
    re = to_dev(uniform_slots(g, n // 2))
    im = to_dev(uniform_slots(g, n // 2))
    ge = rng(cfg.index, 4, extra=77)
    L = cfg.n_q
    a = to_dev(uniform_residues(ge, ctx.q[:L], n))
    e = to_dev(gaussian_error(ge, n))
    gk = rng(cfg.index, 5, extra=77)
    ka = to_dev(uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,)))
    ke = to_dev(gaussian_error(gk, (cfg.dnum, n)))
    return dict(torch=torch, ctx=ctx, cfg=cfg, s=s, re=re, im=im, a=a, e=e, ka=ka, ke=ke, L=L)


def _ws(env, nbytes):
    torch = env["torch"]
    assert nbytes > 0 and nbytes % 256 == 0
    return torch.empty(nbytes // 8, dtype=torch.uint64, device="cuda")


def _ops(env):
    """(name, op code, shape, fn) with fn() -> list of output tensors."""
    ctx, s, L = env["ctx"], env["s"], env["L"]
    pt = ctx.encode(env["re"], env["im"], 2.0 ** 30, L)
    ct = ctx.encrypt(s, pt, env["a"], env["e"])
    rlk = ctx.keygen_relin(s, env["ka"], env["ke"])
    keys = [ctx.keygen_galois(s, ctx.galois_elt(st), env["ka"], env["ke"]) for st in (1, 5, -3)]
    level = L - 1
    c1 = ct.data[1].contiguous()
    x = ctx.modup(c1, level)[0].contiguous()
    return [
        ("encode", ctx.OP_ENCODE, (), lambda: [ctx.encode(env["re"], env["im"], 2.0 ** 30, L).data]),
        ("decode", ctx.OP_DECODE, (L,), lambda: list(ctx.decode(pt))),
        ("encrypt", ctx.OP_ENCRYPT, (L,), lambda: [ctx.encrypt(s, pt, env["a"], env["e"]).data]),
        ("decrypt", ctx.OP_DECRYPT, (L,), lambda: [ctx.decrypt(s, ct).data]),
        ("keygen", ctx.OP_KEYGEN, (), lambda: [ctx.keygen_galois(s, ctx.galois_elt(7), env["ka"], env["ke"])]),
        ("rescale", ctx.OP_RESCALE, (L,), lambda: [ctx.rescale(ct).data]),
        ("rotate", ctx.OP_ROTATE, (L, 1), lambda: [ctx.rotate(ct, 1, keys[0]).data]),
        ("rotate_hoisted", ctx.OP_ROTATE, (L, 3),
         lambda: [o.data for o in ctx.rotate_hoisted(ct, [1, 5, -3], keys)]),
        ("mul_relin", ctx.OP_MUL_RELIN, (L,), lambda: [ctx.mul_relin(ct, ct, rlk).data]),
        ("modup", ctx.OP_MODUP, (level,), lambda: [ctx.modup(c1, level)]),
        ("moddown", ctx.OP_MODDOWN, (level,), lambda: [ctx.moddown(x, level)]),
    ]


def test_every_op_with_exact_workspace(env):
    ctx = env["ctx"]
    ops = _ops(env)
    want = {name: [to_host(t) for t in fn()] for name, _, _, fn in ops}
    for name, op, shape, fn in ops:
        nbytes = ctx.workspace_bytes(op, shape)
        say(name, "workspace bytes", nbytes)
        ws = _ws(env, nbytes)
        ctx.set_workspace(ws)
        got = [to_host(t) for t in fn()]
        ctx.set_workspace(None)
        for g, w in zip(got, want[name]):
            assert np.array_equal(g, w), name


def test_too_small_workspace_fails_before_launch(env):
    from paper_2609_12378_amd import Buf, CkksError
    ctx, s, L = env["ctx"], env["s"], env["L"]
    pt = ctx.encode(env["re"], env["im"], 2.0 ** 30, L)
    ct = ctx.encrypt(s, pt, env["a"], env["e"])
    keys = [ctx.keygen_galois(s, ctx.galois_elt(st), env["ka"], env["ke"]) for st in (1, 2)]
    nbytes = ctx.workspace_bytes(ctx.OP_ROTATE, (L, 2))
    ws = _ws(env, nbytes - 256)
    ctx.set_workspace(ws)
    outs = [Buf(ctx.zeros(2, L), ct.scale) for _ in range(2)]
    with pytest.raises(CkksError, match="too small"):
        ctx.rotate_hoisted(ct, [1, 2], keys, outs)
    for o in outs:
        assert not to_host(o.data).any()
    # the exact size works, and so does the library's arena again
    ctx.set_workspace(_ws(env, nbytes))
    r1 = [to_host(o.data) for o in ctx.rotate_hoisted(ct, [1, 2], keys)]
    ctx.set_workspace(None)
    r2 = [to_host(o.data) for o in ctx.rotate_hoisted(ct, [1, 2], keys)]
    for a, b in zip(r1, r2):
        assert np.array_equal(a, b)


def test_invalid_workspace_shapes_are_rejected(env):
    from paper_2609_12378_amd import CkksError
    ctx = env["ctx"]
    with pytest.raises(CkksError):
        ctx.workspace_bytes(99, (1,))
    with pytest.raises(CkksError):
        ctx.workspace_bytes(ctx.OP_DECRYPT, (ctx.n_q + 1,))
    with pytest.raises(CkksError):
        ctx.workspace_bytes(ctx.OP_LINEAR_PROJECT, (env["L"], 3, 128, 128, 8))  # 3 tokens do not divide the slots


def test_projection_with_exact_workspace(env):
    torch = env["torch"]
    ctx, s, cfg = env["ctx"], env["s"], env["cfg"]
    T, D, n1, L = cfg.tokens, cfg.feats, 16, cfg.level + 1
    d_in, d_out = 2 * D, 3 * D
    X = uniform_slots(rng(cfg.index, 1, extra=78), (T, d_in))
    W = to_dev(gaussian_weights(rng(cfg.index, 2, extra=78), (d_in, d_out)))
    ge = rng(cfg.index, 4, extra=78)
    cts = []
    for i in range(d_in // D):
        x = X[:, i * D:(i + 1) * D].T.reshape(-1)
        pt = ctx.encode(to_dev(x), None, 2.0 ** cfg.scale_log2, L)
        cts.append(ctx.encrypt(s, pt, to_dev(uniform_residues(ge, ctx.q[:L], ctx.n)), to_dev(gaussian_error(ge, ctx.n))))
    n2 = -(-D // n1)
    keys = {st: ctx.keygen_galois(s, ctx.galois_elt(st), env["ka"], env["ke"])
            for st in [T * b for b in range(1, n1)] + [T * n1 * g for g in range(1, n2)]}
    # the lazy ModDown's accumulators make the scratch larger: both modes, each against its own arena result
    for lazy in (False, True):
        ctx.set_lazy_moddown(lazy)
        ctx.set_proj_batch(0)
        want = [to_host(o.data) for o in ctx.linear_project(cts, W, T, n1, keys)]
        for max_pairs in (0, 5):
            ctx.set_proj_batch(max_pairs)
            nbytes = ctx.workspace_bytes(ctx.OP_LINEAR_PROJECT, (L, T, d_in, d_out, n1))
            say("projection workspace bytes", nbytes, "max pairs", max_pairs, "lazy", lazy)
            ctx.set_workspace(_ws(env, nbytes))
            got = [to_host(o.data) for o in ctx.linear_project(cts, W, T, n1, keys)]
            ctx.set_workspace(None)
            for g, w in zip(got, want):
                assert np.array_equal(g, w)
    ctx.set_proj_batch(0)
    ctx.set_lazy_moddown(False)
    torch.cuda.synchronize()
