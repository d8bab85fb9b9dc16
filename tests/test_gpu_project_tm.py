"""GPU parity of the token-major (periodic) projection against the oracle.

Every output ciphertext compared is identical bit for bit to the oracle's, its
decrypted slots agree with the oracle's within 2^-20 of the scale, and with X @ W
within the stated bound:

* toy ring (N = 2^12, 16 tokens x 128 features), n1 = 16, two inputs and three
  outputs, at most five (input, baby step) pairs per launch so the sums are
  carried across launches;
* toy ring with the plain diagonal split (n1 = 128, no giant step), and with n1 = 24,
  which does not divide D (runs of 16 values: the matrix-core multiply-accumulate
  except for n1 = 24, which takes the vector-ALU one);
* a ring of degree 2^10 with 4 tokens (runs of four equal plaintext values: the
  vector-ALU multiply-accumulate, one block meeting many runs);
* the projection parameters at full degree (N = 2^16, 24 + 8 limbs, level 12, 128
  tokens x 256 features, n1 = 32: 31 + 32 baby and 7 giant rotations) on a
  256 x 512 slice (runs of 128 values: the matrix-core multiply-accumulate);
* the token-major benchmark call itself (4096 x 14336, n1 = 32, lazy ModDown): outputs 0,
  27 and 55 against the oracle's stored digests.
"""
import dataclasses

import numpy as np
import pytest

from gpu_common import require_gpu, say, to_dev, to_host
from oracle import Ckks
from workloads import (PROJECTION, TOY, gaussian_error, gaussian_weights, rng, ternary_secret,
                       uniform_residues, uniform_slots)

pytestmark = pytest.mark.gpu


def tm_pack(X, T, D, i):
    return X[:, i * D:(i + 1) * D].reshape(-1)


def run_case(cfg, d_in, d_out, n1, oracle_outputs, max_pairs=0, lazy=False):
    require_gpu()
    from paper_2609_12378_amd import Context
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    ctx.set_proj_batch(max_pairs)
    ctx.set_lazy_moddown(lazy)
    ck = Ckks(cfg.log_n, ctx.q, ctx.p, cfg.dnum)
    n, T, level = ctx.n, cfg.tokens, cfg.level
    D = (n // 2) // T
    n2 = -(-D // n1)
    s = ternary_secret(rng(cfg.index, 3, extra=40), n)
    X = uniform_slots(rng(cfg.index, 1, extra=40), (T, d_in))
    W = gaussian_weights(rng(cfg.index, 2, extra=40), (d_in, d_out))
    delta = float(2 ** cfg.scale_log2)
    ge = rng(cfg.index, 4, extra=40)
    s_dev = to_dev(s)
    cts_o, cts_g = [], []
    for i in range(d_in // D):
        x = tm_pack(X, T, D, i)
        a = uniform_residues(ge, ctx.q[:level + 1], n)
        e = gaussian_error(ge, n)
        cts_o.append(ck.encrypt(s, ck.encode(x, None, delta, level + 1), a, e))
        cts_g.append(ctx.encrypt(s_dev, ctx.encode(to_dev(x), None, delta, level + 1), to_dev(a), to_dev(e)))
    steps = [b for b in range(1, n1)] + [b - D for b in range(n1)] + [n1 * g for g in range(1, n2)]
    gk = rng(cfg.index, 5, extra=40)
    keys_o, keys_g = {}, {}
    for st in steps:
        a = uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,))
        e = gaussian_error(gk, (cfg.dnum, n))
        g = ck.galois_elt(st)
        keys_o[st] = ck.keygen_galois(s, g, a, e)
        keys_g[st] = ctx.keygen_galois(s_dev, g, to_dev(a), to_dev(e))
    say("keys ready", len(steps))
    ctx.profile(True)
    ctx.profile_reset()
    outs = ctx.linear_project(cts_g, to_dev(W), T, n1, keys_g, layout="tm")
    moddowns = ctx.profile_read("moddown")[1]
    ctx.profile(False)
    say("gpu projection done; ModDown launches", moddowns)
    if lazy and n2 > 1:
        # the hoisted baby steps b and b - D (batches of 32 per input), then one ModDown per output tile of 32
        expect = (d_in // D) * -(-(2 * n1 - 1) // 32) + -(-(d_out // D) // 32)
        assert moddowns == expect, (moddowns, expect)
    want = ck.linear_project_tm(cts_o, W, T, n1, keys_o, out_blocks=oracle_outputs, lazy=lazy)
    say("oracle projection done")
    for j, wo in zip(oracle_outputs, want):
        got = to_host(outs[j].data)
        assert got.shape == wo.shape
        bad = np.argwhere(got != wo)
        assert bad.size == 0, "output %d: first mismatches %s" % (j, bad[:5].tolist())
        assert outs[j].scale == delta
        re, im = ctx.decode(ctx.decrypt(s_dev, outs[j]))
        zo = ck.decode(ck.decrypt(s, wo), delta)
        assert np.max(np.abs(to_host(re) - zo.real)) <= 2.0 ** -20
        assert np.max(np.abs(to_host(im) - zo.imag)) <= 2.0 ** -20
    Y = X @ W
    errs = []
    for j, o in enumerate(outs):
        re, _ = ctx.decode(ctx.decrypt(s_dev, o))
        errs.append(np.max(np.abs(to_host(re) - tm_pack(Y, T, D, j))))
    return max(errs)


def test_toy_tm_projection_carried_sums():
    err = run_case(TOY, 2 * TOY.feats, 3 * TOY.feats, 16, [0, 2], max_pairs=5)
    say("toy tm max error vs X@W", err)
    assert err <= 2.0 ** -12


def test_toy_tm_projection_plain_diagonals():
    err = run_case(TOY, TOY.feats, TOY.feats, TOY.feats, [0])
    say("toy tm (n1 = D) max error vs X@W", err)
    assert err <= 2.0 ** -12


def test_toy_tm_projection_uneven_baby_steps():
    # n1 = 24 does not divide D = 128 (the last giant step has 8 baby steps): the vector-ALU multiply-accumulate
    err = run_case(TOY, 2 * TOY.feats, TOY.feats, 24, [0])
    say("toy tm (n1 = 24) max error vs X@W", err)
    assert err <= 2.0 ** -12


def test_small_ring_tm_projection_short_runs():
    cfg = dataclasses.replace(TOY, name="ring10", log_n=10, tokens=4)
    err = run_case(cfg, 256, 384, 16, [0, 2])
    say("N=2^10 tm max error vs X@W", err)
    assert err <= 2.0 ** -12


def test_tm_projection_parameters_full_degree_slice():
    say("full-degree tm slice")
    err = run_case(PROJECTION, 256, 512, 32, [0, 1])
    say("tm slice max error vs X@W", err)
    assert err <= 2.0 ** -18


def test_tm_projection_rejects_bad_shapes_and_missing_keys():
    """Host-side validation fails before any launch; the output buffers keep their contents."""
    require_gpu()
    from paper_2609_12378_amd import Buf, CkksError, Context
    cfg = TOY
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    n, L = ctx.n, cfg.level + 1
    ct = Buf(ctx.zeros(2, L), 2.0 ** 30)
    W = to_dev(np.zeros((128, 128)))
    key = ctx.keygen_galois(to_dev(ternary_secret(rng(1, 3), n)), ctx.galois_elt(1),
                            to_dev(uniform_residues(rng(1, 5), ctx.primes, n, lead=(cfg.dnum,))),
                            to_dev(gaussian_error(rng(1, 5), (cfg.dnum, n))))
    out = Buf(ctx.zeros(2, L - 1), 1.0)
    # 3 tokens do not divide the 2048 slots
    with pytest.raises(CkksError, match="tokens"):
        ctx.linear_project([ct], W, 3, 4, {1: key}, outs=[out], layout="tm")
    # 4 tokens give 512 features per ciphertext, above the periodic encode's limit
    with pytest.raises(CkksError, match="features"):
        ctx.linear_project([ct], to_dev(np.zeros((512, 512))), 4, 4, {1: key}, outs=[out], layout="tm")
    # n1 = 2 needs the steps 1, -128, -127 and the giant steps 2g
    with pytest.raises(CkksError, match="no key"):
        ctx.linear_project([ct], W, 16, 2, {1: key}, outs=[out], layout="tm")
    assert not to_host(out.data).any()
    assert ctx.workspace_bytes(ctx.OP_LINEAR_PROJECT_TM, (L, 16, 128, 128, 2)) > 0
    with pytest.raises(CkksError):
        ctx.workspace_bytes(ctx.OP_LINEAR_PROJECT_TM, (L, 4, 512, 512, 2))


def test_tm_projection_with_exact_workspace():
    require_gpu()
    import torch
    from paper_2609_12378_amd import Context
    cfg = TOY
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    n, T, L, n1 = ctx.n, cfg.tokens, cfg.level + 1, 16
    D = (n // 2) // T
    s = to_dev(ternary_secret(rng(1, 3, extra=41), n))
    X = uniform_slots(rng(1, 1, extra=41), (T, 2 * D))
    W = to_dev(gaussian_weights(rng(1, 2, extra=41), (2 * D, D)))
    ge = rng(1, 4, extra=41)
    cts = [ctx.encrypt(s, ctx.encode(to_dev(tm_pack(X, T, D, i)), None, 2.0 ** 30, L),
                       to_dev(uniform_residues(ge, ctx.q[:L], n)), to_dev(gaussian_error(ge, n))) for i in range(2)]
    gk = rng(1, 5, extra=41)
    keys = {}
    for st in [b for b in range(1, n1)] + [b - D for b in range(n1)] + [n1 * g for g in range(1, D // n1)]:
        keys[st] = ctx.keygen_galois(s, ctx.galois_elt(st), to_dev(uniform_residues(gk, ctx.primes, n, lead=(2,))),
                                     to_dev(gaussian_error(gk, (2, n))))
    want = to_host(ctx.linear_project(cts, W, T, n1, keys, layout="tm")[0].data)
    nbytes = ctx.workspace_bytes(ctx.OP_LINEAR_PROJECT_TM, (L, T, 2 * D, D, n1))
    ctx.set_workspace(torch.empty(nbytes // 8, dtype=torch.uint64, device="cuda"))
    got = to_host(ctx.linear_project(cts, W, T, n1, keys, layout="tm")[0].data)
    ctx.set_workspace(None)
    assert np.array_equal(got, want)


def test_toy_tm_projection_lazy_moddown():
    err = run_case(TOY, 2 * TOY.feats, 3 * TOY.feats, 16, [0, 2], lazy=True)
    say("toy tm lazy-ModDown max error vs X@W", err)
    assert err <= 2.0 ** -12


def test_toy_tm_projection_lowest_level():
    cfg = dataclasses.replace(TOY, level=1)
    err = run_case(cfg, TOY.feats, TOY.feats, 8, [0])
    say("toy tm level-1 max error vs X@W", err)
    assert err <= 2.0 ** -10


def test_tm_projection_benchmark_shape_bit_exact():
    """The token-major benchmark call (n1 = 32): 4096 x 14336 weights, 16 input ciphertexts at level 12 with slot
    t * 256 + f, the lazy ModDown and the default sub-batching, with the benchmark's seeded inputs.  Output
    ciphertexts 0, 27 and 55 are compared in full against the oracle's, stored as SHA-256 digests (with 32
    residues per row) by tests/golden/make_projection_golden.py --layout tm; their decrypted slots must also
    agree with X @ W within 2^-20."""
    require_gpu()
    import hashlib
    import json
    import os
    from paper_2609_12378_amd import Context
    from workloads import projection_inputs
    golden_path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                               "projection_tm_4096x14336_outputs.json")
    with open(golden_path) as f:
        golden = json.load(f)
    cfg = PROJECTION
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q_bits=cfg.q_bits)
    ctx.set_lazy_moddown(True)
    n, T, D, n1, level = ctx.n, cfg.tokens, cfg.feats, cfg.n1, cfg.level
    inp = projection_inputs(cfg, ctx.q, ctx.primes, layout="tm")
    s_dev = to_dev(inp.s)
    delta = float(2 ** cfg.scale_log2)
    cts = []
    for i, (a, e) in enumerate(inp.enc):
        pt = ctx.encode(to_dev(tm_pack(inp.X, T, D, i)), None, delta, level + 1)
        cts.append(ctx.encrypt(s_dev, pt, to_dev(a), to_dev(e)))
    keys = {st: ctx.keygen_galois(s_dev, ctx.galois_elt(st), to_dev(a), to_dev(e)) for st, (a, e) in inp.keys.items()}
    say("token-major benchmark-shape projection: keys ready", len(keys))
    outs = ctx.linear_project(cts, to_dev(inp.W), T, n1, keys, layout="tm")
    assert len(outs) == cfg.d_out // D
    pos = golden["positions"]
    for j in (0, 27, 55):
        rec = golden["outputs"][str(j)]
        assert outs[j].scale == delta and outs[j].n_limbs == level
        got = to_host(outs[j].data)
        assert list(got.shape) == rec["shape"]
        samples = np.array([got[c, r, pos] for c in range(2) for r in range(level)], dtype=np.uint64)
        bad = np.argwhere(samples != np.array(rec["samples"], dtype=np.uint64))
        assert bad.size == 0, "output %d: sampled residues differ at (row, sample) %s" % (j, bad[:5].tolist())
        digest = hashlib.sha256(np.ascontiguousarray(got, dtype="<u8").tobytes()).hexdigest()
        assert digest == rec["sha256"], "output %d: full ciphertext differs from the oracle's" % j
        re, _ = ctx.decode(ctx.decrypt(s_dev, outs[j]))
        want = tm_pack(inp.X @ inp.W[:, j * D:(j + 1) * D], T, D, 0)
        err = float(np.max(np.abs(to_host(re) - want)))
        say("output", j, "bit-exact against the oracle; max error vs X@W", err)
        assert err <= 2.0 ** -20
