"""GPU parity of the batched negacyclic NTT / INTT against the oracle, bit for bit.

Shapes span several thread blocks per row and both kernel passes at N = 2^16
(36 limbs of 50-bit primes, as the NTT microbenchmark), every supported ring
degree from 2^4, a batch whose size is not a multiple of anything the
launcher tiles by, and 60-bit primes (the paper's own modulus sizes).
"""
import numpy as np
import pytest

from gpu_common import require_gpu, say, to_dev, to_host
from oracle import Ckks, gen_primes
from workloads import NTT_BENCH, rng, uniform_residues

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx16():
    require_gpu()
    from paper_2609_12378_amd import Context
    return Context(16, NTT_BENCH.n_q, 0, 1, q_bits=50)


def test_context_primes_match_oracle(ctx16):
    assert ctx16.q == gen_primes(50, 1 << 17, NTT_BENCH.n_q)
    ck = Ckks(16, ctx16.q[:4])
    assert ctx16.psi[:4] == ck.psi


@pytest.mark.parametrize("arith", [0, 1], ids=["fp64", "int"])
@pytest.mark.parametrize("batch,limb0,n_limbs", [(1, 0, 36), (3, 5, 7)])
def test_ntt_n16_parity(ctx16, batch, limb0, n_limbs, arith):
    say("ntt n=2^16 batch", batch, "limbs", limb0, n_limbs, "arith", arith)
    ctx16.set_ntt_arith(arith)
    ck = Ckks(16, ctx16.q)
    primes = ctx16.q[limb0:limb0 + n_limbs]
    a = uniform_residues(rng(2, 1, extra=batch), primes, 1 << 16, lead=(batch,))
    t = to_dev(a)
    ctx16.ntt(t, limb0)
    got = to_host(t)
    idx = list(range(limb0, limb0 + n_limbs))
    want = np.stack([ck.ntt(a[b], idx) for b in range(batch)])
    assert np.array_equal(got, want)
    ctx16.intt(t, limb0)
    assert np.array_equal(to_host(t), a)
    # inverse alone against the oracle's inverse
    t2 = to_dev(a)
    ctx16.intt(t2, limb0)
    want_inv = np.stack([ck.intt(a[b], idx) for b in range(batch)])
    assert np.array_equal(to_host(t2), want_inv)
    ctx16.set_ntt_arith(0)


def test_ntt_benchmark_shape_sampled(ctx16):
    """The NTT benchmark's own launch: 64 polynomials x 36 limbs x 2^16 in one call. Sampled rows bit for bit
    against the oracle's transform; the round trip INTT(NTT(x)) == x on every row."""
    say("ntt benchmark shape 64 x 36 x 2^16")
    ck = Ckks(16, ctx16.q)
    batch = NTT_BENCH.batch
    a = uniform_residues(rng(2, 1, extra=640), ctx16.q, 1 << 16, lead=(batch,))
    t = to_dev(a)
    ctx16.ntt(t)
    got = to_host(t)
    for b, l in ((0, 0), (17, 35), (batch - 1, 18)):
        assert np.array_equal(got[b, l], ck.ntt(a[b, l:l + 1], [l])[0]), (b, l)
    ctx16.intt(t)
    assert np.array_equal(to_host(t), a)


@pytest.mark.parametrize("arith", [0, 1], ids=["fp64", "int"])
@pytest.mark.parametrize("log_n", list(range(4, 16)))
def test_ntt_all_degrees(log_n, arith):
    require_gpu()
    from paper_2609_12378_amd import Context
    say("ntt log_n", log_n, "arith", arith)
    ctx = Context(log_n, 3, 0, 1, q_bits=50)
    ctx.set_ntt_arith(arith)
    ck = Ckks(log_n, ctx.q)
    a = uniform_residues(rng(2, 2, extra=log_n), ctx.q, ctx.n, lead=(5,))
    t = to_dev(a)
    ctx.ntt(t)
    want = np.stack([ck.ntt(a[b], [0, 1, 2]) for b in range(5)])
    assert np.array_equal(to_host(t), want)
    ctx.intt(t)
    assert np.array_equal(to_host(t), a)


def test_ntt_sixty_bit_primes():
    require_gpu()
    from paper_2609_12378_amd import Context
    qs = gen_primes(60, 1 << 17, 2) + gen_primes(61, 1 << 17, 1)
    ctx = Context(16, 3, 0, 1, q=qs)
    ck = Ckks(16, qs)
    a = uniform_residues(rng(2, 3), qs, ctx.n)
    # the largest residues stress the lazy [0, 4q) butterflies
    a[:, :8] = np.array(qs, dtype=np.uint64)[:, None] - 1
    t = to_dev(a)
    ctx.ntt(t)
    assert np.array_equal(to_host(t), ck.ntt(a, [0, 1, 2]))
    ctx.intt(t)
    assert np.array_equal(to_host(t), a)


def test_fp64_extreme_residues():
    # residues 0, 1, q-1 and (q-1)/2 everywhere: the fp64 butterflies' range reductions at their edges
    require_gpu()
    from paper_2609_12378_amd import Context
    ctx = Context(16, 2, 0, 1, q_bits=50)
    ck = Ckks(16, ctx.q)
    for fill in ("zero", "one", "max", "half"):
        a = np.empty((2, ctx.n), dtype=np.uint64)
        for r, q in enumerate(ctx.q):
            a[r] = {"zero": 0, "one": 1, "max": q - 1, "half": (q - 1) // 2}[fill]
        a[:, 1::3] = np.array(ctx.q, dtype=np.uint64)[:, None] - 1
        t = to_dev(a)
        ctx.ntt(t)
        assert np.array_equal(to_host(t), ck.ntt(a, [0, 1])), fill
        ctx.intt(t)
        assert np.array_equal(to_host(t), a), fill


def test_empty_batch_is_a_no_op(ctx16):
    import torch
    t = torch.zeros((0, 36, 1 << 16), dtype=torch.uint64, device="cuda")
    ctx16.ntt(t)
