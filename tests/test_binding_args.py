"""The binding checks every tensor it hands to the library before any call.

The C ABI takes raw device pointers and sizes, so a host tensor, a wrong dtype or a short buffer would be read out
of bounds by a kernel.  These checks run on the CPU: a context object whose library handle fails the test if it is
ever reached stands in for a real one, so each case must be rejected by the binding itself with CkksError.
"""
import ctypes

import pytest
import torch

import paper_2609_12378_amd as pkg
from paper_2609_12378_amd import Buf, CkksError, Context


class _NoLibrary:
    def __getattr__(self, name):
        def call(*args):
            raise AssertionError("the library was called (%s) with arguments the binding should have rejected" % name)
        return call


def _host_ptr(t):
    """The binding's pointer step without its device check, so host tensors reach every other check."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise CkksError("expected a torch tensor, got %s" % type(t).__name__)
    return ctypes.c_void_p(t.data_ptr())


def test_host_tensors_rejected():
    with pytest.raises(CkksError, match="device tensor"):
        pkg._ptr(torch.zeros(4, dtype=torch.uint64))
    with pytest.raises(CkksError, match="secret: expected a device tensor"):
        pkg._arg(torch.zeros(4, dtype=torch.int8), "secret", torch.int8, numel=4)
    with pytest.raises(CkksError, match="device tensor"):
        Buf(torch.zeros((2, 1, 16), dtype=torch.uint64), 1.0).c(16)


@pytest.fixture
def ctx(monkeypatch):
    monkeypatch.setattr(pkg, "_ptr", _host_ptr)
    c = Context.__new__(Context)
    c.lib, c.h = _NoLibrary(), None
    c.log_n, c.n = 4, 16
    c.n_q, c.n_p, c.dnum = 3, 1, 2
    c.alpha = 2
    c.q = [97, 193, 257]
    c.p = [353]
    c.primes = c.q + c.p
    c.zeros = lambda n_polys, n_limbs: torch.zeros((n_polys, n_limbs, c.n), dtype=torch.uint64)
    return c


def ct(c, limbs=2, n=None, dtype=torch.uint64):
    return Buf(torch.zeros((2, limbs, n or c.n), dtype=dtype), 2.0 ** 20)


def key(c, dtype=torch.uint64, shape=None):
    return torch.zeros(shape or c.key_shape(), dtype=dtype)


def test_switching_key_checked(ctx):
    with pytest.raises(CkksError, match="dtype"):
        ctx.rotate(ct(ctx), 1, key(ctx, dtype=torch.int64))
    with pytest.raises(CkksError, match="shape"):
        ctx.rotate(ct(ctx), 1, key(ctx, shape=(2, 2, 3, 16)))
    with pytest.raises(AssertionError, match="library was called"):
        ctx.rotate(ct(ctx), 1, key(ctx))       # well-formed arguments reach the library
    with pytest.raises(CkksError, match="relinearisation key: dtype"):
        ctx.mul_relin(ct(ctx), ct(ctx), key(ctx, dtype=torch.float64))
    with pytest.raises(CkksError, match="3 steps but 2 keys"):
        ctx.rotate_hoisted(ct(ctx), [1, 2, 3], [key(ctx), key(ctx)])
    with pytest.raises(CkksError, match="shape"):
        ctx.rotate_hoisted(ct(ctx), [1, 2], [key(ctx), key(ctx, shape=(2, 2, 4, 8))])


def test_buffers_checked(ctx):
    with pytest.raises(CkksError, match="ring degree"):
        ctx.rescale(ct(ctx, n=32))
    with pytest.raises(CkksError, match="uint64"):
        ctx.add(ct(ctx, dtype=torch.int64), ct(ctx))
    with pytest.raises(CkksError, match="shape"):
        ctx.add(Buf(torch.zeros((4, 2, 16), dtype=torch.uint64), 1.0), ct(ctx))
    with pytest.raises(AssertionError, match="library was called"):
        ctx.add(ct(ctx), ct(ctx))


def test_weights_checked(ctx):
    cts = [ct(ctx), ct(ctx)]
    with pytest.raises(CkksError, match="weights W: dtype"):
        ctx.linear_project(cts, torch.zeros((8, 8), dtype=torch.float32), 2, 2, {})
    with pytest.raises(CkksError, match="2-d"):
        ctx.linear_project(cts, torch.zeros(64, dtype=torch.float64), 2, 2, {})
    with pytest.raises(CkksError, match="key for step 2: dtype"):
        ctx.linear_project(cts, torch.zeros((8, 8), dtype=torch.float64), 2, 2, {2: key(ctx, dtype=torch.int64)})


def test_encode_and_encryption_inputs_checked(ctx):
    with pytest.raises(CkksError, match="encode re: dtype"):
        ctx.encode(torch.zeros(8, dtype=torch.float32), None, 2.0 ** 20, 2)
    with pytest.raises(CkksError, match="encode re: 16 elements, expected 8"):
        ctx.encode(torch.zeros(16, dtype=torch.float64), None, 2.0 ** 20, 2)
    with pytest.raises(CkksError, match="encode im: dtype"):
        ctx.encode(torch.zeros(8, dtype=torch.float64), torch.zeros(8, dtype=torch.int64), 2.0 ** 20, 2)
    pt = Buf(torch.zeros((1, 2, 16), dtype=torch.uint64), 2.0 ** 20)
    a = torch.zeros((2, 16), dtype=torch.uint64)
    e = torch.zeros(16, dtype=torch.int32)
    with pytest.raises(CkksError, match="secret: dtype"):
        ctx.encrypt(torch.zeros(16, dtype=torch.int32), pt, a, e)
    with pytest.raises(CkksError, match="encryption a: 16 elements, expected 32"):
        ctx.encrypt(torch.zeros(16, dtype=torch.int8), pt, a[:1], e)
    with pytest.raises(CkksError, match="encryption error: dtype"):
        ctx.encrypt(torch.zeros(16, dtype=torch.int8), pt, a, e.to(torch.int64))
    with pytest.raises(CkksError, match="secret: 8 elements"):
        ctx.decrypt(torch.zeros(8, dtype=torch.int8), ct(ctx))


def test_keygen_inputs_checked(ctx):
    s = torch.zeros(16, dtype=torch.int8)
    a = torch.zeros((2, 4, 16), dtype=torch.uint64)
    e = torch.zeros((2, 16), dtype=torch.int32)
    with pytest.raises(CkksError, match="key randomness a: shape"):
        ctx.keygen_galois(s, 5, a[:, :3], e, out=key(ctx))
    with pytest.raises(CkksError, match="key error: 16 elements"):
        ctx.keygen_relin(s, a, e[0], out=key(ctx))
    with pytest.raises(CkksError, match="key output: shape"):
        ctx.keygen_relin(s, a, e, out=key(ctx, shape=(2, 2, 4, 8)))


def test_stage_inputs_checked(ctx):
    with pytest.raises(CkksError, match="modup input: 16 elements, expected 32"):
        ctx.modup(torch.zeros(16, dtype=torch.uint64), 1)
    with pytest.raises(CkksError, match="moddown input: dtype"):
        ctx.moddown(torch.zeros((3, 16), dtype=torch.int64), 1)
    with pytest.raises(CkksError, match="whole number of rows"):
        ctx.automorph(torch.zeros(24, dtype=torch.uint64), 5)
    with pytest.raises(CkksError, match="rows of 16 residues"):
        ctx.ntt(torch.zeros((2, 8), dtype=torch.uint64))
    with pytest.raises(CkksError, match="ntt input: dtype"):
        ctx.ntt(torch.zeros((2, 16), dtype=torch.int64))


def test_probe_buffers_checked(ctx):
    src = torch.zeros(64, dtype=torch.uint64)
    with pytest.raises(CkksError, match="calib_copy dst: 32 elements, expected 64"):
        ctx.calib_copy(torch.zeros(32, dtype=torch.uint64), src)
    with pytest.raises(CkksError, match="calib_copy src: dtype"):
        ctx.calib_copy(torch.zeros(64, dtype=torch.uint64), torch.zeros(64, dtype=torch.int64))
    with pytest.raises(CkksError, match="calib_modmul out: dtype"):
        ctx.calib_modmul(torch.zeros(64, dtype=torch.float64), 4, 1)


def test_every_library_call_is_declared():
    assert "ckks_rotate" in pkg.EXPORTED and "ckks_linear_project" in pkg.EXPORTED
