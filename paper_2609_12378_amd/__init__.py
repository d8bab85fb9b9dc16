"""Python binding of libckks_mi.so (RNS-CKKS on MI355X).

Argument marshalling only: every computation runs in the library's HIP
kernels.  Device memory comes from torch tensors (``torch.uint64`` residues,
``torch.float64`` slots and weights, ``torch.int8`` secrets, ``torch.int32``
errors); calls are enqueued on the context's HIP stream, which defaults to the
current torch stream at context creation.  The library must be built first
(``python -m paper_2609_12378_amd.build``); importing this package on a machine
without the built library raises instead of falling back to anything else.
"""
import ctypes
import os
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libckks_mi.so")

__all__ = ["Context", "Buf", "CkksError", "load_library", "LIB_PATH"]


class CkksError(RuntimeError):
    pass


class _Params(ctypes.Structure):
    _fields_ = [("log_n", ctypes.c_uint32), ("n_q", ctypes.c_uint32), ("n_p", ctypes.c_uint32),
                ("dnum", ctypes.c_uint32), ("q", ctypes.POINTER(ctypes.c_uint64)),
                ("p", ctypes.POINTER(ctypes.c_uint64)), ("q_bits", ctypes.c_uint32), ("p_bits", ctypes.c_uint32)]


class _Buf(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n_polys", ctypes.c_uint32), ("n_limbs", ctypes.c_uint32),
                ("scale", ctypes.c_double)]


class _ProjShape(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_uint32), ("d_in", ctypes.c_uint32), ("d_out", ctypes.c_uint32),
                ("n1", ctypes.c_uint32)]


class _AttnShape(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_uint32), ("head_dim", ctypes.c_uint32)]


_LIB = None

# name -> (restype, argtypes)
_VP, _U32, _I32, _U64, _DBL, _SZ = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint64, \
    ctypes.c_double, ctypes.c_size_t
_BP = ctypes.POINTER(_Buf)
_SIGS = {
    "ckks_ctx_create": (ctypes.c_int, [ctypes.POINTER(_Params), _VP, ctypes.POINTER(_VP)]),
    "ckks_ctx_destroy": (None, [_VP]),
    "ckks_ctx_set_stream": (ctypes.c_int, [_VP, _VP]),
    "ckks_ctx_set_ntt_arith": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ckks_ctx_set_proj_batch": (ctypes.c_int, [_VP, _U32]),
    "ckks_ctx_set_lazy_moddown": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ckks_ctx_tables": (ctypes.c_int, [_VP, _VP, _VP, _VP]),
    "ckks_workspace_bytes": (ctypes.c_size_t, [_VP, ctypes.c_int, _VP]),
    "ckks_set_workspace": (ctypes.c_int, [_VP, _VP, ctypes.c_size_t]),
    "ckks_galois_elt": (_U32, [_VP, _I32]),
    "ckks_last_error": (ctypes.c_char_p, []),
    "ckks_ntt": (ctypes.c_int, [_VP, _VP, _U32, _U32, _U32]),
    "ckks_intt": (ctypes.c_int, [_VP, _VP, _U32, _U32, _U32]),
    "ckks_encode": (ctypes.c_int, [_VP, _VP, _VP, _DBL, _U32, _BP]),
    "ckks_decode": (ctypes.c_int, [_VP, _BP, _VP, _VP]),
    "ckks_encrypt_sk": (ctypes.c_int, [_VP, _VP, _BP, _VP, _VP, _BP]),
    "ckks_decrypt": (ctypes.c_int, [_VP, _VP, _BP, _BP]),
    "ckks_keygen_galois": (ctypes.c_int, [_VP, _VP, _U32, _VP, _VP, _VP]),
    "ckks_keygen_relin": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP]),
    "ckks_add": (ctypes.c_int, [_VP, _BP, _BP, _BP]),
    "ckks_mul_plain": (ctypes.c_int, [_VP, _BP, _BP, _BP]),
    "ckks_mul_relin": (ctypes.c_int, [_VP, _BP, _BP, _VP, _BP]),
    "ckks_rescale": (ctypes.c_int, [_VP, _BP, _BP]),
    "ckks_rotate": (ctypes.c_int, [_VP, _BP, _I32, _VP, _BP]),
    "ckks_rotate_hoisted": (ctypes.c_int, [_VP, _BP, _VP, _U32, _VP, _BP]),
    "ckks_rotate_noalloc": (ctypes.c_int, [_VP, _BP, _I32, _VP, _BP]),
    "ckks_expand_key_a": (ctypes.c_int, [_VP, _VP, _VP]),
    "ckks_keygen_galois_seeded": (ctypes.c_int, [_VP, _VP, _U32, _VP, _VP, _VP]),
    "ckks_rotate_hoisted_seeded": (ctypes.c_int, [_VP, _BP, _VP, _U32, _VP, _VP, _BP]),
    "ckks_modup": (ctypes.c_int, [_VP, _VP, _U32, _VP]),
    "ckks_moddown": (ctypes.c_int, [_VP, _VP, _U32, _VP]),
    "ckks_automorph": (ctypes.c_int, [_VP, _VP, _U32, _U32, _VP]),
    "ckks_linear_project": (ctypes.c_int, [_VP, _BP, _VP, ctypes.POINTER(_ProjShape), _VP, _VP, _U32, _BP]),
    "ckks_linear_project_tm": (ctypes.c_int, [_VP, _BP, _VP, ctypes.POINTER(_ProjShape), _VP, _VP, _U32, _BP]),
    "ckks_attention_scores": (ctypes.c_int, [_VP, _BP, _U32, _BP, _U32, _VP, ctypes.POINTER(_AttnShape), _VP, _VP,
                                             _VP, _U32, _BP]),
    "ckks_attention_apply": (ctypes.c_int, [_VP, _BP, _U32, _BP, _U32, _VP, ctypes.POINTER(_AttnShape), _VP, _VP,
                                            _VP, _U32, _BP]),
    "ckks_profile_enable": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ckks_profile_read": (ctypes.c_int, [_VP, ctypes.c_char_p, ctypes.POINTER(_DBL), ctypes.POINTER(_U64),
                                         ctypes.POINTER(_DBL), ctypes.POINTER(_DBL)]),
    "ckks_profile_name": (ctypes.c_char_p, [ctypes.c_int]),
    "ckks_profile_reset": (ctypes.c_int, [_VP]),
    "ckks_calib_copy": (ctypes.c_int, [_VP, _VP, _VP, _SZ]),
    "ckks_calib_modmul": (ctypes.c_int, [_VP, _VP, _U32, _U32, ctypes.c_int]),
}
EXPORTED = tuple(_SIGS)


def load_library(path: str = LIB_PATH):
    """Load libckks_mi.so and declare every exported call; raise if it is missing."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(path):
            raise CkksError("libckks_mi.so is not built (%s); run python -m paper_2609_12378_amd.build" % path)
        L = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name, None)
            if fn is None:
                continue
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def missing_symbols(path: str = LIB_PATH) -> List[str]:
    """Declared calls that the built library does not export."""
    L = load_library(path)
    return [n for n in _SIGS if getattr(L, n, None) is None]


def _check(st: int, what: str):
    if st != 0:
        msg = load_library().ckks_last_error().decode(errors="replace")
        raise CkksError("%s failed (status %d): %s" % (what, st, msg))


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise CkksError("expected a torch tensor, got %s" % type(t).__name__)
    if not t.is_cuda:
        raise CkksError("expected a device tensor")
    if not t.is_contiguous():
        raise CkksError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _arg(t, what: str, dtype: torch.dtype, shape=None, numel: Optional[int] = None):
    """Device pointer of t after checking what the kernels will assume of it: dtype, then shape (a tuple, or
    only the element count), then device residency and contiguity.  A wrong host tensor, dtype or size would
    otherwise be read out of bounds by a kernel, which the C ABI cannot detect."""
    if not isinstance(t, torch.Tensor):
        raise CkksError("%s: expected a torch tensor, got %s" % (what, type(t).__name__))
    if t.dtype != dtype:
        raise CkksError("%s: dtype %s, expected %s" % (what, t.dtype, dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise CkksError("%s: shape %s, expected %s" % (what, tuple(t.shape), tuple(shape)))
    if numel is not None and t.numel() != numel:
        raise CkksError("%s: %d elements, expected %d" % (what, t.numel(), numel))
    try:
        return _ptr(t)
    except CkksError as e:
        raise CkksError("%s: %s" % (what, e)) from None


@dataclass
class Buf:
    """A plaintext ([1][limbs][N]) or ciphertext ([2][limbs][N]) tensor with its scale."""
    data: torch.Tensor
    scale: float

    @property
    def n_polys(self) -> int:
        return self.data.shape[0]

    @property
    def n_limbs(self) -> int:
        return self.data.shape[1]

    @property
    def level(self) -> int:
        return self.n_limbs - 1

    def c(self, n: Optional[int] = None) -> _Buf:
        """The C descriptor; with n, the ring degree the rows must have."""
        d = self.data
        if not isinstance(d, torch.Tensor) or d.dtype != torch.uint64 or d.dim() != 3:
            raise CkksError("buffer must be a 3-d uint64 tensor")
        if n is not None and d.shape[2] != n:
            raise CkksError("buffer rows have %d entries, the ring degree is %d" % (d.shape[2], n))
        if not 1 <= d.shape[0] <= 3 or d.shape[1] < 1:
            raise CkksError("buffer shape %s: 1-3 polynomials of at least one limb expected" % (tuple(d.shape),))
        return _Buf(_ptr(d), d.shape[0], d.shape[1], float(self.scale))


class Context:
    """A libckks_mi context on the current HIP device and stream."""

    def __init__(self, log_n: int, n_q: int, n_p: int = 0, dnum: int = 1, q_bits: int = 50, p_bits: int = 0,
                 q: Optional[Sequence[int]] = None, p: Optional[Sequence[int]] = None, stream=None):
        L = load_library()
        self.lib = L
        qa = (ctypes.c_uint64 * n_q)(*q) if q is not None else None
        pa = (ctypes.c_uint64 * n_p)(*p) if p is not None else None
        prm = _Params(log_n, n_q, n_p, dnum, qa, pa, q_bits, p_bits or q_bits)
        if stream is None:
            stream = torch.cuda.current_stream()
        self._stream = stream
        h = ctypes.c_void_p()
        _check(L.ckks_ctx_create(ctypes.byref(prm), ctypes.c_void_p(stream.cuda_stream), ctypes.byref(h)),
               "ckks_ctx_create")
        self.h = h
        self.log_n, self.n = log_n, 1 << log_n
        self.n_q, self.n_p, self.dnum = n_q, n_p, dnum
        self.alpha = -(-n_q // dnum)
        qo = (ctypes.c_uint64 * max(n_q, 1))()
        po = (ctypes.c_uint64 * max(n_p, 1))()
        so = (ctypes.c_uint64 * (n_q + n_p))()
        _check(L.ckks_ctx_tables(h, qo, po, so), "ckks_ctx_tables")
        self.q = list(qo)[:n_q]
        self.p = list(po)[:n_p]
        self.psi = list(so)
        self.primes = self.q + self.p

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and h.value:
            try:
                self.lib.ckks_ctx_destroy(h)
            except Exception:
                pass
            self.h = None

    # ---------------- helpers ----------------
    def set_ntt_arith(self, mode: int):
        """0: fp64 butterflies where every prime is below 2^50 (default); 1: integer Shoup everywhere."""
        _check(self.lib.ckks_ctx_set_ntt_arith(self.h, mode), "ckks_ctx_set_ntt_arith")

    def set_proj_batch(self, max_pairs: int):
        """Cap the (input, baby step) pairs per projection launch (0 = by the library's staging budget)."""
        _check(self.lib.ckks_ctx_set_proj_batch(self.h, max_pairs), "ckks_ctx_set_proj_batch")

    def set_lazy_moddown(self, on: bool):
        """Sum the rotations of the projections' giant steps and of the attention outer sum with one ModDown."""
        _check(self.lib.ckks_ctx_set_lazy_moddown(self.h, int(bool(on))), "ckks_ctx_set_lazy_moddown")

    # workspace op codes (ckks_op)
    OP_ENCODE, OP_DECODE, OP_ENCRYPT, OP_DECRYPT, OP_KEYGEN, OP_RESCALE, OP_ROTATE, OP_MUL_RELIN, OP_MODUP, \
        OP_MODDOWN, OP_LINEAR_PROJECT, OP_LINEAR_PROJECT_TM, OP_ATTN_SCORES, OP_ATTN_APPLY = range(1, 15)

    def workspace_bytes(self, op: int, shape=()) -> int:
        """Device bytes one call of `op` takes from the arena or workspace, for the given shape."""
        arr = (_U32 * max(1, len(shape)))(*shape)
        b = int(self.lib.ckks_workspace_bytes(self.h, op, arr if shape else None))
        if b == (1 << 64) - 1:
            raise CkksError("ckks_workspace_bytes: " + self.lib.ckks_last_error().decode(errors="replace"))
        return b

    def set_workspace(self, buf: Optional[torch.Tensor]):
        """Use buf (a device tensor the caller keeps alive) as the scratch arena; None: library-managed."""
        if buf is None:
            _check(self.lib.ckks_set_workspace(self.h, None, 0), "ckks_set_workspace")
        else:
            _check(self.lib.ckks_set_workspace(self.h, _ptr(buf), buf.numel() * buf.element_size()),
                   "ckks_set_workspace")
        self._workspace = buf

    def galois_elt(self, steps: int) -> int:
        return int(self.lib.ckks_galois_elt(self.h, steps))

    def n_digits(self, level: int) -> int:
        return level // self.alpha + 1

    def zeros(self, n_polys: int, n_limbs: int) -> torch.Tensor:
        return torch.zeros((n_polys, n_limbs, self.n), dtype=torch.uint64, device="cuda")

    # ---------------- transforms ----------------
    def ntt(self, t: torch.Tensor, limb0: int = 0, inverse: bool = False):
        """In-place (inverse) NTT of t viewed as [batch][limbs][N]; limbs use primes limb0.."""
        if t.dim() < 2 or t.shape[-1] != self.n:
            raise CkksError("ntt: rows of %d residues expected, shape %s" % (self.n, tuple(t.shape)))
        nl = t.shape[-2]
        batch = t.numel() // (nl * self.n)
        ptr = _arg(t, "ntt input", torch.uint64)
        fn = self.lib.ckks_intt if inverse else self.lib.ckks_ntt
        _check(fn(self.h, ptr, batch, limb0, nl), "ckks_intt" if inverse else "ckks_ntt")
        return t

    def intt(self, t: torch.Tensor, limb0: int = 0):
        return self.ntt(t, limb0, inverse=True)

    # ---------------- encoding ----------------
    def encode(self, re: torch.Tensor, im: Optional[torch.Tensor], scale: float, n_limbs: int,
               out: Optional[torch.Tensor] = None) -> Buf:
        out = self.zeros(1, n_limbs) if out is None else out
        b = Buf(out, scale)
        cb = b.c(self.n)
        if out.shape[1] != n_limbs or out.shape[0] != 1:
            raise CkksError("encode: output shape %s, expected (1, %d, %d)" % (tuple(out.shape), n_limbs, self.n))
        pr = _arg(re, "encode re", torch.float64, numel=self.n // 2)
        pi = None if im is None else _arg(im, "encode im", torch.float64, numel=self.n // 2)
        _check(self.lib.ckks_encode(self.h, pr, pi, float(scale), n_limbs, ctypes.byref(cb)), "ckks_encode")
        return b

    def decode(self, pt: Buf):
        re = torch.empty(self.n // 2, dtype=torch.float64, device="cuda")
        im = torch.empty(self.n // 2, dtype=torch.float64, device="cuda")
        cb = pt.c(self.n)
        _check(self.lib.ckks_decode(self.h, ctypes.byref(cb), _ptr(re), _ptr(im)), "ckks_decode")
        return re, im

    # ---------------- encryption ----------------
    def encrypt(self, s: torch.Tensor, pt: Buf, a: torch.Tensor, e: torch.Tensor) -> Buf:
        out = Buf(self.zeros(2, pt.n_limbs), pt.scale)
        cp, co = pt.c(self.n), out.c(self.n)
        ps = _arg(s, "secret", torch.int8, numel=self.n)
        pa = _arg(a, "encryption a", torch.uint64, numel=pt.n_limbs * self.n)
        pe = _arg(e, "encryption error", torch.int32, numel=self.n)
        _check(self.lib.ckks_encrypt_sk(self.h, ps, ctypes.byref(cp), pa, pe, ctypes.byref(co)), "ckks_encrypt_sk")
        return out

    def decrypt(self, s: torch.Tensor, ct: Buf) -> Buf:
        out = Buf(self.zeros(1, ct.n_limbs), ct.scale)
        ci, co = ct.c(self.n), out.c(self.n)
        ps = _arg(s, "secret", torch.int8, numel=self.n)
        _check(self.lib.ckks_decrypt(self.h, ps, ctypes.byref(ci), ctypes.byref(co)), "ckks_decrypt")
        return out

    def key_shape(self):
        return (self.dnum, 2, self.n_q + self.n_p, self.n)

    def keygen_galois(self, s, g: int, a, e, out=None) -> torch.Tensor:
        out = torch.empty(self.key_shape(), dtype=torch.uint64, device="cuda") if out is None else out
        ps, pa, pe, pk = self._keygen_args(s, a, e, out)
        _check(self.lib.ckks_keygen_galois(self.h, ps, g, pa, pe, pk), "ckks_keygen_galois")
        return out

    # ---------------- seed-expanded keys ----------------
    def key_b_shape(self):
        return (self.dnum, self.n_q + self.n_p, self.n)

    @staticmethod
    def _seed(seed):
        if len(seed) != 2:
            raise CkksError("a key seed is two 64-bit words")
        return (ctypes.c_uint64 * 2)(*[int(x) & ((1 << 64) - 1) for x in seed])

    def expand_key_a(self, seed, out=None) -> torch.Tensor:
        """The a half [dnum][n_q+n_p][N] a seed stands for."""
        out = torch.empty(self.key_b_shape(), dtype=torch.uint64, device="cuda") if out is None else out
        po = _arg(out, "expanded a", torch.uint64, shape=self.key_b_shape())
        _check(self.lib.ckks_expand_key_a(self.h, self._seed(seed), po), "ckks_expand_key_a")
        return out

    def keygen_galois_seeded(self, s, g: int, seed, e, out=None) -> torch.Tensor:
        """The b half [dnum][n_q+n_p][N] of the Galois key for g whose a half is expand_key_a(seed)."""
        out = torch.empty(self.key_b_shape(), dtype=torch.uint64, device="cuda") if out is None else out
        ps = _arg(s, "secret", torch.int8, numel=self.n)
        pe = _arg(e, "key error", torch.int32, numel=self.dnum * self.n)
        pk = _arg(out, "key b half", torch.uint64, shape=self.key_b_shape())
        _check(self.lib.ckks_keygen_galois_seeded(self.h, ps, g, self._seed(seed), pe, pk), "ckks_keygen_galois_seeded")
        return out

    def rotate_hoisted_seeded(self, ct: Buf, steps: Sequence[int], keys_b: Sequence[torch.Tensor], seeds,
                              outs: Optional[Sequence[Buf]] = None) -> List[Buf]:
        """rotate_hoisted with seeded keys: keys_b[r] the b half, seeds[r] the seed of rotation r's key."""
        cnt = len(steps)
        if len(keys_b) != cnt or len(seeds) != cnt:
            raise CkksError("rotate_hoisted_seeded: %d steps, %d keys, %d seeds" % (cnt, len(keys_b), len(seeds)))
        if outs is not None and len(outs) < cnt:
            raise CkksError("rotate_hoisted_seeded: %d outputs for %d steps" % (len(outs), cnt))
        kp = (ctypes.c_void_p * max(1, cnt))(*[_arg(k, "key b half", torch.uint64, shape=self.key_b_shape()).value
                                               for k in keys_b])
        sd = (ctypes.c_uint64 * max(2, 2 * cnt))(*[int(w) & ((1 << 64) - 1) for sd_ in seeds for w in sd_])
        if any(len(sd_) != 2 for sd_ in seeds):
            raise CkksError("a key seed is two 64-bit words")
        if outs is None:
            outs = [Buf(self.zeros(2, ct.n_limbs), ct.scale) for _ in range(cnt)]
        st = (ctypes.c_int32 * max(1, cnt))(*steps)
        ob = (_Buf * max(1, cnt))(*[o.c(self.n) for o in outs])
        ci = ct.c(self.n)
        _check(self.lib.ckks_rotate_hoisted_seeded(self.h, ctypes.byref(ci), st, cnt, kp, sd, ob),
               "ckks_rotate_hoisted_seeded")
        for o, b in zip(outs, ob):
            o.scale = b.scale
        return list(outs[:cnt])

    def keygen_relin(self, s, a, e, out=None) -> torch.Tensor:
        out = torch.empty(self.key_shape(), dtype=torch.uint64, device="cuda") if out is None else out
        _check(self.lib.ckks_keygen_relin(self.h, *self._keygen_args(s, a, e, out)), "ckks_keygen_relin")
        return out

    def _keygen_args(self, s, a, e, out):
        ext = self.n_q + self.n_p
        return (_arg(s, "secret", torch.int8, numel=self.n),
                _arg(a, "key randomness a", torch.uint64, shape=(self.dnum, ext, self.n)),
                _arg(e, "key error", torch.int32, numel=self.dnum * self.n),
                self._key(out, "key output"))

    def _key(self, k, what: str = "switching key"):
        """Pointer of a switching key after checking it is a [dnum][2][n_q+n_p][N] uint64 device tensor."""
        return _arg(k, what, torch.uint64, shape=self.key_shape())

    # ---------------- ciphertext operations ----------------
    def _binop(self, name, a: Buf, b: Buf, out_scale: float, out_limbs: int) -> Buf:
        out = Buf(self.zeros(2, out_limbs), out_scale)
        ca, cb, co = a.c(self.n), b.c(self.n), out.c(self.n)
        _check(getattr(self.lib, name)(self.h, ctypes.byref(ca), ctypes.byref(cb), ctypes.byref(co)), name)
        return out

    def add(self, a: Buf, b: Buf) -> Buf:
        return self._binop("ckks_add", a, b, a.scale, a.n_limbs)

    def mul_plain(self, ct: Buf, pt: Buf) -> Buf:
        return self._binop("ckks_mul_plain", ct, pt, ct.scale * pt.scale, ct.n_limbs)

    def mul_relin(self, a: Buf, b: Buf, rlk: torch.Tensor) -> Buf:
        out = Buf(self.zeros(2, a.n_limbs), a.scale * b.scale)
        ca, cb, co = a.c(self.n), b.c(self.n), out.c(self.n)
        _check(self.lib.ckks_mul_relin(self.h, ctypes.byref(ca), ctypes.byref(cb), self._key(rlk, "relinearisation key"),
                                       ctypes.byref(co)), "ckks_mul_relin")
        return out

    def rescale(self, ct: Buf) -> Buf:
        out = Buf(self.zeros(2, ct.n_limbs - 1), ct.scale / self.q[ct.level])
        ci, co = ct.c(self.n), out.c(self.n)
        _check(self.lib.ckks_rescale(self.h, ctypes.byref(ci), ctypes.byref(co)), "ckks_rescale")
        return out

    def rotate(self, ct: Buf, steps: int, key: torch.Tensor) -> Buf:
        out = Buf(self.zeros(2, ct.n_limbs), ct.scale)
        ci, co = ct.c(self.n), out.c(self.n)
        _check(self.lib.ckks_rotate(self.h, ctypes.byref(ci), steps, self._key(key), ctypes.byref(co)), "ckks_rotate")
        return out

    def rotate_noalloc(self, ct: Buf, steps: int, key: torch.Tensor, out: Buf) -> Buf:
        """ckks_rotate without any device allocation by the library (static scratch); out is the caller's."""
        ci, co = ct.c(self.n), out.c(self.n)
        _check(self.lib.ckks_rotate_noalloc(self.h, ctypes.byref(ci), steps, self._key(key), ctypes.byref(co)),
               "ckks_rotate_noalloc")
        out.scale = co.scale
        return out

    def rotate_hoisted(self, ct: Buf, steps: Sequence[int], keys: Sequence[torch.Tensor],
                       outs: Optional[Sequence[Buf]] = None) -> List[Buf]:
        cnt = len(steps)
        if len(keys) != cnt:
            raise CkksError("rotate_hoisted: %d steps but %d keys" % (cnt, len(keys)))
        if outs is not None and len(outs) < cnt:
            raise CkksError("rotate_hoisted: %d outputs for %d steps" % (len(outs), cnt))
        if outs is None:
            outs = [Buf(self.zeros(2, ct.n_limbs), ct.scale) for _ in range(cnt)]
        st = (ctypes.c_int32 * cnt)(*steps)
        kp = (ctypes.c_void_p * cnt)(*[self._key(k).value for k in keys])
        ob = (_Buf * cnt)(*[o.c(self.n) for o in outs])
        ci = ct.c(self.n)
        _check(self.lib.ckks_rotate_hoisted(self.h, ctypes.byref(ci), st, cnt, kp, ob), "ckks_rotate_hoisted")
        return list(outs)

    def modup(self, c: torch.Tensor, level: int) -> torch.Tensor:
        pc = _arg(c, "modup input", torch.uint64, numel=(level + 1) * self.n)
        out = torch.empty((self.n_digits(level), level + 1 + self.n_p, self.n), dtype=torch.uint64, device="cuda")
        _check(self.lib.ckks_modup(self.h, pc, level, _ptr(out)), "ckks_modup")
        return out

    def moddown(self, x: torch.Tensor, level: int) -> torch.Tensor:
        px = _arg(x, "moddown input", torch.uint64, numel=(level + 1 + self.n_p) * self.n)
        out = torch.empty((level + 1, self.n), dtype=torch.uint64, device="cuda")
        _check(self.lib.ckks_moddown(self.h, px, level, _ptr(out)), "ckks_moddown")
        return out

    def automorph(self, x: torch.Tensor, g: int) -> torch.Tensor:
        if x.numel() % self.n:
            raise CkksError("automorph: %d residues is not a whole number of rows of %d" % (x.numel(), self.n))
        px = _arg(x, "automorph input", torch.uint64)
        out = torch.empty_like(x)
        rows = x.numel() // self.n
        _check(self.lib.ckks_automorph(self.h, px, rows, g, _ptr(out)), "ckks_automorph")
        return out

    def linear_project(self, cts: Sequence[Buf], W: torch.Tensor, tokens: int, n1: int,
                       keys: Dict[int, torch.Tensor], outs: Optional[Sequence[Buf]] = None,
                       layout: str = "fm") -> List[Buf]:
        """Y = X W on packed ciphertexts; layout "fm" (slot f*tokens + t) or "tm" (slot t*D + f)."""
        if not isinstance(W, torch.Tensor) or W.dim() != 2:
            raise CkksError("linear_project: W must be a 2-d (d_in, d_out) tensor")
        d_in, d_out = W.shape
        pw = _arg(W, "weights W", torch.float64)
        D = (self.n // 2) // tokens
        n_out = d_out // D
        level = cts[0].level
        if outs is None:
            outs = [Buf(self.zeros(2, level), cts[0].scale) for _ in range(n_out)]
        # the library reads d_in/D input and d_out/D output descriptors: never hand it shorter arrays
        if D > 0 and d_in % D == 0 and d_out % D == 0 and (len(cts) < d_in // D or len(outs) < n_out):
            raise ValueError("linear_project: %d inputs and %d outputs given, the shape needs %d and %d"
                             % (len(cts), len(outs), d_in // D, n_out))
        inb = (_Buf * len(cts))(*[c.c(self.n) for c in cts])
        ob = (_Buf * max(1, len(outs)))(*[o.c(self.n) for o in outs])
        steps = sorted(keys)
        ks = (ctypes.c_int32 * len(steps))(*steps)
        kp = (ctypes.c_void_p * len(steps))(*[self._key(keys[s], "key for step %d" % s).value for s in steps])
        shape = _ProjShape(tokens, d_in, d_out, n1)
        if layout not in ("fm", "tm"):
            raise ValueError("layout must be 'fm' or 'tm'")
        fn = "ckks_linear_project" if layout == "fm" else "ckks_linear_project_tm"
        _check(getattr(self.lib, fn)(self.h, inb, pw, ctypes.byref(shape), ks, kp, len(steps), ob), fn)
        for o, b in zip(outs, ob):
            o.scale = b.scale
        return list(outs)

    def _attention(self, fn: str, a_cts: Sequence[Buf], b_cts: Sequence[Buf], b_of_a: Sequence[int], tokens: int,
                   head_dim: int, rlk: torch.Tensor, keys: Dict[int, torch.Tensor], outs: Optional[Sequence[Buf]]):
        if len(b_of_a) != len(a_cts):
            raise ValueError("%s: %d ciphertexts but %d indices" % (fn, len(a_cts), len(b_of_a)))
        if outs is None:
            outs = [Buf(self.zeros(2, a_cts[0].n_limbs - (2 if fn == "ckks_attention_scores" else 1)), 0.0)
                    for _ in a_cts]
        if len(outs) < len(a_cts):
            raise ValueError("%s: %d outputs for %d inputs" % (fn, len(outs), len(a_cts)))
        ab = (_Buf * len(a_cts))(*[c.c(self.n) for c in a_cts])
        bb = (_Buf * len(b_cts))(*[c.c(self.n) for c in b_cts])
        ob = (_Buf * len(a_cts))(*[o.c(self.n) for o in outs[:len(a_cts)]])
        idx = (_U32 * len(a_cts))(*b_of_a)
        steps = sorted(keys)
        ks = (ctypes.c_int32 * max(1, len(steps)))(*steps)
        kp = (ctypes.c_void_p * max(1, len(steps)))(*[self._key(keys[s], "key for step %d" % s).value
                                                       for s in steps])
        shape = _AttnShape(tokens, head_dim)
        prlk = self._key(rlk, "relinearisation key")
        _check(getattr(self.lib, fn)(self.h, ab, len(a_cts), bb, len(b_cts), idx, ctypes.byref(shape), prlk, ks,
                                     kp, len(steps), ob), fn)
        for o, b in zip(outs, ob):
            o.scale = b.scale
        return list(outs[:len(a_cts)])

    def attention_scores(self, q_cts: Sequence[Buf], k_cts: Sequence[Buf], k_of_q: Sequence[int], tokens: int,
                         head_dim: int, rlk: torch.Tensor, keys: Dict[int, torch.Tensor],
                         outs: Optional[Sequence[Buf]] = None) -> List[Buf]:
        """Scores on token diagonals: out[c] slot t*D + h*hd + delta = sum_d Q_c[t, h, d] K[(t + delta) mod T, d]."""
        return self._attention("ckks_attention_scores", q_cts, k_cts, k_of_q, tokens, head_dim, rlk, keys, outs)

    def attention_apply(self, p_cts: Sequence[Buf], v_cts: Sequence[Buf], v_of_p: Sequence[int], tokens: int,
                        head_dim: int, rlk: torch.Tensor, keys: Dict[int, torch.Tensor],
                        outs: Optional[Sequence[Buf]] = None) -> List[Buf]:
        """Weighted sums: out[c] slot t*D + h*hd + d = sum_delta P_c[t, h, delta] V[(t + delta) mod T, d]."""
        return self._attention("ckks_attention_apply", p_cts, v_cts, v_of_p, tokens, head_dim, rlk, keys, outs)

    @staticmethod
    def attention_steps(slots: int, tokens: int, head_dim: int) -> List[int]:
        """Every rotation step the two attention calls need for this shape."""
        D = slots // tokens
        st = set(-d for d in range(1, tokens)) | set(d * (D - 1) for d in range(1, tokens)) | set(range(1, head_dim))
        st |= set(d * D for d in range(1, tokens)) | set(j for j in range(-head_dim + 1, tokens) if j)
        return sorted(st)

    # ---------------- measurement ----------------
    def profile(self, on: bool = True):
        _check(self.lib.ckks_profile_enable(self.h, int(on)), "ckks_profile_enable")

    def profile_reset(self):
        _check(self.lib.ckks_profile_reset(self.h), "ckks_profile_reset")

    def profile_read(self, kernel: str):
        """(total ms, launches, algorithmic bytes, nominal VALU instructions) of one kernel since the last reset."""
        ms, cnt, by, ops = ctypes.c_double(), ctypes.c_uint64(), ctypes.c_double(), ctypes.c_double()
        _check(self.lib.ckks_profile_read(self.h, kernel.encode(), ctypes.byref(ms), ctypes.byref(cnt),
                                          ctypes.byref(by), ctypes.byref(ops)), "ckks_profile_read")
        return ms.value, cnt.value, by.value, ops.value

    def profile_all(self):
        """{kernel: (total ms, launches, algorithmic bytes, VALU instructions)} for every kernel that ran."""
        out, i = {}, 0
        while True:
            name = self.lib.ckks_profile_name(i)
            if name is None:
                return out
            r = self.profile_read(name.decode())
            if r[1]:
                out[name.decode()] = r
            i += 1

    def calib_copy(self, dst: torch.Tensor, src: torch.Tensor):
        ps = _arg(src, "calib_copy src", torch.uint64)
        pd = _arg(dst, "calib_copy dst", torch.uint64, numel=src.numel())
        _check(self.lib.ckks_calib_copy(self.h, pd, ps, src.numel() * 8), "ckks_calib_copy")

    def calib_modmul(self, out: torch.Tensor, iters: int, mode: int):
        po = _arg(out, "calib_modmul out", torch.uint64)
        _check(self.lib.ckks_calib_modmul(self.h, po, out.numel(), iters, mode), "ckks_calib_modmul")
