"""The C ABI without a GPU: the library builds for gfx950, loads, and exports every call
that include/ckks_mi.h declares; the Python binding declares the same set."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ckks_mi.h")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ckks_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib_path():
    from paper_2609_12378_amd import LIB_PATH, build
    if not os.path.exists(LIB_PATH):
        build.build()
    return LIB_PATH


def test_header_declares_the_api():
    names = declared()
    for must in ("ckks_ntt", "ckks_intt", "ckks_encode", "ckks_encrypt_sk", "ckks_decrypt", "ckks_add",
                 "ckks_mul_plain", "ckks_mul_relin", "ckks_rescale", "ckks_rotate", "ckks_rotate_hoisted",
                 "ckks_linear_project", "ckks_keygen_galois", "ckks_modup", "ckks_moddown"):
        assert must in names


def test_library_exports_every_declared_call(lib_path):
    lib = ctypes.CDLL(lib_path)
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_matches_header(lib_path):
    import paper_2609_12378_amd as m
    assert sorted(m.EXPORTED) == declared()
    assert m.missing_symbols() == []


def test_error_text_without_gpu(lib_path):
    lib = ctypes.CDLL(lib_path)
    lib.ckks_last_error.restype = ctypes.c_char_p
    lib.ckks_ntt.restype = ctypes.c_int
    lib.ckks_ntt.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32]
    # a null context is rejected on the host before anything touches a device
    assert lib.ckks_ntt(None, None, 1, 0, 1) == -1
    assert b"context" in lib.ckks_last_error()
