"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark.

This module holds random-number generation and workload shapes only; it does
none of the scheme's arithmetic.  Every random quantity the scheme draws
(secret, encryption and key randomness, errors) is produced here and passed
explicitly to both the oracle and the GPU library, so the two see identical
inputs.

Seeding convention: ``numpy.random.default_rng(100 * config + role)`` with
roles 1 data, 2 weights, 3 secret, 4 encryption randomness, 5 keys.

The paper evaluates on Meta-Llama-3-8B weights and WikiText-2/C4 text; none of
that is used.  Activations are uniform on [-1, 1] and weights are N(0, 0.02^2),
at the shapes of the paper's projections (Evaluation, Table linear-performance).
"""
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

ROLE_DATA, ROLE_WEIGHTS, ROLE_SECRET, ROLE_ENC, ROLE_KEYS = 1, 2, 3, 4, 5


def rng(config: int, role: int, extra: int = 0) -> np.random.Generator:
    return np.random.default_rng(100 * config + role + 1000 * extra)


def ternary_secret(g: np.random.Generator, n: int) -> np.ndarray:
    """Uniform ternary coefficients, P(-1) = P(0) = P(1) = 1/3, as int8."""
    return g.integers(-1, 2, size=n, dtype=np.int64).astype(np.int8)


def gaussian_error(g: np.random.Generator, shape, sigma: float = 3.2, bound: int = 19) -> np.ndarray:
    """Rounded centred Gaussian with standard deviation sigma, clipped to +-bound, as int32."""
    e = np.rint(g.normal(0.0, sigma, size=shape))
    return np.clip(e, -bound, bound).astype(np.int32)


def uniform_residues(g: np.random.Generator, moduli: Sequence[int], n: int, lead=()) -> np.ndarray:
    """Uniform integers in [0, m) for each modulus m: shape lead + (len(moduli), n), uint64."""
    lead = tuple(lead)
    out = np.empty(lead + (len(moduli), n), dtype=np.uint64)
    for k, m in enumerate(moduli):
        out[..., k, :] = g.integers(0, int(m), size=lead + (n,), dtype=np.uint64)
    return out


def uniform_slots(g: np.random.Generator, shape, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    return g.uniform(lo, hi, size=shape)


def gaussian_weights(g: np.random.Generator, shape, std: float = 0.02) -> np.ndarray:
    return g.normal(0.0, std, size=shape)


@dataclass(frozen=True)
class Config:
    """Shape of one workload: ring, modulus chain, and projection geometry."""
    name: str
    index: int
    log_n: int
    q_bits: int
    n_q: int
    n_p: int
    dnum: int
    scale_log2: int = 40
    level: Optional[int] = None          # ciphertext level (limbs = level + 1); None = top
    tokens: int = 0                       # T, tokens per ciphertext
    d_in: int = 0
    d_out: int = 0
    n1: int = 0                           # baby-step count
    batch: int = 0                        # polynomials per NTT batch / rotations per hoisted batch
    head_dim: int = 0                     # attention: features per head
    heads: int = 0                        # attention: query heads
    kv_heads: int = 0                     # attention: key/value heads (grouped-query attention)
    notes: str = ""

    @property
    def n(self) -> int:
        return 1 << self.log_n

    @property
    def feats(self) -> int:
        return (self.n // 2) // self.tokens if self.tokens else 0


# Toy end-to-end case: N = 2^12, 4 limbs of 36-bit primes, scale 2^30, 16 tokens x 128 features,
# 128 x 128 weights through the plain diagonal method (127 rotations).
TOY = Config("toy", 1, 12, 36, 4, 2, 2, scale_log2=30, level=3, tokens=16, d_in=128, d_out=128, n1=128)
# NTT microbench: N = 2^16, 36 limbs of 50-bit primes, 64 polynomials.
NTT_BENCH = Config("ntt", 2, 16, 50, 36, 0, 1, batch=64)
# Hybrid key switching: N = 2^16, 24 + 8 limbs, dnum 3, 32 hoisted rotations by 1..32.
KEYSWITCH = Config("keyswitch", 3, 16, 50, 24, 8, 3, scale_log2=40, level=23, batch=32)
# Llama-3-8B-shaped projection: 4096 -> 14336 at level 12, 128 tokens x 256 features per ciphertext.
PROJECTION = Config("projection", 4, 16, 50, 24, 8, 3, scale_log2=40, level=12, tokens=128,
                    d_in=4096, d_out=14336, n1=32)
# The other projection shapes of a Llama-3-8B block, same ring and level: QKV (4096 -> 4096 + 2 x 1024),
# attention output (4096 -> 4096) and down (14336 -> 4096; 56 inputs, so n1 = 8, n2 = 32: 392 baby + 496 giant
# rotations).
PROJ_QKV = Config("proj_qkv", 5, 16, 50, 24, 8, 3, scale_log2=40, level=12, tokens=128,
                  d_in=4096, d_out=6144, n1=32)
PROJ_WO = Config("proj_wo", 6, 16, 50, 24, 8, 3, scale_log2=40, level=12, tokens=128,
                 d_in=4096, d_out=4096, n1=32)
PROJ_DOWN = Config("proj_down", 7, 16, 50, 24, 8, 3, scale_log2=40, level=12, tokens=128,
                   d_in=14336, d_out=4096, n1=8)
# Attention block, toy ring: N = 2^12, 6 + 2 limbs of 50-bit primes, scale 2^50 (close to the primes, so a
# ciphertext product rescaled by one prime keeps it), 16 tokens x 128 features = two heads of 64 per
# ciphertext, inputs at level 5.
ATTN_TOY = Config("attn_toy", 8, 12, 50, 6, 2, 3, scale_log2=50, level=5, tokens=16, head_dim=64, heads=4,
                  kv_heads=2)
# One Llama-3-8B attention block's ciphertext work: 128 tokens x 256 features (two heads of 128) per
# ciphertext, 32 query heads (16 ciphertexts) and 8 key/value heads (each repeated in both head positions of
# its own ciphertext: 8 key and 8 value ciphertexts), projections 4096 -> 4096 (Q, O) and 4096 -> 2 x 1024
# (K, V, each head written twice), token-major layout, inputs at level 12, scale 2^50; the projections use n1 = 16
# (with 32 and 16 outputs, half the hoisted baby steps of n1 = 32 save more than the extra giant steps cost).
ATTENTION = Config("attention", 9, 16, 50, 24, 8, 3, scale_log2=50, level=12, tokens=128, d_in=4096,
                   d_out=4096, n1=16, head_dim=128, heads=32, kv_heads=8)


def fm_pack(X: np.ndarray, tokens: int, feats: int, i: int) -> np.ndarray:
    """Slot vector of input ciphertext i in the feature-major layout: slot f*tokens + t holds X[t, i*feats + f]."""
    return X[:, i * feats:(i + 1) * feats].T.reshape(-1)


@dataclass
class ProjectionInputs:
    """Every random quantity one feature-major projection workload draws, in the order the tests and the stored
    expected values draw them: the secret, X, W, per input ciphertext the encryption randomness (a, e), and per
    rotation step the key randomness (a, e) of its Galois key."""
    s: np.ndarray
    X: np.ndarray
    W: np.ndarray
    enc: list                      # [(a [level+1][N] uint64, e [N] int32)] per input ciphertext
    keys: dict                     # step -> (a [dnum][n_q+n_p][N] uint64, e [dnum][N] int32)
    steps: list


def tm_pack(X: np.ndarray, tokens: int, feats: int, i: int) -> np.ndarray:
    """Slot vector of input ciphertext i in the token-major layout: slot t*feats + f holds X[t, i*feats + f]."""
    return X[:, i * feats:(i + 1) * feats].reshape(-1)


def projection_inputs(cfg: Config, q: Sequence[int], primes: Sequence[int], d_in: Optional[int] = None,
                      d_out: Optional[int] = None, layout: str = "fm") -> ProjectionInputs:
    """Seeded inputs of a projection with cfg's ring, level, tokens and n1 (d_in x d_out weights, default cfg's).
    Rotation steps, in drawing order: feature-major ("fm") T*b (0 < b < n1) then T*n1*g (0 < g < n2); token-major
    ("tm") b (0 < b < n1), b - D (0 <= b < n1), then n1*g (0 < g < n2)."""
    d_in = cfg.d_in if d_in is None else d_in
    d_out = cfg.d_out if d_out is None else d_out
    n, T, D, n1, level = cfg.n, cfg.tokens, cfg.feats, cfg.n1, cfg.level
    n2 = -(-D // n1)
    s = ternary_secret(rng(cfg.index, ROLE_SECRET), n)
    X = uniform_slots(rng(cfg.index, ROLE_DATA), (T, d_in))
    W = gaussian_weights(rng(cfg.index, ROLE_WEIGHTS), (d_in, d_out))
    ge = rng(cfg.index, ROLE_ENC)
    enc = []
    for _ in range(d_in // D):
        a = uniform_residues(ge, q[:level + 1], n)
        enc.append((a, gaussian_error(ge, n)))
    if layout == "fm":
        steps = [T * b for b in range(1, n1)] + [T * n1 * g for g in range(1, n2)]
    else:
        steps = [b for b in range(1, n1)] + [b - D for b in range(n1)] + [n1 * g for g in range(1, n2)]
    gk = rng(cfg.index, ROLE_KEYS)
    keys = {}
    for st in steps:
        a = uniform_residues(gk, primes, n, lead=(cfg.dnum,))
        keys[st] = (a, gaussian_error(gk, (cfg.dnum, n)))
    return ProjectionInputs(s, X, W, enc, keys, steps)


@dataclass
class AttentionInputs:
    """Every random quantity of one attention-block parity workload, in the order the tests and the stored
    expected values draw them: the secret; the query blocks Q [T][D], key and value heads K, V [T][hd]; per
    ciphertext (queries, then keys, then values) its encryption randomness (a, e); per rotation step (ascending)
    the Galois-key randomness (a, e); last the relinearisation-key randomness."""
    s: np.ndarray
    Q: list
    K: list
    V: list
    enc: list
    keys: dict
    rlk: tuple


def attention_steps(slots: int, tokens: int, head_dim: int) -> list:
    """Every rotation step of the scores and weighted sums for T tokens and heads of hd (D = slots / T): -delta
    and delta (D - 1), 1 .. hd - 1, delta D (0 < delta < T), and j (-hd < j < T, j != 0)."""
    D = slots // tokens
    st = set(-d for d in range(1, tokens)) | set(d * (D - 1) for d in range(1, tokens)) | set(range(1, head_dim))
    st |= set(d * D for d in range(1, tokens)) | set(j for j in range(-head_dim + 1, tokens) if j)
    return sorted(st)


def attention_inputs(cfg: Config, q: Sequence[int], primes: Sequence[int], n_q: int, n_kv: int,
                     extra: int = 50) -> AttentionInputs:
    n, T, hd, level = cfg.n, cfg.tokens, cfg.head_dim, cfg.level
    D = (n // 2) // T
    s = ternary_secret(rng(cfg.index, ROLE_SECRET, extra=extra), n)
    g = rng(cfg.index, ROLE_DATA, extra=extra)
    Q = [g.uniform(-1, 1, (T, D)) for _ in range(n_q)]
    K = [g.uniform(-1, 1, (T, hd)) for _ in range(n_kv)]
    V = [g.uniform(-1, 1, (T, hd)) for _ in range(n_kv)]
    ge = rng(cfg.index, ROLE_ENC, extra=extra)
    enc = []
    for _ in range(n_q + 2 * n_kv):
        a = uniform_residues(ge, q[:level + 1], n)
        enc.append((a, gaussian_error(ge, n)))
    gk = rng(cfg.index, ROLE_KEYS, extra=extra)
    keys = {}
    for st in attention_steps(n // 2, T, hd):
        a = uniform_residues(gk, primes, n, lead=(cfg.dnum,))
        keys[st] = (a, gaussian_error(gk, (cfg.dnum, n)))
    a = uniform_residues(gk, primes, n, lead=(cfg.dnum,))
    return AttentionInputs(s, Q, K, V, enc, keys, (a, gaussian_error(gk, (cfg.dnum, n))))


# The attention parity case at the benchmark's correlation lengths: N = 2^13, 6 + 2 limbs of 50-bit primes, 16 tokens
# x 256 features = two heads of 128 per ciphertext (scores correlate over 128 positions, the weighted sums over 256),
# inputs at level 5, scale 2^50, one query, key and value ciphertext.
ATTN_HD128 = Config("attn13_hd128", 8, 13, 50, 6, 2, 3, scale_log2=50, level=5, tokens=16, head_dim=128, heads=2,
                    kv_heads=1)


# The paper's own CKKS parameters (Evaluation, "Experimental Setup"): N = 2^16, modulus depth 37 with a 60-bit
# first modulus and 59-bit others, dnum = 5; here with 8 special primes of 60 bits (alpha = 8).  Every prime is at
# least 2^50, so every transform, inner product and conversion takes the integer (64-bit Shoup) path.  The
# hoisted batch at the top level: 32 rotations by 1..32 of a level-36 ciphertext.
KEYSWITCH_PAPER = Config("keyswitch_paper", 10, 16, 59, 37, 8, 5, scale_log2=40, level=36, batch=32,
                         notes="q_0 60-bit, q_1..q_36 59-bit, p 60-bit")


def paper_chain(primes60: Sequence[int], primes59: Sequence[int], n_q: int, n_p: int):
    """(q, p) of the paper's chain from the descending 60- and 59-bit prime lists: q_0 the largest 60-bit prime,
    q_1.. the 59-bit ones, p the next 60-bit primes."""
    return [primes60[0]] + list(primes59[:n_q - 1]), list(primes60[1:1 + n_p])
