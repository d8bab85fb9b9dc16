"""Write the expected outputs of the attention parity case with heads of 128 (N = 2^13, 16 tokens).

Calls only the oracle and the seeded generators: inputs from
``workloads.attention_inputs(ATTN_HD128, ..., n_q=1, n_kv=1)`` (the arrays the GPU
test draws), encrypted and keyed by the oracle; outputs are
``Ckks.attention_scores`` and ``Ckks.attention_apply`` (Section "C--Delta Attention
Layout and Computation" and Table ccmm-performance for what they stand for; the
construction is the scores on cyclic token diagonals and the weighted sums that
consume them), eager and with the lazy ModDown of the scores' outer sum.

For each mode and output it stores the SHA-256 of the full ciphertext (uint64,
little-endian, C order), the residues at 32 fixed positions of each row, the
scale, and the oracle's decrypted error against the plain definitions.  About ten
minutes of CPU time:

    python tests/golden/make_attention_golden.py
"""
import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import Ckks, gen_primes  # noqa: E402
from workloads import ATTN_HD128, attention_inputs  # noqa: E402

OUT = os.path.join(HERE, "attention_n13_hd128_outputs.json")


def sample_positions(n: int, k: int = 32):
    g = np.random.default_rng(20261)
    mid = np.sort(g.choice(np.arange(2, n - 2), k - 4, replace=False))
    return [0, 1] + [int(x) for x in mid] + [n - 2, n - 1]


def scores_def(Q, K, T, D, hd):
    """S[t, h*hd + delta] = sum_d Q[t, h*hd + d] K[(t + delta) mod T, d] for delta < T, zero elsewhere."""
    out = np.zeros((T, D))
    for h in range(D // hd):
        for delta in range(T):
            out[:, h * hd + delta] = np.sum(Q[:, h * hd:(h + 1) * hd] * np.roll(K, -delta, axis=0), axis=1)
    return out


def apply_def(P, V, T, D, hd):
    """O[t, h*hd + d] = sum_{delta < T} P[t, h*hd + delta] V[(t + delta) mod T, d]."""
    out = np.zeros((T, D))
    for h in range(D // hd):
        for delta in range(T):
            out[:, h * hd:(h + 1) * hd] += P[:, h * hd + delta:h * hd + delta + 1] * np.roll(V, -delta, axis=0)
    return out


def record(ck, s, ct, scale, want, pos):
    z = ck.decode(ck.decrypt(s, ct), scale).real.reshape(want.shape)
    return {"sha256": hashlib.sha256(np.ascontiguousarray(ct, dtype="<u8").tobytes()).hexdigest(),
            "shape": list(ct.shape), "scale": scale,
            "samples": [[int(x) for x in ct[c, r, pos]] for c in range(ct.shape[0]) for r in range(ct.shape[1])],
            "decrypted_max_err": float(np.max(np.abs(z - want)))}


def main():
    cfg = ATTN_HD128
    t0 = time.time()
    pr = gen_primes(cfg.q_bits, 2 * cfg.n, cfg.n_q + cfg.n_p)
    ck = Ckks(cfg.log_n, pr[:cfg.n_q], pr[cfg.n_q:], cfg.dnum)
    inp = attention_inputs(cfg, ck.q, ck.primes, 1, 1)
    n, T, hd, level = ck.n, cfg.tokens, cfg.head_dim, cfg.level
    D = (n // 2) // T
    delta = float(2 ** cfg.scale_log2)
    plain = [inp.Q[0], np.tile(inp.K[0], (1, D // hd)), np.tile(inp.V[0], (1, D // hd))]
    q, k, v = [ck.encrypt(inp.s, ck.encode(x.reshape(-1), None, delta, level + 1), a, e)
               for x, (a, e) in zip(plain, inp.enc)]
    keys = {st: ck.keygen_galois(inp.s, ck.galois_elt(st), a, e) for st, (a, e) in inp.keys.items()}
    rlk = ck.keygen_relin(inp.s, *inp.rlk)
    print("inputs and %d keys after %.0f s" % (len(keys), time.time() - t0), flush=True)
    s_scale = delta * delta / ck.q[level - 1]
    o_scale = s_scale * delta / ck.q[level - 2]
    Sd = scores_def(inp.Q[0], inp.K[0], T, D, hd)
    Od = apply_def(Sd, inp.V[0], T, D, hd)
    pos = sample_positions(n)
    data = {"workload": "attention scores and weighted sums, N=2^13, 6+2 50-bit primes, dnum 3, 16 tokens, "
                        "two heads of 128, level 5, scale 2^50, seeds of config 8 (extra 50)",
            "generator": "tests/golden/make_attention_golden.py (oracle only)", "positions": pos, "modes": {}}
    for lazy in (False, True):
        S = ck.attention_scores([q], [k], [0], T, hd, rlk, keys, lazy=lazy)
        O = ck.attention_apply(S, [v], [0], T, hd, rlk, keys)
        mode = "lazy" if lazy else "eager"
        data["modes"][mode] = {"scores": record(ck, inp.s, S[0], s_scale, Sd, pos),
                               "sums": record(ck, inp.s, O[0], o_scale, Od, pos)}
        print("%s after %.0f s: scores %s (err %.3g), sums %s (err %.3g)"
              % (mode, time.time() - t0, data["modes"][mode]["scores"]["sha256"][:16],
                 data["modes"][mode]["scores"]["decrypted_max_err"], data["modes"][mode]["sums"]["sha256"][:16],
                 data["modes"][mode]["sums"]["decrypted_max_err"]), flush=True)
    with open(OUT + ".tmp", "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
    os.replace(OUT + ".tmp", OUT)


if __name__ == "__main__":
    main()
