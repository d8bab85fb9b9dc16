"""Write the expected outputs of the 4096 x 14336 projection calls of the benchmark: the feature-major one (the
headline) and, with --layout tm, the token-major one.

Calls only the oracle and the seeded generators: the inputs are those of
``workloads.projection_inputs(PROJECTION, ...)`` (the same arrays the GPU test
draws), encrypted and keyed by the oracle, and the outputs are
``Ckks.linear_project(..., lazy=True)`` (``linear_project_tm`` for the token-major
layout; the giant steps summed with one ModDown, as the benchmark runs it)
restricted to the requested output ciphertexts
(Eq. slot-diagonal-matvec with BSGS; Table linear-performance, gate/up row, for
the shape).

For each output j it stores the SHA-256 of the full ciphertext ([2][12][N]
uint64, little-endian, C order), the residues at 32 fixed positions of each of
its 24 rows (to locate a mismatch), and the oracle's decrypted error against
X @ W.  Hours of CPU time per output; outputs can be computed by separate
processes and are merged into the JSON file:

    python tests/golden/make_projection_golden.py --outputs 0
    python tests/golden/make_projection_golden.py --outputs 27
    python tests/golden/make_projection_golden.py --outputs 55
    python tests/golden/make_projection_golden.py --layout tm --outputs 0   (and 27, 55)
"""
import argparse
import fcntl
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
from workloads import PROJECTION, fm_pack, projection_inputs, tm_pack  # noqa: E402

OUT = {"fm": os.path.join(HERE, "projection_4096x14336_outputs.json"),
       "tm": os.path.join(HERE, "projection_tm_4096x14336_outputs.json")}
N_SAMPLES = 32


def sample_positions(n: int):
    """32 fixed positions of a row: both ends and a spread of interior indices."""
    g = np.random.default_rng(20260)
    mid = np.sort(g.choice(np.arange(2, n - 2), N_SAMPLES - 4, replace=False))
    return [0, 1] + [int(x) for x in mid] + [n - 2, n - 1]


def digest(ct: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(ct, dtype="<u8").tobytes()).hexdigest()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--outputs", type=int, nargs="+", default=[0, 27, 55])
    ap.add_argument("--layout", choices=["fm", "tm"], default="fm")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    out_path = args.out or OUT[args.layout]
    pack = fm_pack if args.layout == "fm" else tm_pack
    cfg = PROJECTION
    t0 = time.time()
    pr = gen_primes(cfg.q_bits, 2 * cfg.n, cfg.n_q + cfg.n_p)
    ck = Ckks(cfg.log_n, pr[:cfg.n_q], pr[cfg.n_q:], cfg.dnum)
    inp = projection_inputs(cfg, ck.q, ck.primes, layout=args.layout)
    T, D, level = cfg.tokens, cfg.feats, cfg.level
    delta = float(2 ** cfg.scale_log2)
    cts = []
    for i, (a, e) in enumerate(inp.enc):
        cts.append(ck.encrypt(inp.s, ck.encode(pack(inp.X, T, D, i), None, delta, level + 1), a, e))
    keys = {st: ck.keygen_galois(inp.s, ck.galois_elt(st), a, e) for st, (a, e) in inp.keys.items()}
    print("inputs and %d keys ready after %.0f s" % (len(keys), time.time() - t0), flush=True)
    project = ck.linear_project if args.layout == "fm" else ck.linear_project_tm
    outs = project(cts, inp.W, T, cfg.n1, keys, out_blocks=args.outputs, lazy=True)
    print("outputs %s after %.0f s" % (args.outputs, time.time() - t0), flush=True)
    pos = sample_positions(ck.n)
    Y = inp.X @ inp.W
    rec = {}
    for j, ct in zip(args.outputs, outs):
        assert ct.shape == (2, level, ck.n) and ct.dtype == np.uint64
        z = ck.decode(ck.decrypt(inp.s, ct), delta)
        err = float(np.max(np.abs(z.real - pack(Y, T, D, j))))
        rec[str(j)] = {"sha256": digest(ct), "shape": list(ct.shape),
                       "samples": [[int(x) for x in ct[c, r, pos]] for c in range(2) for r in range(level)],
                       "decrypted_max_err_vs_xw": err}
        print("output %d: sha256 %s, decrypted error %.3g" % (j, rec[str(j)]["sha256"], err), flush=True)
    with open(out_path + ".lock", "w") as lock:
        fcntl.flock(lock, fcntl.LOCK_EX)     # processes computing different outputs merge into one file
        merge(out_path, rec, pos, args.layout)
    os.unlink(out_path + ".lock")


def merge(path, rec, pos, layout):
    data = {}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    data.setdefault("workload", "4096x14336 %s projection, N=2^16, 24+8 50-bit primes, dnum 3, level 12, "
                                "128 tokens x 256 features, n1 = 32, lazy ModDown, seeds of config 4"
                    % ("feature-major" if layout == "fm" else "token-major"))
    data.setdefault("generator", "tests/golden/make_projection_golden.py (oracle only)")
    data["positions"] = pos
    data.setdefault("outputs", {}).update(rec)
    with open(path + ".tmp%d" % os.getpid(), "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
    os.replace(path + ".tmp%d" % os.getpid(), path)


if __name__ == "__main__":
    main()
