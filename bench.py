#!/usr/bin/env python3
"""Benchmark of the RNS-CKKS projection path on one MI355X.

One step is one full Llama-3-8B-shaped ciphertext x plaintext projection
(4096 -> 14336, 128 tokens x 256 features per ciphertext, N = 2^16, level 12,
24 + 8 limbs of 50-bit primes, dnum 3, BSGS n1 = 32 / n2 = 8): 16 hoisted
ModUps and 496 baby-step rotations, 229,376 weight plaintexts encoded on the
fly from W (FFT, rounding, RNS, NTT) and multiply-accumulated, 392 giant-step
rotations and 56 rescales.  Inputs (W, ciphertexts, keys) are resident in HBM
before the timed region.  The same JSON line also carries the hoisted
key-switching rate (32 rotations of a level-23 ciphertext) and the batched NTT
microbenchmark (64 polynomials x 36 limbs).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
Prints exactly one JSON line on stdout; progress goes to stderr.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "rotations/s at N=2^16 (keyswitch) and s per 4096x14336 ct-pt projection"
# sums of rotations (giant steps, the attention outer sum) with one ModDown per output (--lazy-moddown)
LAZY = {"on": False}
PROJ_BATCH = {"pairs": 0}   # --proj-batch: pairs per multiply-accumulate launch (0: library default)


def make_context(cfg, n_p=None, dnum=None):
    from paper_2609_12378_amd import Context
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p if n_p is None else n_p, cfg.dnum if dnum is None else dnum,
                  q_bits=cfg.q_bits)
    ctx.set_lazy_moddown(LAZY["on"])
    if PROJ_BATCH["pairs"]:
        ctx.set_proj_batch(PROJ_BATCH["pairs"])
    return ctx
HBM_PEAK_GBS = 8000.0
# 256 CUs x 64 lanes x 2.4 GHz of VALU issue (fp64 FMA and 32-bit integer ops are full rate)
LANE_OPS = 256 * 64 * 2.4e9


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def fm_pack(X, T, D, i):
    return X[:, i * D:(i + 1) * D].T.reshape(-1)


class Timer:
    def __init__(self, torch):
        self.torch = torch

    def __enter__(self):
        self.torch.cuda.synchronize()
        self.a = self.torch.cuda.Event(enable_timing=True)
        self.b = self.torch.cuda.Event(enable_timing=True)
        self.a.record()
        return self

    def __exit__(self, *exc):
        self.b.record()
        self.torch.cuda.synchronize()
        self.ms = self.a.elapsed_time(self.b)


def setup_projection(torch, np, cfg, ctx=None):
    from workloads import (gaussian_error, gaussian_weights, rng, ternary_secret, uniform_residues,
                           uniform_slots)
    ctx = make_context(cfg) if ctx is None else ctx
    n, T, D, level, n1 = ctx.n, cfg.tokens, cfg.feats, cfg.level, cfg.n1
    n2 = -(-D // n1)
    s = torch.from_numpy(ternary_secret(rng(cfg.index, 3), n)).cuda()
    X = uniform_slots(rng(cfg.index, 1), (T, cfg.d_in))
    W = gaussian_weights(rng(cfg.index, 2), (cfg.d_in, cfg.d_out))
    Wd = torch.from_numpy(W).cuda()
    delta = float(2 ** cfg.scale_log2)
    ge = rng(cfg.index, 4)
    cts = []
    for i in range(cfg.d_in // D):
        pt = ctx.encode(torch.from_numpy(fm_pack(X, T, D, i)).cuda(), None, delta, level + 1)
        a = torch.from_numpy(uniform_residues(ge, ctx.q[:level + 1], n)).cuda()
        e = torch.from_numpy(gaussian_error(ge, n)).cuda()
        cts.append(ctx.encrypt(s, pt, a, e))
    steps = [T * b for b in range(1, n1)] + [T * n1 * g for g in range(1, n2)]
    gk = rng(cfg.index, 5)
    keys = {}
    for st in steps:
        a = torch.from_numpy(uniform_residues(gk, ctx.primes, n, lead=(ctx.dnum,))).cuda()
        e = torch.from_numpy(gaussian_error(gk, (ctx.dnum, n))).cuda()
        keys[st] = ctx.keygen_galois(s, ctx.galois_elt(st), a, e)
    torch.cuda.synchronize()
    return dict(ctx=ctx, s=s, X=X, W=W, Wd=Wd, cts=cts, keys=keys, T=T, D=D, n1=n1, delta=delta)


def tm_pack(X, T, D, i):
    return X[:, i * D:(i + 1) * D].reshape(-1)


def setup_projection_tm(torch, np, cfg, n1):
    """Inputs and keys of the token-major projection (slot t*D + f): steps b, b - D (0 <= b < n1) and n1 g."""
    from workloads import (gaussian_error, gaussian_weights, rng, ternary_secret, uniform_residues,
                           uniform_slots)
    ctx = make_context(cfg)
    n, T, level = ctx.n, cfg.tokens, cfg.level
    D = (n // 2) // T
    n2 = -(-D // n1)
    s = torch.from_numpy(ternary_secret(rng(cfg.index, 3), n)).cuda()
    X = uniform_slots(rng(cfg.index, 1), (T, cfg.d_in))
    W = gaussian_weights(rng(cfg.index, 2), (cfg.d_in, cfg.d_out))
    Wd = torch.from_numpy(W).cuda()
    delta = float(2 ** cfg.scale_log2)
    ge = rng(cfg.index, 4)
    cts = []
    for i in range(cfg.d_in // D):
        pt = ctx.encode(torch.from_numpy(tm_pack(X, T, D, i)).cuda(), None, delta, level + 1)
        a = torch.from_numpy(uniform_residues(ge, ctx.q[:level + 1], n)).cuda()
        e = torch.from_numpy(gaussian_error(ge, n)).cuda()
        cts.append(ctx.encrypt(s, pt, a, e))
    steps = [b for b in range(1, n1)] + [b - D for b in range(n1)] + [n1 * g for g in range(1, n2)]
    gk = rng(cfg.index, 5)
    keys = {}
    for st in steps:
        a = torch.from_numpy(uniform_residues(gk, ctx.primes, n, lead=(ctx.dnum,))).cuda()
        e = torch.from_numpy(gaussian_error(gk, (ctx.dnum, n))).cuda()
        keys[st] = ctx.keygen_galois(s, ctx.galois_elt(st), a, e)
    torch.cuda.synchronize()
    return dict(ctx=ctx, s=s, X=X, W=W, Wd=Wd, cts=cts, keys=keys, T=T, D=D, n1=n1, delta=delta)


def bench_tm(torch, np, steps, warmup, n1s=(16, 32)):
    """The 4096x14336 projection in the token-major layout (periodic weight plaintexts), per baby-step size."""
    from workloads import PROJECTION as cfg
    res = {}
    for n1 in n1s:
        st = setup_projection_tm(torch, np, cfg, n1)
        ctx = st["ctx"]
        outs = None
        for _ in range(warmup):
            outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], n1, st["keys"], outs, layout="tm")
        # timed with the library's profiler off; the per-kernel figures from as many profiled steps afterwards
        with Timer(torch) as t:
            for _ in range(steps):
                outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], n1, st["keys"], outs, layout="tm")
        ctx.profile(True)
        ctx.profile_reset()
        for _ in range(steps):
            outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], n1, st["keys"], outs, layout="tm")
        torch.cuda.synchronize()
        prof = ctx.profile_all()
        ctx.profile(False)
        T, D = st["T"], st["D"]
        errs = []
        for j in (0, 27, 55):
            re, _ = ctx.decode(ctx.decrypt(st["s"], outs[j]))
            want = tm_pack(st["X"] @ st["W"][:, j * D:(j + 1) * D], T, D, 0)
            errs.append(float(np.max(np.abs(re.cpu().numpy() - want))))
        n2 = -(-D // n1)
        res["n1=%d" % n1] = {
            "workload": "4096x14336 token-major (slot t*256 + f), N=2^16, level 12, n1=%d n2=%d, %d rotations"
                        % (n1, n2, 16 * (2 * n1 - 1) + 56 * (n2 - 1)),
            "s_per_projection": t.ms / steps / 1e3, "decrypt_max_abs_err": max(errs),
            "kernels_ms": {k: round(v[0] / steps, 3) for k, v in sorted(prof.items(), key=lambda kv: -kv[1][0])}}
        log("token-major n1=%d: %.1f ms" % (n1, t.ms / steps))
        del st, outs, ctx
        torch.cuda.empty_cache()
    return res


def device_keys(torch, ctx, s, steps, seed):
    """Galois keys for `steps` and the relinearisation key from device randomness (uniform residues, rounded
    Gaussian errors): generating the attention block's ~550 keys from host randomness would take minutes."""
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

    keys = {st: ctx.keygen_galois(s, ctx.galois_elt(st), rand_a(), rand_e()) for st in steps}
    return keys, ctx.keygen_relin(s, rand_a(), rand_e())


def attention_plain(np, X, Wq, Wk, Wv, Wo, T, hd, heads, kv_heads):
    """The block in fp64 on the host, scores on cyclic token diagonals (no Softmax: P = S)."""
    Q, K, V = X @ Wq, X @ Wk, X @ Wv
    O = np.zeros((T, heads * hd))
    grp = heads // kv_heads
    for h in range(heads):
        q, k, v = Q[:, h * hd:(h + 1) * hd], K[:, (h // grp) * hd:(h // grp + 1) * hd], \
            V[:, (h // grp) * hd:(h // grp + 1) * hd]
        S = np.stack([np.sum(q * np.roll(k, -d, axis=0), axis=1) for d in range(T)], axis=1)  # [t][delta]
        for d in range(T):
            O[:, h * hd:(h + 1) * hd] += S[:, d:d + 1] * np.roll(v, -d, axis=0)
    return O @ Wo


def bench_attention(torch, np, steps, warmup):
    """One Llama-3-8B attention block's ciphertext work in the token-major layout: Q, K, V projections, scores
    on token diagonals, weighted sums of values (consuming the scores; the Softmax between them is not part of
    this library) and the output projection, timed as one step."""
    from paper_2609_12378_amd import Context
    from workloads import ATTENTION as cfg, gaussian_error, gaussian_weights, rng, ternary_secret, \
        uniform_residues, uniform_slots
    ctx = make_context(cfg)
    n, T, hd, level, n1 = ctx.n, cfg.tokens, cfg.head_dim, cfg.level, cfg.n1
    D = (n // 2) // T
    hpc = D // hd
    d_kv = cfg.kv_heads * hd
    s = torch.from_numpy(ternary_secret(rng(cfg.index, 3), n)).cuda()
    X = uniform_slots(rng(cfg.index, 1), (T, cfg.d_in))
    gw = rng(cfg.index, 2)
    # 1/sqrt(hd) folded into W_Q, as the block scales its scores
    Wq = gaussian_weights(gw, (cfg.d_in, cfg.heads * hd)) / np.sqrt(hd)
    Wk = gaussian_weights(gw, (cfg.d_in, d_kv))
    Wv = gaussian_weights(gw, (cfg.d_in, d_kv))
    Wo = gaussian_weights(gw, (cfg.heads * hd, cfg.d_out))
    # K and V projections emit each head in every head position of its own ciphertext
    dup = np.concatenate([np.arange(m * hd, (m + 1) * hd) for m in range(cfg.kv_heads) for _ in range(hpc)])
    Wk2, Wv2 = np.ascontiguousarray(Wk[:, dup]), np.ascontiguousarray(Wv[:, dup])
    # one projection for Q, K' and V' (one set of baby-step rotations of the inputs, full output tiles)
    Wqkv = np.ascontiguousarray(np.concatenate([Wq, Wk2, Wv2], axis=1))
    Wd = {k: torch.from_numpy(v).cuda() for k, v in (("qkv", Wqkv), ("o", Wo))}
    delta = float(2 ** cfg.scale_log2)
    ge = rng(cfg.index, 4)
    cts = []
    for i in range(cfg.d_in // D):
        pt = ctx.encode(torch.from_numpy(tm_pack(X, T, D, i)).cuda(), None, delta, level + 1)
        a = torch.from_numpy(uniform_residues(ge, ctx.q[:level + 1], n)).cuda()
        e = torch.from_numpy(gaussian_error(ge, n)).cuda()
        cts.append(ctx.encrypt(s, pt, a, e))
    n2 = -(-D // n1)
    steps_p = [b for b in range(1, n1)] + [b - D for b in range(n1)] + [n1 * g for g in range(1, n2)]
    all_steps = sorted(set(steps_p) | set(Context.attention_steps(n // 2, T, hd)))
    keys, rlk = device_keys(torch, ctx, s, all_steps, cfg.index)
    torch.cuda.synchronize()
    log("attention: %d keys ready" % len(keys))
    n_q, n_kv = cfg.heads * hd // D, cfg.kv_heads
    grp = cfg.heads // cfg.kv_heads
    kv_of_q = [c * hpc // grp for c in range(n_q)]
    ev = {k: torch.cuda.Event(enable_timing=True) for k in ("a", "b", "c", "d", "e")}

    def step():
        ev["a"].record()
        QKV = ctx.linear_project(cts, Wd["qkv"], T, n1, keys, layout="tm")
        Q, K, V = QKV[:n_q], QKV[n_q:n_q + n_kv], QKV[n_q + n_kv:]
        ev["b"].record()
        S = ctx.attention_scores(Q, K, kv_of_q, T, hd, rlk, keys)
        ev["c"].record()
        O = ctx.attention_apply(S, V, kv_of_q, T, hd, rlk, keys)
        ev["d"].record()
        Y = ctx.linear_project(O, Wd["o"], T, n1, keys, layout="tm")
        ev["e"].record()
        return Y

    for w in range(warmup):
        Y = step()
        torch.cuda.synchronize()
        log("attention warmup", w, "done")
    # timed with the library's profiler off; the per-kernel figures from as many profiled steps afterwards
    phase = {"qkv_projection": 0.0, "scores": 0.0, "weighted_sums": 0.0, "output_projection": 0.0}
    with Timer(torch) as t:
        for _ in range(steps):
            Y = step()
            torch.cuda.synchronize()
            for name, (a, b) in zip(phase, (("a", "b"), ("b", "c"), ("c", "d"), ("d", "e"))):
                phase[name] += ev[a].elapsed_time(ev[b]) / steps
    ctx.profile(True)
    ctx.profile_reset()
    for _ in range(steps):
        Y = step()
    torch.cuda.synchronize()
    prof = ctx.profile_all()
    ctx.profile(False)
    want = attention_plain(np, X, Wq, Wk, Wv, Wo, T, hd, cfg.heads, cfg.kv_heads)
    errs = []
    for j in (0, 7, 15):
        re, _ = ctx.decode(ctx.decrypt(s, Y[j]))
        errs.append(float(np.max(np.abs(re.cpu().numpy() - tm_pack(want, T, D, j)))))
    res = {
        "workload": "one Llama-3-8B attention block, token-major (slot t*256 + f): 128 tokens, 32 query / 8 key-value "
                    "heads of 128, N=2^16, 24+8 x 50-bit primes, dnum 3, scale 2^50, inputs at level 12; Q/K/V/O "
                    "projections (n1=%d; Q, K, V as one 4096x8192 projection, K and V heads written twice), scores on token "
                    "diagonals, weighted sums consuming them (no Softmax)" % n1,
        "s_per_block": t.ms / steps / 1e3,
        "phases_ms": {k: round(v, 3) for k, v in phase.items()},
        "decrypt_max_abs_err": max(errs), "output_max_abs": float(np.max(np.abs(want))),
        "keys": len(keys),
        "kernels_ms": {k: round(v[0] / steps, 3) for k, v in sorted(prof.items(), key=lambda kv: -kv[1][0])}}
    log("attention block: %.1f ms (%s), max err %.3g" % (t.ms / steps, res["phases_ms"], max(errs)))
    del keys, rlk, cts, ctx
    torch.cuda.empty_cache()
    return res


def check_projection(np, st, outs, blocks=(0, 27, 55)):
    """Decrypt sampled outputs and compare with X @ W (property check at full size)."""
    ctx, T, D = st["ctx"], st["T"], st["D"]
    errs = []
    for j in blocks:
        if j >= len(outs):
            continue
        re, _ = ctx.decode(ctx.decrypt(st["s"], outs[j]))
        want = fm_pack(st["X"] @ st["W"][:, j * D:(j + 1) * D], T, D, 0)
        errs.append(float(np.max(np.abs(re.cpu().numpy() - want))))
    return max(errs) if errs else None


COPY = {"GBps": None}


def measure_copy(torch, ctx, mib=1024, reps=3):
    """Measured HBM rate of a plain device copy (read + write bytes over time) of a buffer far larger than the
    caches: the practical ceiling next to the nominal 8 TB/s."""
    src = torch.ones(mib << 17, dtype=torch.uint64, device="cuda")
    dst = torch.empty_like(src)
    ctx.calib_copy(dst, src)
    with Timer(torch) as t:
        for _ in range(reps):
            ctx.calib_copy(dst, src)
    del src, dst
    COPY["GBps"] = 2.0 * (mib << 20) * reps / (t.ms * 1e-3) / 1e9
    return COPY["GBps"]


def measure_modmul(torch, ctx, lanes=1 << 21, iters=512):
    """Measured fp64 modular-multiply rate (the library's probe: eight independent product chains per lane,
    exact FMA products, q < 2^50), the ALU reference for the projection's modmul-class work."""
    out = torch.empty(lanes, dtype=torch.uint64, device="cuda")
    ctx.calib_modmul(out, iters, 1)
    with Timer(torch) as t:
        ctx.calib_modmul(out, iters, 1)
    del out
    return lanes * iters * 8 / (t.ms * 1e-3)


def projection_modmuls(cfg, ks_rotations):
    """Modmul-class operations of one projection: one modular product per encode-NTT butterfly (every weight
    plaintext, every limb), two per multiply-accumulated residue, and about 2.5e7 per key-switched rotation at
    level 12 (inner product, conversions and the ModDown transforms)."""
    D = cfg.feats
    plaintexts = (cfg.d_out // D) * (cfg.d_in // D) * D
    limbs = cfg.level + 1
    n, log_n = 1 << cfg.log_n, cfg.log_n
    return plaintexts * limbs * (n // 2) * log_n + plaintexts * limbs * n * 2 + ks_rotations * 2.5e7


def hbm_fracs(gbs):
    out = {"frac": gbs / HBM_PEAK_GBS}
    if COPY["GBps"]:
        out["copy_GBps"] = COPY["GBps"]
        out["frac_of_copy"] = gbs / COPY["GBps"]
    return out


def roofline(prof):
    """The kernel with the most total time, against the HBM roof and the VALU issue roof.

    HBM: algorithmic bytes per launch / average launch time vs 8 TB/s.  VALU: the kernel's nominal lane
    instructions (its arithmetic model, reported by the library) per second vs 256 CUs x 64 lanes x 2.4 GHz
    (fp64 FMA and 32-bit integer instructions issue at full rate).  "bound" names the roof the kernel is
    nearer to; the top-level achieved/peak/frac are for that roof.
    """
    name, (ms, cnt, by, ops) = max(prof.items(), key=lambda kv: kv[1][0])
    sec = ms * 1e-3
    gbs = by / sec / 1e9
    hbm = {"achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", **hbm_fracs(gbs)}
    out = {"kernel": name, "launches": cnt, "avg_ms": ms / cnt, "bytes_per_launch": by / cnt}
    alu = None
    if ops:
        gops = ops / sec / 1e9
        alu = {"achieved": gops, "peak": LANE_OPS / 1e9, "unit": "G VALU lane-instr/s", "frac": gops * 1e9 / LANE_OPS,
               "instr_per_launch": ops / cnt}
    bound = "alu" if alu and alu["frac"] > hbm["frac"] else "hbm"
    out["bound"] = bound
    out.update(alu if bound == "alu" else hbm)
    out["hbm"] = hbm
    if alu:
        out["alu"] = alu
    return out


# sources whose text determines a kernel's memory traffic; a recorded counter value applies only while
# their hash is unchanged
KERNEL_SOURCES = {
    "ntt_row_mac": ["project.hip", "ntt_core.h", "modarith.h", "ckks_internal.h"],
    "ntt_fwd_col": ["encode.hip", "ntt.hip", "ntt_core.h", "modarith.h", "ckks_internal.h"],
}


def sources_sha(kernel):
    names = KERNEL_SOURCES.get(kernel)
    if not names:
        return None
    h = hashlib.sha256()
    for f in names:
        with open(os.path.join(ROOT, "paper_2609_12378_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(kernel):
    """HBM bytes per launch measured with rocprofv3 FETCH_SIZE + WRITE_SIZE (copy-calibrated), if recorded
    in profiles/pmc_traffic.md for the current text of the kernel's sources; else None."""
    path = os.path.join(ROOT, "profiles", "pmc_traffic.md")
    sha = sources_sha(kernel)
    if sha is None or not os.path.exists(path):
        return None
    for line in open(path):
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 6 and cells[0] == kernel and cells[2] == sha:
            try:
                return float(cells[5])
            except ValueError:
                return None
    return None


def paper_context(cfg):
    """A context with the paper's chain (q_0 of 60 bits, q_1.. of 59 bits, special primes of 60 bits), the prime
    lists taken from the library's own generator."""
    from paper_2609_12378_amd import Context
    from workloads import paper_chain
    p60 = Context(cfg.log_n, 1 + cfg.n_p, 0, 1, q_bits=60).q
    p59 = Context(cfg.log_n, cfg.n_q - 1, 0, 1, q_bits=59).q
    q, p = paper_chain(p60, p59, cfg.n_q, cfg.n_p)
    ctx = Context(cfg.log_n, cfg.n_q, cfg.n_p, cfg.dnum, q=q, p=p)
    ctx.set_lazy_moddown(LAZY["on"])
    return ctx


def bench_keyswitch(torch, np, steps, warmup, seeded=False, paper=False):
    """The hoisted batch; with `seeded`, seed-expanded keys (b halves in HBM, the a halves generated in the kernels);
    with `paper`, the paper's parameters (N = 2^16, 37 limbs of 60/59 bits + 8 of 60 bits, dnum 5, level 36)."""
    from workloads import KEYSWITCH, KEYSWITCH_PAPER, gaussian_error, rng, ternary_secret, uniform_residues, \
        uniform_slots
    cfg = KEYSWITCH_PAPER if paper else KEYSWITCH
    ctx = paper_context(cfg) if paper else make_context(cfg)
    n, L = ctx.n, cfg.level + 1
    s = torch.from_numpy(ternary_secret(rng(cfg.index, 3), n)).cuda()
    z = uniform_slots(rng(cfg.index, 1), n // 2)
    pt = ctx.encode(torch.from_numpy(z).cuda(), None, float(2 ** cfg.scale_log2), L)
    ge = rng(cfg.index, 4)
    ct = ctx.encrypt(s, pt, torch.from_numpy(uniform_residues(ge, ctx.q[:L], n)).cuda(),
                     torch.from_numpy(gaussian_error(ge, n)).cuda())
    rsteps = list(range(1, cfg.batch + 1))
    gk = rng(cfg.index, 5)
    keys, seeds = [], []
    for r in rsteps:
        if seeded:
            seeds.append([int(x) for x in gk.integers(0, 1 << 63, 2)])
            e = torch.from_numpy(gaussian_error(gk, (cfg.dnum, n))).cuda()
            keys.append(ctx.keygen_galois_seeded(s, ctx.galois_elt(r), seeds[-1], e))
        else:
            a = torch.from_numpy(uniform_residues(gk, ctx.primes, n, lead=(cfg.dnum,))).cuda()
            e = torch.from_numpy(gaussian_error(gk, (cfg.dnum, n))).cuda()
            keys.append(ctx.keygen_galois(s, ctx.galois_elt(r), a, e))

    def batch(outs=None):
        if seeded:
            return ctx.rotate_hoisted_seeded(ct, rsteps, keys, seeds, outs)
        return ctx.rotate_hoisted(ct, rsteps, keys, outs)

    outs = batch()
    for _ in range(warmup):
        batch(outs)
    # each batch bracketed by its own events, the library's profiler off: the median over the runs; then the same
    # number of batches again with the profiler on (two events around every launch) for the per-kernel figures
    runs = []
    for _ in range(steps):
        with Timer(torch) as t:
            batch(outs)
        runs.append(t.ms)
    ctx.profile(True)
    ctx.profile_reset()
    for _ in range(steps):
        batch(outs)
    torch.cuda.synchronize()
    prof = ctx.profile_all()
    ctx.profile(False)
    re, _ = ctx.decode(ctx.decrypt(s, outs[-1]))
    err = float(np.max(np.abs(re.cpu().numpy() - np.roll(z, -rsteps[-1]))))
    ms = float(np.median(runs))
    # HBM roofline of the batch.  Algorithmic bytes: what any hoisted batch must move once, the 32 keys
    # [dnum][2][L+K][N], the 32 outputs [2][L][N], the input [2][L][N], and the ModUp digits [dnum][L+K][N]
    # written and read once; over the batch's median time.  Beside it, the bytes the library's profiler tags on
    # its launches (each word a launch reads or writes, once; intermediate rows included) over the kernels'
    # summed time: how close the kernels run to the rate HBM sustains.
    word = 8.0 * n
    nd = cfg.dnum
    # keys: both halves, or the b half of a seeded key
    khalves = 1 if seeded else 2
    abytes = (cfg.batch * nd * khalves * (L + cfg.n_p) + cfg.batch * 2 * L + 2 * L + 2 * nd * (L + cfg.n_p)) * word
    kbytes = sum(v[2] for v in prof.values()) / steps
    kms = sum(v[0] for v in prof.values()) / steps
    res = {"workload": ("32 hoisted rotations by 1..32 of one level-36 ciphertext, N=2^16, L=37 (60/59-bit) + K=8 "
                        "(60-bit), dnum=5 (the paper's parameters)" if paper else
                        "32 hoisted rotations by 1..32 of one level-23 ciphertext, N=2^16, L=24+K=8, dnum=3")
                       + (", seed-expanded keys" if seeded else ""),
           "ms_per_batch": ms, "rotations_per_s": cfg.batch / (ms * 1e-3), "decrypt_err_last": err,
           "runs": steps, "warmup": warmup, "ms_min": min(runs), "ms_max": max(runs),
           "roofline": {"bound": "hbm", "algorithmic_bytes_per_batch": abytes,
                        "achieved": abytes / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        **hbm_fracs(abytes / (ms * 1e-3) / 1e9)},
           "kernel_traffic": {"bytes_per_batch": kbytes, "GBps": kbytes / (kms * 1e-3) / 1e9,
                              **hbm_fracs(kbytes / (kms * 1e-3) / 1e9)},
           "kernels_ms": {k: v[0] / steps for k, v in prof.items()},
           "kernels_GBps": {k: v[2] / (v[0] * 1e-3) / 1e9 for k, v in prof.items() if v[0] > 0}}
    del keys, outs, ct, ctx
    return res


def bench_projection_paper(torch, np):
    """The 4096x14336 projection (its shapes, level 12, n1 = 32) with the paper's modulus chain (60/59-bit q, 60-bit
    special primes, dnum 5): every prime is at least 2^50, so the encode transforms, the multiply-accumulate (128-bit
    integer sums) and the key switching run on the integer path.  One timed step after one warm-up."""
    from workloads import KEYSWITCH_PAPER, PROJECTION
    st = setup_projection(torch, np, PROJECTION, ctx=paper_context(KEYSWITCH_PAPER))
    ctx = st["ctx"]
    outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"])
    with Timer(torch) as t:
        outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
    ctx.profile(True)
    ctx.profile_reset()
    outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
    prof = ctx.profile_all()
    ctx.profile(False)
    err = check_projection(np, st, outs)
    res = {"workload": "4096x14336 feature-major projection, N=2^16, level 12 of the paper's chain (q_0 60-bit, "
                       "q_1.. 59-bit, 8 x 60-bit special primes, dnum 5), n1 = 32: the integer path",
           "s_per_projection": t.ms / 1e3, "decrypt_max_abs_err": err,
           "kernels_ms": {k: round(v[0], 2) for k, v in sorted(prof.items(), key=lambda kv: -kv[1][0])}}
    del st, outs, ctx
    torch.cuda.empty_cache()
    return res


def bench_ntt(torch, steps, bits=50):
    """The batched NTT microbenchmark; bits = 59: the same shape over 59-bit primes (the paper's size; integer
    butterflies)."""
    import numpy as np
    from paper_2609_12378_amd import Context
    from workloads import NTT_BENCH as cfg
    ctx = Context(cfg.log_n, cfg.n_q, 0, 1, q_bits=bits)
    g = torch.Generator(device="cuda").manual_seed(202)
    x = torch.randint(0, 1 << (bits - 1), (cfg.batch, cfg.n_q, ctx.n), generator=g, device="cuda",
                      dtype=torch.int64).view(torch.uint64)
    ctx.ntt(x)
    ctx.intt(x)
    for _ in range(2):
        ctx.ntt(x)
        ctx.intt(x)
    # timed with the library's profiler off; the per-kernel figures from as many profiled runs afterwards
    fwd, inv = [], []
    for _ in range(steps):
        with Timer(torch) as tf:
            ctx.ntt(x)
        fwd.append(tf.ms)
        with Timer(torch) as ti:
            ctx.intt(x)
        inv.append(ti.ms)
    ctx.profile(True)
    ctx.profile_reset()
    for _ in range(steps):
        ctx.ntt(x)
        ctx.intt(x)
    torch.cuda.synchronize()
    prof = ctx.profile_all()
    ctx.profile(False)
    fms, ims = float(np.median(fwd)), float(np.median(inv))
    algo = 16.0 * cfg.batch * cfg.n_q * ctx.n
    res = {"workload": "64 polys x 36 limbs x 2^16, %d-bit primes" % bits, "fwd_ms": fms, "inv_ms": ims,
           "runs": steps, "warmup": 3, "algorithmic_bytes_per_direction": algo,
           "fwd_GBps": algo / (fms * 1e-3) / 1e9, "inv_GBps": algo / (ims * 1e-3) / 1e9,
           "kernels": {k: {"avg_ms": v[0] / v[1], "GBps": v[2] / (v[0] * 1e-3) / 1e9,
                           **hbm_fracs(v[2] / (v[0] * 1e-3) / 1e9)} for k, v in prof.items()}}
    # per transform (one read and one write of every residue) against 8 TB/s; each two-pass transform moves twice that
    res["fwd_hbm"] = hbm_fracs(res["fwd_GBps"])
    res["inv_hbm"] = hbm_fracs(res["inv_GBps"])
    del x, ctx
    return res


def bench_tile(torch, np, steps, warmup, calib_mib):
    """One output tile of the projection: 4096 -> 28 x 256 features, the same launches as the full one.

    A smaller process for hardware-counter passes; per-launch figures of its kernels apply to the full
    projection, whose launches have the same shapes.
    """
    import dataclasses
    from workloads import PROJECTION
    cfg = dataclasses.replace(PROJECTION, d_out=28 * PROJECTION.feats)
    st = setup_projection(torch, np, cfg)
    ctx = st["ctx"]
    if calib_mib:
        src = torch.ones(calib_mib << 17, dtype=torch.uint64, device="cuda")
        dst = torch.empty_like(src)
        ctx.calib_copy(dst, src)
        torch.cuda.synchronize()
        del src, dst
    outs = None
    for _ in range(warmup):
        outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
    ctx.profile(True)
    ctx.profile_reset()
    with Timer(torch) as t:
        for _ in range(steps):
            outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
    prof = ctx.profile_all()
    ctx.profile(False)
    err = check_projection(np, st, outs, blocks=(0, 27))
    return {"workload": "projection 4096x7168 (one tile of 28 output ciphertexts of the 4096x14336 projection)",
            "ms_per_step": t.ms / steps, "decrypt_max_abs_err": err,
            "kernels": {k: {"launches": v[1] / steps, "avg_ms": v[0] / v[1], "bytes_per_launch": v[2] / v[1],
                            "GBps": v[2] / (v[0] * 1e-3) / 1e9} for k, v in prof.items()}}


def bench_shapes(torch, np, steps):
    """The other projection shapes of a Llama-3-8B block (QKV, attention output, down), same ring and level."""
    from workloads import PROJ_DOWN, PROJ_QKV, PROJ_WO
    res = {}
    for cfg in (PROJ_QKV, PROJ_WO, PROJ_DOWN):
        st = setup_projection(torch, np, cfg)
        ctx = st["ctx"]
        outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"])
        with Timer(torch) as t:
            for _ in range(steps):
                outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
        n_out = cfg.d_out // st["D"]
        err = check_projection(np, st, outs, blocks=(0, n_out - 1))
        D, n1 = st["D"], cfg.n1
        n2 = -(-D // n1)
        res[cfg.name] = {"workload": "%dx%d, n1=%d n2=%d, %d rotations" % (
                             cfg.d_in, cfg.d_out, n1, n2, (cfg.d_in // D) * (n1 - 1) + n_out * (n2 - 1)),
                         "s_per_projection": t.ms / steps / 1e3, "decrypt_max_abs_err": err}
        log("shape %s: %.1f ms" % (cfg.name, t.ms / steps))
        del st, outs, ctx
        torch.cuda.empty_cache()
    return res


def cpu_baseline(np, cfg, budget_s=20.0):
    """The oracle on a bounded sample of the projection, extrapolated to one full projection."""
    from oracle import Ckks, gen_primes
    from workloads import gaussian_error, gaussian_weights, rng, ternary_secret, uniform_residues, uniform_slots
    pr = gen_primes(cfg.q_bits, 2 * cfg.n, cfg.n_q + cfg.n_p)
    ck = Ckks(cfg.log_n, pr[:cfg.n_q], pr[cfg.n_q:], cfg.dnum)
    n, T, D, level, n1 = ck.n, cfg.tokens, cfg.feats, cfg.level, cfg.n1
    s = ternary_secret(rng(cfg.index, 3), n)
    W = gaussian_weights(rng(cfg.index, 2), (D, D))
    X = uniform_slots(rng(cfg.index, 1), (T, D))
    ge = rng(cfg.index, 4)
    ct = ck.encrypt(s, ck.encode(fm_pack(X, T, D, 0), None, 2.0 ** 40, level + 1),
                    uniform_residues(ge, ck.q[:level + 1], n), gaussian_error(ge, n))
    gk = rng(cfg.index, 5)
    key = ck.keygen_galois(s, ck.galois_elt(T), uniform_residues(gk, ck.primes, n, lead=(cfg.dnum,)),
                           gaussian_error(gk, (cfg.dnum, n)))
    qd = float(ck.q[level])
    n_in, n_out = cfg.d_in // D, cfg.d_out // D
    n2 = -(-D // n1)

    def sample(budget, min_pts):
        t0 = time.time()
        n_pts, acc = 0, None
        while time.time() - t0 < budget or n_pts < min_pts:
            z = Ckks.diag_slot_vector(W, T, D, 0, 0, n1, 0, n_pts % n1)
            term = ck.ct_mul_plain(ct, ck.encode(z, None, qd, level + 1))
            acc = term if acc is None else ck.ct_add(acc, term)
            n_pts += 1
        t_pt = (time.time() - t0) / n_pts
        t1 = time.time()
        ck.rotate(ct, T, key)
        t_rot = time.time() - t1
        t2 = time.time()
        ck.rescale(acc)
        t_rs = time.time() - t2
        total = (n_out * n_in * D) * t_pt + (n_in * (n1 - 1) + n_out * (n2 - 1)) * t_rot + n_out * t_rs
        return total, n_pts, t_pt, t_rot, t_rs

    L = oracle_lib()
    threads = L.or_threads()
    total, n_pts, t_pt, t_rot, t_rs = sample(budget_s * 0.5, 2)
    # the same sample on one thread (the oracle's loops run over limb rows, so this is its serial rate)
    L.or_set_threads(1)
    try:
        total1, n1_pts, t_pt1, t_rot1, _ = sample(budget_s * 0.15, 2)
    finally:
        L.or_set_threads(threads)
    return {"value": total, "unit": "s/projection (extrapolated)", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "host_threads": os.cpu_count(),
            "single_thread": {"value": total1, "unit": "s/projection (extrapolated)",
                              "sample": "%d plaintexts (%.3f s each), 1 rotation (%.2f s)" % (n1_pts, t_pt1, t_rot1)},
            "sample": "%d weight plaintexts encoded+multiplied+accumulated (%.3f s each), 1 rotation (%.2f s), "
                      "1 rescale (%.2f s) at N=2^16 level 12, %d threads; scaled by 229376 plaintexts, 888 rotations, "
                      "56 rescales" % (n_pts, t_pt, t_rot, t_rs, threads)}


def oracle_lib():
    from oracle.ckks import lib
    return lib()


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo, as lscpu reports it)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_oracle_secondary(np):
    """The oracle on the NTT and key-switching workloads in full, with its OpenMP threads (rows of the transform
    in parallel; the key switch's limb loops): the 64 x 36 x 2^16 forward and inverse transforms (round trip
    checked), and the 32 hoisted rotations of the key-switching batch; plus the NTT's single-threaded rate from
    one row."""
    from oracle import Ckks, gen_primes
    from oracle.ckks import lib as oracle_lib
    from workloads import KEYSWITCH as kcfg, NTT_BENCH as ncfg, gaussian_error, rng, ternary_secret, \
        uniform_residues, uniform_slots
    out = {}
    threads = oracle_lib().or_threads()
    pr = gen_primes(ncfg.q_bits, 2 * ncfg.n, ncfg.n_q)
    ck = Ckks(ncfg.log_n, pr)
    a = uniform_residues(rng(ncfg.index, 1), pr, ck.n, lead=(ncfg.batch,))
    idx = list(range(ncfg.n_q)) * ncfg.batch
    t0 = time.time()
    fa = ck.ntt(a, idx)
    t_fwd = time.time() - t0
    t0 = time.time()
    back = ck.intt(fa, idx)
    t_inv = time.time() - t0
    assert np.array_equal(back, a), "oracle NTT round trip failed"
    del fa, back
    oracle_lib().or_set_threads(1)
    try:
        t0 = time.time()
        ck.ntt(a[0, :1], [0])
        t_row1 = time.time() - t0
    finally:
        oracle_lib().or_set_threads(threads)
    out["ntt"] = {"s_per_direction": t_fwd, "inv_s": t_inv, "threads": threads,
                  "single_thread_s_per_direction": t_row1 * ncfg.batch * ncfg.n_q,
                  "sample": "the full 64 x 36 x 2^16 forward and inverse (round trip checked), %d threads; single "
                            "thread: one row (%.3f s) scaled by 64 x 36" % (threads, t_row1)}
    del a
    pr = gen_primes(kcfg.q_bits, 2 * kcfg.n, kcfg.n_q + kcfg.n_p)
    ck = Ckks(kcfg.log_n, pr[:kcfg.n_q], pr[kcfg.n_q:], kcfg.dnum)
    n, L = ck.n, kcfg.level + 1
    s = ternary_secret(rng(kcfg.index, 3), n)
    ge = rng(kcfg.index, 4)
    ct = ck.encrypt(s, ck.encode(uniform_slots(rng(kcfg.index, 1), n // 2), None, 2.0 ** 40, L),
                    uniform_residues(ge, ck.q[:L], n), gaussian_error(ge, n))
    gk = rng(kcfg.index, 5)
    steps = list(range(1, kcfg.batch + 1))
    keys = [ck.keygen_galois(s, ck.galois_elt(r), uniform_residues(gk, ck.primes, n, lead=(kcfg.dnum,)),
                             gaussian_error(gk, (kcfg.dnum, n))) for r in steps]
    t0 = time.time()
    ck.rotate_hoisted(ct, steps, keys)
    batch = time.time() - t0
    out["keyswitch"] = {"rotations_per_s": kcfg.batch / batch, "s_per_batch": batch, "threads": threads,
                        "sample": "the full batch: 32 hoisted rotations by 1..32 at level 23, %d threads" % threads}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--only", choices=["keyswitch", "keyswitch_seeded", "paper", "ntt", "tile", "shapes", "tm",
                                       "attention"],
                    default=None,
                    help="run only this secondary workload (for profiling); prints its JSON")
    ap.add_argument("--lazy-moddown", type=int, default=1, choices=[0, 1],
                    help="1 (default): sums of rotations with one ModDown per output (the library's lazy mode); "
                         "0: one ModDown per rotation")
    ap.add_argument("--proj-batch", type=int, default=0,
                    help="at most this many (input, baby step) pairs per multiply-accumulate launch of a projection "
                         "(0: the library's default, 128); for schedule experiments")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (for hardware-counter calibration)")
    args = ap.parse_args()
    LAZY["on"] = bool(args.lazy_moddown)
    PROJ_BATCH["pairs"] = args.proj_batch
    if args.gpus != 1:
        print("bench.py runs on one GPU: the library drives a single GPU (--gpus %d requested)"
              % args.gpus, file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from workloads import PROJECTION as cfg
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.calib_copy_mib and args.only not in (None, "tile"):
        # one plain copy of known size, for scaling the counter passes of these workloads
        from paper_2609_12378_amd import Context
        src = torch.ones(args.calib_copy_mib << 17, dtype=torch.uint64, device="cuda")
        dst = torch.empty_like(src)
        Context(12, 2, 1, 1).calib_copy(dst, src)
        torch.cuda.synchronize()
        del src, dst
    if args.only == "keyswitch":
        print(json.dumps(bench_keyswitch(torch, np, args.steps, args.warmup)), flush=True)
        return
    if args.only == "keyswitch_seeded":
        print(json.dumps(bench_keyswitch(torch, np, args.steps, args.warmup, seeded=True)), flush=True)
        return
    if args.only == "paper":
        print(json.dumps({"keyswitch": bench_keyswitch(torch, np, args.steps, args.warmup, paper=True),
                          "ntt": bench_ntt(torch, args.steps, bits=59),
                          "projection": bench_projection_paper(torch, np)}), flush=True)
        return
    if args.only == "ntt":
        print(json.dumps(bench_ntt(torch, args.steps)), flush=True)
        return
    if args.only == "tm":
        print(json.dumps(bench_tm(torch, np, args.steps, args.warmup)), flush=True)
        return
    if args.only == "attention":
        print(json.dumps(bench_attention(torch, np, args.steps, args.warmup)), flush=True)
        return
    if args.only == "shapes":
        print(json.dumps(bench_shapes(torch, np, args.steps)), flush=True)
        return
    if args.only == "tile":
        print(json.dumps(bench_tile(torch, np, args.steps, args.warmup, args.calib_copy_mib)), flush=True)
        return
    log("setup: projection 4096 -> 14336")
    st = setup_projection(torch, np, cfg)
    ctx = st["ctx"]
    log("copy calibration: %.0f GB/s" % measure_copy(torch, ctx))
    modmul_peak = measure_modmul(torch, ctx)
    log("modmul calibration: %.2f T/s" % (modmul_peak / 1e12))
    if args.calib_copy_mib:
        src = torch.ones(args.calib_copy_mib << 17, dtype=torch.uint64, device="cuda")
        dst = torch.empty_like(src)
        ctx.calib_copy(dst, src)
        torch.cuda.synchronize()
        log("calibration copy of %d MiB done" % args.calib_copy_mib)
        del src, dst
    outs = None
    for w in range(args.warmup):
        outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
        torch.cuda.synchronize()
        log("warmup", w, "done")
    # the timed steps run with the library's event profiler off; one more step with it on gives the per-kernel
    # figures and the roofline of the dominant kernel
    with Timer(torch) as t:
        for _ in range(args.steps):
            outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
    ms = t.ms / args.steps
    log("projection: %.1f ms/step" % ms)
    ctx.profile(True)
    ctx.profile_reset()
    with Timer(torch) as tp:
        outs = ctx.linear_project(st["cts"], st["Wd"], st["T"], st["n1"], st["keys"], outs)
    prof = ctx.profile_all()
    ctx.profile(False)
    log("profiled step: %.1f ms" % tp.ms)
    err = check_projection(np, st, outs)
    log("decrypted outputs 0/27/55: max |err| vs X@W = %.3g" % err)
    roof = roofline(prof)
    roof["traffic"] = load_traffic(roof["kernel"])
    roof["profiled_step_ms"] = tp.ms
    kernels_ms = {k: round(v[0], 3) for k, v in sorted(prof.items(), key=lambda kv: -kv[1][0])}
    del st, outs, ctx
    torch.cuda.empty_cache()
    secondary = {}
    if not args.no_secondary:
        log("keyswitch batch")
        secondary["keyswitch"] = bench_keyswitch(torch, np, max(args.steps, 10), 3)
        torch.cuda.empty_cache()
        log("keyswitch batch, seed-expanded keys")
        secondary["keyswitch_seeded"] = bench_keyswitch(torch, np, max(args.steps, 10), 3, seeded=True)
        torch.cuda.empty_cache()
        log("ntt microbench")
        secondary["ntt"] = bench_ntt(torch, max(args.steps, 10))
        torch.cuda.empty_cache()
        log("the paper's parameters: keyswitch batch and 59-bit NTT")
        secondary["keyswitch_paper_params"] = bench_keyswitch(torch, np, max(args.steps, 10), 3, paper=True)
        torch.cuda.empty_cache()
        secondary["ntt_59bit"] = bench_ntt(torch, max(args.steps, 10), bits=59)
        torch.cuda.empty_cache()
        log("the paper's parameters: 4096x14336 projection (integer path)")
        secondary["projection_paper_params"] = bench_projection_paper(torch, np)
        log("other projection shapes")
        secondary["shapes"] = bench_shapes(torch, np, 1)
        torch.cuda.empty_cache()
        log("token-major projection")
        secondary["projection_tm"] = bench_tm(torch, np, 1, 1, n1s=(32,))["n1=32"]
        torch.cuda.empty_cache()
        log("attention block")
        secondary["attention"] = bench_attention(torch, np, 1, 1)
    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle sample)")
        cpu = cpu_baseline(np, cfg)
        if secondary:
            log("oracle samples: NTT and key switching")
            for k, v in cpu_oracle_secondary(np).items():
                v["cores"] = cpu["cores"]
                v["cpu_model"] = cpu["cpu_model"]
                secondary[k]["cpu_oracle"] = v
    line = {
        "metric": METRIC,
        "value": ms / 1e3,
        "unit": "s/projection",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": "Llama-3-8B-shaped ct-pt projection 4096x14336, N=2^16, level 12 (13 limbs), "
                               "24+8 x 50-bit primes, dnum 3, 128 tokens x 256 features, BSGS n1=32 n2=8",
                   "rotations_per_s": secondary.get("keyswitch", {}).get("rotations_per_s")},
        "roofline": roof,
        "cpu_baseline": cpu,
        "decrypt_max_abs_err": err,
        "copy_GBps": COPY["GBps"],
        "modmul": {"ops_per_projection": projection_modmuls(cfg, 888),
                   "achieved_per_s": projection_modmuls(cfg, 888) / (ms * 1e-3),
                   "measured_peak_per_s": modmul_peak,
                   "frac": projection_modmuls(cfg, 888) / (ms * 1e-3) / modmul_peak,
                   "note": "encode-NTT butterflies + multiply-accumulate products + key switching, against the "
                           "library's fp64 modmul probe (8 independent chains per lane)"},
        "kernels_ms_per_step": kernels_ms,
        "secondary": secondary,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
