"""The fp64 NTT passes skip range reductions in some forward stages; the masks in csrc/ntt.hip must keep every value
below 8q (q < 2^50, so below 2^53, where the fp64 products are exact) and the column pass's output below 2q (the
bound the fused key-switching kernels assume for a first pass's rows).

Bounds in units of q, from the arithmetic in csrc/ntt_core.h (Ar<true>): mul(a, w) <= 0.5 + 0.375|a| for |a| <= 8,
red(x) <= 0.5 (+2^-52|x|), so a reducing stage maps b to 1 + 0.375b and a lazy one to b + 0.5 + 0.375b.
"""
import os
import re

import pytest

SRC = os.path.join(os.path.dirname(__file__), "..", "paper_2609_12378_amd", "csrc", "ntt.hip")
SLOP = 1 + 2.0 ** -40   # the 2^-52 relative terms, generously


def masks():
    """The three mask tables of csrc/ntt.hip, indexed by log2 of the sub-transform size."""
    text = open(SRC).read()
    out = {}
    for name in ("kFwdColMask", "kFwdRowMask", "kFwdSingleMask"):
        body = re.search(r"constexpr unsigned %s\[9\] = \{([^}]*)\};" % name, text).group(1)
        out[name] = [int(v.strip(), 16) for v in body.split(",")]
    return out


def run(b, mask, stages):
    peak = b
    for s in range(stages):
        b = (1 + 0.375 * b if (mask >> s) & 1 else 1.375 * b + 0.5) * SLOP
        peak = max(peak, b)
    return b, peak


@pytest.mark.parametrize("logs", [4, 5, 6, 7, 8])
def test_forward_masks_stay_exact(logs):
    m = masks()
    out, peak = run(1.0, m["kFwdColMask"][logs], logs)        # canonical input
    assert peak < 8 and out < 2, (logs, out, peak)
    out_r, peak_r = run(2.0, m["kFwdRowMask"][logs], logs)    # after a column pass
    assert peak_r < 8 and out_r < 8
    out_s, peak_s = run(1.0, m["kFwdSingleMask"][logs], logs)  # single-pass transform
    assert peak_s < 8 and out_s < 8


def test_masks_are_lazy_somewhere():
    m = masks()
    assert bin(m["kFwdColMask"][8]).count("1") == 4 and bin(m["kFwdRowMask"][8]).count("1") == 3


def test_a_wrong_mask_is_caught():
    # every stage lazy in a 256-point column pass overflows the exact range
    assert run(1.0, 0x00, 8)[1] > 8


CORE = os.path.join(os.path.dirname(__file__), "..", "paper_2609_12378_amd", "csrc", "ntt_core.h")


def masks8():
    """kColMask8 and kRowMask8 of csrc/ntt_core.h: the 8-residue passes of the projection and key switching."""
    m = re.search(r"constexpr unsigned kColMask8 = (0x[0-9a-fA-F]+), kRowMask8 = (0x[0-9a-fA-F]+);",
                  open(CORE).read())
    return int(m.group(1), 16), int(m.group(2), 16)


def test_eight_residue_masks_and_their_consumers():
    """Column pass from inputs reduced to q/2, then the row pass; the consumers of the row pass's outputs: the
    multiply-accumulate (four products onto a reduced sum) and the fused ModDown (digit products reduced every
    four terms, minus the transformed conversion, times P^-1)."""
    col, row = masks8()
    out_c, peak_c = run(0.5, col, 8)
    out_r, peak_r = run(out_c, row, 8)
    assert peak_c < 8 and peak_r < 8, (peak_c, peak_r)
    prod = 0.5 + 0.375 * out_r
    assert 0.5 + 4 * prod < 8                        # k_row_mac8's sums
    diff = 0.5 + 4 * 0.875 + out_r                   # k_ks_finish8: u - v
    assert diff < 8 and 0.5 + 0.375 * diff + 1 < 8    # (u - v) P^-1 + c0
    # the bounds the kernels' comments state
    assert out_c < 4.3 and peak_c < 5.3 and out_r < 2.6 and peak_r < 6.4 and 0.5 + 4 * prod < 6.4


def test_eight_residue_masks_are_minimal():
    """No pair of masks with fewer reducing stages in total keeps the same bounds below 7.9 q (the best such pair
    leaves the multiply-accumulate's sums within 0.5% of the exact range)."""
    col, row = masks8()
    used = bin(col).count("1") + bin(row).count("1")
    for c in range(256):
        oc, pc = run(0.5, c, 8)
        if pc >= 7.9:
            continue
        for r in range(256):
            if bin(c).count("1") + bin(r).count("1") >= used:
                continue
            orr, pr = run(oc, r, 8)
            ok = pr < 7.9 and 0.5 + 4 * (0.5 + 0.375 * orr) < 7.9 and 4.0 + orr < 7.9
            assert not ok, (hex(c), hex(r))
