"""Writes moduli_fp64_k16384.txt: the residue set used for the FP64-significand workload.

It calls only the oracle: the per-modulus scheme search and the smallest-count
selection of pairwise-coprime moduli whose product exceeds 2 K B^2 with
K = 16384 and B = 2^53 - 1 (Sec. 5.3).  Run from the repository root:
    python tests/golden/make_moduli.py
"""
import math
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from oracle import modm  # noqa: E402

K, WIDTH = 16384, 54
moduli, total = modm.select_moduli(K, WIDTH)
lines = [
    "# Pairwise-coprime moduli and their total FP4 product count for the FP64 significand",
    "# (width 54) at reduction length 16384, written by make_moduli.py from the oracle.",
    "# Sum of log2(m) = %.3f > log2(2 K B^2) = %.3f." % (sum(math.log2(m) for m in moduli),
                                                       modm.crt_bits_needed(K, WIDTH)),
    "# Per modulus: " + " ".join("%d:r%d" % (m, modm.find_scheme(m).r) for m in moduli),
    " ".join(str(m) for m in moduli),
    str(total),
]
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "moduli_fp64_k16384.txt"), "w") as f:
    f.write("\n".join(lines) + "\n")
print("\n".join(lines))
