"""Writes full_oracle_sha256.txt: the SHA-256 of the oracle's whole C for the workloads whose
full product is too slow to recompute inside a GPU test.

* The headline product at 8192^3: operands ``inputs.int8_pair(8192, 8192, 8192, seed=0)``, C = A B
  exactly as int32 (Alg. 1, its postcondition; |C| <= 8192 * 128^2 fits), and the INT4 x INT8
  product on ``inputs.int8_pair(8192, 8192, 8192, seed=0, a_range=(-8, 7))`` (Sec. 5.2).

* Residue products at 4096^3, one per modulus of moduli_fp64_k16384.txt: operands
  ``inputs.residue_pair(4096, 4096, 4096, m)`` (seed m), C = (A B) mod m as int32 in [0, m)
  (Sec. 5.3, the congruence relaxation).
* The accumulation stress 4096 x 4096 x 65,536: operands ``inputs.stress_operands(4096, 4096,
  65536, seed=0)``, C = A B exactly as int64 (Alg. 1, its postcondition).

Each hash covers the C-contiguous little-endian bytes of C.  It calls only the oracle and the
seeded input generators.  Run from the repository root (minutes on a few cores):
    python tests/golden/make_full_oracle_hashes.py
"""
import hashlib
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
import numpy as np  # noqa: E402

from oracle import gemm as og  # noqa: E402
from paper_2609_24519_amd import inputs  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def moduli():
    with open(os.path.join(HERE, "moduli_fp64_k16384.txt")) as f:
        rows = [l for l in f if l.strip() and not l.startswith("#")]
    return [int(x) for x in rows[0].split()]


def digest(C):
    return hashlib.sha256(np.ascontiguousarray(C).tobytes()).hexdigest()


def main():
    lines = ["# SHA-256 of the oracle's full C (C-contiguous little-endian bytes), written by",
             "# make_full_oracle_hashes.py from oracle/ and the seeded inputs only.",
             "# workload | M N K | dtype | sha256"]
    for name, a_range in (("int8 8192", None), ("int4xint8 8192", (-8, 7))):
        t0 = time.time()
        A, B = (inputs.int8_pair(8192, 8192, 8192, seed=0) if a_range is None else
                inputs.int8_pair(8192, 8192, 8192, seed=0, a_range=a_range))
        C = og.gemm_i64(A, B)
        assert np.abs(C).max() < 2**31
        lines.append("%s | 8192 8192 8192 | int32 | %s" % (name, digest(C.astype(np.int32))))
        print(lines[-1], "(%.0f s)" % (time.time() - t0), flush=True)
        del A, B, C
    for m in moduli():
        t0 = time.time()
        A, B = inputs.residue_pair(4096, 4096, 4096, m)
        C = og.gemm_mod(m, A, B)
        assert C.dtype == np.int32
        lines.append("residues mod %d | 4096 4096 4096 | int32 | %s" % (m, digest(C)))
        print(lines[-1], "(%.0f s)" % (time.time() - t0), flush=True)
    t0 = time.time()
    A, B = inputs.stress_operands(4096, 4096, 65536, seed=0)
    C = og.gemm_i64(np.ascontiguousarray(A), B)
    lines.append("stress | 4096 4096 65536 | int64 | %s" % digest(C))
    print(lines[-1], "(%.0f s)" % (time.time() - t0), flush=True)
    with open(os.path.join(HERE, "full_oracle_sha256.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
