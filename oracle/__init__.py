"""Oracle for the exact FP4-GEMM integer product (test infrastructure only).

This package is a plain, slow, CPU-only restatement of what the method
computes, written from the paper and independent of the HIP library: it shares
no code, table, header or constant generator with ``paper_2609_24519_amd``,
and neither imports the other.  Only ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import or execute it.

* ``gemm``    -- the plain definition C = A B (and C mod m), a C triple loop
                 with a 64-bit accumulator (128-bit for int64 operands),
                 loaded through ctypes.
* ``schemes`` -- the paper's encodings (storable set, limb tables, planes,
                 reconstruction coefficients, coverage, K*), the scheme
                 identity and the run-time procedure in plain numpy int64;
                 also the INT8 x INT8 variants in E2M3 (FP6) products: 3 by
                 the Karatsuba step that Sec. 3.3 admits, and 4 whose limb
                 weights ride in the E8M0 block scales (Sec. 4.5).
* ``modm``    -- the congruence (mod m) schemes and their tables.
* ``crt``     -- residues and the Chinese-remainder reconstruction of a
                 residue number system, in Python integers.
"""
