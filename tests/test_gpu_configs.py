"""GPU parity at the benchmark workloads' full sizes, in the launch configuration the
benchmark times, against the oracle (bit-exact).

* 256^3 int8, base-13 and AWE6 (in test_gpu_gemm.py).
* 8192^3 int8, AWE6 and base-13, int32 C: the whole C against the oracle's (its SHA-256 in
  tests/golden/full_oracle_sha256.txt, written from the oracle by make_full_oracle_hashes.py),
  64 random 128 x 128 output tiles plus the 4 corner tiles against the oracle restricted to
  those tiles (which locate a difference), and a full 2048^3 product against the full oracle.
* 8192^3 int4 x int8, AWE4: the same checks.
* 4096^3 residues for every modulus of the FP64-significand residue set
  (tests/golden/moduli_fp64_k16384.txt): the whole C against the oracle's (its SHA-256 in
  tests/golden/full_oracle_sha256.txt, written from the oracle by
  make_full_oracle_hashes.py), sampled tiles to locate a difference, and a full 512^3.
* 4096 x 4096 x 65536 accumulation stress, AWE6, int64 C, default and forced fold
  segment: the whole C against the oracle's (SHA-256 as above), closed forms over the whole
  of C where they exist, plus sampled tiles.
"""
import os

import numpy as np
import pytest
import torch

from oracle import gemm as og
from paper_2609_24519_amd import awe, inputs
from tests.gpu_helpers import full_oracle_match, to_dev

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _moduli():
    with open(os.path.join(GOLDEN, "moduli_fp64_k16384.txt")) as f:
        lines = [l for l in f if l.strip() and not l.startswith("#")]
    return [int(x) for x in lines[0].split()]


def _check_tiles(C, A, B, tiles, mod=None):
    for rows, cols in tiles:
        a = np.ascontiguousarray(A[rows])
        b = np.ascontiguousarray(B[:, cols])
        ref = og.gemm_mod(mod, a, b) if mod else og.gemm_i64(a, b)
        got = C[rows][:, cols]
        assert np.array_equal(got.astype(np.int64), ref.astype(np.int64)), (rows[0], cols[0])


def _exact_on_gpu(enc, A, B, out=torch.int32):
    C = awe.matmul_exact(to_dev(A), to_dev(B), enc, out)
    torch.cuda.synchronize()
    host = C.cpu().numpy()
    del C
    torch.cuda.empty_cache()
    return host


@pytest.fixture(scope="module")
def int8_8192():
    return inputs.int8_pair(8192, 8192, 8192, seed=0)


@pytest.mark.parametrize("enc", [awe.ENC_AWE6, awe.ENC_B13])
def test_config2_int8_8192(int8_8192, enc):
    A, B = int8_8192
    C = _exact_on_gpu(enc, A, B)
    full_ok = full_oracle_match(C, "int8 8192", (8192, 8192), "int32")
    _check_tiles(C, A, B, inputs.sample_tiles(8192, 8192, 64, 128, seed=1))
    assert full_ok, "whole C differs from the oracle's (sampled tiles agree)"


@pytest.mark.parametrize("enc", [awe.ENC_AWE6, awe.ENC_B13])
def test_config2_full_2048(enc):
    A, B = inputs.int8_pair(2048, 2048, 2048, seed=0)
    C = _exact_on_gpu(enc, A, B)
    assert np.array_equal(C.astype(np.int64), og.gemm_i64(A, B))


def test_config3_int4_int8_8192():
    A, B = inputs.int8_pair(8192, 8192, 8192, seed=0, a_range=(-8, 7))
    C = _exact_on_gpu(awe.ENC_AWE4, A, B)
    full_ok = full_oracle_match(C, "int4xint8 8192", (8192, 8192), "int32")
    _check_tiles(C, A, B, inputs.sample_tiles(8192, 8192, 64, 128, seed=1))
    assert full_ok, "whole C differs from the oracle's (sampled tiles agree)"


def test_config3_full_2048():
    A, B = inputs.int8_pair(2048, 2048, 2048, seed=0, a_range=(-8, 7))
    C = _exact_on_gpu(awe.ENC_AWE4, A, B)
    assert np.array_equal(C.astype(np.int64), og.gemm_i64(A, B))


@pytest.mark.parametrize("m", _moduli())
def test_config4_residues_4096(m):
    A, B = inputs.residue_pair(4096, 4096, 4096, m)
    C = awe.matmul_mod(m, to_dev(A), to_dev(B))
    torch.cuda.synchronize()
    Ch = C.cpu().numpy()
    del C
    assert Ch.min() >= 0 and Ch.max() < m
    full_ok = full_oracle_match(Ch, "residues mod %d" % m, (4096, 4096), "int32")
    # sampled tiles locate a difference; the whole C must match the oracle's in any case
    _check_tiles(Ch, A, B, inputs.sample_tiles(4096, 4096, 12, 128, seed=m), mod=m)
    assert full_ok, "C mod %d differs from the oracle's full product" % m
    a, b = inputs.residue_pair(512, 512, 512, m, seed=m + 1000)
    Cs = awe.matmul_mod(m, to_dev(a), to_dev(b))
    torch.cuda.synchronize()
    assert np.array_equal(Cs.cpu().numpy(), og.gemm_mod(m, a, b))


@pytest.fixture(scope="module")
def stress():
    return inputs.stress_operands(4096, 4096, 65536, seed=0)


def _stress_closed_forms(C, A, B, K):
    lo, hi = -128, 127
    h = K // 2
    t = np.arange(C.shape[0]) % 4
    u = np.arange(C.shape[1]) % 4
    closed = {(0, 0): K * lo * lo, (0, 1): K * lo * hi, (1, 1): K * hi * hi,
              (3, 3): h * (lo * lo + hi * hi), (0, 3): h * (lo * lo + lo * hi),
              (1, 3): h * (hi * lo + hi * hi)}
    for (x, y), val in closed.items():
        for p, q in ((x, y), (y, x)):
            blk = C[np.ix_(t == p, u == q)]
            assert (blk == val).all(), (p, q)
    # random-sign rows against constant columns: the row sum times the constant
    rs = A[t == 2].astype(np.int64).sum(axis=1)
    assert np.array_equal(C[np.ix_(t == 2, u == 0)], np.outer(rs, np.ones((u == 0).sum(), np.int64)) * lo)
    cs = B[:, u == 2].astype(np.int64).sum(axis=0)
    assert np.array_equal(C[np.ix_(t == 1, u == 2)], np.outer(np.ones((t == 1).sum(), np.int64), cs) * hi)
    assert C.max() == 2 ** 30  # -128 * -128 * 65536


@pytest.mark.parametrize("kseg", [0, 4096])
def test_config5_stress_65536(stress, kseg):
    A, B = stress
    M, K = A.shape
    N = B.shape[1]
    enc = awe.ENC_AWE6
    pa = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_A, M, K), dtype=torch.uint8, device="cuda")
    pb = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_B, N, K), dtype=torch.uint8, device="cuda")
    Ad, Bd = to_dev(A), to_dev(B)
    awe.encode(enc, 0, awe.SIDE_A, Ad, M, K, K, pa)
    awe.encode(enc, 0, awe.SIDE_B, Bd, N, K, N, pb)
    del Ad, Bd
    C = torch.empty((M, N), dtype=torch.int64, device="cuda")
    awe.gemm_planes(enc, 0, M, N, K, pa, pb, C, N, awe.I64, kseg)
    torch.cuda.synchronize()
    Ch = C.cpu().numpy()
    del C, pa, pb
    torch.cuda.empty_cache()
    full_ok = full_oracle_match(Ch, "stress", (4096, 4096), "int64")
    _stress_closed_forms(Ch, A, B, K)
    _check_tiles(Ch, A, B, inputs.sample_tiles(M, N, 4, 64, seed=5))
    assert full_ok, "the stress product differs from the oracle's full product"
