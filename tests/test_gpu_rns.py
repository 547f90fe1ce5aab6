"""GPU parity of the residue-number-system route (Sec. 5.3) against the oracle:
residues of int64 matrices, the Chinese-remainder reconstruction (128-bit words and
nearest double), and the exact product of 53-bit integer matrices through the FP64
residue set (23 moduli) at K = 16,384."""
import os

import numpy as np
import pytest
import torch

from oracle import crt as ocrt
from oracle import gemm as og
from paper_2609_24519_amd import awe, inputs
from tests.gpu_helpers import to_dev

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
B53 = (1 << 53) - 1


def _moduli():
    with open(os.path.join(GOLDEN, "moduli_fp64_k16384.txt")) as f:
        lines = [l for l in f if l.strip() and not l.startswith("#")]
    return [int(x) for x in lines[0].split()]


def _words_to_ints(c128):
    w = c128.cpu().numpy().reshape(-1, 2)
    return np.array([(int(h) << 64) + (int(l) & ((1 << 64) - 1)) for l, h in w],
                    dtype=object).reshape(c128.shape[:-1])


@pytest.mark.parametrize("bits", [63, 53])
@pytest.mark.parametrize("shape", [(1, 1), (37, 129), (300, 65), (64, 1000), (3, 16, 0), (70, 256, 0),
                                   (5, 48, 16), (4, 40, 8)])
def test_residues(shape, bits):
    # (rows, cols[, ld - cols]): ld = cols + 3 reads entry by entry; cols and ld multiples
    # of 16 take the 16-entry vector path, whose groups of entries below 2^53 in magnitude
    # take the double-precision route (bits = 53: mostly those, with 2^53 itself and the
    # int64 ends mixed in)
    rows, cols = shape[:2]
    pad = shape[2] if len(shape) > 2 else 3
    # every modulus of the FP64 set, plus the extremes of the allowed range (residues
    # need no coprimality)
    ms = _moduli() + [2, 3, 255, 256]
    rng = np.random.default_rng(rows * 7 + cols + bits)
    lim = (1 << bits) - 1
    x = rng.integers(-lim - (bits == 63), lim, size=(rows, cols), dtype=np.int64, endpoint=True)
    edges = [-(1 << 63), (1 << 63) - 1, -1, 0, B53, -B53, 1 << 53, -(1 << 53)]
    x.ravel()[: min(len(edges), x.size)] = edges[: min(len(edges), x.size)]
    ld = cols + pad
    xp = np.zeros((rows, ld), dtype=np.int64)
    xp[:, :cols] = x
    xd = to_dev(xp)
    for chunk in (ms[:12], ms[12:]):
        if not chunk:
            continue
        out = torch.empty(len(chunk) * rows * cols, dtype=torch.uint8, device="cuda")
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        awe.residues(xd, rows, cols, ld, (1 << 63) - 1, chunk, out, rows * cols, flag)
        torch.cuda.synchronize()
        got = out.cpu().numpy().reshape(len(chunk), rows, cols)
        for j, m in enumerate(chunk):
            assert np.array_equal(got[j], ocrt.residues(x, m).astype(np.uint8)), m
        # the bound 2^63 - 1 excludes only -2^63, which the first entry holds
        assert int(flag.item()) == int(bool((x == np.iinfo(np.int64).min).any()))


def test_residues_range_flag():
    x = np.array([[B53, -B53, 0, B53 + 1]], dtype=np.int64)
    out = torch.empty(4, dtype=torch.uint8, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    awe.residues(to_dev(x), 1, 4, 4, B53, [13], out, 4, flag)
    torch.cuda.synchronize()
    assert int(flag.item()) != 0
    assert np.array_equal(out.cpu().numpy(), ocrt.residues(x[0], 13))


@pytest.mark.parametrize("moduli", ["fp64", "fp64_12", [3, 5, 7], [256, 255, 253, 251], [97], [256, 255],
                                    [13, 11, 9, 7, 5, 256, 251, 241, 239, 233]])
def test_crt_reconstruction(moduli):
    # 1 to 23 moduli: every digit-group shape of the Horner step (1, 2 or 3 digits in the top
    # group) and all three kernel widths (up to 8, 16 and 32 moduli)
    ms = _moduli() if moduli == "fp64" else (_moduli()[:12] if moduli == "fp64_12" else moduli)
    M = ocrt.modulus_product(ms)
    rng = np.random.default_rng(len(ms))
    rows, cols = 33, 70
    vals = [int.from_bytes(rng.bytes(16), "little") % M - M // 2 for _ in range(rows * cols)]
    edge = [0, 1, -1, M // 2, -(M // 2) + 1, M // 2 - 1]
    vals[: len(edge)] = edge
    X = np.array(vals, dtype=object).reshape(rows, cols)
    ld = cols + 5
    stride = rows * ld + 7
    res = np.zeros((len(ms), stride), dtype=np.int32)
    for j, m in enumerate(ms):
        r = np.vectorize(lambda v: v % m, otypes=[np.int64])(X)
        res[j, : rows * ld].reshape(rows, ld)[:, :cols] = r
    c128 = torch.empty((rows, cols, 2), dtype=torch.int64, device="cuda")
    c64 = torch.empty((rows, cols), dtype=torch.float64, device="cuda")
    awe.crt(to_dev(res), stride, rows, cols, ld, ms, c128, c64, cols)
    torch.cuda.synchronize()
    assert (_words_to_ints(c128) == X).all()
    assert np.array_equal(c64.cpu().numpy(), ocrt.to_double(X))


def test_crt_double_rounding_edges():
    # integers just around ties at several magnitudes: the double must be the
    # correctly rounded one (ties to even), including values with a nonzero high word
    ms = _moduli()
    vals = []
    for e in (53, 60, 64, 65, 80, 100, 118):
        base = 1 << e
        ulp = 1 << (e - 52)
        for d in (0, 1, ulp // 2 - 1, ulp // 2, ulp // 2 + 1, ulp - 1, ulp + ulp // 2):
            vals += [base + d, -(base + d)]
    X = np.array(vals, dtype=object).reshape(1, -1)
    n = X.shape[1]
    res = np.stack([np.vectorize(lambda v: v % m, otypes=[np.int64])(X).astype(np.int32).ravel()
                    for m in ms])
    c64 = torch.empty((1, n), dtype=torch.float64, device="cuda")
    awe.crt(to_dev(res), n, 1, n, n, ms, None, c64, n)
    torch.cuda.synchronize()
    assert np.array_equal(c64.cpu().numpy(), ocrt.to_double(X))


def _int53_pair(M, N, K, seed):
    rng = np.random.default_rng(seed)
    A = rng.integers(-B53, B53, size=(M, K), dtype=np.int64, endpoint=True)
    B = rng.integers(-B53, B53, size=(K, N), dtype=np.int64, endpoint=True)
    return A, B


@pytest.mark.parametrize("shape", [(40, 24, 16384), (33, 65, 1000), (5, 7, 1)])
def test_gemm_crt_full(shape):
    M, N, K = shape
    ms = _moduli()
    A, B = _int53_pair(M, N, K, seed=M + N + K)
    c128, c64 = awe.matmul_crt(to_dev(A), to_dev(B), ms, B53, B53)
    torch.cuda.synchronize()
    ref = og.gemm_i128(A, B)
    assert (_words_to_ints(c128) == ref).all()
    assert np.array_equal(c64.cpu().numpy(), ocrt.to_double(ref))


@pytest.mark.parametrize("grouped,cfg", [("1", None), ("0", None), ("1", "4"), ("1", "1"), ("1", "6"), ("1", "13"),
                                          ("1", "16"), ("1", "17")])
def test_gemm_crt_grouped_launch(monkeypatch, grouped, cfg):
    # the moduli's GEMMs run as one grouped launch (jobs with the most products first) or,
    # with AWE_GEMM_GROUPED=0 or a tile configuration the grouped kernel lacks (6, 17), one launch
    # per modulus; 9 tiles per modulus (256 x 128) are not a multiple of the 8 XCDs
    monkeypatch.setenv("AWE_GEMM_GROUPED", grouped)
    if cfg is not None:
        monkeypatch.setenv("AWE_GEMM_CFG", cfg)
    ms = _moduli()
    M, N, K = 700, 300, 2000
    A, B = _int53_pair(M, N, K, seed=5)
    c128, c64 = awe.matmul_crt(to_dev(A), to_dev(B), ms, B53, B53)
    torch.cuda.synchronize()
    ref = og.gemm_i128(A, B)
    assert (_words_to_ints(c128) == ref).all()
    assert np.array_equal(c64.cpu().numpy(), ocrt.to_double(ref))


def test_gemm_crt_split_reduction():
    # K beyond what one launch of modulus 147's scheme may reduce (about 165,000 indices for its
    # int32 partial sums): its residue product takes two launches, the second adding mod 147 into
    # the byte residues of the first; the other moduli take one launch each, so nothing is grouped
    ms = [147, 149, 151, 157, 139]
    M, N, K, bound = 32, 40, 200_000, 100
    rng = np.random.default_rng(7)
    A = rng.integers(-bound, bound, size=(M, K), dtype=np.int64, endpoint=True)
    B = rng.integers(-bound, bound, size=(K, N), dtype=np.int64, endpoint=True)
    c128, c64 = awe.matmul_crt(to_dev(A), to_dev(B), ms, bound, bound)
    torch.cuda.synchronize()
    ref = og.gemm_i128(A, B)
    assert (_words_to_ints(c128) == ref).all()
    assert np.array_equal(c64.cpu().numpy(), ocrt.to_double(ref))


def test_gemm_crt_extremes():
    # every product at the bound: C = -K B^2 needs 120 bits and the top of the range
    ms = _moduli()
    K = 16384
    A = np.full((32, K), B53, dtype=np.int64)
    B = np.full((K, 16), -B53, dtype=np.int64)
    B[:, 1::2] = B53
    c128, c64 = awe.matmul_crt(to_dev(A), to_dev(B), ms, B53, B53)
    torch.cuda.synchronize()
    got = _words_to_ints(c128)
    assert (got[:, 0::2] == -K * B53 * B53).all() and (got[:, 1::2] == K * B53 * B53).all()
    assert (c64.cpu().numpy()[:, 1] == float(K * B53 * B53)).all()


def test_gemm_crt_4096_sampled():
    # the FP64-significand workload: 4096 x 4096 x 16384, |entries| <= 2^53 - 1, 23 moduli
    ms = _moduli()
    M = N = 4096
    K = 16384
    A, B = _int53_pair(M, N, K, seed=0)
    c128, c64 = awe.matmul_crt(to_dev(A), to_dev(B), ms, B53, B53)
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    rows = np.concatenate([[0, M - 1], rng.choice(M, 30, replace=False)])
    cols = np.concatenate([[0, N - 1], rng.choice(N, 30, replace=False)])
    ref = og.gemm_i128_sampled(A, B, rows, cols)
    sub = c128[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")]
    assert (_words_to_ints(sub) == ref).all()
    sub64 = c64[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")]
    assert np.array_equal(sub64.cpu().numpy(), ocrt.to_double(ref))


def test_gemm_crt_range_flag_and_large_entries():
    # entries beyond the stated bound set the flag (both operands), and entries at or beyond
    # 2^53 (the integer residue route instead of the double one) still give exact residues;
    # the product stays within the moduli's range, so C is exact too
    ms = _moduli()
    M, N, K = 33, 40, 300
    rng = np.random.default_rng(21)
    A = rng.integers(-1000, 1000, size=(M, K), dtype=np.int64, endpoint=True)
    B = rng.integers(-1000, 1000, size=(K, N), dtype=np.int64, endpoint=True)
    for bound_a, bound_b, big in ((1000, 1000, False), (999, 1000, False), (1000, 999, False),
                                  (1 << 60, 1000, True)):
        Ai = A.copy()
        if big:
            Ai[3, 7] = (1 << 53) + 5  # a wave of A entries takes the integer route
            Ai[4, 9] = -(1 << 60)
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        c128, c64 = awe.matmul_crt(to_dev(Ai), to_dev(B), ms, bound_a, bound_b, flag)
        torch.cuda.synchronize()
        expect_flag = bool((np.abs(Ai) > bound_a).any() or (np.abs(B) > bound_b).any())
        assert bool(flag.item()) == expect_flag, (bound_a, bound_b)
        assert (_words_to_ints(c128) == og.gemm_i128(Ai, B)).all()
