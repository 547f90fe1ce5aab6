"""GPU parity of the exact product against the oracle's plain int64 GEMM (bit-exact).

Small and ragged shapes that span several 256 x 128 tiles and a ragged tail,
every encoding, both output types, forced small fold segments, reduction
lengths that need several launches, the FP32 partial near its 2^23 bound,
and the degenerate sizes.
"""
import numpy as np
import pytest
import torch

from oracle import gemm as og
from paper_2609_24519_amd import awe, inputs
from tests.gpu_helpers import full_oracle_match, to_dev

pytestmark = pytest.mark.gpu

EXACT = [awe.ENC_B13, awe.ENC_AWE6, awe.ENC_AWE6ALT, awe.ENC_AWE4, awe.ENC_TERNARY, awe.ENC_FP8FP4,
         awe.ENC_FP6K3, awe.ENC_FP6P4]


def _run_exact(enc, A, B, out=torch.int32):
    Ad, Bd = to_dev(A), to_dev(B)
    C = awe.matmul_exact(Ad, Bd, enc, out)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def _operands(enc, M, N, K, seed):
    a_range = {awe.ENC_AWE4: (-8, 7), awe.ENC_TERNARY: (-1, 1)}.get(enc, (-128, 127))
    return inputs.int8_pair(M, N, K, seed, a_range=a_range)


def test_config1_256_cubed():
    A, B = inputs.int8_pair(256, 256, 256, seed=0)
    ref = og.gemm_i64(A, B)
    for enc in (awe.ENC_B13, awe.ENC_AWE6):
        C = _run_exact(enc, A, B)
        assert C.dtype == np.int32
        assert np.array_equal(C.astype(np.int64), ref), enc


@pytest.mark.parametrize("enc", EXACT)
@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (33, 65, 129), (300, 200, 333), (513, 129, 1000),
                                   (64, 256, 64), (31, 17, 4097)])
def test_ragged_shapes(enc, M, N, K):
    A, B = _operands(enc, M, N, K, seed=M + N + K)
    C = _run_exact(enc, A, B)
    assert np.array_equal(C.astype(np.int64), og.gemm_i64(A, B))


@pytest.mark.parametrize("enc", EXACT)
def test_int64_output(enc):
    A, B = _operands(enc, 97, 300, 700, seed=5)
    C = _run_exact(enc, A, B, torch.int64)
    assert C.dtype == np.int64 and np.array_equal(C, og.gemm_i64(A, B))


def test_extremes():
    # every entry at an end of the int8 range; the two's-complement end -128 included
    M, N, K = 64, 96, 2048
    A, B = inputs.stress_operands(M, N, K, seed=3)
    ref = og.gemm_i64(A, B)
    for enc in (awe.ENC_B13, awe.ENC_AWE6, awe.ENC_AWE6ALT, awe.ENC_FP8FP4, awe.ENC_FP6K3, awe.ENC_FP6P4):
        assert np.array_equal(_run_exact(enc, A, B).astype(np.int64), ref), enc
    A4 = np.where(A < 0, -8, 7).astype(np.int8)
    assert np.array_equal(_run_exact(awe.ENC_AWE4, A4, B).astype(np.int64), og.gemm_i64(A4, B))


def test_zero_k_and_empty():
    A = np.zeros((40, 0), np.int8)
    B = np.zeros((0, 50), np.int8)
    C = _run_exact(awe.ENC_AWE6, A, B)
    assert C.shape == (40, 50) and not C.any()
    C = awe.matmul_exact(to_dev(np.zeros((0, 8), np.int8)), to_dev(np.zeros((8, 5), np.int8)))
    assert tuple(C.shape) == (0, 5)


def _planes(enc, m, A, B):
    M, K = A.shape
    N = B.shape[1]
    pa = torch.empty(max(awe.plane_bytes(enc, m, awe.SIDE_A, M, K), 1), dtype=torch.uint8, device="cuda")
    pb = torch.empty(max(awe.plane_bytes(enc, m, awe.SIDE_B, N, K), 1), dtype=torch.uint8, device="cuda")
    Ad, Bd = to_dev(A), to_dev(B)
    awe.encode(enc, m, awe.SIDE_A, Ad, M, K, K, pa)
    awe.encode(enc, m, awe.SIDE_B, Bd, N, K, N, pb)
    return pa, pb


@pytest.mark.parametrize("enc", EXACT)
@pytest.mark.parametrize("kseg", [awe.K_PAD, 2 * awe.K_PAD, 4 * awe.K_PAD])
def test_forced_fold_segments(enc, kseg):
    # (capped at the encoding's own segment: the weights-in-scales scheme folds every 768)
    kseg = min(kseg, awe.get_encoding_info(enc)["k_seg"])
    M, N, K = 130, 260, 2000
    A, B = _operands(enc, M, N, K, seed=11)
    pa, pb = _planes(enc, 0, A, B)
    C = torch.empty((M, N), dtype=torch.int32, device="cuda")
    awe.gemm_planes(enc, 0, M, N, K, pa, pb, C, N, awe.I32, kseg)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy().astype(np.int64), og.gemm_i64(A, B))


def test_concurrent_streams():
    # the library keeps no device state between calls: two GEMMs of different encodings and
    # shapes enqueued on two streams at once (default priority) both stay exact
    A1, B1 = _operands(awe.ENC_AWE6, 700, 500, 3000, seed=31)
    A2, B2 = _operands(awe.ENC_FP6P4, 600, 900, 2100, seed=32)
    pa1, pb1 = _planes(awe.ENC_AWE6, 0, A1, B1)
    pa2, pb2 = _planes(awe.ENC_FP6P4, 0, A2, B2)
    torch.cuda.synchronize()
    C1 = torch.empty((700, 500), dtype=torch.int32, device="cuda")
    C2 = torch.empty((600, 900), dtype=torch.int64, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(3):
        awe.gemm_planes(awe.ENC_AWE6, 0, 700, 500, 3000, pa1, pb1, C1, 500, awe.I32, 0, s1)
        awe.gemm_planes(awe.ENC_FP6P4, 0, 600, 900, 2100, pa2, pb2, C2, 900, awe.I64, 0, s2)
    torch.cuda.synchronize()
    assert np.array_equal(C1.cpu().numpy().astype(np.int64), og.gemm_i64(A1, B1))
    assert np.array_equal(C2.cpu().numpy(), og.gemm_i64(A2, B2))


def test_graph_capture_replays():
    # encode A, encode B and the GEMM captured into one HIP graph (after an eager call, which
    # also sets the kernels' LDS limits): every replay, with eager work and synchronisations in
    # between, gives the exact product; nothing in these calls records a memset
    M, N, K = 520, 300, 1500
    A, B = _operands(awe.ENC_AWE6, M, N, K, seed=41)
    Ad, Bd = to_dev(A), to_dev(B)
    pa = torch.empty(awe.plane_bytes(awe.ENC_AWE6, 0, awe.SIDE_A, M, K), dtype=torch.uint8, device="cuda")
    pb = torch.empty(awe.plane_bytes(awe.ENC_AWE6, 0, awe.SIDE_B, N, K), dtype=torch.uint8, device="cuda")
    C = torch.empty((M, N), dtype=torch.int32, device="cuda")

    def step():
        awe.encode(awe.ENC_AWE6, 0, awe.SIDE_A, Ad, M, K, K, pa)
        awe.encode(awe.ENC_AWE6, 0, awe.SIDE_B, Bd, N, K, N, pb)
        awe.gemm_planes(awe.ENC_AWE6, 0, M, N, K, pa, pb, C, N, awe.I32)

    ref = og.gemm_i64(A, B)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        step()
    for rep in range(3):
        C.fill_(-7)
        pa.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(C.cpu().numpy().astype(np.int64), ref), rep


def test_ldc_larger_than_n():
    M, N, K = 70, 50, 300
    A, B = inputs.int8_pair(M, N, K, seed=2)
    pa, pb = _planes(awe.ENC_AWE6, 0, A, B)
    C = torch.full((M, 64), -7, dtype=torch.int32, device="cuda")
    awe.gemm_planes(awe.ENC_AWE6, 0, M, N, K, pa, pb, C, 64, awe.I32)
    torch.cuda.synchronize()
    Cn = C.cpu().numpy()
    assert np.array_equal(Cn[:, :N].astype(np.int64), og.gemm_i64(A, B))
    assert (Cn[:, N:] == -7).all()


def test_multi_launch_reduction():
    # K beyond what one launch's int32 accumulator may hold (130816 for int8 x int8): the
    # host splits the reduction and the launches add into the int64 output
    M, N, K = 40, 72, 300_000
    A, B = inputs.int8_pair(M, N, K, seed=9)
    ref = og.gemm_i64(A, B)
    for enc in (awe.ENC_AWE6, awe.ENC_FP6K3, awe.ENC_FP6P4):
        C = _run_exact(enc, A, B, torch.int64)
        assert np.array_equal(C, ref), enc


def test_fp32_partial_near_bound_fp6k3():
    # the 3-product E2M3 scheme: c_A c_B = 15 * 15 (the sum plane of x = -120 is -8 - 7 = -15),
    # default fold segment 37,120, so with A = B = -120 the sum plane's FP32 partial reaches
    # 225 * 37120 = 8,352,000, just below 2^23, before its fold with coefficient 16
    info = awe.get_encoding_info(awe.ENC_FP6K3)
    K = info["k_seg"]
    assert 225 * K < 2 ** 23 <= 225 * (K + awe.K_PAD)
    lo, T = awe.get_plane_table(awe.ENC_FP6K3, 0, awe.SIDE_A)
    assert list(T[-120 - lo]) == [-8, -7, -15]
    A = np.full((32, K), -120, np.int8)
    B = np.full((K, 48), -120, np.int8)
    B[:, 1::2] = 127
    C = _run_exact(awe.ENC_FP6K3, A, B, torch.int32)
    assert np.array_equal(C.astype(np.int64), og.gemm_i64(A, B))


def test_fp32_partial_near_bound():
    # AWE4: c_A c_B = 24, default fold segment = the largest multiple of K_PAD not above
    # (2^23 - 1) / 24 (349440), so one FP32 partial reaches 24 * 349440 = 8386560, just below
    # 2^23; constant operands put every product at its largest magnitude
    info = awe.get_encoding_info(awe.ENC_AWE4)
    K = info["k_seg"]
    assert K % awe.K_PAD == 0 and 24 * K < 2 ** 23 <= 24 * (K + awe.K_PAD)
    loa, TA = awe.get_plane_table(awe.ENC_AWE4, 0, awe.SIDE_A)
    lob, TB = awe.get_plane_table(awe.ENC_AWE4, 0, awe.SIDE_B)
    xs = [x for x in range(loa, loa + TA.shape[0]) if np.abs(TA[x - loa]).max() == 3]
    ys = [y for y in range(lob, lob + TB.shape[0]) if np.abs(TB[y - lob]).max() == 8]
    M = N = 32
    A = np.empty((M, K), np.int8)
    B = np.empty((K, N), np.int8)
    for i in range(M):
        A[i] = xs[i % len(xs)]
    for j in range(N):
        B[:, j] = ys[(7 * j) % len(ys)]
    C = _run_exact(awe.ENC_AWE4, A, B, torch.int64)
    ref = np.outer(A[:, 0].astype(np.int64), B[0].astype(np.int64)) * K
    assert np.array_equal(C, ref)


@pytest.mark.parametrize("m", [2, 9, 13, 31, 53, 89, 149, 157])
def test_mod_parity(m):
    A, B = inputs.residue_pair(190, 140, 777, m)
    Ad, Bd = to_dev(A), to_dev(B)
    C = awe.matmul_mod(m, Ad, Bd)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy(), og.gemm_mod(m, A, B))


def test_mod_forced_segments():
    m = 157
    A, B = inputs.residue_pair(64, 200, 3000, m)
    pa, pb = _planes(awe.ENC_MOD, m, A, B)
    C = torch.empty((64, 200), dtype=torch.int32, device="cuda")
    awe.gemm_planes(awe.ENC_MOD, m, 64, 200, 3000, pa, pb, C, 200, awe.I32, awe.K_PAD)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy(), og.gemm_mod(m, A, B))


@pytest.mark.parametrize("cfg", ["1", "2", "4", "5", "6", "7", "8", "9", "10", "12", "13", "15", "16", "17"])
@pytest.mark.parametrize("enc", [awe.ENC_AWE6, awe.ENC_AWE4, awe.ENC_B13, awe.ENC_TERNARY])
def test_every_tile_configuration(monkeypatch, cfg, enc):
    # AWE_GEMM_CFG forces one of the GEMM's tile configurations (256x128 on 8 waves with
    # 2 or 4 k-steps per stage, 256x192 on 8 waves in 2 or 5 stages, fragments read one or
    # three k-steps ahead or in place, 32x32x64 or 16x16x128 MFMAs, 256x256 with part of
    # the int32 fold accumulators in LDS, copies issued before or after the first MFMAs of a
    # stage); every one must give the exact product
    monkeypatch.setenv("AWE_GEMM_CFG", cfg)
    monkeypatch.setenv("AWE_GEMM_ALLPAIRS", "0")  # base-13 on the product-major stream here
    M, N, K = 300, 420, 1100
    A, B = _operands(enc, M, N, K, seed=int(cfg) + 40)
    C = _run_exact(enc, A, B)
    assert np.array_equal(C.astype(np.int64), og.gemm_i64(A, B))
    m = 89
    Ar, Br = inputs.residue_pair(130, 270, 600, m)
    Cm = awe.matmul_mod(m, to_dev(Ar), to_dev(Br))
    torch.cuda.synchronize()
    assert np.array_equal(Cm.cpu().numpy(), og.gemm_mod(m, Ar, Br))



@pytest.mark.parametrize("cfg", ["16", "17"])
@pytest.mark.parametrize("shape,kseg,out", [
    ((256, 256, 1), 0, torch.int32),        # the whole reduction in 2 stages: copies past its end
    ((300, 420, 257), 0, torch.int32),      # 4 stages, ragged tiles
    ((512, 512, 1024), 0, torch.int32),     # whole 256 x 256 tiles (16-byte row epilogue)
    ((512, 256, 3000), 256, torch.int32),   # a fold every 2 stages, whole tiles
    ((260, 520, 1500), 512, torch.int64),   # int64 C, ragged, a fold every 4 stages
])
def test_long_reduction_schedules_edges(monkeypatch, cfg, shape, kseg, out):
    # configs 16 and 17 (256 x 256, copies between the MFMAs, fragments read during the k-step
    # before, config 17's barrier inside the second k-step; 17 is the default for long
    # reductions): reductions of a few stages, forced fold segments, whole and ragged tiles
    monkeypatch.setenv("AWE_GEMM_CFG", cfg)
    M, N, K = shape
    enc = awe.ENC_AWE6
    A, B = _operands(enc, M, N, K, seed=K % 97 + int(cfg))
    pa, pb = _planes(enc, 0, A, B)
    C = torch.empty((M, N), dtype=out, device="cuda")
    awe.gemm_planes(enc, 0, M, N, K, pa, pb, C, N, awe.I64 if out == torch.int64 else awe.I32, kseg)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy().astype(np.int64), og.gemm_i64(A, B))


def test_ternary_4096_sampled():
    # {0, +-1} x INT8 (Sec. 6.2) at 4096 x 4096 x 8192, int32 C, sampled tiles
    M = N = 4096
    K = 8192
    A, B = inputs.int8_pair(M, N, K, seed=3, a_range=(-1, 1))
    C = awe.matmul_exact(to_dev(A), to_dev(B), awe.ENC_TERNARY, torch.int32)
    torch.cuda.synchronize()
    Ch = C.cpu().numpy()
    for rows, cols in inputs.sample_tiles(M, N, 16, 128, seed=2):
        ref = og.gemm_i64(np.ascontiguousarray(A[rows]), np.ascontiguousarray(B[:, cols]))
        assert np.array_equal(Ch[rows][:, cols].astype(np.int64), ref)



@pytest.mark.parametrize("allpairs", ["1", "0"])
@pytest.mark.parametrize("shape,out", [((70, 45, 500), torch.int32), ((130, 260, 2000), torch.int64),
                                       ((33, 40, 16384), torch.int64), ((16, 24, 120_000), torch.int64),
                                       ((300, 420, 70_000), torch.int64)])
def test_fp16_12_products(monkeypatch, allpairs, shape, out):
    # App. A: 12-bit integers (FP16 significands) in 12 FP4 products, by default one launch per
    # reduction range in which each stage brings planes t and t + 3 of each side for the four
    # products (t, k, l) into one accumulator per outer weight 71^(k+l); with
    # AWE_GEMM_ALLPAIRS=0, one launch per outer weight; the last shapes need several reduction
    # launches (and, the last, several fold segments)
    monkeypatch.setenv("AWE_GEMM_ALLPAIRS", allpairs)
    M, N, K = shape
    rng = np.random.default_rng(M + N + K)
    A = inputs.uniform(rng, (M, K), -2048, 2047, np.int16)
    B = inputs.uniform(rng, (K, N), -2048, 2047, np.int16)
    A[0, :] = -2048
    B[:, 0] = -2048
    C = awe.matmul_exact(to_dev(A), to_dev(B), awe.ENC_FP16, out)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy().astype(np.int64), og.gemm_i64_wide(A, B))



def test_fp8fp4_4096_sampled():
    # App. A's 2 FP8 + 1 FP4 scheme at 4096 x 4096 x 8192, int32 C, sampled tiles; the two
    # E4M3 products and the E2M1 product run as two launches adding into C
    M = N = 4096
    K = 8192
    A, B = inputs.int8_pair(M, N, K, seed=4)
    C = awe.matmul_exact(to_dev(A), to_dev(B), awe.ENC_FP8FP4, torch.int32)
    torch.cuda.synchronize()
    Ch = C.cpu().numpy()
    for rows, cols in inputs.sample_tiles(M, N, 16, 128, seed=6):
        ref = og.gemm_i64(np.ascontiguousarray(A[rows]), np.ascontiguousarray(B[:, cols]))
        assert np.array_equal(Ch[rows][:, cols].astype(np.int64), ref)


@pytest.mark.parametrize("cfg,cus", [("5", "12"), ("6", "16"), ("12", "12"), ("13", "12"), ("15", "12"), ("16", "12"), ("17", "12")])
@pytest.mark.parametrize("enc,out", [(awe.ENC_AWE6, torch.int32), (awe.ENC_AWE4, torch.int64),
                                     (awe.ENC_FP8FP4, torch.int32), (awe.ENC_FP16, torch.int64),
                                     (awe.ENC_FP6K3, torch.int32), (awe.ENC_FP6P4, torch.int32)])
def test_split_last_round(monkeypatch, cfg, cus, enc, out):
    # AWE_GEMM_CUS plans the rounds of workgroups for fewer CUs, so that this shape has a
    # ragged last round (30 tiles on 12 CUs, 20 tiles on 16) whose tiles are split along
    # the reduction into parts that add into C with atomics; the result must stay exact
    # (for D = 2, with launch groups adding into C, and with E4M3 operands)
    monkeypatch.setenv("AWE_GEMM_CFG", cfg)
    monkeypatch.setenv("AWE_GEMM_CUS", cus)
    M, N, K = 1100, 700, 2100
    if enc == awe.ENC_FP16:
        rng = np.random.default_rng(8)
        A = inputs.uniform(rng, (M, K), -2048, 2047, np.int16)
        B = inputs.uniform(rng, (K, N), -2048, 2047, np.int16)
        ref = og.gemm_i64_wide(A, B)
    else:
        A, B = _operands(enc, M, N, K, seed=12)
        ref = og.gemm_i64(A, B)
    C = awe.matmul_exact(to_dev(A), to_dev(B), enc, out)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy().astype(np.int64), ref)


@pytest.mark.parametrize("cfg", ["0", "1", "3", "5", "6"])
def test_every_e2m3_tile_configuration(monkeypatch, cfg):
    # AWE_GEMM_CFG_E2M3 forces one of the E2M3 tile configurations (256x128 on 8 waves
    # in 3 or 4 stages, with 4 k-steps per stage; 256x192 on 8 waves with fragments read in
    # place and the int32 fold accumulators of 1 or 2 blocks per wave in LDS); each must be
    # exact, also with a forced fold segment of one K_PAD
    monkeypatch.setenv("AWE_GEMM_CFG_E2M3", cfg)
    M, N, K = 300, 420, 1100
    A, B = _operands(awe.ENC_FP6K3, M, N, K, seed=int(cfg) + 70)
    ref = og.gemm_i64(A, B)
    assert np.array_equal(_run_exact(awe.ENC_FP6K3, A, B).astype(np.int64), ref)
    pa, pb = _planes(awe.ENC_FP6K3, 0, A, B)
    C = torch.empty((M, N), dtype=torch.int64, device="cuda")
    awe.gemm_planes(awe.ENC_FP6K3, 0, M, N, K, pa, pb, C, N, awe.I64, awe.K_PAD)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy(), ref)


def test_fp6k3_8192():
    # INT8 x INT8 in 3 E2M3 products at 8192^3 (the benchmark's shape and launch), int32 C: the
    # whole C against the oracle's (by its SHA-256), sampled 128 x 128 tiles plus the four corner
    # tiles to locate a difference
    M = N = K = 8192
    A, B = inputs.int8_pair(M, N, K, seed=0)
    C = awe.matmul_exact(to_dev(A), to_dev(B), awe.ENC_FP6K3, torch.int32)
    torch.cuda.synchronize()
    Ch = C.cpu().numpy()
    full_ok = full_oracle_match(Ch, "int8 8192", (M, N), "int32")
    for rows, cols in inputs.sample_tiles(M, N, 16, 128, seed=1):
        ref = og.gemm_i64(np.ascontiguousarray(A[rows]), np.ascontiguousarray(B[:, cols]))
        assert np.array_equal(Ch[rows][:, cols].astype(np.int64), ref)
    assert full_ok, "whole C differs from the oracle's (sampled tiles agree)"


@pytest.mark.parametrize("cfg", ["0", "1"])
def test_shared_accumulator_configurations(monkeypatch, cfg):
    # INT8 x INT8 in 4 E2M3 products with the weights in the block scales: both tile
    # configurations (fragments read ahead or in place), the default fold segment and a
    # forced one of one K_PAD, and the accumulator near its bound: x = y = 120 makes every
    # reduction index add 18,496 in absolute terms, and the default segment (768 indices)
    # brings the FP32 accumulator to 14,400 * 768 = 11,059,200 of 2^24
    monkeypatch.setenv("AWE_GEMM_CFG_SHARED", cfg)
    M, N, K = 300, 420, 1100
    A, B = _operands(awe.ENC_FP6P4, M, N, K, seed=int(cfg) + 90)
    A[:7, :] = 120
    B[:, :5] = 120
    ref = og.gemm_i64(A, B)
    assert np.array_equal(_run_exact(awe.ENC_FP6P4, A, B).astype(np.int64), ref)
    pa, pb = _planes(awe.ENC_FP6P4, 0, A, B)
    C = torch.empty((M, N), dtype=torch.int64, device="cuda")
    awe.gemm_planes(awe.ENC_FP6P4, 0, M, N, K, pa, pb, C, N, awe.I64, awe.K_PAD)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy(), ref)


def test_fp6p4_8192():
    # the weights-in-scales scheme at 8192^3 (the benchmark's shape and launch), int32 C: the
    # whole C against the oracle's (by its SHA-256), sampled tiles to locate a difference
    M = N = K = 8192
    A, B = inputs.int8_pair(M, N, K, seed=0)
    C = awe.matmul_exact(to_dev(A), to_dev(B), awe.ENC_FP6P4, torch.int32)
    torch.cuda.synchronize()
    Ch = C.cpu().numpy()
    full_ok = full_oracle_match(Ch, "int8 8192", (M, N), "int32")
    for rows, cols in inputs.sample_tiles(M, N, 16, 128, seed=3):
        ref = og.gemm_i64(np.ascontiguousarray(A[rows]), np.ascontiguousarray(B[:, cols]))
        assert np.array_equal(Ch[rows][:, cols].astype(np.int64), ref)
    assert full_ok, "whole C differs from the oracle's (sampled tiles agree)"


@pytest.mark.parametrize("allpairs", ["1", "0"])
@pytest.mark.parametrize("shape,out,kseg", [((1, 1, 1), torch.int32, 0), ((300, 420, 1100), torch.int32, 0),
                                            ((129, 513, 3000), torch.int64, 256),
                                            ((700, 300, 2100), torch.int64, 512)])
def test_base13_all_pairs_stream(monkeypatch, allpairs, shape, out, kseg):
    # base-13's nine limb pairs with one accumulator per coefficient 13^(i + j): each stage
    # brings the three planes of each side once (default), or the product-major stream
    # (AWE_GEMM_ALLPAIRS=0); ragged shapes, both outputs, forced fold segments
    monkeypatch.setenv("AWE_GEMM_ALLPAIRS", allpairs)
    M, N, K = shape
    enc = awe.ENC_B13
    A, B = _operands(enc, M, N, K, seed=M + N + K)
    A[0, :] = -128
    B[:, 0] = -128
    pa, pb = _planes(enc, 0, A, B)
    C = torch.empty((M, N), dtype=out, device="cuda")
    awe.gemm_planes(enc, 0, M, N, K, pa, pb, C, N, awe.I64 if out == torch.int64 else awe.I32, kseg)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy().astype(np.int64), og.gemm_i64(A, B))


@pytest.mark.parametrize("cus", ["12", "16"])
def test_base13_all_pairs_split_last_round(monkeypatch, cus):
    # a ragged last round of 128 x 128 all-pairs tiles split along the reduction (atomics into C)
    monkeypatch.setenv("AWE_GEMM_CUS", cus)
    M, N, K = 1100, 700, 2100
    A, B = _operands(awe.ENC_B13, M, N, K, seed=13)
    C = awe.matmul_exact(to_dev(A), to_dev(B), awe.ENC_B13, torch.int32)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy().astype(np.int64), og.gemm_i64(A, B))

