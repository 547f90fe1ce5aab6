"""GPU encoder parity: stored planes, decoded from the documented layout, equal the
oracle's table lookup element by element (Alg. 1, first two loops)."""
import numpy as np
import pytest
import torch

from oracle import modm, schemes as sc
from paper_2609_24519_amd import awe, inputs
from tests.gpu_helpers import decode_planes, to_dev

pytestmark = pytest.mark.gpu

EXACT = {"b13": awe.ENC_B13, "awe6": awe.ENC_AWE6, "awe6_alt": awe.ENC_AWE6ALT, "awe4": awe.ENC_AWE4,
         "ternary": awe.ENC_TERNARY, "fp16_12": awe.ENC_FP16, "fp8fp4": awe.ENC_FP8FP4,
         "fp6k3": awe.ENC_FP6K3, "fp6p4": awe.ENC_FP6P4}


def _dtype(lo, hi):
    return np.int8 if -128 <= lo and hi <= 127 else np.int16


def _encode(enc, m, side, X, rows, K, flag=None):
    info = awe.get_encoding_info(enc, m)
    npl = info["planes_a"] if side == awe.SIDE_A else info["planes_b"]
    nbytes = awe.plane_bytes(enc, m, side, rows, K)
    # garbage first: the encoder must write every byte, padding included
    planes = torch.full((max(nbytes, 1),), 0xAB, dtype=torch.uint8, device="cuda")
    xd = to_dev(X)
    awe.encode(enc, m, side, xd, rows, K, X.shape[1], planes, flag)
    torch.cuda.synchronize()
    fmts = info["formats_a"] if side == awe.SIDE_A else info["formats_b"]
    return decode_planes(planes.cpu().numpy(), npl, rows, K, fmts)


@pytest.mark.parametrize("name", sorted(EXACT))
@pytest.mark.parametrize("rows,K", [(32, 128), (70, 200), (1, 1), (257, 333), (160, 1000)])
def test_encode_matches_oracle(name, rows, K):
    s = sc.ALL_SCHEMES[name]()
    rng = np.random.default_rng(rows * 1000 + K)
    A = inputs.uniform(rng, (rows, K), *s.range_a, dtype=_dtype(*s.range_a))
    got = _encode(EXACT[name], 0, awe.SIDE_A, A, rows, K)
    assert np.array_equal(got, sc.encode_planes(s, "a", A))
    B = inputs.uniform(rng, (K, rows), *s.range_b, dtype=_dtype(*s.range_b))  # K x N, N = rows
    got = _encode(EXACT[name], 0, awe.SIDE_B, B, rows, K)
    assert np.array_equal(got, np.swapaxes(sc.encode_planes(s, "b", B), 1, 2))


@pytest.mark.parametrize("m", [7, 31, 89, 157])
def test_encode_mod_matches_oracle(m):
    sch = modm.find_scheme(m)
    A, B = inputs.residue_pair(45, 37, 150, m)
    got = _encode(awe.ENC_MOD, m, awe.SIDE_A, A, 45, 150)
    assert np.array_equal(got, modm.encode_planes(sch, A))
    got = _encode(awe.ENC_MOD, m, awe.SIDE_B, B, 37, 150)
    assert np.array_equal(got, np.swapaxes(modm.encode_planes(sch, B), 1, 2))


def test_range_flag():
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    A = np.full((32, 64), 3, np.int8)
    _encode(awe.ENC_AWE4, 0, awe.SIDE_A, A, 32, 64, flag)
    assert flag.item() == 0
    A[5, 7] = 9  # outside int4
    got = _encode(awe.ENC_AWE4, 0, awe.SIDE_A, A, 32, 64, flag)
    assert flag.item() != 0
    assert not got[:, 5, 7].any()
    flag.zero_()
    R = np.full((40, 40), 12, np.uint8)
    _encode(awe.ENC_MOD, 13, awe.SIDE_B, R, 40, 40, flag)
    assert flag.item() == 0
    R[0, 0] = 13
    _encode(awe.ENC_MOD, 13, awe.SIDE_B, R, 40, 40, flag)
    assert flag.item() != 0


def test_encode_wide_range_flag():
    # int16 inputs of the FP16 scheme: values outside [-2048, 2047] raise the flag
    A = np.zeros((32, 64), dtype=np.int16)
    A[3, 5] = 2047
    A[7, 9] = -2048
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    _encode(awe.ENC_FP16, 0, awe.SIDE_A, A, 32, 64, flag)
    assert int(flag.item()) == 0
    A[8, 8] = 2048
    _encode(awe.ENC_FP16, 0, awe.SIDE_A, A, 32, 64, flag)
    assert int(flag.item()) != 0
