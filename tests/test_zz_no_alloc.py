"""The allocation-free entry point awe_gemm_exact_noalloc (planes in the library's fixed device
array) against awe_gemm_exact with a caller workspace and against the oracle: two calls in a
row, the second smaller, bit-exact; and the refusal of sizes whose planes exceed the array."""
import numpy as np
import pytest
import torch

from oracle import gemm as og
from paper_2609_24519_amd import awe, inputs
from tests.gpu_helpers import to_dev

pytestmark = pytest.mark.gpu


def _operands(enc, M, N, K, seed):
    if enc == awe.ENC_FP16:
        rng = np.random.default_rng(seed)
        return (inputs.uniform(rng, (M, K), -2048, 2047, np.int16),
                inputs.uniform(rng, (K, N), -2048, 2047, np.int16))
    a_range = (-8, 7) if enc == awe.ENC_AWE4 else (-128, 127)
    return inputs.int8_pair(M, N, K, seed=seed, a_range=a_range)


def _reference(enc, A, B):
    return og.gemm_i64_wide(A, B) if enc == awe.ENC_FP16 else og.gemm_i64(A, B)


@pytest.mark.parametrize("enc,out", [(awe.ENC_AWE6, torch.int32), (awe.ENC_B13, torch.int64),
                                     (awe.ENC_AWE4, torch.int32), (awe.ENC_FP6P4, torch.int32),
                                     (awe.ENC_FP16, torch.int64)])
def test_noalloc_matches_workspace_entry_point(enc, out):
    c_type = awe.I64 if out == torch.int64 else awe.I32
    for (M, N, K), seed in (((700, 900, 1300), 11), ((130, 70, 260), 12)):
        A, B = _operands(enc, M, N, K, seed)
        Ad, Bd = to_dev(A), to_dev(B)
        wsn = awe.workspace_bytes(enc, 0, M, N, K)
        ws = torch.empty(wsn, dtype=torch.uint8, device="cuda")
        Cw = torch.full((M, N), -7, dtype=out, device="cuda")
        awe.gemm_exact(enc, M, N, K, Ad, K, Bd, N, Cw, N, c_type, ws, wsn)
        Cn = torch.full((M, N), -9, dtype=out, device="cuda")
        awe.gemm_exact_noalloc(enc, M, N, K, Ad, K, Bd, N, Cn, N, c_type)
        torch.cuda.synchronize()
        got = Cn.cpu().numpy()
        assert np.array_equal(got, Cw.cpu().numpy()), (enc, M, N, K)
        assert np.array_equal(got.astype(np.int64), _reference(enc, A, B)), (enc, M, N, K)


def test_noalloc_refuses_planes_past_the_array():
    # AWE6 at 4096^3 needs 2 x 6 x 4096 x 4096 / 2 bytes of planes, past the 64 MiB array:
    # the call fails before anything is enqueued and C keeps its contents
    enc, n = awe.ENC_AWE6, 4096
    assert awe.workspace_bytes(enc, 0, n, n, n) > awe.NOALLOC_MAX_BYTES
    A = torch.zeros((n, n), dtype=torch.int8, device="cuda")
    C = torch.full((n, n), 5, dtype=torch.int32, device="cuda")
    with pytest.raises(awe.AweError) as ei:
        awe.gemm_exact_noalloc(enc, n, n, n, A, n, A, n, C, n, awe.I32)
    assert ei.value.status == awe.ERR_WORKSPACE and "fixed planes array" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((C == 5).all())
