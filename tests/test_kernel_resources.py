"""Register budget of the kernels, from the gfx950 code object (hipcc cross-compiles here,
no GPU needed): the GEMM configurations the library picks by default, the grouped GEMM and
every encoder, residue and reconstruction kernel must run without scratch memory (a spill of
the accumulators to scratch costs the GEMM ~20 %)."""
import os
import shutil

import pytest

from paper_2609_24519_amd import build


# the configuration template's defaults, from the read-ahead on
_CFG_DEFAULTS = (4, 2, 2, 2, 2, 3, 1, 0, 1, 32, 0, 0, 0, 0, 1, 0)


def _cfg(*t):
    t = t + _CFG_DEFAULTS[len(t):]
    return "CfgI" + "".join("Li%dE" % v for v in t) + "EE"


# (waves M, waves N, blocks M, blocks N, k-steps per stage, stages, read-ahead, format, planes,
#  MFMA shape, blocks per wave whose int32 fold accumulators live in LDS, schedule, all-pairs planes
#  of A and B, plane step, outer groups)
DEFAULTS = {
    "E2M1 256x128, 3 k-steps ahead (default for smaller shapes)": _cfg(4, 2, 2, 2, 4, 3, 3, 0, 1, 32, 0),
    "E2M1 256x192, 4 k-steps per stage": _cfg(4, 2, 2, 3, 4, 2, 1, 0, 1, 32, 0),
    "E2M1 256x192, 5 stages": _cfg(4, 2, 2, 3, 2, 5, 1, 0, 1, 32, 0),
    "E2M1 256x192, in place": _cfg(4, 2, 2, 3, 4, 2, 0, 0, 1, 32, 0),
    "E2M1 256x128, 16x16x128": _cfg(4, 2, 2, 2, 4, 3, 1, 0, 1, 16, 0),
    "E2M1 256x128, 16x16x128, in place": _cfg(4, 2, 2, 2, 4, 3, 0, 0, 1, 16, 0),
    "E2M1 256x256, int32 fold of 3 blocks per wave in LDS": _cfg(4, 2, 2, 4, 2, 2, 0, 0, 1, 32, 3),
    "E2M1 256x256, int32 fold of 2 blocks per wave in LDS, 3 stages": _cfg(4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2),
    "E4M3": _cfg(4, 2, 2, 2, 2, 3, 1, 1, 1, 32, 0),
    "E2M3 256x128, 4 k-steps per stage": _cfg(4, 2, 2, 2, 4, 2, 1, 2, 1, 32, 0),
    "E2M3 weights in the scales": _cfg(4, 2, 2, 2, 2, 2, 1, 2, 2, 32, 0),
    "E2M1 256x256, copies spread over the stage, fragments read a k-step ahead in place":
        _cfg(4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2, 2),
    "E2M1 256x256, as above with the barrier inside the second k-step (default)":
        _cfg(4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2, 3),
    "E2M1 base-13, all nine plane pairs in one stream": _cfg(4, 2, 1, 2, 2, 3, 0, 0, 1, 32, 0, 0, 3, 3),
    "E2M1 FP16 significands, outer groups": _cfg(4, 2, 1, 2, 2, 3, 0, 0, 1, 32, 0, 3, 2, 2, 3, 1),
}


@pytest.fixture(scope="module")
def rows():
    h = build.hipcc()
    if not (os.path.exists(h) or shutil.which(h)):
        pytest.skip("hipcc not found")
    return build.kernel_resources()


# The E2M3 default (256x192, the fold accumulators of 1 block per wave in LDS) spills one
# 4-byte value: a store before the reduction loop and a reload after it, outside the loop, and
# it runs 6-8 % faster than the E2M3 configuration without spills.  No more than that.
# The E2M1 256x256 tile with the copies spread over the stage and each k-step's fragments read
# right before its MFMAs spills one 4-byte value the same way: its 16-byte row epilogue needs one
# register more than the loop leaves.
SMALL_SPILL = {"E2M3 256x192, 1 fold block per wave in LDS (default)": _cfg(4, 2, 2, 3, 2, 3, 0, 2, 1, 32, 1),
               "E2M1 256x256, the copies spread over the stage": _cfg(4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2, 1)}


def test_default_gemm_configurations_do_not_spill(rows):
    for label, frag in DEFAULTS.items():
        hits = [r for r in rows if "gemm_kernel" in r[0] and "group" not in r[0] and frag in r[0]]
        assert hits, label
        for r in hits:
            assert r[4] == 0 and r[7] == 0, (label, r)
    for label, frag in SMALL_SPILL.items():
        hits = [r for r in rows if "gemm_kernel" in r[0] and "group" not in r[0] and frag in r[0]]
        assert hits, label
        for r in hits:
            assert r[4] <= 1 and r[7] <= 8, (label, r)
    groups = [r for r in rows if "gemm_group_kernel" in r[0]]
    assert groups and all(r[4] == 0 and r[7] == 0 for r in groups), groups


def test_other_kernels_use_no_scratch(rows):
    for r in rows:
        if "gemm" in r[0]:
            continue
        assert r[7] == 0, r


def test_encoders_keep_four_waves_per_simd(rows):
    # The byte encoders are HBM-bound and need four waves per SIMD (at most 128 registers) to keep
    # enough loads in flight: at 148 registers (three waves) the B side took 15 % longer.
    enc = [r for r in rows if "13encode_kernel" in r[0]]
    assert len(enc) == 2, enc
    for r in enc:
        assert r[1] + r[2] <= 128, r
