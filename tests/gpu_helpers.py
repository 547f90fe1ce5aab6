"""Helpers for the GPU tests: device upload and decoding of the stored plane layout.

The decoder follows the plane layout that include/awe.h documents (1 KiB
bricks of 32 rows x 64 reduction indices, stored k-step major, K padded to
a multiple of awe.K_PAD, lane L = 32 h + t owning row t and
indices 32 h .. 32 h + 31, two E2M1 codes per byte, low nibble first).
"""
import hashlib
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _full_hashes():
    out = {}
    with open(os.path.join(GOLDEN, "full_oracle_sha256.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, dims, dtype, digest = [x.strip() for x in line.split("|")]
                out[name] = (tuple(int(v) for v in dims.split()), dtype, digest)
    return out


def full_oracle_match(C, name, shape, dtype):
    """Whether C (host array) equals the oracle's whole C for workload `name`, by the SHA-256 that
    tests/golden/make_full_oracle_hashes.py wrote from the oracle."""
    dims, want_dtype, digest = _full_hashes()[name]
    assert C.shape == shape and str(C.dtype) == want_dtype == dtype, (C.shape, C.dtype)
    return hashlib.sha256(np.ascontiguousarray(C).tobytes()).hexdigest() == digest


E2M1_MAG = np.array([0, 1, 2, 3, 4, 6, 8, 12], dtype=np.int64)


def device():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a GPU")
    return torch.device("cuda", 0)


def to_dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(device())


def _e4m3_table():
    """Value of every E4M3 code (OCP FP8: sign, 4 exponent bits with bias 7, 3 mantissa bits)."""
    v = np.zeros(256)
    for c in range(256):
        e, m = (c >> 3) & 15, c & 7
        mag = (m / 8.0) * 2.0 ** -6 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 7)
        v[c] = -mag if c & 0x80 else mag
    return v


E4M3 = _e4m3_table()


def _e2m3_table():
    """Value of every E2M3 code (OCP MX FP6: sign bit 5, 2 exponent bits with bias 1, 3 mantissa bits)."""
    v = np.zeros(64)
    for c in range(64):
        e, m = (c >> 3) & 3, c & 7
        mag = m / 8.0 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 1)
        v[c] = -mag if c & 0x20 else mag
    return v


E2M3 = _e2m3_table()


def _decode_e2m1(raw, R32, KS, Kp):
    # raw [KS, R32, 64 lanes, 16 bytes] -> [R32*32, Kp] doubled values
    raw = raw.transpose(1, 0, 2, 3)
    nib = np.stack([raw & 0xF, raw >> 4], axis=-1).reshape(R32, KS, 2, 32, 32)
    val = E2M1_MAG[nib & 7] * np.where(nib & 8, -1, 1)
    return val.transpose(0, 3, 1, 2, 4).reshape(R32 * 32, Kp)


def _decode_e4m3(raw, R32, KS, Kp):
    # raw [KS, R32, 64 lanes, 32 bytes] -> [R32*32, Kp] values (integers)
    raw = raw.transpose(1, 0, 2, 3).reshape(R32, KS, 2, 32, 32)
    val = E4M3[raw]
    assert np.array_equal(val, np.round(val)), "E4M3 planes hold integers"
    return val.astype(np.int64).transpose(0, 3, 1, 2, 4).reshape(R32 * 32, Kp)


def _decode_e2m3(raw, R32, KS, Kp):
    # raw [KS/2 units, R32, 3072 bytes] -> [R32*32, Kp] integers n (stored as n / 8)
    U = KS // 2
    lo = raw[:, :, :2048].reshape(U, R32, 2, 64, 16)
    hi = raw[:, :, 2048:].reshape(U, R32, 2, 64, 8)
    words = np.concatenate([lo, hi], axis=-1)                    # [U, R32, i, lane, 24 bytes]
    bits = np.unpackbits(words, axis=-1, bitorder="little")      # [..., 192], bit b of the word
    codes = (bits.reshape(U, R32, 2, 64, 32, 6) << np.arange(6, dtype=np.uint8)).sum(-1)
    val = E2M3[codes] * 8
    assert np.array_equal(val, np.round(val)), "E2M3 planes hold integers / 8"
    val = val.astype(np.int64).reshape(U, R32, 2, 2, 32, 32)    # [u, rb, i, h, t, j]
    return val.transpose(1, 4, 0, 2, 3, 5).reshape(R32 * 32, Kp)


def decode_planes(buf, nplanes, rows, K, formats=None):
    """Stored planes (uint8 numpy) -> int64 array [nplanes, rows, K]: doubled values for E2M1
    planes, the integers for E4M3 and E2M3 planes (formats: list of "e2m1"/"e4m3"/"e2m3",
    default all E2M1); every padding element checked to hold code 0."""
    formats = formats or ["e2m1"] * nplanes
    R32 = -(-rows // 32)
    from paper_2609_24519_amd import awe
    Kp = -(-K // awe.K_PAD) * awe.K_PAD
    KS = Kp // 64
    unit = R32 * KS * 1024
    out = []
    off = 0
    buf = np.asarray(buf, dtype=np.uint8)
    for f in formats:
        # k-step major: brick (rb, ks) at (ks * R32 + rb) * brick bytes
        if f == "e4m3":
            full = _decode_e4m3(buf[off: off + 2 * unit].reshape(KS, R32, 64, 32), R32, KS, Kp)
            off += 2 * unit
        elif f == "e2m3":  # units of two k-steps: unit (rb, u) at (u * R32 + rb) * 3072
            full = _decode_e2m3(buf[off: off + 3 * unit // 2].reshape(KS // 2, R32, 3072), R32, KS, Kp)
            off += 3 * unit // 2
        else:
            full = _decode_e2m1(buf[off: off + unit].reshape(KS, R32, 64, 16), R32, KS, Kp)
            off += unit
        pad = full.copy()
        pad[:rows, :K] = 0
        assert not pad.any(), "padding must hold code 0"
        out.append(full[:rows, :K])
    return np.stack(out) if out else np.zeros((0, rows, K), np.int64)
