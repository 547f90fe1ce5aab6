"""Helpers for the GPU tests: device upload and decoding of the stored plane layout.

The decoder follows the plane layout that include/awe.h documents (1 KiB
bricks of 32 rows x 64 reduction indices, stored k-step major, K padded to
a multiple of awe.K_PAD, lane L = 32 h + t owning row t and
indices 32 h .. 32 h + 31, two E2M1 codes per byte, low nibble first).
"""
import numpy as np

E2M1_MAG = np.array([0, 1, 2, 3, 4, 6, 8, 12], dtype=np.int64)


def device():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a GPU")
    return torch.device("cuda", 0)


def to_dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(device())


def decode_planes(buf, nplanes, rows, K):
    """Stored planes (uint8 numpy) -> int64 array [nplanes, rows, K] of doubled values; padding checked."""
    R32 = -(-rows // 32)
    from paper_2609_24519_amd import awe
    Kp = -(-K // awe.K_PAD) * awe.K_PAD
    KS = Kp // 64
    stride = R32 * KS * 1024
    # k-step major: brick (rb, ks) at (ks * R32 + rb) * 1024
    raw = np.asarray(buf[: nplanes * stride], dtype=np.uint8).reshape(nplanes, KS, R32, 64, 16)
    raw = raw.transpose(0, 2, 1, 3, 4)
    nib = np.stack([raw & 0xF, raw >> 4], axis=-1).reshape(nplanes, R32, KS, 2, 32, 32)
    val = E2M1_MAG[nib & 7] * np.where(nib & 8, -1, 1)
    # [p, rb, ks, h, t, j] -> [p, rb, t, ks, h, j]
    full = val.transpose(0, 1, 4, 2, 3, 5).reshape(nplanes, R32 * 32, Kp)
    pad = full.copy()
    pad[:, :rows, :K] = 0
    assert not pad.any(), "padding must hold code 0"
    return full[:, :rows, :K]
