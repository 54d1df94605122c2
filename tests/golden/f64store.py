"""Compact lossless storage of float64 arrays for the stored oracle runs.

The eight bytes of every value are split into eight planes (all first
bytes, then all second bytes, ...) before zlib compression: the sign,
exponent and leading mantissa bytes of finish times that lie close together
compress well, the trailing mantissa bytes do not.  Loading reverses the
split exactly, so the arrays read back are bit for bit the ones written.
"""

from __future__ import annotations

import numpy as np


def save(path: str, **arrays) -> None:
    planes = {}
    for name, a in arrays.items():
        a = np.ascontiguousarray(a, dtype="<f8")
        planes[name] = a.view(np.uint8).reshape(-1, 8).T.copy()
    np.savez_compressed(path, **planes)


def load(path: str) -> dict:
    out = {}
    with np.load(path, allow_pickle=False) as z:
        for name in z.files:
            p = z[name]
            out[name] = np.ascontiguousarray(p.T).reshape(-1).view("<f8").copy()
    return out
