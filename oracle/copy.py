"""Oracle: single host<->GPU copy and tensor-list copy (test infrastructure only).

Definition followed: a multipath copy must be a drop-in replacement for the native
single-path copy (Abstract; Introduction, contributions), and the logical copy is
complete only once every fragment has arrived (Section 2.3, challenge C2). The
result is therefore exactly ``dst[i] = src[i]`` for every byte of the request, with
all other destination bytes unchanged -- independent of how the copy was split into
micro-transfers or which path carried each one.

The model wake-up workload reloads weights host->GPU (Section 2.1; Section 5.2.2):
a list of independent copies, each with the same definition. Destinations of one
list must not overlap (a reading: concurrent micro-transfers into overlapping bytes
would make the result depend on path timing, which the paper's semantics exclude).
"""
from __future__ import annotations

from typing import Iterable, Sequence, Tuple

import numpy as np


def memcpy(dst_before: np.ndarray, dst_off: int, src: np.ndarray, src_off: int, n: int) -> np.ndarray:
    """Expected destination buffer after copying ``n`` bytes src[src_off:] -> dst[dst_off:]."""
    if n < 0 or dst_off < 0 or src_off < 0:
        raise ValueError("negative size or offset")
    if dst_off + n > dst_before.size or src_off + n > src.size:
        raise ValueError("copy out of bounds")
    out = np.array(dst_before, dtype=np.uint8, copy=True)
    out[dst_off:dst_off + n] = src[src_off:src_off + n]
    return out


def destinations_disjoint(ranges: Iterable[Tuple[int, int]]) -> bool:
    """True iff the half-open byte ranges (offset, length) are pairwise disjoint."""
    spans = sorted((o, o + n) for o, n in ranges if n > 0)
    return all(spans[i][1] <= spans[i + 1][0] for i in range(len(spans) - 1))


def tensor_list(dst_before: np.ndarray, src: np.ndarray,
                descs: Sequence[Tuple[int, int, int]]) -> np.ndarray:
    """Expected destination arena after a list of copies.

    ``descs`` holds (dst_off, src_off, nbytes) into one destination and one source
    arena. Each copy is applied as its own memcpy; the destinations must be disjoint.
    """
    if not destinations_disjoint((d, n) for d, _, n in descs):
        raise ValueError("overlapping destinations")
    out = np.array(dst_before, dtype=np.uint8, copy=True)
    for d, s, n in descs:
        out[d:d + n] = src[s:s + n]
    return out
