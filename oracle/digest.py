"""Oracle: the dependent check kernel's digest (test infrastructure only).

The mixed-contention workload interleaves each weight-group load with a dependent
HBM-bound kernel on the same stream, to show that stream ordering survives the
dummy-task substitution (Section 3.3: downstream work must never see a copy before
all of its fragments have landed). That kernel reduces each freshly loaded tensor
to one 64-bit digest; this module defines it.

For a buffer read as little-endian 32-bit words ``w_0 .. w_{n-1}`` (a trailing
partial word is zero-padded)::

    digest = sum_i (w_i + 1) * (2*i + 1)   mod 2**64

The sum is over integers modulo 2**64, so any reduction order gives the same bits.
A word at the wrong position, a missing word or a zero word all change it.
"""
from __future__ import annotations

import numpy as np


def words_u32(buf: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(buf).view(np.uint8).reshape(-1)
    pad = (-b.size) % 4
    if pad:
        b = np.concatenate([b, np.zeros(pad, dtype=np.uint8)])
    return b.view("<u4")


def digest(buf: np.ndarray) -> int:
    w = words_u32(buf).astype(np.uint64)
    i = np.arange(w.size, dtype=np.uint64)
    terms = (w + np.uint64(1)) * (np.uint64(2) * i + np.uint64(1))
    return int(np.sum(terms, dtype=np.uint64))
