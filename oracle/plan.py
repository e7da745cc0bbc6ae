"""Oracle: the micro-task split and its coverage check (test infrastructure only).

Passages followed (Section 3.4, Task Manager): on the start signal the transfer is
divided into fixed-size micro-tasks; chunk size trades per-task overhead against
load-balancing granularity (Section 5.3). Transfers below a configurable threshold
are not split (Section 3.2, fallback mechanism). Completion of the logical copy means
every chunk has been delivered (Section 4), so a valid plan covers every byte of the
request exactly once.

Readings (the paper gives no remainder rule or threshold values):

* chunks start at offset 0 of each request; the last one is shorter;
* a request (or one tensor of a list) below ``fallback`` bytes is one micro-task;
* a tensor below ``small`` bytes is marked CU-only (a copy-engine command costs more
  than moving it);
* a tensor list is chunked per tensor -- no micro-task spans two tensors;
* a KV micro-task is one logical block's range of consecutive pieces (piece index
  ``p = 2*l + k``), holding ``max(1, chunk // piece_bytes)`` pieces except the last.
"""
from __future__ import annotations

from typing import Iterable, List, Sequence, Tuple

import numpy as np


def plan_linear(nbytes: int, chunk: int, fallback: int) -> List[Tuple[int, int]]:
    """(offset, length) micro-tasks of one contiguous request."""
    if chunk <= 0:
        raise ValueError("chunk must be positive")
    if nbytes == 0:
        return []
    if nbytes < fallback:
        return [(0, nbytes)]
    return [(o, min(chunk, nbytes - o)) for o in range(0, nbytes, chunk)]


def plan_list(sizes: Sequence[int], chunk: int, fallback: int, small: int
              ) -> List[Tuple[int, int, int, bool]]:
    """(tensor, offset, length, cu_only) micro-tasks of a tensor list, in list order."""
    out = []
    for t, n in enumerate(sizes):
        for o, m in plan_linear(int(n), chunk, fallback):
            out.append((t, o, m, int(n) < small))
    return out


def plan_kv(n_blocks: int, pieces_per_block: int, piece_bytes: int, chunk: int
            ) -> List[Tuple[int, int, int]]:
    """(table index i, first piece, piece count) micro-tasks of a KV fetch/offload."""
    per = max(1, chunk // piece_bytes)
    return [(i, p0, min(per, pieces_per_block - p0))
            for i in range(n_blocks) for p0 in range(0, pieces_per_block, per)]


def covers_exactly_once(intervals: Iterable[Tuple[int, int]], total: int) -> bool:
    """Write-count check: every byte of [0, total) lies in exactly one (offset, length) interval."""
    count = np.zeros(total, dtype=np.int64)
    for o, n in intervals:
        if o < 0 or n <= 0 or o + n > total:
            return False
        count[o:o + n] += 1
    return bool(np.all(count == 1))


def kv_covers_exactly_once(tasks: Iterable[Tuple[int, int, int]], n_blocks: int, pieces_per_block: int) -> bool:
    """Every (block, piece) pair appears in exactly one KV micro-task."""
    count = np.zeros((n_blocks, pieces_per_block), dtype=np.int64)
    for i, p0, np_ in tasks:
        if not (0 <= i < n_blocks) or p0 < 0 or np_ <= 0 or p0 + np_ > pieces_per_block:
            return False
        count[i, p0:p0 + np_] += 1
    return bool(np.all(count == 1))
