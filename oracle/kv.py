"""Oracle: paged-KV fetch and offload through block tables (test infrastructure only).

Passages followed: serving systems offload KV caches to host memory and, on a prefix
hit, fetch the cached KV pages back to the GPU before decoding (Section 2.1,
"Fetching cached KV pages..."; Section 5.2.1). The paper does not state the memory
layouts (they are internal to LMCache/vLLM), so this oracle takes the following
reading:

* host pool: ``S`` slots, slot ``s`` = ``[L][2][piece]`` contiguous, where a piece is
  one layer's K (k=0) or V (k=1) of one block: ``block_tokens*kv_heads*head_dim``
  elements;
* GPU cache: one tensor per layer, ``[2][NB][piece]``.

Fetch of n blocks, for every i < n, l < L, k in {0, 1}::

    GPU[l][k][gpu_blocks[i]] = HOST[host_slots[i]][l][k]

Offload is the reverse::

    HOST[host_slots[j]][l][k] = GPU[l][k][gpu_blocks[j]]

Every other GPU block (fetch) or host slot (offload) is unchanged. Table validity (a
reading; the paper is silent): entries in range, and no destination named twice,
since two sources racing into one block would make the result path-dependent.
Sources may repeat.

GPU block layouts (``layout``; the host side is always token-major
``[block_tokens][kv_heads][head_dim]`` per piece):

* ``LAYOUT_PIECE`` (0): the GPU block holds the piece exactly as the host does;
* ``LAYOUT_XPACKED`` (1): the layout of paged-attention decode kernels, where a
  block's key is ``[kv_heads][head_dim / x][block_tokens][x]`` with ``x = 16 //
  elem_bytes`` (16-byte groups of consecutive dims, token-minor), and its value is
  ``[kv_heads][head_dim][block_tokens]`` (token-minor). ``head_dim * elem_bytes``
  must be a multiple of 16;
* ``LAYOUT_HND`` (2): head-major, the transposed layout of some attention kernels: K
  and V blocks are both ``[kv_heads][block_tokens][head_dim]``, i.e. the piece's
  (token, head) rows of ``head_dim`` elements, transposed to (head, token) order.

All three are readings: the paper names the KV-cache systems but not their layouts.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np


def validate_tables(src_idx: Sequence[int], src_count: int,
                    dst_idx: Sequence[int], dst_count: int) -> bool:
    """True iff both tables have equal length, entries are in range and destinations are distinct."""
    if len(src_idx) != len(dst_idx):
        return False
    seen = set()
    for s, d in zip(src_idx, dst_idx):
        s, d = int(s), int(d)
        if not (0 <= s < src_count) or not (0 <= d < dst_count):
            return False
        if d in seen:
            return False
        seen.add(d)
    return True


LAYOUT_PIECE = 0
LAYOUT_XPACKED = 1
LAYOUT_HND = 2


def piece_to_block(piece: np.ndarray, k: int, layout: int, geom) -> np.ndarray:
    """GPU block bytes of one layer's K (k=0) or V (k=1) piece given in the host's
    token-major layout. ``geom`` = (block_tokens, kv_heads, head_dim, elem_bytes)."""
    piece = np.asarray(piece, dtype=np.uint8).reshape(-1)
    if layout == LAYOUT_PIECE:
        return piece.copy()
    if layout == LAYOUT_HND:  # K and V alike: [B][H][row] -> [H][B][row]
        B, H, D, E = geom
        return np.ascontiguousarray(piece.reshape(B, H, D * E).transpose(1, 0, 2)).reshape(-1)
    if layout != LAYOUT_XPACKED:
        raise ValueError("unknown layout")
    B, H, D, E = geom
    if (D * E) % 16:
        raise ValueError("head_dim * elem_bytes must be a multiple of 16")
    x = 16 // E
    a = piece.reshape(B, H, D, E)
    if k == 0:  # key: [H][D/x][B][x]
        return np.ascontiguousarray(a.reshape(B, H, D // x, x, E).transpose(1, 2, 0, 3, 4)).reshape(-1)
    return np.ascontiguousarray(a.transpose(1, 2, 0, 3)).reshape(-1)  # value: [H][D][B]


def block_to_piece(block: np.ndarray, k: int, layout: int, geom) -> np.ndarray:
    """Inverse of piece_to_block: the host (token-major) bytes of a GPU block's K or V."""
    block = np.asarray(block, dtype=np.uint8).reshape(-1)
    if layout == LAYOUT_PIECE:
        return block.copy()
    if layout == LAYOUT_HND:  # [H][B][row] -> [B][H][row]
        B, H, D, E = geom
        return np.ascontiguousarray(block.reshape(H, B, D * E).transpose(1, 0, 2)).reshape(-1)
    if layout != LAYOUT_XPACKED:
        raise ValueError("unknown layout")
    B, H, D, E = geom
    if (D * E) % 16:
        raise ValueError("head_dim * elem_bytes must be a multiple of 16")
    x = 16 // E
    if k == 0:
        a = block.reshape(H, D // x, B, x, E).transpose(2, 0, 1, 3, 4)
    else:
        a = block.reshape(H, D, B, E).transpose(2, 0, 1, 3)
    return np.ascontiguousarray(a).reshape(-1)


def _pool_view(host_pool: np.ndarray, layers: int) -> np.ndarray:
    slots = host_pool.shape[0]
    return host_pool.reshape(slots, layers, 2, -1)


def kv_fetch_layer(host_pool: np.ndarray, layer_before: np.ndarray, l: int, layers: int,
                   host_slots: Sequence[int], gpu_blocks: Sequence[int],
                   layout: int = LAYOUT_PIECE, geom=None) -> np.ndarray:
    """Expected GPU layer tensor ``l`` (shape [2, NB, piece]) after a fetch."""
    pool = _pool_view(host_pool, layers)
    nb = layer_before.shape[1]
    if not validate_tables(host_slots, pool.shape[0], gpu_blocks, nb):
        raise ValueError("invalid block tables")
    out = np.array(layer_before, dtype=np.uint8, copy=True)
    for i in range(len(host_slots)):
        for k in (0, 1):
            out[k, int(gpu_blocks[i])] = piece_to_block(pool[int(host_slots[i]), l, k], k, layout, geom)
    return out


def kv_fetch(host_pool: np.ndarray, layers_before: List[np.ndarray],
             host_slots: Sequence[int], gpu_blocks: Sequence[int],
             layout: int = LAYOUT_PIECE, geom=None) -> List[np.ndarray]:
    """Expected GPU layer tensors after a fetch (all layers)."""
    L = len(layers_before)
    return [kv_fetch_layer(host_pool, layers_before[l], l, L, host_slots, gpu_blocks, layout, geom)
            for l in range(L)]


def kv_offload(host_pool_before: np.ndarray, layers: List[np.ndarray],
               gpu_blocks: Sequence[int], host_slots: Sequence[int],
               layout: int = LAYOUT_PIECE, geom=None) -> np.ndarray:
    """Expected host pool (shape [S, slot_bytes]) after an offload."""
    L = len(layers)
    nb = layers[0].shape[1]
    if not validate_tables(gpu_blocks, nb, host_slots, host_pool_before.shape[0]):
        raise ValueError("invalid block tables")
    out = np.array(host_pool_before, dtype=np.uint8, copy=True)
    pool = _pool_view(out, L)
    for j in range(len(host_slots)):
        for l in range(L):
            for k in (0, 1):
                pool[int(host_slots[j]), l, k] = block_to_piece(layers[l][k, int(gpu_blocks[j])], k, layout, geom)
    return out


def kv_offload_slot(layers_block_pieces: List[np.ndarray]) -> np.ndarray:
    """Expected contents of one destination slot, given the source block's pieces
    ``layers_block_pieces[l][k]`` (shape [2, piece] per layer): the slot layout
    concatenates l-major, then k."""
    return np.concatenate([np.concatenate([p[0], p[1]]) for p in layers_block_pieces])
