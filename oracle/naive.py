"""Oracle: byte-at-a-time KV fetch/offload from the flat index formula (test infrastructure only).

This is a second, independent statement of the paged-KV fetch and offload
(Section 2.1; Section 5.2.1) used to pin ``oracle.kv``: it never slices or
reshapes, it computes the flat byte offset of every element on both sides from
its coordinates and copies one byte at a time. Pure Python loops, tiny shapes only.

Host slot s, layer l, k (0 = K, 1 = V), token t, head h, dim d, byte b::

    host_off = (((((s*L + l)*2 + k)*B + t)*H + h)*D + d)*E + b

GPU layer tensor l, block g, block layout 0 (as on the host)::

    gpu_off  = ((((k*NB + g)*B + t)*H + h)*D + d)*E + b

block layout 1 (x-packed key, token-minor value; x = 16 // E elements)::

    key   (k=0): ((((k*NB + g)*H + h)*(D//x) + d//x)*B + t)*x + d%x) * E + b
    value (k=1): ((((k*NB + g)*H + h)*D + d)*B + t) * E + b

block layout 2 (head-major, K and V alike)::

    gpu_off  = ((((k*NB + g)*H + h)*B + t)*D + d)*E + b
"""
from __future__ import annotations

from typing import List, Sequence


def host_offset(s, l, k, t, h, d, b, L, B, H, D, E):
    return (((((s * L + l) * 2 + k) * B + t) * H + h) * D + d) * E + b


def gpu_offset(k, g, t, h, d, b, NB, B, H, D, E, layout=0):
    if layout == 0:
        return ((((k * NB + g) * B + t) * H + h) * D + d) * E + b
    if layout == 2:
        return ((((k * NB + g) * H + h) * B + t) * D + d) * E + b
    x = 16 // E
    if k == 0:
        return (((((k * NB + g) * H + h) * (D // x) + d // x) * B + t) * x + d % x) * E + b
    return ((((k * NB + g) * H + h) * D + d) * B + t) * E + b


def fetch(host: bytes, layers: List[bytes], host_slots: Sequence[int], gpu_blocks: Sequence[int],
          L: int, B: int, H: int, D: int, E: int, NB: int, layout: int = 0) -> List[bytearray]:
    out = [bytearray(x) for x in layers]
    for i in range(len(host_slots)):
        s, g = host_slots[i], gpu_blocks[i]
        for l in range(L):
            for k in range(2):
                for t in range(B):
                    for h in range(H):
                        for d in range(D):
                            for b in range(E):
                                out[l][gpu_offset(k, g, t, h, d, b, NB, B, H, D, E, layout)] = \
                                    host[host_offset(s, l, k, t, h, d, b, L, B, H, D, E)]
    return out


def offload(host: bytes, layers: List[bytes], gpu_blocks: Sequence[int], host_slots: Sequence[int],
            L: int, B: int, H: int, D: int, E: int, NB: int, layout: int = 0) -> bytearray:
    out = bytearray(host)
    for j in range(len(host_slots)):
        s, g = host_slots[j], gpu_blocks[j]
        for l in range(L):
            for k in range(2):
                for t in range(B):
                    for h in range(H):
                        for d in range(D):
                            for b in range(E):
                                out[host_offset(s, l, k, t, h, d, b, L, B, H, D, E)] = \
                                    layers[l][gpu_offset(k, g, t, h, d, b, NB, B, H, D, E, layout)]
    return out
