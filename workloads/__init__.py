"""Seeded synthetic workloads for the multipath host<->GPU copy path.

This module only *generates inputs*: random bytes, bf16 weights, block tables and
the shapes of the five benchmark workloads. It contains no data-movement logic, so
both the CPU oracle (``oracle/``) and the GPU path's tests and benchmark can use it
without sharing any of the method's arithmetic.

Random streams are keyed by ``(workload, tag, index)`` so that the expected data of
any single tensor or KV block can be regenerated on its own instead of being
mirrored in host memory.

The paper measures on LLM serving workloads (LongBench v2 documents on Qwen models
under LMCache+vLLM, and vLLM sleep-mode weight reloads; Evaluation section). Those
datasets, models and systems are not used here. The transfer cost depends only on
sizes and structure, which these synthetic stand-ins reproduce: a Llama-3-8B-shaped
bf16 tensor list for model wake-up, and a 64k-token GQA paged KV cache.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Tuple

import numpy as np

SEED = 251216056  # the paper's arXiv identifier, used as the root seed

# Tags of the independent random streams.
TAG_DATA = 0          # payload bytes / weight values
TAG_HOST_PERM = 1     # host-slot permutation (KV fetch)
TAG_GPU_PERM = 2      # GPU-block permutation
TAG_DIRTY = 3         # dirty-block subset (KV offload)
TAG_FREE_PERM = 4     # order in which free host slots are used (KV offload)
TAG_OCCUPIED = 5      # which host slots are already occupied (KV offload)
TAG_OCC_DATA = 6      # contents of occupied host slots

KiB = 1024
MiB = 1024 * KiB
GiB = 1024 * MiB


def rng(cfg: int, tag: int, idx: int) -> np.random.Generator:
    """Independent PCG64 stream for (workload, tag, index)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, cfg, tag, idx])))


def uniform_bytes(cfg: int, tag: int, idx: int, n: int) -> np.ndarray:
    """n uniform random bytes (read-only uint8 view)."""
    return np.frombuffer(rng(cfg, tag, idx).bytes(n), dtype=np.uint8)


def f32_to_bf16_rne(f: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns with round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def bf16_normal(cfg: int, tag: int, idx: int, n_elems: int, std: float = 0.02) -> np.ndarray:
    """n_elems bf16 values ~ N(0, std), as uint16 bit patterns."""
    f = rng(cfg, tag, idx).standard_normal(n_elems, dtype=np.float32)
    f *= np.float32(std)
    return f32_to_bf16_rne(f)


# ---------------------------------------------------------------------------
# Workload 1: one contiguous 64 MiB host->GPU copy, 2 MiB micro-transfers.
# ---------------------------------------------------------------------------
COPY64_BYTES = 64 * MiB
COPY64_CHUNK = 2 * MiB


# ---------------------------------------------------------------------------
# Workload 2: Llama-3-8B-shaped bf16 tensor list (model wake-up).
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelShape:
    layers: int = 32
    hidden: int = 4096
    ffn: int = 14336
    q_heads: int = 32
    kv_heads: int = 8
    head_dim: int = 128
    vocab: int = 128256
    elem_bytes: int = 2


LLAMA3_8B = ModelShape()


def weight_tensor_list(m: ModelShape = LLAMA3_8B) -> List[Tuple[str, Tuple[int, ...]]]:
    """(name, shape) of every weight tensor, in load order."""
    kv = m.kv_heads * m.head_dim
    q = m.q_heads * m.head_dim
    out: List[Tuple[str, Tuple[int, ...]]] = [("embed_tokens", (m.vocab, m.hidden))]
    for l in range(m.layers):
        p = f"layers.{l}."
        out += [
            (p + "input_layernorm", (m.hidden,)),
            (p + "q_proj", (q, m.hidden)),
            (p + "k_proj", (kv, m.hidden)),
            (p + "v_proj", (kv, m.hidden)),
            (p + "o_proj", (m.hidden, q)),
            (p + "post_attention_layernorm", (m.hidden,)),
            (p + "gate_proj", (m.ffn, m.hidden)),
            (p + "up_proj", (m.ffn, m.hidden)),
            (p + "down_proj", (m.hidden, m.ffn)),
        ]
    out += [("norm", (m.hidden,)), ("lm_head", (m.vocab, m.hidden))]
    return out


def weight_tensor_bytes(m: ModelShape = LLAMA3_8B) -> List[int]:
    return [int(np.prod(s)) * m.elem_bytes for _, s in weight_tensor_list(m)]


def weight_groups(m: ModelShape = LLAMA3_8B) -> List[List[int]]:
    """Tensor indices grouped as [embed], [layer l's 9 tensors] x L, [norm, lm_head]."""
    n = len(weight_tensor_list(m))
    groups = [[0]]
    for l in range(m.layers):
        groups.append(list(range(1 + 9 * l, 1 + 9 * (l + 1))))
    groups.append([n - 2, n - 1])
    return groups


def arena_offsets(sizes: List[int], align: int = 256) -> Tuple[List[int], int]:
    """Offsets of tensors packed into one arena, each `align`-aligned; returns (offsets, total)."""
    offs, cur = [], 0
    for s in sizes:
        cur = (cur + align - 1) // align * align
        offs.append(cur)
        cur += s
    return offs, (cur + align - 1) // align * align


def weight_values(cfg: int, t: int, n_elems: int) -> np.ndarray:
    """bf16 N(0, 0.02) contents of tensor t of workload cfg."""
    return bf16_normal(cfg, TAG_DATA, t, n_elems)


# ---------------------------------------------------------------------------
# Workloads 3-5: paged KV cache.
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class KVShape:
    """Host slot: [layers][2 (K,V)][block_tokens][kv_heads][head_dim] contiguous.
    GPU layer tensor l: [2][gpu_num_blocks][block_tokens][kv_heads][head_dim]."""
    layers: int = 32
    block_tokens: int = 16
    kv_heads: int = 8
    head_dim: int = 128
    elem_bytes: int = 2
    gpu_num_blocks: int = 4352
    host_num_slots: int = 4096
    n_blocks: int = 4096  # blocks moved by one call (65536 tokens / 16)

    @property
    def piece_bytes(self) -> int:
        return self.block_tokens * self.kv_heads * self.head_dim * self.elem_bytes

    @property
    def pieces_per_block(self) -> int:
        return 2 * self.layers

    @property
    def slot_bytes(self) -> int:
        return self.pieces_per_block * self.piece_bytes

    @property
    def layer_bytes(self) -> int:
        return 2 * self.gpu_num_blocks * self.piece_bytes


KV64K = KVShape()


def kv_fetch_tables(s: KVShape, cfg: int = 3) -> Tuple[np.ndarray, np.ndarray]:
    """(host_slots, gpu_blocks) int32 for a fetch of s.n_blocks logical blocks."""
    host_slots = rng(cfg, TAG_HOST_PERM, 0).permutation(s.host_num_slots)[: s.n_blocks].astype(np.int32)
    gpu_blocks = rng(cfg, TAG_GPU_PERM, 0).permutation(s.gpu_num_blocks)[: s.n_blocks].astype(np.int32)
    return host_slots, gpu_blocks


def kv_block_bytes(cfg: int, i: int, s: KVShape) -> np.ndarray:
    """Contents of logical block i (all layers, K and V), slot layout."""
    return uniform_bytes(cfg, TAG_DATA, i, s.slot_bytes)


@dataclass
class OffloadPlan:
    gpu_blocks_all: np.ndarray   # GPU block of each logical block (int32, n_blocks)
    dirty: np.ndarray            # logical blocks to offload, in call order
    occupied: np.ndarray         # host slots holding other data (must stay untouched)
    free: np.ndarray             # free host slots, ascending
    dest: np.ndarray             # destination slot of each dirty block (int32)

    @property
    def src_blocks(self) -> np.ndarray:
        return self.gpu_blocks_all[self.dirty].astype(np.int32)


def kv_offload_plan(s: KVShape, cfg: int = 4, dirty_frac: float = 0.5) -> OffloadPlan:
    gpu_blocks_all = rng(cfg, TAG_GPU_PERM, 0).permutation(s.gpu_num_blocks)[: s.n_blocks].astype(np.int32)
    n_dirty = int(s.n_blocks * dirty_frac)
    dirty = rng(cfg, TAG_DIRTY, 0).permutation(s.n_blocks)[:n_dirty].astype(np.int64)
    n_occ = s.host_num_slots - n_dirty
    occupied = np.sort(rng(cfg, TAG_OCCUPIED, 0).permutation(s.host_num_slots)[:n_occ]).astype(np.int64)
    mask = np.ones(s.host_num_slots, dtype=bool)
    mask[occupied] = False
    free = np.nonzero(mask)[0].astype(np.int64)
    dest = free[rng(cfg, TAG_FREE_PERM, 0).permutation(len(free))[:n_dirty]].astype(np.int32)
    return OffloadPlan(gpu_blocks_all, dirty, occupied, free, dest)


def kv_occupied_bytes(cfg: int, slot: int, s: KVShape) -> np.ndarray:
    return uniform_bytes(cfg, TAG_OCC_DATA, slot, s.slot_bytes)


GPU_POISON = 0xA5      # untouched GPU KV blocks
HOST_FREE_POISON = 0x5A  # free host slots before an offload
WEIGHT_POISON = 0xFF   # weight destinations before a load


def small_kv_shape(layers=2, block_tokens=2, kv_heads=2, head_dim=16, elem_bytes=2,
                   gpu_num_blocks=40, host_num_slots=32, n_blocks=24) -> KVShape:
    """Reduced KV shape with the same structure, for tests."""
    return KVShape(layers, block_tokens, kv_heads, head_dim, elem_bytes, gpu_num_blocks, host_num_slots, n_blocks)
