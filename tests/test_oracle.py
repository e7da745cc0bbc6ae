"""Pins of the CPU oracle against things other than itself.

Each test checks the oracle against hand-worked fixtures, closed forms, an
independent formulation (byte-at-a-time index formula, Python bytes slicing,
numpy transposes, torch's bf16 rounding) or invariants -- never against a retyped
copy of its own formula.
"""
import hashlib
import itertools
import os

import numpy as np
import pytest

from conftest import parse_golden, parse_pairs
import workloads as W
from oracle import copy as ocopy
from oracle import digest as odigest
from oracle import kv as okv
from oracle import naive as onaive
from oracle import plan as oplan


# ----------------------------------------------------------------------------- copy
def test_memcpy_bruteforce_vs_bytes_slicing():
    src = np.frombuffer(bytes(range(256)) * 2, dtype=np.uint8)
    dst0 = np.full(64, 0xEE, dtype=np.uint8)
    for n in range(0, 41):
        for so in range(0, 6):
            for do in range(0, 64 - n + 1, 7):
                got = ocopy.memcpy(dst0, do, src, so, n)
                want = bytes(dst0[:do]) + bytes(src)[so:so + n] + bytes(dst0[do + n:])
                assert got.tobytes() == want


def test_memcpy_rejects_out_of_bounds():
    with pytest.raises(ValueError):
        ocopy.memcpy(np.zeros(8, np.uint8), 4, np.zeros(8, np.uint8), 0, 5)
    with pytest.raises(ValueError):
        ocopy.memcpy(np.zeros(8, np.uint8), 0, np.zeros(8, np.uint8), 4, 5)


def test_memcpy_preserves_checksum():
    src = W.uniform_bytes(1, 0, 0, 1 << 20)
    out = ocopy.memcpy(np.zeros(1 << 20, np.uint8), 0, src, 0, 1 << 20)
    assert hashlib.blake2b(out.tobytes(), digest_size=16).digest() == \
        hashlib.blake2b(src.tobytes(), digest_size=16).digest()


def test_tensor_list_vs_bytearray_loop():
    r = np.random.default_rng(5)
    src = r.integers(0, 256, 4096, dtype=np.uint8)
    dst0 = np.full(4096, 0xFF, np.uint8)
    descs = [(0, 100, 17), (17, 0, 1), (300, 2000, 500), (1000, 3000, 1096)]
    want = bytearray(dst0.tobytes())
    s = src.tobytes()
    for d, so, n in descs:
        for j in range(n):
            want[d + j] = s[so + j]
    assert ocopy.tensor_list(dst0, src, descs).tobytes() == bytes(want)


def test_tensor_list_rejects_overlap():
    with pytest.raises(ValueError):
        ocopy.tensor_list(np.zeros(64, np.uint8), np.zeros(64, np.uint8), [(0, 0, 10), (9, 20, 5)])
    assert ocopy.destinations_disjoint([(0, 10), (10, 5), (30, 0), (30, 1)])


# ----------------------------------------------------------------------------- kv
def _golden_kv(golden_dir):
    return parse_golden(os.path.join(golden_dir, "kv_tiny.txt"))


@pytest.mark.parametrize("name", ["fetch1", "fetch2"])
def test_kv_fetch_golden(golden_dir, name):
    g = _golden_kv(golden_dir)[name]
    L, B, H, D, E, NB = g["L"], g["B"], g["H"], g["D"], g["E"], g["NB"]
    piece = B * H * D * E
    host = np.array(g["host"], np.uint8).reshape(-1, L * 2 * piece)
    before = np.array(g["gpu_before"], np.uint8).reshape(L, 2, NB, piece)
    layers = okv.kv_fetch(host, [before[l] for l in range(L)], g["host_slots"], g["gpu_blocks"])
    for l in range(L):
        assert layers[l].reshape(-1).tolist() == g[f"gpu_after.{l}"]


def test_kv_offload_golden(golden_dir):
    g = _golden_kv(golden_dir)["offload1"]
    L, NB, S = g["L"], g["NB"], g["S"]
    piece = g["B"] * g["H"] * g["D"] * g["E"]
    layers = [np.array(g[f"gpu.{l}"], np.uint8).reshape(2, NB, piece) for l in range(L)]
    host = np.array(g["host_before"], np.uint8).reshape(S, -1)
    out = okv.kv_offload(host, layers, g["gpu_blocks"], g["host_slots"])
    assert out.reshape(-1).tolist() == g["host_after"]


def _tiny(L=2, B=2, H=1, D=2, E=2, S=4, NB=5, seed=0):
    r = np.random.default_rng(seed)
    piece = B * H * D * E
    host = r.integers(0, 256, (S, L * 2 * piece), dtype=np.uint8)
    layers = [r.integers(0, 256, (2, NB, piece), dtype=np.uint8) for _ in range(L)]
    return host, layers


def test_kv_fetch_matches_naive_all_permutations():
    L, B, H, D, E, S, NB = 2, 2, 1, 2, 2, 4, 5
    host, layers = _tiny(L, B, H, D, E, S, NB)
    for perm in itertools.permutations(range(4)):
        slots = list(perm)
        blocks = [4, 0, 2, 3]
        got = okv.kv_fetch(host, layers, slots, blocks)
        want = onaive.fetch(host.tobytes(), [x.tobytes() for x in layers], slots, blocks, L, B, H, D, E, NB)
        for l in range(L):
            assert got[l].tobytes() == bytes(want[l])


def test_kv_offload_matches_naive_all_permutations():
    L, B, H, D, E, S, NB = 2, 1, 2, 2, 1, 4, 4
    host, layers = _tiny(L, B, H, D, E, S, NB, seed=1)
    for perm in itertools.permutations(range(4)):
        got = okv.kv_offload(host, layers, [1, 3, 0, 2], list(perm))
        want = onaive.offload(host.tobytes(), [x.tobytes() for x in layers], [1, 3, 0, 2], list(perm),
                              L, B, H, D, E, NB)
        assert got.tobytes() == bytes(want)


@pytest.mark.parametrize("shape", [(1, 1, 1, 8, 1), (2, 2, 2, 16, 2), (3, 16, 1, 8, 2)])
def test_kv_fetch_matches_naive_shapes(shape):
    L, B, H, D, E = shape
    S, NB = 3, 4
    host, layers = _tiny(L, B, H, D, E, S, NB, seed=sum(shape))
    slots, blocks = [2, 0, 1], [3, 1, 0]
    got = okv.kv_fetch(host, layers, slots, blocks)
    want = onaive.fetch(host.tobytes(), [x.tobytes() for x in layers], slots, blocks, L, B, H, D, E, NB)
    assert all(got[l].tobytes() == bytes(want[l]) for l in range(L))


def test_kv_identity_tables_are_a_transpose():
    # With host_slots = gpu_blocks = identity over all blocks, fetch is the
    # transpose [S][L][2][piece] -> [L][2][S][piece].
    L, S, piece = 3, 5, 12
    r = np.random.default_rng(3)
    host = r.integers(0, 256, (S, L * 2 * piece), dtype=np.uint8)
    layers = [np.zeros((2, S, piece), np.uint8) for _ in range(L)]
    got = np.stack(okv.kv_fetch(host, layers, list(range(S)), list(range(S))))
    assert np.array_equal(got, host.reshape(S, L, 2, piece).transpose(1, 2, 0, 3))
    pool = okv.kv_offload(np.zeros_like(host), list(got), list(range(S)), list(range(S)))
    assert np.array_equal(pool, host)


def test_kv_roundtrip_and_untouched():
    s = W.small_kv_shape()
    r = np.random.default_rng(11)
    host = r.integers(0, 256, (s.host_num_slots, s.slot_bytes), dtype=np.uint8)
    layers = [np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8) for _ in range(s.layers)]
    slots, blocks = W.kv_fetch_tables(s)
    fetched = okv.kv_fetch(host, layers, slots, blocks)
    untouched = np.setdiff1d(np.arange(s.gpu_num_blocks), blocks)
    for l in range(s.layers):
        assert np.all(fetched[l][:, untouched] == W.GPU_POISON)
    # per-piece digests: the multiset moved is the multiset of sources, mapped by the tables
    for i in range(len(slots)):
        for l in range(s.layers):
            for k in (0, 1):
                src = host.reshape(s.host_num_slots, s.layers, 2, -1)[slots[i], l, k]
                assert odigest.digest(fetched[l][k, blocks[i]]) == odigest.digest(src)
    back = okv.kv_offload(np.zeros_like(host), fetched, blocks, slots)
    assert np.array_equal(back[slots], host[slots])
    others = np.setdiff1d(np.arange(s.host_num_slots), slots)
    assert np.all(back[others] == 0)


def test_kv_table_validation():
    assert okv.validate_tables([0, 1, 1], 2, [3, 2, 0], 4)       # repeated source is fine
    assert not okv.validate_tables([0, 1], 2, [3, 3], 4)         # duplicate destination
    assert not okv.validate_tables([0, 2], 2, [0, 1], 4)         # source out of range
    assert not okv.validate_tables([0, 1], 2, [0, 4], 4)         # destination out of range
    assert not okv.validate_tables([0, -1], 2, [0, 1], 4)        # negative
    assert not okv.validate_tables([0], 2, [0, 1], 4)            # length mismatch
    host, layers = _tiny()
    with pytest.raises(ValueError):
        okv.kv_fetch(host, layers, [0, 1], [2, 2])


def test_kv_offload_slot_layout():
    L, piece = 3, 4
    pieces = [np.arange(2 * piece, dtype=np.uint8).reshape(2, piece) + 10 * l for l in range(L)]
    slot = okv.kv_offload_slot(pieces)
    assert slot.tolist() == [x for l in range(L) for x in pieces[l].reshape(-1).tolist()]


# ----------------------------------------------------------------------------- x-packed KV layout
XP = okv.LAYOUT_XPACKED


@pytest.mark.parametrize("name", ["bytes1", "elem2"])
def test_kv_xpacked_golden(golden_dir, name):
    g = parse_golden(os.path.join(golden_dir, "kv_xpacked_tiny.txt"))[name]
    geom = (g["B"], g["H"], g["D"], g["E"])
    host = np.array(g["host"], np.uint8)
    assert okv.piece_to_block(host, 0, XP, geom).tolist() == g["key"]
    assert okv.piece_to_block(host, 1, XP, geom).tolist() == g["value"]
    assert okv.block_to_piece(np.array(g["key"], np.uint8), 0, XP, geom).tolist() == g["host"]
    assert okv.block_to_piece(np.array(g["value"], np.uint8), 1, XP, geom).tolist() == g["host"]


XP_SHAPES = [(1, 2, 1, 8, 2), (2, 2, 2, 16, 2), (1, 3, 2, 16, 1), (2, 4, 1, 4, 4), (1, 16, 2, 8, 2), (1, 5, 3, 32, 1)]


@pytest.mark.parametrize("shape", XP_SHAPES)
def test_kv_xpacked_matches_naive(shape):
    L, B, H, D, E = shape
    S, NB = 3, 4
    host, layers = _tiny(L, B, H, D, E, S, NB, seed=7 + sum(shape))
    slots, blocks = [2, 0, 1], [3, 1, 0]
    geom = (B, H, D, E)
    got = okv.kv_fetch(host, layers, slots, blocks, XP, geom)
    want = onaive.fetch(host.tobytes(), [x.tobytes() for x in layers], slots, blocks, L, B, H, D, E, NB, layout=1)
    assert all(got[l].tobytes() == bytes(want[l]) for l in range(L))
    got = okv.kv_offload(host, layers, blocks, slots, XP, geom)
    want = onaive.offload(host.tobytes(), [x.tobytes() for x in layers], blocks, slots, L, B, H, D, E, NB, layout=1)
    assert got.tobytes() == bytes(want)


def test_kv_xpacked_all_permutations_naive():
    L, B, H, D, E, S, NB = 1, 2, 2, 8, 2, 4, 5
    host, layers = _tiny(L, B, H, D, E, S, NB, seed=21)
    geom = (B, H, D, E)
    for perm in itertools.permutations(range(4)):
        got = okv.kv_fetch(host, layers, list(perm), [4, 0, 2, 3], XP, geom)
        want = onaive.fetch(host.tobytes(), [x.tobytes() for x in layers], list(perm), [4, 0, 2, 3],
                            L, B, H, D, E, NB, layout=1)
        assert got[0].tobytes() == bytes(want[0])


def test_kv_xpacked_single_token_block_is_the_host_layout():
    # With one token per block, [H][D/x][1][x] and [H][D][1] are the host order [1][H][D].
    r = np.random.default_rng(5)
    for H, D, E in [(1, 8, 2), (4, 16, 2), (3, 16, 1), (2, 4, 4)]:
        piece = r.integers(0, 256, H * D * E, dtype=np.uint8)
        for k in (0, 1):
            assert np.array_equal(okv.piece_to_block(piece, k, XP, (1, H, D, E)), piece)


def test_kv_xpacked_value_is_a_per_head_transpose():
    # Per head, the value block [D][B] is the transpose of the host's [B][D] rows taken at
    # stride H*D elements -- written with explicit Python loops over elements.
    B, H, D, E = 4, 3, 8, 2
    r = np.random.default_rng(9)
    piece = r.integers(0, 256, B * H * D * E, dtype=np.uint8)
    blk = okv.piece_to_block(piece, 1, XP, (B, H, D, E))
    for h in range(H):
        for d in range(D):
            for t in range(B):
                src = ((t * H + h) * D + d) * E
                dst = ((h * D + d) * B + t) * E
                assert blk[dst:dst + E].tolist() == piece[src:src + E].tolist()


def test_kv_xpacked_roundtrip_and_rejects():
    r = np.random.default_rng(13)
    for B, H, D, E in [(16, 8, 128, 2), (3, 2, 16, 1), (2, 2, 8, 4)]:
        piece = r.integers(0, 256, B * H * D * E, dtype=np.uint8)
        for k in (0, 1):
            blk = okv.piece_to_block(piece, k, XP, (B, H, D, E))
            assert sorted(blk.tolist()) == sorted(piece.tolist())
            assert np.array_equal(okv.block_to_piece(blk, k, XP, (B, H, D, E)), piece)
    with pytest.raises(ValueError):
        okv.piece_to_block(np.zeros(2 * 1 * 6 * 2, np.uint8), 0, XP, (2, 1, 6, 2))  # 12-byte rows
    s = W.small_kv_shape(head_dim=16)
    geom = (s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes)
    host = r.integers(0, 256, (s.host_num_slots, s.slot_bytes), dtype=np.uint8)
    layers = [np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8) for _ in range(s.layers)]
    slots, blocks = W.kv_fetch_tables(s)
    fetched = okv.kv_fetch(host, layers, slots, blocks, XP, geom)
    untouched = np.setdiff1d(np.arange(s.gpu_num_blocks), blocks)
    assert all(np.all(fetched[l][:, untouched] == W.GPU_POISON) for l in range(s.layers))
    back = okv.kv_offload(np.zeros_like(host), fetched, blocks, slots, XP, geom)
    assert np.array_equal(back[slots], host[slots])


# ----------------------------------------------------------------------------- head-major (HND) KV layout
HND = okv.LAYOUT_HND


@pytest.mark.parametrize("name", ["rows16", "rows3"])
def test_kv_hnd_golden(golden_dir, name):
    g = parse_golden(os.path.join(golden_dir, "kv_hnd_tiny.txt"))[name]
    geom = (g["B"], g["H"], g["D"], g["E"])
    host = np.array(g["host"], np.uint8)
    for k in (0, 1):  # K and V share the layout
        assert okv.piece_to_block(host, k, HND, geom).tolist() == g["block"]
        assert okv.block_to_piece(np.array(g["block"], np.uint8), k, HND, geom).tolist() == g["host"]


HND_SHAPES = [(1, 2, 2, 8, 2), (2, 3, 2, 8, 2), (1, 2, 3, 16, 1), (2, 1, 4, 4, 4), (1, 4, 1, 8, 2), (1, 3, 5, 2, 1)]


@pytest.mark.parametrize("shape", HND_SHAPES)
def test_kv_hnd_matches_naive(shape):
    L, B, H, D, E = shape
    S, NB = 3, 4
    host, layers = _tiny(L, B, H, D, E, S, NB, seed=11 + sum(shape))
    slots, blocks = [1, 2, 0], [0, 3, 2]
    geom = (B, H, D, E)
    got = okv.kv_fetch(host, layers, slots, blocks, HND, geom)
    want = onaive.fetch(host.tobytes(), [x.tobytes() for x in layers], slots, blocks, L, B, H, D, E, NB, layout=2)
    assert all(got[l].tobytes() == bytes(want[l]) for l in range(L))
    got = okv.kv_offload(host, layers, blocks, slots, HND, geom)
    want = onaive.offload(host.tobytes(), [x.tobytes() for x in layers], blocks, slots, L, B, H, D, E, NB, layout=2)
    assert got.tobytes() == bytes(want)


def test_kv_hnd_all_permutations_naive():
    L, B, H, D, E, S, NB = 1, 2, 3, 8, 2, 4, 5
    host, layers = _tiny(L, B, H, D, E, S, NB, seed=23)
    geom = (B, H, D, E)
    for perm in itertools.permutations(range(4)):
        got = okv.kv_fetch(host, layers, list(perm), [1, 4, 0, 2], HND, geom)
        want = onaive.fetch(host.tobytes(), [x.tobytes() for x in layers], list(perm), [1, 4, 0, 2],
                            L, B, H, D, E, NB, layout=2)
        assert got[0].tobytes() == bytes(want[0])


def test_kv_hnd_one_token_or_one_head_is_the_host_layout():
    # [H][1][D] and [1][B][D] are the host's [1][H][D] and [B][1][D].
    r = np.random.default_rng(17)
    for B, H, D, E in [(1, 4, 8, 2), (1, 3, 16, 1), (5, 1, 8, 2), (16, 1, 128, 2)]:
        piece = r.integers(0, 256, B * H * D * E, dtype=np.uint8)
        for k in (0, 1):
            assert np.array_equal(okv.piece_to_block(piece, k, HND, (B, H, D, E)), piece)


def test_kv_hnd_rows_move_whole():
    # Every (token, head) row of D*E bytes lands intact at row (head, token) -- explicit loops.
    B, H, D, E = 4, 3, 8, 2
    R = D * E
    r = np.random.default_rng(19)
    piece = r.integers(0, 256, B * H * R, dtype=np.uint8)
    blk = okv.piece_to_block(piece, 0, HND, (B, H, D, E))
    for t in range(B):
        for h in range(H):
            assert blk[(h * B + t) * R:(h * B + t + 1) * R].tolist() == piece[(t * H + h) * R:(t * H + h + 1) * R].tolist()
    assert np.array_equal(okv.block_to_piece(blk, 1, HND, (B, H, D, E)), piece)


# ----------------------------------------------------------------------------- plan
def test_plan_counts_golden(golden_dir):
    g = dict(parse_pairs(os.path.join(golden_dir, "plan_counts.txt")))
    sizes = W.weight_tensor_bytes()
    assert sum(sizes) == int(g["weights_total_bytes"])
    assert len(sizes) == int(g["weights_tensors"])
    M, K = W.MiB, W.KiB
    assert len(oplan.plan_linear(64 * M, 2 * M, 4 * M)) == int(g["copy64_2MiB"])
    assert len(oplan.plan_list(sizes, 2 * M, 4 * M, 64 * K)) == int(g["weights_2MiB"])
    assert len(oplan.plan_list(sizes, 256 * K, 512 * K, 64 * K)) == int(g["weights_256KiB"])
    s = W.KV64K
    assert len(oplan.plan_kv(4096, s.pieces_per_block, s.piece_bytes, 2 * M)) == int(g["kv_fetch_2MiB"])
    assert len(oplan.plan_kv(2048, s.pieces_per_block, s.piece_bytes, 2 * M)) == int(g["kv_offload_2MiB"])
    assert len(oplan.plan_kv(2048, s.pieces_per_block, s.piece_bytes, 256 * K)) == int(g["kv_offload_256KiB"])


def test_plan_linear_rules():
    assert oplan.plan_linear(0, 16, 32) == []
    assert oplan.plan_linear(31, 16, 32) == [(0, 31)]           # below fallback: one task
    assert oplan.plan_linear(33, 16, 32) == [(0, 16), (16, 16), (32, 1)]
    assert oplan.plan_linear(32, 16, 32) == [(0, 16), (16, 16)]
    for n in range(0, 200, 3):
        for c in (1, 7, 16, 64):
            p = oplan.plan_linear(n, c, 2 * c)
            assert (n == 0 and p == []) or oplan.covers_exactly_once(p, n)
            if n >= 2 * c:
                assert len(p) == -(-n // c)
                assert all(m == c for _, m in p[:-1])


def test_plan_list_small_tensors_cu_only():
    p = oplan.plan_list([100, 10, 0, 70], 32, 64, 64)
    assert [(t, o, m, cu) for t, o, m, cu in p] == [
        (0, 0, 32, False), (0, 32, 32, False), (0, 64, 32, False), (0, 96, 4, False),
        (1, 0, 10, True), (3, 0, 32, False), (3, 32, 32, False), (3, 64, 6, False)]


def test_plan_kv_cover():
    for ppb, pb, chunk in [(64, 32768, 2 << 20), (64, 32768, 256 << 10), (6, 100, 250), (4, 1000, 10)]:
        p = oplan.plan_kv(7, ppb, pb, chunk)
        assert oplan.kv_covers_exactly_once(p, 7, ppb)
        assert all(np_ * pb <= max(chunk, pb) for _, _, np_ in p)


def test_coverage_check_catches_mistakes():
    p = oplan.plan_linear(100, 16, 32)
    assert oplan.covers_exactly_once(p, 100)
    assert not oplan.covers_exactly_once(p[:-1], 100)                 # dropped chunk
    assert not oplan.covers_exactly_once(p + [p[0]], 100)              # duplicated chunk
    assert not oplan.covers_exactly_once([(o + 1, m) for o, m in p], 100)  # shifted
    k = oplan.plan_kv(3, 4, 10, 20)
    assert not oplan.kv_covers_exactly_once(k[1:], 3, 4)
    assert not oplan.kv_covers_exactly_once(k + [(0, 0, 1)], 3, 4)


# ----------------------------------------------------------------------------- digest
def test_digest_golden(golden_dir):
    for lhs, rhs in parse_pairs(os.path.join(golden_dir, "digest.txt")):
        words = np.array([int(x) for x in lhs.split(",")], dtype="<u4")
        assert odigest.digest(words.view(np.uint8)) == int(rhs)


def test_digest_closed_forms():
    for n in (1, 2, 3, 100, 4096):
        assert odigest.digest(np.zeros(4 * n, np.uint8)) == n * n            # sum of odd numbers
        c = 12345
        assert odigest.digest(np.full(n, c, "<u4").view(np.uint8)) == (c + 1) * n * n
    n = 1 << 16                                                             # wraps to exactly 0
    assert odigest.digest(np.full(n, 0xFFFFFFFF, "<u4").view(np.uint8)) == 0


def test_digest_bruteforce_python_ints():
    r = np.random.default_rng(2)
    for nb in (1, 3, 4, 5, 63, 64, 257):
        b = r.integers(0, 256, nb, dtype=np.uint8)
        padded = b.tobytes() + b"\0" * ((-nb) % 4)
        want = 0
        for i in range(len(padded) // 4):
            w = int.from_bytes(padded[4 * i:4 * i + 4], "little")
            want = (want + (w + 1) * (2 * i + 1)) % (1 << 64)
        assert odigest.digest(b) == want


def test_digest_sensitive_to_position():
    a = np.array([1, 2, 3, 4], "<u4")
    b = np.array([2, 1, 3, 4], "<u4")
    assert odigest.digest(a.view(np.uint8)) != odigest.digest(b.view(np.uint8))


# ----------------------------------------------------------------------------- inputs
def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(9)
    f = (r.standard_normal(100000).astype(np.float32) * np.float32(0.02))
    ties = np.array([0x3F808000, 0x3F818000, 0x3F80FFFF, 0x3F807FFF, 0xBF808000], np.uint32).view(np.float32)
    f = np.concatenate([f, ties, np.array([0.0, -0.0, 1.0, -3.5], np.float32)])
    ours = W.f32_to_bf16_rne(f)
    theirs = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, theirs)


def test_workload_generators_deterministic():
    a = W.uniform_bytes(3, 0, 17, 1000)
    b = W.uniform_bytes(3, 0, 17, 1000)
    c = W.uniform_bytes(3, 0, 18, 1000)
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    s = W.KV64K
    hs, gb = W.kv_fetch_tables(s)
    assert len(hs) == 4096 and len(set(hs.tolist())) == 4096 and hs.max() < s.host_num_slots
    assert len(set(gb.tolist())) == 4096 and gb.max() < s.gpu_num_blocks
    op = W.kv_offload_plan(s)
    assert len(op.dirty) == 2048 and len(set(op.dest.tolist())) == 2048
    assert not set(op.dest.tolist()) & set(op.occupied.tolist())
    assert s.piece_bytes == 32768 and s.slot_bytes == 2 << 20
