"""Host-side checks of the GEMM work schedule (persistent workgroups, and the
stream-K split of the last rounds of tiles), through the library's own
schedule routine: the same header code the kernel runs.  No GPU needed.  The
routine also walks the kernel's incremental cursor for every workgroup and
fails (-2) unless it yields exactly the segments checked here, with a
pipeline step count that covers them.  Both tile shapes are covered: 128 x
256 (tiles = 0, the linear layer's kernel) and 256 x 128 (tiles = 1, the
kernel template of the other GEMM entry points).

For every shape and persistent grid size, with and without the split: every (tile, 64-group) unit of the
output is computed exactly once; whole-tile rounds use whole tiles; the
split part is balanced to within one group per workgroup; each shared tile's
contributors are exactly the workgroups the finisher will read, each with a
distinct slot inside the workspace layout (2 slots per workgroup, one counter
set per split tile); and the finisher's slot lookup matches the slot each
contributor writes.  These are the invariants the kernel's partial-sum
protocol relies on for both correctness and in-bounds workspace accesses.
"""
import collections

import numpy as np
import pytest

import paper_2509_26436_amd as q

TILE_SHAPES = {0: (128, 256), 1: (256, 128)}

SHAPES = [
    # (M, K, N): FLUX.1 joint block, batched FLUX MLP, PixArt, SDXL im2col, single layer
    (4608, 3072, 9216), (4608, 3072, 3072), (4608, 3072, 12288), (4608, 12288, 3072),
    (18432, 3072, 12288), (18432, 12288, 3072),
    (4096, 1152, 3456), (4096, 1152, 1152), (4096, 1152, 4608), (4096, 4608, 1152),
    (16384, 2880, 320), (4096, 5760, 640), (1024, 11520, 1280),
    (256, 1152, 1152),
    # ragged and tiny
    (1, 64, 1), (300, 192, 200), (257, 128, 129), (4000, 640, 1000), (33, 4096, 70),
]
BLOCKS = [256, 304, 80, 32, 7, 1]


def _tiles(M, N, tiles):
    BM, BN = TILE_SHAPES[tiles]
    return -(-M // BM) * -(-N // BN)


def _check(M, K, N, blocks, split=True, tiles=0):
    s, seg = q.linear_schedule(M, N, K, blocks, split, tiles)
    BN = TILE_SHAPES[tiles][1]
    T, G = _tiles(M, N, tiles), K // 64
    assert s["groups"] == G
    assert 1 <= s["blocks"] <= blocks and s["sk_blocks"] <= s["blocks"]
    assert s["split"] or s["blocks"] <= T
    assert s["sk_first"] + s["sk_tiles"] == T
    if not s["split"]:
        assert s["sk_tiles"] == 0
    else:
        assert s["sk_first"] % s["blocks"] == 0
    assert s["tiles_n"] == -(-N // BN)
    f = {name: i for i, name in enumerate(q.SEGMENT_FIELDS)}

    # exactly-once coverage of every (tile, group)
    cover = np.zeros((T, G), dtype=np.int32)
    for r in seg:
        assert 0 <= r[f["tile"]] < T and 0 <= r[f["g0"]] < r[f["g1"]] <= G
        cover[r[f["tile"]], r[f["g0"]]:r[f["g1"]]] += 1
    assert (cover == 1).all()

    # segments of a workgroup: whole-tile rounds first (tile r * blocks + b), then its range
    per_block = collections.defaultdict(list)
    for r in seg:
        per_block[int(r[f["block"]])].append(r)
    units = {}
    for b, rows in per_block.items():
        assert 0 <= b < s["blocks"]
        assert [int(r[f["index"]]) for r in rows] == list(range(len(rows)))
        n_dp = sum(1 for r in rows if r[f["tile"]] < s["sk_first"])
        for j, r in enumerate(rows[:n_dp]):
            assert r[f["tile"]] == j * s["blocks"] + b
            assert (r[f["g0"]], r[f["g1"]], r[f["sk_tile"]]) == (0, G, -1)
        sk_rows = rows[n_dp:]
        units[b] = sum(int(r[f["g1"]] - r[f["g0"]]) for r in sk_rows)
        # at most two partial segments per workgroup: its first and its last
        for r in sk_rows[1:-1]:
            assert r[f["sk_tile"]] == -1
    if s["split"]:
        sk_units = [units.get(b, 0) for b in range(s["sk_blocks"])]
        assert sum(sk_units) == s["sk_tiles"] * G
        assert max(sk_units) - min(sk_units) <= 1
    # whole-tile work: the workgroups' tile counts differ by one at most
    dp = collections.Counter(int(r[f["block"]]) for r in seg if r[f["tile"]] < s["sk_first"])
    if dp:
        assert max(dp.values()) - min(dp.get(b, 0) for b in range(s["blocks"])) <= 1

    # partial segments: slots, counters, contributor sets, finisher lookup
    slots_seen = set()
    by_tile = collections.defaultdict(list)
    for r in seg:
        t = int(r[f["sk_tile"]])
        tile_full = (r[f["g0"]], r[f["g1"]]) == (0, G)
        if t < 0:
            assert tile_full
            continue
        assert not tile_full
        assert t == r[f["tile"]] - s["sk_first"] and 0 <= t < s["sk_tiles"]
        slot = int(r[f["slot"]])
        assert 0 <= slot < 2 * s["sk_blocks"] and slot not in slots_seen
        slots_seen.add(slot)
        assert r[f["finisher_slot"]] == slot
        by_tile[t].append(int(r[f["block"]]))
    for r in seg:
        t = int(r[f["sk_tile"]])
        if t >= 0:
            assert sorted(by_tile[t]) == list(range(r[f["b_first"]], r[f["b_last"]] + 1))
            assert len(by_tile[t]) >= 2
    return s


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("blocks", BLOCKS)
@pytest.mark.parametrize("split", [True, False])
@pytest.mark.parametrize("tiles", [0, 1])
def test_schedule_invariants(shape, blocks, split, tiles):
    M, K, N = shape
    _check(M, K, N, blocks, split, tiles)


@pytest.mark.parametrize("tiles", [0, 1])
def test_schedule_choices_on_256_compute_units(tiles):
    # Split where the idle part of the last round of whole tiles is worth at
    # least 16 groups per workgroup: FLUX qkv (1296 tiles = 5.06 rounds of 48
    # groups: 45 groups saved) and fc2 (432 tiles of 192 groups: 60), not out
    # (432 tiles of 48 groups: 15) nor fc1 (1728 tiles = 6.75 rounds: 12); a
    # multiple of 256 tiles needs no split
    # (both tile shapes give these layers the same tile counts)
    s = _check(4608, 3072, 9216, 256, tiles=tiles)
    assert s["split"] == 1 and (s["dp_tiles_b0"], s["sk_tiles"]) == (4, 272)
    assert _check(4608, 3072, 3072, 256, tiles=tiles)["split"] == 0
    assert _check(4608, 12288, 3072, 256, tiles=tiles)["split"] == 1
    assert _check(4608, 3072, 12288, 256, tiles=tiles)["split"] == 0
    assert _check(18432, 3072, 12288, 256, tiles=tiles)["split"] == 0   # 6912 tiles = 27 rounds
    # without a workspace nothing is split: 1296 tiles over 256 workgroups
    s = _check(4608, 3072, 9216, 256, split=False, tiles=tiles)
    assert s["split"] == 0 and s["blocks"] == 256 and s["dp_tiles_b0"] == 6
    # fewer tiles than workgroups: at least 16 groups per workgroup and at
    # least 1/8 of a tile's groups (so about 8 workgroups share a tile at
    # most), and no split at all when that leaves under two workgroups per
    # tile: the single 256 x 1152 x 1152 linear (10 tiles of 128 x 256 or 9 of
    # 256 x 128, 18 groups each) stays whole, as measured faster (20 against
    # 36 us with the 256 x 128 tiles)
    T1 = _tiles(256, 1152, tiles)
    s = _check(256, 1152, 1152, 256, tiles=tiles)
    assert s["split"] == 0 and s["blocks"] == T1
    s = _check(160, 4608, 448, 256, tiles=tiles)
    assert s["split"] == 1 and s["sk_q"] >= 16 and s["sk_blocks"] >= 2 * _tiles(160, 448, tiles)
    s = _check(257, 12288, 129, 256, tiles=tiles)
    assert s["split"] == 1 and s["sk_q"] >= 192 // 8
    s = _check(256, 1152, 1152, 256, split=False, tiles=tiles)
    assert s["split"] == 0 and s["blocks"] == T1


def test_schedule_rejects_bad_arguments():
    import numpy as np
    sched = np.zeros(10, dtype=np.int32)
    assert q.quartz_w4a4_linear_schedule(0, 64, 64, 256, 1, 0, sched.ctypes.data, None, 0) == -1
    assert q.quartz_w4a4_linear_schedule(64, 64, 100, 256, 1, 0, sched.ctypes.data, None, 0) == -1
    assert q.quartz_w4a4_linear_schedule(64, 64, 64, 256, 1, 0, None, None, 0) == -1
    assert q.quartz_w4a4_linear_schedule(64, 64, 64, 0, 1, 0, sched.ctypes.data, None, 0) == -1
    assert q.quartz_w4a4_linear_schedule(64, 64, 64, 256, 1, 2, sched.ctypes.data, None, 0) == -1
