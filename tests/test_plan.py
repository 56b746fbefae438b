"""The host planner of hb_run_iteration (paper_2503_22562_amd/csrc/hb_plan.cpp,
no HIP), built with g++ against a small driver: every query row of every
request and kv head must see each key of [0, position] in exactly one work
unit, with key ranges on the 64-key step grid, and split results must land
in disjoint partial slots."""
import os
import subprocess
from collections import defaultdict

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2503_22562_amd", "csrc")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("plan") / "plan_driver")
    cmd = ["g++", "-O1", "-std=c++17", f"-I{CSRC}", f"-I{os.path.join(ROOT, 'include')}",
           os.path.join(ROOT, "tests", "plan_driver.cpp"), os.path.join(CSRC, "hb_plan.cpp"), "-o", exe]
    subprocess.run(cmd, check=True)
    return exe


def run_plan(exe, shape, cu, reqs, split_item=0):
    H, nq, nkv, hd, F = shape
    lines = [f"{H} {nq} {nkv} {hd} {F} {cu} {len(reqs)} {split_item}"]
    nxt = 0
    for c, x in reqs:
        nb = -(-(c + x) // 16)
        lines.append(f"{c} {x} {nb} " + " ".join(str(nxt + i) for i in range(nb)))
        nxt += nb
    out = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True, check=True).stdout
    plan = defaultdict(list)
    for ln in out.splitlines():
        k, *v = ln.split()
        plan[k].append([int(t) for t in v])
    return plan


def check(plan, shape, reqs):
    H, nq, nkv, hd, F = shape
    G = nq // nkv
    starts = np.concatenate([[0], np.cumsum([c for c, _ in reqs])])
    tok_req = np.repeat(np.arange(len(reqs)), [c for c, _ in reqs])
    # token metadata
    toks = plan["tok"]
    assert len(toks) == starts[-1]
    for t, (pos, r) in enumerate(toks):
        assert r == tok_req[t] and pos == reqs[r][1] + t - starts[r]
    assert all(o[0] % 16 == 0 for o in plan["off"])
    # units: each tile once, each group of per_unit items once; a merged unit's
    # items are consecutive key ranges (some possibly empty) of one (request,
    # kv head, positions) with one destination, and it yields one result
    tile_cols, per_unit = plan["geom"][0]
    MERGED = 1 << 29
    units = [u[0] for u in plan["unit"]]
    tiles = sorted(u for u in units if u >= 0)
    item_units = sorted((-1 - u) & ~MERGED for u in units if u < 0)
    assert tiles == list(range(len(plan["tile"])))
    assert len(plan["item"]) % per_unit == 0
    assert item_units == list(range(len(plan["item"]) // per_unit))
    merged = {(-1 - u) & ~MERGED for u in units if u < 0 and (-1 - u) & MERGED}
    results = [("tile", tile_cols, it) for it in plan["tile"]]
    for v in range(len(plan["item"]) // per_unit):
        its = plan["item"][per_unit * v:per_unit * (v + 1)]
        if v in merged:
            assert len({tuple(it[:5]) + (it[7],) for it in its}) == 1, "merged unit mixes columns or destinations"
            full = [it for it in its if it[5] < it[6]]
            assert full and all(x[6] == y[5] for x, y in zip(full, full[1:])), "merged ranges not consecutive"
            assert all(it[5] % 64 == 0 for it in full)
            assert all(it[5] == it[6] for it in its[len(full):]), "empty ranges must come last"
            req, g, tok0, pos0, npos, _, _, part = its[0]
            results.append(("item", 16, [req, g, tok0, pos0, npos, full[0][5], full[-1][6], part]))
        else:
            results += [("item", 16, it) for it in its if it[5] < it[6]]
    # coverage: (token, kv head) -> list of key ranges
    cover = defaultdict(list)
    slots = []
    for kind, width, (req, g, tok0, pos0, npos, kb, ke, part) in results:
        assert kb % 64 == 0 and kb < ke and npos * G <= width
        assert tok0 == starts[req] + pos0 - reqs[req][1]
        assert ke <= pos0 + npos and ke <= reqs[req][0] + reqs[req][1]
        for i in range(npos):
            cover[(tok0 + i, g)].append((kb, ke, part))
        if part >= 0:
            slots.append((part, part + width))
    for t in range(starts[-1]):
        pos = toks[t][0]
        for g in range(nkv):
            rng = sorted(cover[(t, g)])
            assert rng, f"token {t} head {g} not covered"
            assert rng[0][0] == 0
            for (a0, a1, _), (b0, b1, _) in zip(rng, rng[1:]):
                assert a1 == b0, f"token {t} head {g}: gap or overlap {rng}"
            assert rng[-1][1] >= pos + 1
            # a later split of a tile may hold only keys past this row's position:
            # the row then contributes l = 0 to the merge, which drops it
            assert (len(rng) == 1) == (rng[0][2] < 0)
    slots.sort()
    for (a0, a1), (b0, b1) in zip(slots, slots[1:]):
        assert a1 <= b0, "partial slots overlap"
    # merge groups and their 16-column merge units
    want = []
    for gi, (p0, n, stride, tok0, npos, g, _, _) in enumerate(plan["group"]):
        assert n > 1 and stride in (16, tile_cols) and npos * G <= stride
        want += [gi * 16 + cb for cb in range(-(-npos * G // 16))]
    assert sorted(u[0] for u in plan["merge"]) == want


SHAPES = {"tiny": (256, 4, 2, 64, 688), "8b": (4096, 32, 8, 128, 14336), "70b": (8192, 64, 8, 128, 28672),
          "g16": (1024, 16, 1, 64, 512), "g1": (512, 4, 4, 128, 336),
          "8b-tp2": (4096, 16, 4, 128, 7168), "70b-tp8": (8192, 8, 1, 128, 3584)}


@pytest.mark.parametrize("name,reqs,cu", [
    ("tiny", [(64, 128)] + [(1, 256)] * 8, 256),
    ("8b", [(512, 3431)] + [(1, int(c)) for c in np.linspace(512, 4096, 64)], 256),
    ("8b", [(2048, 0)], 256),
    ("8b", [(128, 0)] + [(1, int(c)) for c in np.geomspace(256, 8192, 256)], 256),
    ("70b", [(2048, 30720)] + [(1, 32768)] * 32, 256),
    ("70b-tp8", [(2048, 30720)] + [(1, 32768)] * 32, 256),
    ("8b-tp2", [(512, 3431)] + [(1, int(c)) for c in np.linspace(512, 4096, 64)], 256),
    ("g16", [(37, 21), (1, 0), (300, 5), (5, 3)], 8),
    ("g1", [(129, 0), (1, 15), (1, 16), (7, 1000)], 4),
    ("8b", [(33, 0), (32, 40), (31, 1)], 1),
    ("8b", [(1, 519), (1, 599), (1, 4100), (1, 2049), (1, 8191), (1, 511), (3, 700)], 256),
])
def test_plan_covers_every_key_once(driver, name, reqs, cu):
    plan = run_plan(driver, SHAPES[name], cu, reqs)
    check(plan, SHAPES[name], reqs)


def test_plan_merged_units_with_short_item_splits(driver):
    """A short forced item split: merged workgroups with an empty wave range,
    and ranges spread over several merged workgroups and a merge group."""
    reqs = [(1, 519), (1, 599), (1, 4100), (1, 2049), (1, 8191), (1, 511), (3, 700), (512, 3000)]
    plan = run_plan(driver, SHAPES["8b"], 256, reqs, split_item=512)
    check(plan, SHAPES["8b"], reqs)
    merged = [(-1 - u[0]) & ~(1 << 29) for u in plan["unit"] if u[0] < 0 and (-1 - u[0]) & (1 << 29)]
    assert any(it[5] == it[6] for v in merged for it in plan["item"][4 * v:4 * v + 4]), "no empty wave range"
    assert any(g[2] == 16 for g in plan["group"]), "no merge group of item workgroups"


def test_plan_random_batches(driver):
    """Seeded random batches (shape, CU count, request mix and forced item
    split drawn per case): the coverage and slot invariants hold for every
    plan, including merged units, empty wave ranges and merge groups."""
    rng = np.random.default_rng(2503)
    names = sorted(SHAPES)
    for case in range(12):
        name = names[rng.integers(len(names))]
        cu = int(rng.choice([1, 4, 8, 64, 256]))
        reqs, T = [], 0
        for _ in range(int(rng.integers(1, 41))):
            kind = rng.integers(3)
            c = 1 if kind == 0 else int(rng.integers(2, 65)) if kind == 1 else int(rng.integers(65, 513))
            if T + c > 1024:
                break
            reqs.append((c, int(rng.integers(0, 9000))))
            T += c
        if not reqs:
            reqs = [(1, 100)]
        split_item = int(rng.choice([0, 256, 512, 1024]))
        plan = run_plan(driver, SHAPES[name], cu, reqs, split_item=split_item)
        try:
            check(plan, SHAPES[name], reqs)
        except AssertionError as e:
            raise AssertionError(f"case {case}: {name} cu={cu} split_item={split_item} reqs={reqs}: {e}") from e


def _split_tile_pieces(plan):
    """Key ranges of the split tiles, grouped by (request, kv head, first
    position): {group: sorted [(kv_begin, kv_end)]}."""
    groups = defaultdict(list)
    for req, g, tok0, pos0, npos, kb, ke, part in plan["tile"]:
        if part >= 0:
            groups[(req, g, pos0)].append((kb, ke))
    return {k: sorted(v) for k, v in groups.items()}


def test_split_tiles_are_even_when_every_unit_has_a_slot(driver):
    """Mixed launch of the 8B layer's TP2 shard (64 tiles, 256 item units on
    512 workgroup slots): the longest piece of each split tile is as short as
    the 64-key step grid allows for its piece count, since the longest piece
    sets the launch's length."""
    reqs = [(512, 3431)] + [(1, int(c)) for c in np.linspace(512, 4096, 64)]
    plan = run_plan(driver, SHAPES["8b-tp2"], 256, reqs)
    check(plan, SHAPES["8b-tp2"], reqs)
    pieces = _split_tile_pieces(plan)
    assert pieces, "no tile was split"
    for k, v in pieces.items():
        kv, n = v[-1][1], len(v)
        assert max(e - b for b, e in v) == -(-(-(-kv // n)) // 64) * 64, (k, v)


def test_split_tiles_keep_full_pieces_when_units_queue(driver):
    """Mixed launch of the 70B layer's TP8 shard (more units than slots):
    every piece of a split tile but the last spans exactly the split length."""
    reqs = [(2048, 30720)] + [(1, 32768)] * 32
    plan = run_plan(driver, SHAPES["70b-tp8"], 256, reqs)
    check(plan, SHAPES["70b-tp8"], reqs)
    S = plan["T"][0][1]
    pieces = _split_tile_pieces(plan)
    assert pieces, "no tile was split"
    for k, v in pieces.items():
        assert all(e - b == S for b, e in v[:-1]) and 0 < v[-1][1] - v[-1][0] <= S, (k, S, v)
