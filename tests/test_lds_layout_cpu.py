"""Host-side check of the GEMM tile's LDS layout: the 16-byte chunk swizzle (``row_swizzle`` in
``qgemm_kernels.hpp``) keeps the tile's LDS accesses free of bank conflicts.

Chunk c of tile row r (128-byte rows) sits at byte ``128 r + 16 (c ^ row_swizzle(r))``. The
accesses that matter are (per instruction, 64 lanes, 16 bytes each):

* fragment reads: lane l reads row (block base + l % 32) at logical chunk 2 kk + l / 32;
* Q4 dequant writes: lane t writes row t / 2, logical chunk 4 (t % 2) + u;
* Q8 dequant writes: lane t writes row t / 4, logical chunk 2 (t % 4) + u.

Two bank models are checked: 16 lanes per access phase over 64 four-byte banks, and 8 lanes per
phase over 32 banks (what the hardware counters point to on gfx950). No test here touches a GPU.
"""
import os
import re

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "..", "paper_2607_19438_amd", "csrc", "qgemm_kernels.hpp")
MODELS = ((64, 16), (32, 8))     # (banks, lanes per 16-byte access phase)


def table():
    text = open(SRC).read()
    m = re.search(r"kRowSwizzleTable\s*=\s*(0x[0-9a-fA-F]+)ull", text)
    assert m, "kRowSwizzleTable not found"
    t = int(m.group(1), 16)
    return [(t >> (4 * r)) & 7 for r in range(16)]


def worst_degree(addrs, banks, lanes):
    worst = 1
    for g in range(0, len(addrs), lanes):
        seen = {}
        for a in addrs[g:g + lanes]:
            for dw in range(a // 4, a // 4 + 4):
                seen.setdefault(dw % banks, set()).add(dw)
        worst = max(worst, max(len(v) for v in seen.values()))
    return worst


def patterns(sw):
    chunk = lambda r, c: 128 * r + 16 * (c ^ sw[r % 16])
    for base in (0, 32, 64, 96):
        for kk in range(2):
            yield f"fragment read base={base} kk={kk}", [chunk(base + l % 32, 2 * kk + l // 32) for l in range(64)]
    for base in (0, 32, 64):
        for u in range(4):
            yield f"Q4 write base={base} u={u}", [chunk(base + t // 2, 4 * (t % 2) + u) for t in range(64)]
        for u in range(2):
            yield f"Q8 write base={base} u={u}", [chunk(base + t // 4, 2 * (t % 4) + u) for t in range(64)]


def test_swizzle_is_a_permutation_per_row():
    sw = table()
    assert all(0 <= v < 8 for v in sw)
    for r in range(16):
        assert sorted(c ^ sw[r] for c in range(8)) == list(range(8))


@pytest.mark.parametrize("banks,lanes", MODELS)
def test_tile_accesses_conflict_free(banks, lanes):
    sw = table()
    for name, addrs in patterns(sw):
        assert worst_degree(addrs, banks, lanes) == 1, f"{name}: conflict with {banks} banks, {lanes} lanes"


def test_row_pair_swizzle_conflicts_in_the_narrow_model():
    """The model check bites: the earlier swizzle by row pair is conflict-free with 64 banks and
    16 lanes per phase but 2-way conflicted with 32 banks and 8 lanes."""
    pair = [(r >> 1) & 7 for r in range(16)]
    degrees = {m: max(worst_degree(a, *m) for _, a in patterns(pair)) for m in MODELS}
    assert degrees[(64, 16)] == 1 and degrees[(32, 8)] == 2
