"""Index arithmetic of the kernels' launch shapes, emulated on the CPU.

For every batch size and cell count the library launches with, the mapping
from (workgroup, wave, lane) to offspring or cell is replayed here from the
kernels' own constants (read from the sources): every offspring / cell is
taken by exactly one lane, every LDS slot index stays inside its array, and
what a later phase reads is what an earlier phase wrote for the same
offspring.  This is the host-side check of the launch shapes, covering the
two-phase LDS insertion on small four-dimensional CVTs (its final phase must
run on the workgroup's own lanes only).
"""
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2202_01258_amd", "csrc")


def constants():
    src = "".join(open(os.path.join(CSRC, f)).read()
                  for f in ("qd_kernels.hpp", "qd_rollout.hpp"))
    out = {}
    for m in re.finditer(r"constexpr int ([^;]+);", src):
        for part in m.group(1).split(","):
            name, _, val = part.partition("=")
            name, val = name.strip(), val.strip()
            if re.fullmatch(r"\d+", val):
                out[name] = int(val)
            elif re.fullmatch(r"(\d+) \* (\w+)", val):
                a, b = re.fullmatch(r"(\d+) \* (\w+)", val).groups()
                out[name] = int(a) * out[b]
    return out


K = constants()
BATCHES = sorted(set(list(range(1, 130)) + [255, 256, 257, 600, 1000, 1023, 1024, 1025, 2049,
                                            3000, 8191, 8192, 8193, 16384, 65536, 131072]))


def test_constants_found():
    for name in ("kOffspringPerWave", "kOneOffspringBatch", "kTwoOffspringBatch",
                 "kInsertLdsOffspring", "kCvtLdsCells", "kRegenCellsPerWave",
                 "kRegenCells", "kRegenCellsMlp", "kInsertBlock", "kInsertSlots"):
        assert name in K, name


def ceil_div(a, b):
    return (a + b - 1) // b


@pytest.mark.parametrize("nb", BATCHES)
def test_lds_cvt_insertion_lanes(nb):
    """k_insert_cvt_lds: grid ceil(nb / KO) x 256 threads.  Phase 1: row
    `row` (lane >> 4) of wave w measures offspring first + t, t = 16 r +
    4 w + row, and lane sub = 0 of the row stores its cell in s_cell[t].
    Phase 2: lanes 0 .. KO - 1 of wave 0 with j = first + lane < nb read
    s_cell[lane]."""
    KO = K["kInsertLdsOffspring"]
    assert KO % 16 == 0 and KO <= 64
    blocks = ceil_div(nb, KO)
    tid = np.arange(256)
    wave, lane = tid >> 6, tid & 63
    row, sub = lane >> 4, lane & 15
    taken = np.zeros(nb, np.int64)
    for b in range(blocks):
        first = b * KO
        written = {}
        for r in range(KO // 16):
            t = r * 16 + wave * 4 + row
            assert t.min() >= 0 and t.max() < KO           # s_cell bounds
            for tt in np.unique(t[sub == 0]):
                assert tt not in written
                written[int(tt)] = first + int(tt)          # offspring whose cell it holds
        assert sorted(written) == list(range(KO))            # every slot written
        # phase 2: wave 0 only
        l2 = lane[wave == 0]
        j = first + l2
        live = (l2 < KO) & (j < nb)
        for ll, jj in zip(l2[live], j[live]):
            assert written[int(ll)] == jj                    # reads its own offspring's slot
            taken[jj] += 1
    np.testing.assert_array_equal(taken, 1)


def offspring_per_wave(nb):
    """The library's choice (offspring_per_wave in qd_kernels.hpp)."""
    if nb <= K["kOneOffspringBatch"]:
        return 1
    return 2 if nb <= K["kTwoOffspringBatch"] else K["kOffspringPerWave"]


def test_offspring_per_wave_choice():
    """Four per wave in large batches, fewer in small ones; the selection and
    cell-search lanes (0 .. P-1, rows of 16 lanes for four offspring) hold P."""
    assert K["kOffspringPerWave"] == 4
    assert 0 < K["kOneOffspringBatch"] < K["kTwoOffspringBatch"]
    assert [offspring_per_wave(nb) for nb in (1, 2048, 2049, 8192, 8193, 65536)] == [1, 1, 2, 2, 4, 4]
    from paper_2202_01258_amd import qd     # the binding names kernel instances by it
    assert (qd.OFFSPRING_PER_WAVE, qd.ONE_OFFSPRING_BATCH, qd.TWO_OFFSPRING_BATCH) == (
        K["kOffspringPerWave"], K["kOneOffspringBatch"], K["kTwoOffspringBatch"])
    assert all(qd.offspring_per_wave(nb) == offspring_per_wave(nb) for nb in BATCHES)


@pytest.mark.parametrize("nb", BATCHES)
def test_vary_eval_offspring_lanes(nb):
    """k_vary_eval: grid ceil(nb / (4 P)) x 256; wave w of workgroup b takes
    offspring j0 = (4 b + w) P .. j0 + nmine - 1, lane i < nmine speaking for
    j0 + i."""
    P = offspring_per_wave(nb)
    blocks = ceil_div(nb, 4 * P)
    taken = np.zeros(nb, np.int64)
    for b in range(blocks):
        for w in range(4):
            j0 = (b * 4 + w) * P
            if j0 >= nb:
                continue
            nmine = min(P, nb - j0)
            for i in range(nmine):
                taken[j0 + i] += 1
    np.testing.assert_array_equal(taken, 1)


@pytest.mark.parametrize("C", [1, 13, 31, 32, 33, 500, 625, 1024, 2048, 2049, 10000])
@pytest.mark.parametrize("kind", ["testfn", "mlp"])
def test_regen_cells(C, kind):
    """k_regen / k_regen_mlp: ceil(C / cells) workgroups take cells, one
    more compacts; a cell past C reads key 0 and is skipped."""
    cells = K["kRegenCells"] if kind == "testfn" else K["kRegenCellsMlp"]
    blocks = ceil_div(C, cells) + 1
    taken = np.zeros(C, np.int64)
    for b in range(blocks - 1):
        for t in range(cells):
            c = b * cells + t
            if c < C:
                taken[c] += 1
    np.testing.assert_array_equal(taken, 1)
    if kind == "testfn":
        assert K["kRegenCells"] == 4 * K["kRegenCellsPerWave"] and K["kRegenCells"] <= 256


def test_insert_hash_always_has_a_free_slot():
    """k_insert: a workgroup of kInsertBlock offspring sees at most that many
    distinct cells, so its open-addressing table of kInsertSlots entries
    (a power of two) never fills."""
    assert K["kInsertSlots"] >= 2 * K["kInsertBlock"]
    assert K["kInsertSlots"] & (K["kInsertSlots"] - 1) == 0
