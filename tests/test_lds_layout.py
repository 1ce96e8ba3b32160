"""LDS layout of the extend kernel's 128-key steps (tile_attn.hpp, tile_attend_dl),
checked on the CPU against the properties the kernel relies on:

* each row load fills one contiguous 1 KB block (lane l -> slot l / 16, chunk l % 16)
  whose four rows lie in one 64-key half of the step, so one page base serves the
  wave's whole instruction;
* every row and chunk of the step is loaded exactly once by the 8 waves x 4 blocks;
* the K operand read and the transposed V read are a per-lane base plus offsets that
  depend only on the (compile-time) operand index, and address the rows and columns
  the MFMA operands need;
* no LDS bank is hit twice by one hardware lane group: 16 lanes for the 16-byte K
  reads, 32 lanes for the 8-byte transposed reads (64 banks of 4 bytes);
* both buffers of K and V fit the 160 KB of LDS.

The pitches are read from the kernel header, so a change there is checked here.
"""

import os
import re
from collections import Counter

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "paper_2609_08368_amd", "csrc", "tile_attn.hpp")


def constants():
    src = open(HDR).read()
    out = {}
    for name in ("kDlKeys", "kDlKPitch", "kDlVPitch"):
        m = re.search(rf"constexpr int {name} = ([0-9 +]+);", src)
        assert m, name
        out[name] = sum(int(x) for x in m.group(1).split("+"))
    return out


C = constants()
KP, VP, KEYS = C["kDlKPitch"], C["kDlVPitch"], C["kDlKeys"]


def block(r):
    return r % 16 + 16 * (r // 64)


def slot(r):
    return (r // 16) % 4


def addr(r, byte, pitch):
    return block(r) * pitch + slot(r) * 256 + byte


def worst_bank_load(addrs, width, group):
    """Largest number of distinct 4-byte words one bank serves within a lane group."""
    worst = 0
    for g0 in range(0, 64, group):
        words = {a // 4 + k for a in addrs[g0:g0 + group] for k in range(width // 4)}
        worst = max(worst, max(Counter(w % 64 for w in words).values()))
    return worst


def test_step_and_pitches():
    assert KEYS == 128
    assert KP >= 1024 and VP >= 1024 and KP % 16 == 0 and VP % 16 == 0
    assert 2 * 32 * (KP + VP) <= 160 * 1024


def test_row_loads_cover_the_step_once_from_one_half_per_block():
    seen = Counter()
    for wave in range(8):
        for i in range(4):
            b = wave + 8 * i
            halves = set()
            for lane in range(64):
                # the kernel's lane mapping: row in its half, 16-byte chunk
                row_in_half = wave + 8 * (i & 1) + 16 * (lane >> 4)
                r = 64 * (i >> 1) + row_in_half
                chunk = lane & 15
                assert addr(r, 16 * chunk, KP) == b * KP + 16 * lane
                assert addr(r, 16 * chunk, VP) == b * VP + 16 * lane
                halves.add(r // 64)
                seen[(r, chunk)] += 1
            assert len(halves) == 1
    assert len(seen) == KEYS * 16 and set(seen.values()) == {1}


def test_operand_reads_are_base_plus_constant_and_address_the_right_rows():
    for lane in range(64):
        col, kg = lane & 31, lane >> 5
        kbase = (col & 15) * KP + (col >> 4) * 256 + 16 * kg
        for kb in range(4):                      # S^T: key rows 32 kb + col, dims 16 c + 8 kg ..
            for c in range(8):
                want = addr(32 * kb + col, 2 * (16 * c + 8 * kg), KP)
                assert want == kbase + 16 * (kb >> 1) * KP + 512 * (kb & 1) + 32 * c
        tr_row = 4 * kg + ((lane & 15) >> 2)
        tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3)
        vbase = tr_row * VP + 2 * tr_col
        for h in range(8):                       # O^T += V^T P^T: keys 16 h .., dims 32 jd ..
            for u in range(2):                   # the two transposed reads of one operand
                for jd in range(4):
                    want = addr(16 * h + tr_row + 8 * u, 2 * (32 * jd + tr_col), VP)
                    assert want == vbase + (16 * (h >> 2) + 8 * u) * VP + 256 * (h & 3) + 64 * jd


def test_operand_reads_are_bank_conflict_free():
    for kb in range(4):
        for c in range(8):
            a = [addr(32 * kb + (l & 31), 2 * (16 * c + 8 * (l >> 5)), KP) for l in range(64)]
            assert worst_bank_load(a, 16, 16) == 1
    for h in range(8):
        for u in range(2):
            for jd in range(4):
                a = []
                for l in range(64):
                    kg = l >> 5
                    r = 16 * h + 4 * kg + ((l & 15) >> 2) + 8 * u
                    col = 32 * jd + 16 * ((l >> 4) & 1) + 4 * (l & 3)
                    a.append(addr(r, 2 * col, VP))
                assert worst_bank_load(a, 8, 32) == 1


def test_unpadded_blocks_would_conflict():
    """The padding is what spreads the rows over the banks (a mistake there shows)."""
    a = [addr(l & 31, 16 * (l >> 5), 1024) for l in range(64)]
    assert worst_bank_load(a, 16, 16) > 1
