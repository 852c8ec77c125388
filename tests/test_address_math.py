"""The kernels' address arithmetic, restated on the host (CPU only).

The HIP kernels read spd through 32-bit buffer offsets and index per-lane
LDS tables and histograms by spd bytes. These tests restate each address
expression of the kernels (the constants are read from the sources) and
check the extremes the host validation admits: every spd offset stays below
the buffer range 2^31 - 1 at the largest row stride, every byte value
0..255 lands on a table/histogram entry inside its LDS object, and the
128-bucket layout's remap sends every byte >= 128 to the padding bucket."""
import re
from pathlib import Path

import pytest

CSRC = Path(__file__).resolve().parents[1] / "paper_2609_34420_amd" / "csrc"
RANGE = 0x7FFFFFFF                     # num_records of the kernels' buffer resources


def _const(name, fname="api.hip"):
    text = (CSRC / fname).read_text()
    m = re.search(rf"constexpr int64_t {name} = \(1LL << (\d+)\) - (\d+);", text)
    return (1 << int(m.group(1))) - int(m.group(2))


K_MAX_LD = _const("kMaxLd")


def perm(s0, s1, sel):
    """v_perm_b32: byte i of the result is byte sel_i of (s0:s1), where
    selectors 0..3 pick s1's bytes, 4..7 s0's, and 0x0c gives 0."""
    b = [(s1 >> (8 * i)) & 0xFF for i in range(4)] + [(s0 >> (8 * i)) & 0xFF for i in range(4)]
    out = 0
    for i in range(4):
        s = (sel >> (8 * i)) & 0xFF
        out |= (0 if s == 0x0C else b[s]) << (8 * i)
    return out


def test_max_stride_constant_matches_the_header():
    text = (Path(__file__).resolve().parents[1] / "include" / "gt_attn.h").read_text()
    assert "2^25 - 16" in text and K_MAX_LD == 2 ** 25 - 16


@pytest.mark.parametrize("ld", [K_MAX_LD, K_MAX_LD - 16, 131072, 64])
def test_query_stationary_spd_offsets(ld):
    """Forward and dQ: a wave's resource starts at its first query row; lane
    offset (row - first) ld + 16 g, key offset jt + 32 kb as the scalar part;
    a 16-byte load. Forward waves own 64 rows, dQ waves 32."""
    Sk = ld                              # the widest key block the stride admits
    for rows in (64, 32):
        v = (rows - 1) * ld + 16          # largest lane offset (g = 1)
        s = (Sk - 64) + 32                # last tile, second 32-key block
        assert v + s + 15 <= RANGE, (ld, rows)


@pytest.mark.parametrize("ld", [K_MAX_LD, 131072, 4096])
def test_key_stationary_spd_offsets(ld):
    """dK/dV: column gathers read bytes i_base + 16 g + r (r < 16) of the
    key's column from a resource at row i_base: lane offset 16 g ld + key,
    scalar offset r ld; the transposed rows (spd_t) are used only when
    256 ld < 2^31, lane offset (key - key0) ld + 16 g, scalar offset i_base
    <= ld - 16, one 16-byte load."""
    key = 255
    assert 16 * ld + key + 15 * ld <= RANGE
    if 256 * ld < 2 ** 31:
        assert (255 * ld + 16) + (ld - 16) + 15 <= RANGE


def test_forward_lane_table_addresses():
    """Forward and dQ: entry (b, lane) at byte 256 b + 4 lane of a 64 KiB
    per-lane table, from one permute: every byte value has an entry."""
    for lane in (0, 1, 31, 32, 63):
        for r in range(4):
            for b in (0, 1, 127, 128, 255):
                w = b << (8 * r)
                a = perm(w, lane * 4, 0x0C0C0000 | ((4 + r) << 8))
                assert a == 256 * b + 4 * lane
                assert 0 <= a and a + 4 <= 256 * 64 * 4


def _clamp128(b):
    return 0x7F if b & 0x80 else b


def test_key_stationary_table_and_histogram_128():
    """dK/dV with at most 127 buckets: 32 copies (lane & 31) of a 128-bucket
    layout at byte 64 KiB, 8-byte entries; the histogram entry 32 KiB past
    the table entry. Bytes >= 128 are first mapped to the padding bucket 127.
    Every (byte, lane) lands inside the table and histogram of its copy."""
    tab_base, ent = 1 << 16, 128 * 32
    seen = set()
    for lane in range(64):
        cpyb = (lane & 31) * 8 | tab_base
        for b in range(256):
            bc = _clamp128(b)
            assert bc < 128 and (bc == b or bc == 127)
            a = perm(bc, cpyb, 0x0C020400)
            assert a == tab_base + 256 * bc + 8 * (lane & 31)
            idx = (a - tab_base) // 8
            assert 0 <= idx < ent and idx % 32 == (lane & 31)
            hist = a + ent * 8
            assert tab_base + ent * 8 <= hist < tab_base + 2 * ent * 8
            seen.add(idx)
    assert len(seen) == ent


def test_key_stationary_table_and_histogram_256():
    """Past 127 buckets: 16 copies (lane & 15) of a 256-bucket layout,
    entry address (b << 7) | copy offset | base."""
    tab_base, ent = 1 << 16, 256 * 16
    for lane in range(64):
        cpyb = (lane & 15) * 8 | tab_base
        for b in range(256):
            a = (b << 7) | cpyb
            idx = (a - tab_base) // 8
            assert 0 <= idx < ent and idx == b * 16 + (lane & 15)
            assert a + ent * 8 < tab_base + 2 * ent * 8


def test_histogram_fixed_point_range():
    """Every histogram term is round(dS 2^F) with |dS| 2^F <= 2^30: a copy's
    64-bit sum of the 2 lanes x 8 waves x N queries that can share it stays
    below 2^63 for every N the stride limit admits."""
    terms = 2 * 8 * K_MAX_LD
    assert terms * 2 ** 30 < 2 ** 63
