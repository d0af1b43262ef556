"""Bounds of the long-segment chain's buffer offsets, checked on the CPU.

The producers of a long-segment chain read ids and gradient rows through raw
buffer resources with the whole byte offset in the vector offset, which the
hardware range-checks against the resource size (reads past it return 0
without touching memory). Ids of chunks ahead of the segment's end are read on
purpose and come back as 0; rows past the end are read at an offset of
kOutOfRange. This checks, from the constants in the kernel source, that every
offset a chain forms fits the signed 32-bit vector offset and that the
out-of-range ones really lie past every resource, for every segment length
and row width the buffer path accepts (longer segments and wider row spans
take the 64-bit fallback).
"""
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2010_13100_amd", "csrc")

INT32_MAX = 2 ** 31 - 1


def _source(name):
    with open(os.path.join(CSRC, name)) as f:
        return f.read()


def _const(src, name):
    m = re.search(r"constexpr\s+int(?:32_t)?\s+" + name + r"\s*=\s*([^;]+);", src)
    assert m, name
    value = m.group(1).strip()
    return 64 if value == "kWave" else int(value, 0)  # the wavefront width, or a literal


def test_constants_are_what_the_check_assumes():
    src = _source("tc_backward.hip")
    assert _const(src, "kChunkRows") == 64
    assert _const(src, "kPartCols") == 64
    # the buffer path is left for the 64-bit fallback at this length
    assert "len >= (1 << 28)" in src
    assert "span > uint64_t(kOutOfRange)" in src
    # the id resource spans exactly the segment's ids, the offset sits in
    # the vector offset and the scalar offset is 0
    assert "make_buffer_rsrc(const_cast<int32_t *>(sid), 0, len * 4, kBufferWord3)" in src
    assert "raw_buffer_load_b32(id_rsrc, c * (kChunkRows * 4) + lane * 4, 0," in src


def test_id_reads_fit_and_past_the_end_are_range_checked():
    src = _source("tc_backward.hip")
    rows, ahead = _const(src, "kChunkRows"), _const(src, "kIdAhead")
    for length in (80, 81, 2047, 2048, 10 ** 6, (1 << 28) - 1):
        nchunks = (length + rows - 1) // rows
        # the producers read the ids of chunks 0 .. nchunks - 1 + kIdAhead
        last_chunk = nchunks - 1 + ahead
        top = last_chunk * rows * 4 + 63 * 4
        assert top <= INT32_MAX, length
        assert length * 4 <= INT32_MAX  # the resource size
        # every read of a chunk at or past the end starts at or past len*4
        first_past = nchunks * rows * 4
        assert first_past >= length * 4


def test_row_reads_fit_and_out_of_range_rows_read_zero():
    src = _source("tc_backward.hip")
    oor = _const(src, "kOutOfRange")
    max_dim = _const(_source("tc_internal.h"), "kMaxDim")
    parts = (max_dim + 63) // 64
    # a lane's byte offset within a row: its part's columns plus its own 4
    lane_bytes_max = (parts - 1) * 64 * 4 + (64 // 4 - 1) * 4 * 4
    assert lane_bytes_max < max_dim * 4
    # rows of a segment lie within span <= kOutOfRange bytes of its first row
    # (else the fallback runs), so in-range offsets stay below span and the
    # out-of-range offset kOutOfRange + lane bytes is past the resource
    assert oor + lane_bytes_max <= INT32_MAX
    assert oor % 16 == 0  # 16-byte loads stay aligned
    # the whole-array window is used only when grad fits below kOutOfRange
    assert "gb <= kOutOfRange ? int32_t(gb) : 0" in src
