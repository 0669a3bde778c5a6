"""Oracle of the session-state copy path (offload to host memory, resume, compaction).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU-baseline leg may use
it; the product path never imports it.

What it computes.  The paper's runtime suspends an idle session by copying its persistent state
from GPU memory to host memory and resumes it by copying the state back to the GPU chosen for it
(Sec. 3.1, "GPU-CPU state offloading"); the state is the session's isolated region, so only that
region moves (Sec. 6.1, "Session memory layout").  In a packed token-major batch a session's
cached keys (or values) are one contiguous byte range.  The operation is therefore a list of
range copies between two byte buffers:

    for every range r = (src_offset, dst_offset, nbytes):
        dst[dst_offset : dst_offset + nbytes] = src[src_offset : src_offset + nbytes]

with every other byte of dst left as it was.  Written out byte by byte in plain Python for tiny
buffers, and with numpy slice assignment (the same definition, one range at a time) for larger
ones.
"""
import numpy as np


def copy_ranges_bytewise(src, dst, ranges):
    """The definition, one byte at a time (tiny buffers only).  src, dst: bytes-like / bytearray.
    Returns a new bytearray."""
    out = bytearray(dst)
    for so, do, n in ranges:
        for i in range(int(n)):
            out[int(do) + i] = src[int(so) + i]
    return out


def copy_ranges(src, dst, ranges):
    """The same definition with one numpy slice assignment per range.  src, dst: 1-D uint8 arrays.
    Returns a new array; dst is not modified."""
    out = np.array(dst, dtype=np.uint8, copy=True)
    for so, do, n in ranges:
        so, do, n = int(so), int(do), int(n)
        out[do:do + n] = src[so:so + n]
    return out


def session_ranges(cu_rows, sessions, row_bytes, dst_start=0):
    """(src_offset, dst_offset, nbytes) ranges that pack the rows of the given sessions (segment
    indices into cu_rows) of one token-major tensor back to back from dst_start, in the order
    given.  Returns (ranges, end offset)."""
    ranges, off = [], int(dst_start)
    for s in sessions:
        a, b = int(cu_rows[s]), int(cu_rows[s + 1])
        n = (b - a) * int(row_bytes)
        ranges.append((a * int(row_bytes), off, n))
        off += n
    return ranges, off
