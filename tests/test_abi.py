"""The C ABI without a GPU: the library loads, exports every declared symbol, and rejects bad
arguments on the host before any HIP call (fake pointers are never dereferenced)."""
import ctypes
import math
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ts_attn.h")

ts = pytest.importorskip("paper_2606_19271_amd")
from paper_2606_19271_amd import _lib  # noqa: E402


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ts_attn_\w+)\s*\(", text)))


def header_macro(name):
    m = re.search(r"#define\s+%s\s+(\d+)" % name, open(HEADER).read())
    return int(m.group(1))


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert names == ["ts_attn_abi_version", "ts_attn_fwd", "ts_attn_fwd_kvcache",
                     "ts_attn_fwd_kvcache_noalloc", "ts_attn_fwd_varlen", "ts_attn_status_str"]
    copy_names = sorted(set(re.findall(r"\b(ts_state_\w+)\s*\(",
                                       re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S))))
    assert copy_names == ["ts_state_copy"]
    names = names + copy_names
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (ts_\w+)", out))
    assert set(names) <= exported
    # nothing else: the C++ launch layer and the kernel stubs stay local to the library
    defined = set(re.findall(r"^[0-9a-fA-F]+ [A-Za-z] (\S+)$", out, flags=re.M))
    assert defined == set(names), sorted(defined - set(names))


def test_abi_version_matches_header(lib):
    assert lib.ts_attn_abi_version() == header_macro("TS_ATTN_ABI_VERSION")


def test_header_compiles_as_c_and_cxx(tmp_path):
    src = tmp_path / "use.c"
    src.write_text('#include "ts_attn.h"\nint main(void){return ts_attn_abi_version() - TS_ATTN_ABI_VERSION;}\n')
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-I", os.path.dirname(HEADER),
                    str(src)], check=True)
    subprocess.run(["g++", "-std=c++11", "-Wall", "-Werror", "-fsyntax-only", "-x", "c++",
                    "-I", os.path.dirname(HEADER), str(src)], check=True)


def test_plain_c_client_builds_and_links(tmp_path):
    # the C client of tests/c_abi (HIP runtime + this header, -Werror) compiles and links against
    # the built library; it runs on the GPU in test_gpu_c_abi.py
    import importlib.util
    spec = importlib.util.spec_from_file_location("c_abi_build", os.path.join(ROOT, "tests", "c_abi", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    exe = mod.build(str(tmp_path / "caller"))
    assert os.access(exe, os.X_OK)


def test_status_strings(lib):
    for code, name in enumerate(_lib.STATUS_NAMES):
        assert ts.status_str(code).startswith(name)
    assert ts.status_str(999) == "unknown ts_status"


A = 0x10000          # fake, 16-byte aligned device addresses; never dereferenced
BIG = 0x100000000000  # far from A: no overlap for the sizes below


def fwd(lib, q=A, k=A, v=A, o=BIG, B=1, L=128, H=2, d=128, scale=0.125, stream=None):
    P = ctypes.c_void_p
    return lib.ts_attn_fwd(P(q), P(k), P(v), P(o), B, L, H, d, scale, P(stream))


def varlen(lib, q=A, k=A, v=A, o=BIG, cu=A, nseq=2, max_seqlen=64, T=128, H=2, d=128,
           scale=0.125):
    P = ctypes.c_void_p
    return lib.ts_attn_fwd_varlen(P(q), P(k), P(v), P(o), P(cu), nseq, max_seqlen, T, H, d, scale,
                                  P(None))


def test_dense_argument_checks(lib):
    assert fwd(lib, q=0) == _lib.TS_ERR_NULL
    assert fwd(lib, o=0) == _lib.TS_ERR_NULL
    assert fwd(lib, B=-1) == _lib.TS_ERR_SHAPE
    assert fwd(lib, L=-5) == _lib.TS_ERR_SHAPE
    assert fwd(lib, H=0) == _lib.TS_ERR_SHAPE
    for d in (0, 32, 96, 256):
        assert fwd(lib, d=d) == _lib.TS_ERR_HEAD_DIM
    for s in (math.nan, math.inf, -math.inf):
        assert fwd(lib, scale=s) == _lib.TS_ERR_SCALE
    assert fwd(lib, k=A + 8) == _lib.TS_ERR_ALIGN
    assert fwd(lib, o=BIG + 2) == _lib.TS_ERR_ALIGN
    assert fwd(lib, o=A) == _lib.TS_ERR_ALIAS                      # o == q
    assert fwd(lib, v=BIG + 4096, o=BIG) == _lib.TS_ERR_ALIAS      # o overlaps v
    assert fwd(lib, L=300000, H=40) == _lib.TS_ERR_SHAPE           # beyond the byte limit
    # head counts whose row size alone passes the byte limit (the check must not overflow)
    for H in (1 << 23, (1 << 31) - 1):
        assert fwd(lib, H=H) == _lib.TS_ERR_SHAPE
        assert fwd(lib, H=H, L=(1 << 31) - 1) == _lib.TS_ERR_SHAPE
        assert varlen(lib, H=H, max_seqlen=(1 << 31) - 1) == _lib.TS_ERR_SHAPE
        assert kvcache(lib, H=H, max_k=(1 << 31) - 1) == _lib.TS_ERR_SHAPE
    # empty problems are no-ops that never touch the device, also with NULL tensors (an empty
    # torch tensor has a NULL data pointer)
    assert fwd(lib, B=0) == _lib.TS_OK
    assert fwd(lib, L=0) == _lib.TS_OK
    assert fwd(lib, q=0, k=0, v=0, o=0, B=0) == _lib.TS_OK
    assert fwd(lib, q=0, k=0, v=0, o=0, L=0) == _lib.TS_OK
    assert fwd(lib, k=0, B=3, L=0) == _lib.TS_OK


def test_varlen_argument_checks(lib):
    assert varlen(lib, cu=0) == _lib.TS_ERR_NULL
    assert varlen(lib, q=0) == _lib.TS_ERR_NULL
    assert varlen(lib, q=0, k=0, v=0, o=0, T=0) == _lib.TS_OK   # empty batch, empty tensors
    assert varlen(lib, q=0, k=0, v=0, o=0, T=0, d=80) == _lib.TS_ERR_HEAD_DIM
    assert varlen(lib, nseq=-1) == _lib.TS_ERR_SHAPE
    assert varlen(lib, max_seqlen=-1) == _lib.TS_ERR_SHAPE
    assert varlen(lib, T=-1) == _lib.TS_ERR_SHAPE
    assert varlen(lib, d=80) == _lib.TS_ERR_HEAD_DIM
    assert varlen(lib, scale=math.nan) == _lib.TS_ERR_SCALE
    assert varlen(lib, q=A + 1) == _lib.TS_ERR_ALIGN
    assert varlen(lib, o=A) == _lib.TS_ERR_ALIAS
    assert varlen(lib, nseq=1 << 24, T=1 << 24) == _lib.TS_ERR_SHAPE  # grid too large
    assert varlen(lib, nseq=0) == _lib.TS_OK
    assert varlen(lib, T=0) == _lib.TS_OK


def kvcache(lib, q=A, k=A, v=A, o=BIG, lse=None, cuq=A, cuk=A, nseq=2, max_q=64, max_k=256,
            tq=128, tk=512, H=2, d=128, scale=0.125, splits=0, entry="ts_attn_fwd_kvcache"):
    P = ctypes.c_void_p
    return getattr(lib, entry)(P(q), P(k), P(v), P(o), P(lse), P(cuq), P(cuk), nseq, max_q,
                               max_k, tq, tk, H, d, scale, splits, P(None))


def test_kvcache_noalloc_argument_checks(lib):
    """The allocation-free chunk call makes every check of ts_attn_fwd_kvcache, and refuses a
    forced split count whose partial results exceed its 32 MiB scratch before any HIP call."""
    def noalloc(**kw):
        return kvcache(lib, entry="ts_attn_fwd_kvcache_noalloc", **kw)
    assert noalloc(cuk=0) == _lib.TS_ERR_NULL
    assert noalloc(splits=17) == _lib.TS_ERR_SHAPE
    assert noalloc(d=96) == _lib.TS_ERR_HEAD_DIM
    assert noalloc(scale=math.nan) == _lib.TS_ERR_SCALE
    assert noalloc(o=A + 300 * 2 * 128 * 2) == _lib.TS_ERR_ALIAS
    assert noalloc(nseq=0) == _lib.TS_OK and noalloc(tq=0) == _lib.TS_OK
    # plan (256 B) + lse (align256(4 n tq H)) + partial O (4 n tq H d) against 32 MiB
    tq, H, d = 8192, 2, 128
    assert 256 + 4 * 3 * tq * H + 4 * 3 * tq * H * d <= 32 << 20 < 256 + 4 * 4 * tq * H + 4 * 4 * tq * H * d
    big = BIG * 4
    assert noalloc(tq=tq, max_q=tq, o=big, splits=4) == _lib.TS_ERR_SCRATCH
    assert noalloc(tq=tq, max_q=tq, o=big, splits=16) == _lib.TS_ERR_SCRATCH
    assert noalloc(tq=tq, max_q=tq, o=big, splits=4, d=80) == _lib.TS_ERR_HEAD_DIM  # checks first


def test_kvcache_argument_checks(lib):
    assert kvcache(lib, cuk=0) == _lib.TS_ERR_NULL
    assert kvcache(lib, cuq=0) == _lib.TS_ERR_NULL
    assert kvcache(lib, v=0) == _lib.TS_ERR_NULL
    assert kvcache(lib, nseq=-1) == _lib.TS_ERR_SHAPE
    assert kvcache(lib, max_k=-1) == _lib.TS_ERR_SHAPE
    assert kvcache(lib, tk=-1) == _lib.TS_ERR_SHAPE
    assert kvcache(lib, splits=-1) == _lib.TS_ERR_SHAPE
    assert kvcache(lib, splits=17) == _lib.TS_ERR_SHAPE
    assert kvcache(lib, d=96) == _lib.TS_ERR_HEAD_DIM
    assert kvcache(lib, scale=math.inf) == _lib.TS_ERR_SCALE
    assert kvcache(lib, k=A + 8) == _lib.TS_ERR_ALIGN
    assert kvcache(lib, lse=BIG * 2 + 2) == _lib.TS_ERR_ALIGN
    # o holds tq rows; k/v hold tk rows: o placed inside k's range aliases
    row = 2 * 128 * 2
    assert kvcache(lib, o=A + 300 * row) == _lib.TS_ERR_ALIAS       # inside k/v (512 rows)
    assert kvcache(lib, lse=BIG + 64) == _lib.TS_ERR_ALIAS          # lse inside o
    assert kvcache(lib, max_k=300000, H=40) == _lib.TS_ERR_SHAPE    # beyond the byte limit
    # empty problems are no-ops that never touch the device
    assert kvcache(lib, nseq=0) == _lib.TS_OK
    assert kvcache(lib, tq=0) == _lib.TS_OK
    assert kvcache(lib, q=0, o=0, tq=0) == _lib.TS_OK
    assert kvcache(lib, q=0, k=0, v=0, o=0, tq=0, tk=0) == _lib.TS_OK
    # NULL k/v of zero rows pass the pointer check (a later host check, d = 80, shows it without
    # reaching the device); NULL tensors with rows do not
    assert kvcache(lib, k=0, v=0, tk=0, max_k=0, d=80) == _lib.TS_ERR_HEAD_DIM
    assert kvcache(lib, k=0, tk=0, max_k=0, d=80) == _lib.TS_ERR_HEAD_DIM
    assert kvcache(lib, k=0, v=0, d=80) == _lib.TS_ERR_NULL
    assert kvcache(lib, q=0, tq=128) == _lib.TS_ERR_NULL
    assert kvcache(lib, o=0) == _lib.TS_ERR_NULL
    assert kvcache(lib, k=0, tq=0) == _lib.TS_ERR_NULL   # k has rows: its pointer is required


def state_copy(lib, src=A, sb=1 << 20, dst=BIG, db=1 << 20, ranges=((0, 0, 256),), n=None):
    r = np.ascontiguousarray(np.asarray(ranges, dtype=np.int64).reshape(-1, 3))
    P = ctypes.c_void_p
    return lib.ts_state_copy(P(src), sb, P(dst), db, P(r.ctypes.data), r.shape[0] if n is None else n,
                             P(None))


def test_state_copy_argument_checks(lib):
    assert state_copy(lib, n=-1) == _lib.TS_ERR_SHAPE
    assert state_copy(lib, n=0) == _lib.TS_OK
    assert state_copy(lib, src=0) == _lib.TS_ERR_NULL
    assert state_copy(lib, dst=A + 8) == _lib.TS_ERR_ALIGN
    assert state_copy(lib, ranges=((16, 0, 24),)) == _lib.TS_ERR_ALIGN
    assert state_copy(lib, ranges=((0, 8, 16),)) == _lib.TS_ERR_ALIGN
    assert state_copy(lib, ranges=((-16, 0, 16),)) == _lib.TS_ERR_SHAPE
    assert state_copy(lib, ranges=((0, 0, (1 << 20) + 16),)) == _lib.TS_ERR_SHAPE   # past src
    assert state_copy(lib, ranges=((0, (1 << 20) - 16, 32),)) == _lib.TS_ERR_SHAPE  # past dst
    assert state_copy(lib, dst=A + 4096) == _lib.TS_ERR_ALIAS                     # buffers overlap


def test_pack_ranges():
    r, end = ts.pack_ranges([0, 7, 7, 19, 30], [3, 1, 0], 80, dst_start=160)
    assert r == [(19 * 80, 160, 11 * 80), (7 * 80, 160 + 880, 0), (0, 1040, 7 * 80)]
    assert end == 1040 + 560


def test_binding_refuses_ints_that_do_not_fit_int32():
    # ctypes would wrap 2**32 + 64 to 64 without a word; the binding refuses it instead
    for x in (1 << 31, (1 << 32) + 64, -(1 << 31) - 1):
        with pytest.raises(ValueError):
            _lib.i32("L", x)
    for x in (0, 1, (1 << 31) - 1, -(1 << 31)):
        assert _lib.i32("L", x) == x


def test_python_binding_rejects_cpu_tensors():
    import torch
    x = torch.zeros((1, 8, 1, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        ts.ts_attn_fwd(x, x, x)
    with pytest.raises(ValueError):
        ts.ts_attn_fwd_varlen(x[0], x[0], x[0], torch.tensor([0, 8], dtype=torch.int32), 8)

    with pytest.raises(ValueError):
        cu = torch.tensor([0, 8], dtype=torch.int32)
        ts.ts_attn_fwd_kvcache(x[0], x[0], x[0], cu, cu, 8, 8)
