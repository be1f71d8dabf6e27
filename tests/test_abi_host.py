"""The C-ABI library on the host: it builds, loads, exports every declared
symbol, validates segment metadata, and rejects bad arguments before any
launch. No test here launches a kernel."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2408_00539_amd import ops
from paper_2408_00539_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ism_attn.h")
NO_GPU = not os.path.exists("/dev/kfd")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(ops.LIB_PATH):
        from paper_2408_00539_amd import build
        build.build()
    return ops.lib()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ism_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert {"ism_attn_fwd", "ism_attn_bwd", "ism_attn_prefill_cached",
            "ism_attn_decode"} <= set(names)
    for n in names:
        assert hasattr(L, n), n
    out = os.popen(f"nm -D --defined-only {ops.LIB_PATH}").read()
    for n in names:
        assert re.search(rf"\bT {n}\b", out), n


def test_status_strings(L):
    for s in range(9):
        assert L.ism_status_string(s)
    assert L.ism_version().decode().count(".") == 2


def test_validator_accepts_workloads(L):
    for i in (0, 1, 2, 4):
        s = W.make_segments(i, i)
        st, msg = ops.check_segments_host(s.cu_seqlens, s.cu_segs, s.seg_is_query)
        assert st == 0, msg


@pytest.mark.parametrize("case,cu,cs,fl,want", [
    ("empty segment", [0, 5], [0, 2, 2, 5], [1, 0, 1], 4),
    ("reversed", [0, 5], [0, 3, 2, 5], [1, 0, 1], 4),
    ("seq boundary not a segment boundary", [0, 3, 6], [0, 2, 6], [1, 0], 4),
    ("last != total", [0, 6], [0, 2, 5], [1, 0], 4),
    ("not starting at 0", [1, 6], [1, 2, 6], [1, 0], 4),
    ("empty dialogue", [0, 0, 4], [0, 4], [1], 2),
])
def test_validator_rejects(L, case, cu, cs, fl, want):
    st, msg = ops.check_segments_host(np.array(cu), np.array(cs), np.array(fl),
                                      max_seqlen=100)
    assert st == want, (case, st, msg)
    assert msg


def test_validator_max_seqlen(L):
    st, msg = ops.check_segments_host(np.array([0, 10]), np.array([0, 4, 10]),
                                      np.array([1, 0]), max_seqlen=9)
    assert st == 2 and "max_seqlen" in msg


def _segs(cu, cs, fl, batch, nseg, total, maxlen):
    return ops.ism_segments(cu, cs, fl, batch, nseg, total, maxlen)


FAKE = 0x1000  # never dereferenced: every call below fails a host check first


def test_fwd_argument_errors(L):
    sg = _segs(FAKE, FAKE, FAKE, 1, 1, 10, 10)
    ws = ctypes.c_void_p(FAKE * 256)
    big = 1 << 20
    # null q
    assert L.ism_attn_fwd(ctypes.byref(sg), None, FAKE, FAKE, FAKE, None, 1, 1,
                          64, 0.125, ws, big, None) == 1
    # null segments struct
    assert L.ism_attn_fwd(None, FAKE, FAKE, FAKE, FAKE, None, 1, 1, 64, 0.125,
                          ws, big, None) == 1
    # hq not a multiple of hkv
    assert L.ism_attn_fwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, None, 3, 2,
                          64, 0.125, ws, big, None) == 2
    # unsupported head dim
    assert L.ism_attn_fwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, None, 1, 1,
                          96, 0.125, ws, big, None) == 3
    # bad scale
    assert L.ism_attn_fwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, None, 1, 1,
                          64, -1.0, ws, big, None) == 2
    # workspace too small / missing / misaligned
    assert L.ism_attn_fwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, None, 1, 1,
                          64, 0.125, ws, 4, None) == 5
    assert L.ism_attn_fwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, None, 1, 1,
                          64, 0.125, None, 0, None) == 5
    assert L.ism_attn_fwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, None, 1, 1,
                          64, 0.125, ctypes.c_void_p(FAKE * 256 + 4), big, None) == 5
    # max_seqlen > total
    sg2 = _segs(FAKE, FAKE, FAKE, 1, 1, 10, 11)
    assert L.ism_attn_fwd(ctypes.byref(sg2), FAKE, FAKE, FAKE, FAKE, None, 1, 1,
                          64, 0.125, ws, big, None) == 2
    assert L.ism_last_error()


def test_cache_argument_errors(L):
    ws = ctypes.c_void_p(FAKE * 256)
    # decode: query heads not a multiple of the KV heads
    assert L.ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 1, 0, FAKE,
                             None, 3, 2, 64, 0.125, 0, ws, 1 << 20, None) == 2
    # allocation-free decode: partials beyond the fixed scratch, bad
    # max_seqlen, bad head dim (all refused before any device access)
    assert L.ism_attn_decode_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 64, 0,
                                     FAKE, None, 64, 64, 128, 0.125, 64, None) == 5
    assert L.ism_attn_decode_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 1, 65,
                                     FAKE, None, 1, 1, 64, 0.125, 0, None) == 6
    assert L.ism_attn_decode_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 1, 0,
                                     FAKE, None, 1, 1, 96, 0.125, 0, None) == 3
    # visibility: outputs required
    sgv = _segs(FAKE, FAKE, FAKE, 1, 1, 10, 10)
    assert L.ism_visibility(ctypes.byref(sgv), None, FAKE, None) == 1
    # decode: max_seqlen beyond capacity
    assert L.ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 1, 65, FAKE,
                             None, 1, 1, 64, 0.125, 0, ws, 1 << 20, None) == 6
    # decode: workspace too small
    assert L.ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 1, 0, FAKE,
                             None, 1, 1, 64, 0.125, 0, ws, 8, None) == 5
    # prefill: capacity smaller than the new segment
    assert L.ism_attn_prefill_cached(FAKE, 1, 10, 10, FAKE, FAKE, FAKE, FAKE,
                                     FAKE, 8, FAKE, FAKE, None, 1, 1, 64, 0.125,
                                     None, 0, None) == 6
    # prefill: null cache
    assert L.ism_attn_prefill_cached(FAKE, 1, 10, 10, FAKE, FAKE, FAKE, None,
                                     FAKE, 64, FAKE, FAKE, None, 1, 1, 64, 0.125,
                                     None, 0, None) == 1
    # prefill of an answer segment: the same checks
    for flag in (0, 1):
        assert L.ism_attn_prefill_cached_segment(
            FAKE, 1, 10, 10, flag, FAKE, FAKE, FAKE, FAKE, FAKE, 8, FAKE, FAKE,
            None, 1, 1, 64, 0.125, None, 0, None) == 6
        assert L.ism_attn_prefill_cached_segment(
            FAKE, 1, 10, 10, flag, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE,
            None, None, 1, 1, 64, 0.125, None, 0, None) == 1
    # paged cache: page size not a multiple of 64, no table, empty pool
    for ps, tab, npages, want in ((96, FAKE, 4, 3), (64, None, 4, 1), (64, FAKE, 0, 2)):
        assert L.ism_attn_prefill_paged(
            FAKE, 1, 10, 10, 1, FAKE, FAKE, FAKE, FAKE, FAKE, npages, ps, tab, 2, FAKE,
            FAKE, None, 1, 1, 64, 0.125, None, 0, None) == want
        assert L.ism_attn_decode_paged(
            FAKE, FAKE, FAKE, FAKE, FAKE, npages, ps, tab, 2, FAKE, 1, 0, FAKE, None,
            1, 1, 64, 0.125, 0, ws, 1 << 20, None) == want
    # paged prefill: new segment longer than max_pages * page_size
    assert L.ism_attn_prefill_paged(
        FAKE, 1, 200, 200, 1, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 64, FAKE, 2, FAKE, FAKE,
        None, 1, 1, 64, 0.125, None, 0, None) == 6
    # bwd: null gradient output
    sg = _segs(FAKE, FAKE, FAKE, 1, 1, 10, 10)
    assert L.ism_attn_bwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                          None, FAKE, FAKE, 1, 1, 64, 0.125, 0, ws, 1 << 20,
                          None) == 1


def test_rope_argument_errors(L):
    # rotation: null tensor / positions, bad dtype, unsupported head dim, bad base
    assert L.ism_rope2d(None, 0, 4, 1, 64, FAKE, FAKE, 10000.0, 0, None) == 1
    assert L.ism_rope2d(FAKE, 0, 4, 1, 64, None, FAKE, 10000.0, 0, None) == 1
    assert L.ism_rope2d(FAKE, 2, 4, 1, 64, FAKE, FAKE, 10000.0, 0, None) == 3
    assert L.ism_rope2d(FAKE, 0, 4, 1, 96, FAKE, FAKE, 10000.0, 0, None) == 3
    assert L.ism_rope2d(FAKE, 1, -1, 1, 64, FAKE, FAKE, 10000.0, 0, None) == 2
    for base in (1.0, 0.5, float("inf"), float("nan")):
        assert L.ism_rope2d(FAKE, 0, 4, 1, 64, FAKE, FAKE, base, 0, None) == 2
    # positions: segments checked as for the forward
    sg = _segs(FAKE, FAKE, FAKE, 2, 1, 10, 10)
    assert L.ism_positions_2d(ctypes.byref(sg), FAKE, FAKE, None) == 2
    sg = _segs(FAKE, FAKE, FAKE, 1, 1, 10, 10)
    assert L.ism_positions_2d(ctypes.byref(sg), None, FAKE, None) == 1
    # fused prefill: the prefill checks, then the positions and the base
    assert L.ism_attn_prefill_cached_rope2d(
        FAKE, 1, 10, 10, 1, FAKE, FAKE, FAKE, FAKE, FAKE, 8, FAKE, FAKE, FAKE, 10000.0,
        FAKE, None, 1, 1, 64, 0.125, None, 0, None) == 6
    assert L.ism_attn_prefill_cached_rope2d(
        FAKE, 1, 10, 10, 1, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, None, FAKE, 10000.0,
        FAKE, None, 1, 1, 64, 0.125, None, 0, None) == 1
    assert L.ism_attn_prefill_cached_rope2d(
        FAKE, 1, 10, 10, 0, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, FAKE, FAKE, 1.0,
        FAKE, None, 1, 1, 64, 0.125, None, 0, None) == 2
    assert L.ism_last_error()


@pytest.mark.skipif(not NO_GPU, reason="only meaningful where no GPU exists")
def test_no_device_is_reported(L):
    sg = _segs(FAKE, FAKE, FAKE, 1, 1, 10, 10)
    ws = ctypes.c_void_p(FAKE * 256)
    assert L.ism_attn_fwd(ctypes.byref(sg), FAKE, FAKE, FAKE, FAKE, None, 1, 1,
                          64, 0.125, ws, 1 << 20, None) == 7
    assert L.ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 1, 0, FAKE,
                             None, 1, 1, 64, 0.125, 0, ws, 1 << 20, None) == 7


def test_workspace_sizes(L):
    assert ops.workspace_size(ops.ISM_OP_FWD, 1, 1000, 1000, 4, 4, 64) >= 4000
    assert ops.workspace_size(ops.ISM_OP_FWD, 1, 1000, 1000, 4, 4, 64) % 256 == 0
    assert ops.workspace_size(ops.ISM_OP_PREFILL_CACHED, 1, 10, 10, 4, 4, 64) == 0
    a = ops.workspace_size(ops.ISM_OP_DECODE, 2, 0, 4096, 8, 2, 128, 4)
    assert a >= 2 * 8 * 4 * 128 * 4 + 2 * 8 * 4 * 2 * 4
    # any head grouping has a decode workspace (groups above 8 run in sets)
    for hq, hkv in ((3, 1), (12, 1), (32, 1), (6, 2)):
        assert ops.workspace_size(ops.ISM_OP_DECODE, 2, 0, 4096, hq, hkv, 128) > 0


def test_product_path_has_no_fallback():
    """The binding must fail loudly without the library and never import the
    oracle."""
    src = open(os.path.join(ROOT, "paper_2408_00539_amd", "ops.py")).read()
    assert "oracle" not in src.replace("no oracle", "")
    for f in os.listdir(os.path.join(ROOT, "paper_2408_00539_amd")):
        if f.endswith(".py"):
            text = open(os.path.join(ROOT, "paper_2408_00539_amd", f)).read()
            assert "import oracle" not in text and "from oracle" not in text, f
