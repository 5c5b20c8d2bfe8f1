"""The C ABI on the host side (no GPU needed): the library loads, exports every
entry point the header declares, and rejects bad arguments before any device
work."""
import ctypes
import os
import re

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "dg.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dg_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    from paper_2405_05231_amd import _lib
    return _lib.load()


def test_header_declares_the_three_path_calls():
    names = declared_functions()
    for want in ("dg_sample_group", "dg_pack_group", "dg_assemble_batch"):
        assert want in names


def test_library_exports_every_declared_symbol(L):
    from paper_2405_05231_amd import _lib
    names = declared_functions()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.SIGNATURES), "binding signatures out of sync with dg.h"
    assert L.dg_version().decode().startswith("libdg")


def test_no_fallback_when_library_missing(tmp_path, monkeypatch):
    from paper_2405_05231_amd import _lib
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(ImportError):
        _lib.load()


def test_sample_bounds(L):
    import paper_2405_05231_amd as dg
    assert dg.sample_bounds(10_000, 105_000, 64, [5, 5]) == (64 * 31, 64 * 30)
    assert dg.sample_bounds(100_000_000, 1_600_000_000, 1024, [15, 10, 5]) == (937_984, 936_960)
    assert dg.sample_bounds(1000, 5000, 4, [-1, 2]) == (1000, 5000)
    assert dg.sample_bounds(50, 10**9, 8, [10, 10]) == (50, 580)  # hop-1 frontier <= N
    # layered: every node so far samples again at each hop
    assert dg.sample_bounds(10**6, 10**9, 4, [2, 3], layered=True) == (4 * 3 * 4, 8 + 12 * 3)
    assert dg.sample_bounds(1000, 5000, 4, [-1, 2], layered=True) == (1000, 7000)
    with pytest.raises(dg.DGError):
        dg.sample_bounds(0, 10, 1, [1])
    # the sampling call's whole flags word is accepted; only LAYERED changes
    # the bounds, and unknown bits are rejected
    import ctypes
    from paper_2405_05231_amd import _lib
    fo = (ctypes.c_int32 * 2)(2, 3)
    nc, ec = ctypes.c_int64(), ctypes.c_int64()
    for flags, want in ((_lib.DG_SAMPLE_DIRECT | _lib.DG_SAMPLE_EXIT_CLEAR
                         | _lib.DG_SAMPLE_ENTRY_CLEAR, dg.sample_bounds(10**6, 10**9, 4, [2, 3])),
                        (_lib.DG_SAMPLE_LAYERED | _lib.DG_SAMPLE_DIRECT,
                         dg.sample_bounds(10**6, 10**9, 4, [2, 3], layered=True))):
        assert L.dg_sample_bounds(10**6, 10**9, 4, fo, 2, flags, ctypes.byref(nc),
                                  ctypes.byref(ec)) == 0
        assert (nc.value, ec.value) == want
    assert L.dg_sample_bounds(10**6, 10**9, 4, fo, 2, 1 << 20, ctypes.byref(nc),
                              ctypes.byref(ec)) == -1


def test_workspace_queries(L):
    a = L.dg_sample_workspace_bytes(10_000, 4, 2000, 2000, 0)
    b = L.dg_sample_workspace_bytes(20_000, 4, 2000, 2000, 0)
    assert 0 < a < b and a % 256 == 0
    assert L.dg_sample_workspace_bytes(10_000, 65, 2000, 2000, 0) == 0
    assert L.dg_sample_workspace_bytes(10_000, 4, 2000, 2000, 16) == 0  # unknown flag
    # the clear flags do not change the workspace size
    assert L.dg_sample_workspace_bytes(10_000, 4, 2000, 2000, 2 | 4 | 8) == \
        L.dg_sample_workspace_bytes(10_000, 4, 2000, 2000, 2)
    # the direct relabelling table replaces the hash table: 4*N*B bytes, plus the
    # last hop's segments (at most node_cap + 192 per batch) and sparse indices
    # (16384 entries per batch), 4 bytes each
    d = L.dg_sample_workspace_bytes(10_000_000, 64, 2000, 2000, 2)
    h = L.dg_sample_workspace_bytes(10_000_000, 64, 2000, 2000, 0)
    search = 4 * 64 * (2000 + 192) + 4 * 64 * 16384
    assert d > h and d - 4 * 10_000_000 * 64 - search < h
    assert L.dg_sample_workspace_bytes(10_000, 4, 2000, 2000, 3) == \
        L.dg_sample_workspace_bytes(10_000, 4, 2000, 2000, 2)
    p = L.dg_pack_workspace_bytes(10_000, 4, 8000)
    assert p > 8 * 10_000 and p % 256 == 0
    assert L.dg_pack_workspace_bytes(10_000, 0, 10) == 0
    # the fused call's packing workspace: packing's for B*node_cap entries, plus
    # a list slot per entry and a member-lines map
    f = L.dg_sample_pack_workspace_bytes(10_000, 4, 2000)
    assert f % 256 == 0
    assert f >= p + 4 * 8000 + L.dg_member_lines_bytes(10_000)
    assert L.dg_sample_pack_workspace_bytes(10_000, 65, 2000) == 0
    assert L.dg_sample_pack_workspace_bytes(0, 4, 2000) == 0
    assert L.dg_sample_pack_workspace_bytes(10_000, 4, 0) == 0


def test_sample_pack_host_side_argument_errors(L):
    from paper_2405_05231_amd import _lib
    sizes = _lib.Sizes()
    g = _lib.Csr(10, 0, 0x1000, 0)
    hop = (ctypes.c_int64 * 4)()
    ep = (ctypes.c_int64 * 3)()
    ph = (ctypes.c_int64 * 2)()
    fo = (ctypes.c_int32 * 1)(2)
    fake = ctypes.c_void_p(0x1000)
    pws = L.dg_sample_pack_workspace_bytes(10, 1, 4)

    def call(cache_slot=fake, loc=fake, feats=fake, row_bytes=16, pack_flags=0, ws=fake,
             ws_bytes=1 << 30, pack_ws=fake, pack_ws_bytes=pws, timing=None):
        return L.dg_sample_pack_group(
            ctypes.byref(g), fake, 1, 1, 0, fo, 1, 0, _lib.DG_SAMPLE_DIRECT, 4, fake, hop, 4,
            fake, fake, ep, None, cache_slot, loc, feats, row_bytes, 0, None, None, fake, ph,
            None, 0, pack_flags, ws, ws_bytes, pack_ws, pack_ws_bytes, None, None,
            ctypes.byref(sizes), timing)

    # packing needs the cache slots, the address tables and the features
    for kw in ({"cache_slot": None}, {"loc": None}, {"feats": None}):
        assert call(**kw) == _lib.DG_EINVAL and b"null" in L.dg_last_error()
    assert call(row_bytes=0) == _lib.DG_EINVAL
    assert call(pack_flags=_lib.DG_PACK_CLEAR_MEMBERSHIP) == _lib.DG_EINVAL
    assert b"pack flags" in L.dg_last_error()
    tm = _lib.Timing()
    assert call(pack_flags=_lib.DG_PACK_ROWS_STREAM, timing=ctypes.byref(tm)) == _lib.DG_EINVAL
    assert b"timing" in L.dg_last_error()
    # packing's workspace: missing, small or misaligned
    assert call(pack_ws=None) == _lib.DG_EWORKSPACE
    assert call(pack_ws_bytes=pws - 256) == _lib.DG_EWORKSPACE
    assert call(pack_ws=ctypes.c_void_p(0x1010)) == _lib.DG_EWORKSPACE
    assert b"packing workspace" in L.dg_last_error()
    # sampling's workspace is checked by sampling, before any device work
    assert call(ws=None, ws_bytes=0) == _lib.DG_EWORKSPACE


def test_host_side_argument_errors(L):
    from paper_2405_05231_amd import _lib
    sizes = _lib.Sizes()
    # null CSR / outputs: rejected before any device call
    rc = L.dg_sample_group(None, None, 1, 1, 0, None, 0, 0, 0, 1, None, None, 1, None, None,
                           None, None, None, None, None, None, 0, None, ctypes.byref(sizes),
                           None)
    assert rc == _lib.DG_EINVAL
    assert b"null" in L.dg_last_error()
    g = _lib.Csr(10, 0, 0x1000, 0)
    hop = (ctypes.c_int64 * 4)()
    ep = (ctypes.c_int64 * 3)()
    fo = (ctypes.c_int32 * 1)(2)
    fake = ctypes.c_void_p(0x1000)
    # B out of range
    rc = L.dg_sample_group(ctypes.byref(g), fake, 65, 1, 0, fo, 1, 0, 0, 4, fake, hop, 4, fake,
                           fake, ep, None, None, None, None, fake, 1 << 20, None,
                           ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL
    # workspace missing
    rc = L.dg_sample_group(ctypes.byref(g), fake, 1, 1, 0, fo, 1, 0, 0, 4, fake, hop, 4, fake,
                           fake, ep, None, None, None, None, None, 0, None, ctypes.byref(sizes),
                           None)
    assert rc == _lib.DG_EWORKSPACE
    # the cached address-table entries need both the cache slots and the table
    rc = L.dg_sample_group(ctypes.byref(g), fake, 1, 1, 0, fo, 1, 0, 0, 4, fake, hop, 4, fake,
                           fake, ep, None, None, fake, None, fake, 1 << 20, None,
                           ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"cache_slot and loc" in L.dg_last_error()
    # unknown flags
    rc = L.dg_sample_group(ctypes.byref(g), fake, 1, 1, 0, fo, 1, 0, 16, 4, fake, hop, 4, fake,
                           fake, ep, None, None, None, None, fake, 1 << 20, None,
                           ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"flags" in L.dg_last_error()
    # DG_SAMPLE_ENTRY_CLEAR asserts something about `membership`, so it needs one
    rc = L.dg_sample_group(ctypes.byref(g), fake, 1, 1, 0, fo, 1, 0,
                           _lib.DG_SAMPLE_ENTRY_CLEAR, 4, fake, hop, 4, fake,
                           fake, ep, None, None, None, None, fake, 1 << 20, None,
                           ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"membership" in L.dg_last_error()
    # pack: B = 0, row_bytes = 0, counts beyond the stride
    cnt = (ctypes.c_int64 * 2)(3, 9)
    ph = (ctypes.c_int64 * 3)()
    rc = L.dg_pack_group(fake, 10, 0, fake, 2, fake, 8, cnt, 0, None, None, fake, ph, fake, None,
                         0, None, None, None, 0, None, 0, fake, 1 << 20, None, None,
                         ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL
    rc = L.dg_pack_group(fake, 10, 4, fake, 2, fake, 8, cnt, 0, None, None, fake, ph, fake, None,
                         0, None, None, None, 0, None, 0, fake, 1 << 20, None, None,
                         ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"node_count" in L.dg_last_error()
    # pack flags: unknown bits, and a clear request without a membership mask
    ok_cnt = (ctypes.c_int64 * 2)(3, 5)
    rc = L.dg_pack_group(fake, 10, 4, fake, 2, fake, 8, ok_cnt, 0, None, None, fake, ph, fake,
                         None, 0, fake, None, None, 0, None, 8, fake, 1 << 20, None, None,
                         ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"flags" in L.dg_last_error()
    rc = L.dg_pack_group(fake, 10, 4, fake, 2, fake, 8, ok_cnt, 0, None, None, fake, ph, fake,
                         None, 0, None, None, None, 0, None, _lib.DG_PACK_CLEAR_MEMBERSHIP, fake,
                         1 << 20, None, None, ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"membership" in L.dg_last_error()
    # a row copy left on a second stream cannot be timed by the call
    tm = _lib.Timing()
    rc = L.dg_pack_group(fake, 10, 4, fake, 2, fake, 8, ok_cnt, 0, fake, None, fake, ph, fake,
                         None, 0, None, None, None, 0, None, _lib.DG_PACK_ROWS_STREAM, fake,
                         1 << 20, None, None, ctypes.byref(sizes), ctypes.byref(tm))
    assert rc == _lib.DG_EINVAL and b"timing" in L.dg_last_error()
    # member lines come with a membership mask
    rc = L.dg_pack_group(fake, 10, 4, fake, 2, fake, 8, ok_cnt, 0, None, None, fake, ph, fake,
                         None, 0, None, fake, None, 0, None, 0, fake, 1 << 20, None, None,
                         ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"member_lines" in L.dg_last_error()
    # the cache fill needs its node list, a packed buffer and no rows stream
    rc = L.dg_pack_group(fake, 10, 4, fake, 2, fake, 8, ok_cnt, 0, None, None, fake, ph, fake,
                         None, 0, None, None, None, 4, fake, 0, fake, 1 << 20, None, None,
                         ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"cache fill" in L.dg_last_error()
    rc = L.dg_pack_group(fake, 10, 4, fake, 2, fake, 8, ok_cnt, 0, fake, None, fake, ph, fake,
                         None, 0, None, None, fake, 4, fake, _lib.DG_PACK_ROWS_STREAM, fake,
                         1 << 20, None, fake, ctypes.byref(sizes), None)
    assert rc == _lib.DG_EINVAL and b"cache fill" in L.dg_last_error()
    # member-lines map size: a byte per 8 nodes, in blocks of 4096 nodes
    assert L.dg_member_lines_bytes(0) == 0
    assert L.dg_member_lines_bytes(1) == 512
    assert L.dg_member_lines_bytes(4096) == 512
    assert L.dg_member_lines_bytes(4097) == 1024
    # assemble: n_b = 0 is a no-op; negative sizes and overlap are rejected
    assert L.dg_assemble_batch(None, 0, None, 0, None, 0, 16, None, None, None) == _lib.DG_OK
    assert L.dg_assemble_batch(None, 0, None, 0, fake, -1, 16, fake, None, None) == _lib.DG_EINVAL
    buf = ctypes.c_void_p(0x100000)
    rc = L.dg_assemble_batch(buf, 100, ctypes.c_void_p(0x900000), 10, ctypes.c_void_p(0xF00000), 4,
                             16, ctypes.c_void_p(0x100010), None, None)
    assert rc == _lib.DG_EINVAL and b"overlap" in L.dg_last_error()


def test_assemble_batches_host_checks(L):
    from paper_2405_05231_amd import _lib
    ptr = (ctypes.c_int64 * 3)(0, 2, 5)
    cnt = (ctypes.c_int64 * 2)(3, 4)
    outs = (ctypes.c_void_p * 1)(0x100000)
    fake = ctypes.c_void_p(0x200000)
    # B = 0: nothing to do
    assert L.dg_assemble_batches(None, 0, None, ptr, None, 0, cnt, 0, 16, outs, 1, None,
                                 None) == _lib.DG_OK
    # no output buffer, bad row size, negative B
    assert L.dg_assemble_batches(None, 0, fake, ptr, fake, 8, cnt, 2, 16, outs, 0, None,
                                 None) == _lib.DG_EINVAL
    assert L.dg_assemble_batches(None, 0, fake, ptr, fake, 8, cnt, 2, 0, outs, 1, None,
                                 None) == _lib.DG_EINVAL
    assert L.dg_assemble_batches(None, 0, fake, ptr, fake, 8, cnt, -1, 16, outs, 1, None,
                                 None) == _lib.DG_EINVAL
    # n_b beyond the address-table stride (batch 1), decreasing chunk bounds:
    # rejected before any batch is enqueued
    assert L.dg_assemble_batches(None, 0, fake, ptr, fake, 3, cnt, 2, 16, outs, 1, None,
                                 None) == _lib.DG_EINVAL
    bad = (ctypes.c_int64 * 3)(0, 4, 2)
    rc = L.dg_assemble_batches(None, 0, fake, bad, fake, 8, cnt, 2, 16, outs, 1, None, None)
    assert rc == _lib.DG_EINVAL and b"bounds" in L.dg_last_error()

